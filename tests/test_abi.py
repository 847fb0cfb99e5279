"""CPU checks of the C-ABI library: it loads, exports every declared entry point,
its structs have the layout the binding assumes, and argument validation that
needs no GPU rejects bad input."""
import ctypes
import glob
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "stage.h")
HEADERS = sorted(glob.glob(os.path.join(ROOT, "include", "*.h")))


def declared_functions():
    text = "".join(open(h).read() for h in HEADERS)
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(stage_\w+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("stage_init", "stage_load_layer", "stage_prefill", "stage_decode", "stage_kv_append"):
        assert required in names


def test_library_exports_every_declared_symbol():
    import paper_2512_21835_amd as P
    lib = P.lib()
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing
    assert sorted(P.EXPORTED) == declared_functions()


def test_binding_constants_match_header():
    """Every #define STAGE_* of the header is exported by the package with the same value."""
    import paper_2512_21835_amd as P
    defines = [d for h in HEADERS for d in re.findall(r"^#define (STAGE_\w+) (-?\d+)", open(h).read(), flags=re.M)]
    assert len(defines) >= 10
    for name, value in defines:
        assert getattr(P, name, None) == int(value), name


def test_struct_layout_matches_binding(tmp_path):
    import paper_2512_21835_amd as P
    structs = [("stage_config", P.StageConfig), ("stage_layer_weights", P.StageLayerWeights),
               ("stage_plan_input", P.StagePlanInput), ("stage_plan_step", P.StagePlanStep),
               ("stage_alloc_device", P.StageAllocDevice), ("stage_alloc_input", P.StageAllocInput),
               ("stage_alloc_plan", P.StageAllocPlan)]
    src = tmp_path / "layout.c"
    lines = ['#include <stdio.h>', '#include <stddef.h>'] + [f'#include "{os.path.basename(h)}"' for h in HEADERS]
    lines += ['int main(void) {']
    want = []
    for cname, py in structs:
        lines.append(f'printf("%zu\\n", sizeof({cname}));')
        want.append(ctypes.sizeof(py))
        for f in py._fields_:
            lines.append(f'printf("%zu\\n", offsetof({cname}, {f[0]}));')
            want.append(getattr(py, f[0]).offset)
    lines += ['return 0; }']
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.check_call(["gcc", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)])
    out = subprocess.check_output([str(exe)]).decode().split()
    assert [int(x) for x in out] == want


def test_defaults_and_status_strings():
    import paper_2512_21835_amd as P
    cfg = P.stage_config_default()
    assert cfg.rope_theta == 10000.0 and abs(cfg.rms_eps - 1e-5) < 1e-12
    assert cfg.kv_block_tokens == 16 and cfg.n_stream_slots == 2 and cfg.device == 0
    for code in (P.STAGE_OK, P.STAGE_EINVAL, P.STAGE_ENOMEM, P.STAGE_EHIP, P.STAGE_ESTATE, P.STAGE_ERANGE):
        assert P.stage_strerror(code) not in ("", "unknown status")
    assert P.stage_strerror(-99) == "unknown status"


@pytest.mark.parametrize("field,value", [
    ("n_layers", 0), ("hidden", 100), ("n_kv_heads", 3), ("head_dim", 96), ("ffn", 7),
    ("kv_block_tokens", 32), ("max_batch", 0), ("max_microbatches", 65), ("n_resident_max", 3),
    ("kv_fp32", 2), ("timing", 8), ("n_thresholds", 40),
])
def test_init_rejects_bad_config_without_touching_a_gpu(field, value):
    import synth
    import paper_2512_21835_amd as P
    cfg = P.config_for(synth.TINY, max_microbatches=1, max_batch=1, max_context=32, n_resident_max=2)
    setattr(cfg, field, value)
    h = ctypes.c_void_p()
    assert P.lib().stage_init(ctypes.byref(cfg), ctypes.byref(h)) == P.STAGE_EINVAL
    assert h.value is None


def test_null_handles_are_rejected():
    import paper_2512_21835_amd as P
    L = P.lib()
    n = ctypes.c_int32()
    assert L.stage_sync(None) == P.STAGE_EINVAL
    assert L.stage_get_slot_log(None, None, 0, ctypes.byref(n)) == P.STAGE_EINVAL
    assert L.stage_destroy(None) == P.STAGE_OK
    assert L.stage_init(None, None) == P.STAGE_EINVAL


def test_binding_fails_loudly_without_library(monkeypatch):
    from paper_2512_21835_amd import stage as S
    monkeypatch.setattr(S, "_LIB", None)
    monkeypatch.setattr(S, "LIB_PATH", "/nonexistent/libstage.so")
    with pytest.raises(ImportError):
        S.lib()
