"""stage_decode_noalloc, the decode entry point that allocates nothing: it runs stage_decode's
kernels with their workspaces carved out of the library's fixed per-GPU scratch array.

Checked through the C ABI against stage_decode on a twin stage with the same weights and the
same call history: two noalloc calls in a row, the second smaller, give the twin's outputs bit
for bit (same kernels, same launch shapes; the attention partials only use a different stride).
Also: a call that needs more scratch than the array holds is refused with ENOMEM before anything
runs, and a call that would change the residency is refused with ESTATE, leaving the stage as it
was.
"""
import numpy as np
import pytest

import synth
from tests.harness import compute_stream, weights_of

pytestmark = pytest.mark.gpu


def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _stage(P, shape, cs, n_mb, B, ctx, **kw):
    cfg = P.config_for(shape, max_microbatches=n_mb, max_batch=B, max_context=ctx, n_resident_max=shape.n_layers,
                       compute_stream=cs.handle, **kw)
    h = P.stage_init(cfg)
    w = weights_of(shape)
    for l in range(shape.n_layers):
        P.stage_load_layer(h, l, w(l), 1)
    return h


@pytest.mark.parametrize("shape,n_mb,B,prefill", [(synth.TINY, 3, 2, 37), (synth.LLAMA8B_STAGE, 3, 2, 40)])
def test_noalloc_decode_equals_stage_decode(shape, n_mb, B, prefill):
    """Prefill, one stage_decode step, then two noalloc calls in a row -- all micro-batches
    (n_mb x B rows: the matrix-core projections and their split-K area), then one micro-batch (B
    rows: the vector kernels) -- against the same calls through stage_decode on a twin stage."""
    _gpu()
    import torch
    import paper_2512_21835_amd as P

    H = shape.hidden
    wl = synth.Workload("noalloc", 120, shape, n_mb=n_mb, batch=B, prefill=prefill, decode_steps=3)
    xp = torch.from_numpy(np.stack([np.stack([synth.prefill_inputs(wl, m, b, prefill) for b in range(B)])
                                    for m in range(n_mb)])).cuda()
    xd = [torch.from_numpy(np.stack([np.stack([synth.decode_input(wl, m, b, s) for b in range(B)])
                                     for m in range(n_mb)])).cuda() for s in range(3)]
    calls = [("decode", list(range(n_mb))), ("noalloc", list(range(n_mb))), ("noalloc", [1])]
    outs = {}
    with compute_stream() as cs:
        for mode in ("twin", "noalloc"):
            h = _stage(P, shape, cs, n_mb, B, prefill + 8)
            try:
                y = torch.empty_like(xp)
                P.stage_prefill(h, list(range(n_mb)), B, prefill, xp, y)
                got = [y]
                for s, (kind, mbs) in enumerate(calls):
                    x = xd[s][mbs].contiguous()
                    yo = torch.empty_like(x)
                    if kind == "noalloc" and mode == "noalloc":
                        P.stage_decode_noalloc(h, mbs, B, x, yo)
                    else:
                        P.stage_decode(h, mbs, B, x, yo)
                    got.append(yo)
                P.stage_sync(h)
                outs[mode] = [g.cpu().numpy() for g in got]
                lengths = [P.stage_get_length(h, m, b) for m in range(n_mb) for b in range(B)]
                assert lengths == [prefill + 2 + (m == 1) for m in range(n_mb) for _ in range(B)]
            finally:
                P.stage_destroy(h)
    for c, (a, b) in enumerate(zip(outs["noalloc"], outs["twin"])):
        print(f"\n[noalloc {shape.name}] call {c}: max|d| {float(np.abs(a - b).max()):.3g}", flush=True)
        assert np.isfinite(a).all()
        assert np.array_equal(a, b), f"call {c} differs"


def test_noalloc_refuses_what_it_cannot_do_without_allocating():
    """ENOMEM for a call whose workspaces exceed the scratch array (a stage whose FFN is so wide
    that the split-K area alone is 512 MiB; refused before any kernel runs), ESTATE for a call that
    reaches a residency threshold; after either, stage_decode still works and the state is as
    before."""
    _gpu()
    import dataclasses
    import torch
    import paper_2512_21835_amd as P

    wide = dataclasses.replace(synth.TINY, ffn=1 << 19)
    with compute_stream() as cs:
        cfg = P.config_for(wide, max_microbatches=3, max_batch=1, max_context=16, n_resident_max=wide.n_layers,
                           compute_stream=cs.handle)
        h = P.stage_init(cfg)
        try:
            x = torch.zeros(3, 1, wide.hidden, device="cuda")
            with pytest.raises(P.StageError) as e:
                P.stage_decode_noalloc(h, [0, 1, 2], 1, x, torch.empty_like(x))
            assert e.value.code == P.STAGE_ENOMEM
            assert "scratch" in str(e.value)
        finally:
            P.stage_destroy(h)

        shape = synth.TINY
        wl = synth.Workload("noalloc_th", 121, shape, n_mb=1, batch=1, prefill=20, decode_steps=2)
        h = _stage(P, shape, cs, 1, 1, 32, thresholds=[22], n_stream_slots=2)
        try:
            xp = torch.from_numpy(synth.prefill_inputs(wl, 0, 0, 20)).cuda()
            P.stage_prefill(h, [0], 1, 20, xp, torch.empty_like(xp))
            x = torch.from_numpy(synth.decode_input(wl, 0, 0, 0)[None]).cuda()
            y = torch.empty_like(x)
            P.stage_decode_noalloc(h, [0], 1, x, y)                   # length 21: no threshold yet
            with pytest.raises(P.StageError) as e:
                P.stage_decode_noalloc(h, [0], 1, x, y)               # 22 reaches the threshold
            assert e.value.code == P.STAGE_ESTATE
            assert P.stage_get_length(h, 0, 0) == 21 and P.stage_get_residency(h, 2) == [1, 1]
            P.stage_decode(h, [0], 1, x, y)                           # stage_decode demotes layer 1
            P.stage_sync(h)
            assert P.stage_get_residency(h, 2) == [1, 0] and P.stage_get_length(h, 0, 0) == 22
            assert np.isfinite(y.cpu().numpy()).all()
        finally:
            P.stage_destroy(h)
