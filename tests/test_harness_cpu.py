"""The parity harness's bookkeeping, checked on the CPU with the oracle standing in for the GPU."""
import numpy as np

import synth
from oracle.stage_oracle import OracleStage
from tests.harness import RunResult, Scenario, run_oracle, teacher_forced, weights_of

# 2 layers, hidden 256; 3 micro-batches of batch 2 with fresh decode inputs (no feedback)
WL = synth.Workload("tiny_fresh", 102, synth.TINY, n_mb=3, batch=2, prefill=9, decode_steps=3)


def oracle_runner(sc, weights, feed):
    """A one-layer stage run by the oracle through the call plan, on the fed rows (fp32)."""
    orc = OracleStage(sc.shape, weights, kv_dtype="bf16")
    res = RunResult()
    for kind, mbs, _ in sc.call_plan():
        x = feed(kind, mbs, sc.prefill if kind == "prefill" else 1)
        outs = orc.forward([((m, b), x[i, b]) for i, m in enumerate(mbs) for b in range(sc.wl.batch)])
        res.inputs.append(x)
        res.outputs.append(np.stack(outs).reshape(x.shape))
    return res


def test_trace_holds_each_layers_input_rows():
    sc = Scenario(WL, prefill=9, decode_steps=3, calls="one")
    ref = run_oracle(sc, trace=True)
    assert len(ref.layer_rows) == sc.shape.n_layers + 1
    # layer 0 receives the stage inputs and the last entry is the stage output, per sequence
    flat_in = ref.flat_in().reshape(-1, 256)
    got_in = np.concatenate([ref.layer_rows[0][(m, 0)][:9] for m in range(3)])
    assert np.array_equal(flat_in[: 3 * 2 * 9].reshape(3, 2, 9, 256)[:, 0].reshape(-1, 256), got_in)
    assert np.array_equal(ref.outputs[0][0, 1], ref.layer_rows[-1][(0, 1)][:9])


def test_teacher_forcing_with_the_oracle_as_device_is_exact_up_to_fp32_inputs():
    for calls in ("one", "all"):
        sc = Scenario(WL, prefill=9, decode_steps=3, calls=calls)
        ref = run_oracle(sc, trace=True)
        res = teacher_forced(sc, ref, runner=oracle_runner)
        assert len(res) == sc.shape.n_layers
        for m in res:
            assert m["max_abs"] < 1e-4 and m["cos"] > 0.999999, m
            assert m["n"] == 3 * 2 * (9 + 3) * 256
