"""CPU checks of bench.py: the one-GPU contract and the arithmetic behind its roofline figures.

The expected values are counted here by hand from the stage shapes (bf16 weights: 2 bytes per
parameter; fp32 activations; bf16 K/V), not taken from bench.py's formulas.
"""
import os
import subprocess
import sys

import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and "--gpus 2" in r.stderr
    assert r.stdout.strip() == ""


def test_layer_and_stage_bytes():
    # 8B-shaped layer: Wq|Wk|Wv 6144 x 4096, Wo 4096 x 4096, Wg, Wu, Wd 3 x 14336 x 4096, two 4096 gains
    assert synth.LLAMA8B_STAGE.layer_bytes() == 2 * (6144 * 4096 + 4096 * 4096 + 3 * 14336 * 4096 + 2 * 4096)
    assert synth.LLAMA8B_STAGE.layer_bytes() == 436_224_000            # 436.2 MB
    assert 8 * synth.LLAMA8B_STAGE.layer_bytes() == 3_489_792_000      # 3.490 GB per 8-layer stage
    # 70B-shaped layer: Wq|Wk|Wv 10240 x 8192, Wo 8192 x 8192, 3 x 28672 x 8192, two 8192 gains
    assert synth.LLAMA70B_STAGE.layer_bytes() == 1_711_308_800         # 1711.3 MB
    assert 16 * synth.LLAMA70B_STAGE.layer_bytes() == 27_380_940_800   # 27.381 GB per 16-layer stage


def test_roofline_bytes_and_flops():
    import bench
    s8 = synth.LLAMA8B_STAGE
    # gate/up launch, one row: two 14336 x 4096 bf16 matrices, the bf16 gain, x in (fp32), h out (fp32)
    assert bench.gateup_bytes(s8, 1) == 234_881_024 + 8_192 + 16_384 + 57_344 == 234_962_944
    # one batch-1 decode step at a context of 1024 tokens before the step: per layer the weights,
    # K and V of 1025 positions read (2 x 1024 bf16 each), the new K and V written, and the fp32
    # activations every projection reads and writes
    kv = 1025 * 2 * 1024 * 2 + 2 * 1024 * 2
    acts = 4 * (4096 + 6144 + 4096 + 4096 + 4096 + 4096 + 2 * 4096 + 14336 + 14336 + 2 * 4096)
    assert bench.decode_step_bytes(s8, 1024) == 8 * (436_224_000 + kv + acts) == 3_525_705_728
    # prefill of 1024 tokens: 2 flops per projection weight per token; causal attention QK^T and PV,
    # 2 x 2 flops per (query, key <= query, head, dim)
    gemm, attn = bench.prefill_flops(s8, 1024)
    assert gemm == 2 * (6144 * 4096 + 4096 * 4096 + 3 * 14336 * 4096) * 1024 * 8 == 3_573_412_790_272
    assert attn == 4 * (1024 * 1025 // 2) * 32 * 128 * 8 == 68_786_585_600


def test_eq1_total_of_a_given_spread_by_hand():
    """Eq. (1) for the hand-worked two-device instance (whole-layer offloading): compute 1*3 + 2*3,
    hops 2 stages x 2 devices x 1, uncovered max(0, 1*10 - (1*2 + 2*3 + 2), 2*6 - (2*1 + 1*3 + 2))
    = 5; total 18."""
    import bench
    devices = [(25, 1, 3, 7), (15, 2, 2, 4)]
    assert bench.eq1_total(2, devices, [3, 3], [2, 1], [1, 2], 1) == 9 + 4 + 5 == 18
    # nothing offloaded: compute and hops only
    assert bench.eq1_total(1, devices, [2, 1], [2, 1], [0, 0], 3) == 2 + 2 + 1 * 2 * 3
