"""The host-only planner and allocation scheduler under the address and undefined-behaviour
sanitizers (CPU only).

csrc/planner.cpp (Eqs. (6)-(7)) and csrc/alloc.cpp (Alg. 1 with Eqs. (1)-(4)) are plain C++
with no GPU code, so they are rebuilt here with g++ -fsanitize=address,undefined together with
a small driver (tests/native/host_sanitize.cpp) that runs every instance through the C ABI,
both the count-only query and the full one.  The same random instances as the other CPU suites,
plus edge and invalid inputs, go through it; every answer must equal the oracle's
(oracle/planner.py, oracle/allocation.py) and the sanitizers must report nothing.
"""
import os
import random
import shutil
import subprocess

import pytest

from oracle.allocation import Device, allocate
from oracle.planner import PlanInput, plan_steps

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2512_21835_amd", "csrc")

EINVAL, ERANGE = -1, -5


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    exe = str(tmp_path_factory.mktemp("asan") / "host_sanitize")
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-I", os.path.join(ROOT, "include"),
           os.path.join(CSRC, "planner.cpp"), os.path.join(CSRC, "alloc.cpp"),
           os.path.join(ROOT, "tests", "native", "host_sanitize.cpp"), "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    return exe


def run(exe, lines):
    # verify_asan_link_order=0: a library preloaded by the environment may precede the runtime
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:halt_on_error=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe], input="\n".join(lines) + "\n", capture_output=True, text=True, env=env,
                       timeout=300)
    assert r.returncode == 0, r.stderr[-4000:]
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr[-4000:]
    out = r.stdout.splitlines()
    assert len(out) == len(lines)
    return out


def plan_line(p: PlanInput) -> str:
    return "plan " + " ".join(str(int(v)) for v in p)


def plan_expected(p: PlanInput) -> str:
    steps, cap = plan_steps(p)
    return " ".join([f"0 {len(steps)} {cap}"] + [f"{t}:{a}:{b}" for t, a, b in steps])


def alloc_line(n_layers, mha, mlp, comm, devs) -> str:
    vals = [n_layers, mha, mlp, comm, len(devs)] + [v for d in devs for v in d]
    return "alloc " + " ".join(str(int(v)) for v in vals)


def alloc_expected(n_layers, mha, mlp, comm, devs) -> str:
    want = allocate(n_layers, mha, mlp, comm, devs)
    if want is None:
        return str(ERANGE)
    s, t, plans = want
    return " ".join([f"0 {s} {t}"] + [":".join(str(v) for v in p) for p in plans])


def test_planner_under_sanitizers(driver):
    rng = random.Random(77)
    cases = [PlanInput(1000, 10, 300, 700, 300, 700, 1, 1, 2), PlanInput(0, 1, 1, 1, 1, 1, 0, 0, 1),
             PlanInput(-50, 7, 40, 90, 3, 5, 4, 4, 3), PlanInput(5, 10, 1, 1, 1, 1, 0, 0, 2)]
    for _ in range(200):
        cases.append(PlanInput(mem_left=rng.randint(-2000, 4000), kv_bytes_per_token=rng.randint(1, 60),
                               mha_bytes=rng.randint(1, 700), mlp_bytes=rng.randint(1, 1500),
                               mha_cost=rng.randint(1, 900), mlp_cost=rng.randint(1, 900),
                               mha_free=rng.randint(0, 6), mlp_free=rng.randint(0, 6), n_stage=rng.randint(1, 4)))
    bad = [PlanInput(1000, 0, 300, 700, 300, 700, 1, 1, 2), PlanInput(1000, 10, 300, 700, 0, 700, 1, 1, 2),
           PlanInput(1000, 10, 300, 700, 300, 700, -1, 1, 2), PlanInput(1000, 10, 300, 700, 300, 700, 1, 1, 0),
           PlanInput(1000, 10, 1 << 62, 700, 300, 700, 4, 1, 2)]
    out = run(driver, [plan_line(p) for p in cases + bad])
    for p, got in zip(cases, out):
        assert got == plan_expected(p), p
    assert out[len(cases):] == [str(EINVAL)] * len(bad)


def test_allocator_under_sanitizers(driver):
    rng = random.Random(2512)
    cases = [(6, 3, 7, 1, [Device(25, 1, 3, 7), Device(15, 2, 2, 4)]),
             (14, 3, 7, 2, [Device(100, 3, 1, 1), Device(100, 5, 1, 1)]),
             (3, 3, 7, 1, [Device(10, 1, 1, 1)]),
             (1, 1, 1, 0, [Device(0, 0, 1, 1)])]
    for _ in range(300):
        D = rng.randint(1, 5)
        devs = [Device(rng.randint(0, 60), rng.randint(0, 9), rng.randint(1, 9), rng.randint(1, 19)) for _ in range(D)]
        cases.append((rng.randint(1, 20), rng.randint(1, 6), rng.randint(2, 14), rng.randint(0, 5), devs))
    bad = [(0, 3, 7, 1, [Device(25, 1, 3, 7)]), (6, 0, 7, 1, [Device(25, 1, 3, 7)]),
           (6, 3, 7, -1, [Device(25, 1, 3, 7)]), (6, 3, 7, 1, [Device(25, 1, 0, 7)]), (6, 3, 7, 1, [])]
    out = run(driver, [alloc_line(*c) for c in cases + bad])
    for c, got in zip(cases, out):
        assert got == alloc_expected(*c), c
    assert out[len(cases):] == [str(EINVAL)] * len(bad)
