"""The closed-form walk of the scheduled dK/dV kernel (walk_plan / walk_step in
csrc/common.hpp) equals the walk defined step by step: 32-row blocks from the
top of the two query ranges down, at each block every range active there
(range 0 first), each with its head pairs in order.  Host code only: the
harness is compiled with hipcc and run on the CPU."""
import os
import random
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(os.path.dirname(HERE), "paper_2609_19242_amd", "csrc")


def walk_by_definition(r0, r1, npairs):
    """(q, s, hp) of every step, enumerated block by block."""
    spans = (r0, r1)
    blocks = [s for (a, b) in spans for s in range(a, b)]
    out = []
    for s in sorted(set(blocks), reverse=True):
        for q, (a, b) in enumerate(spans):
            if a <= s < b:
                out.extend((q, s, hp) for hp in range(npairs))
    return out


def cases():
    rng = random.Random(7)
    fixed = [((0, 0), (0, 0), 1), ((0, 5), (0, 0), 2), ((0, 0), (3, 9), 1), ((2, 9), (2, 9), 2), ((0, 4), (6, 10), 3),
             ((6, 10), (0, 4), 2), ((0, 10), (3, 6), 4), ((3, 6), (0, 10), 1), ((0, 1), (0, 1), 1), ((5, 6), (0, 1), 2),
             ((0, 1024), (2, 1024), 2), ((0, 4096), (0, 4096), 4), ((7, 8), (8, 9), 3)]
    out = list(fixed)
    for _ in range(3000):
        def span():
            if rng.random() < 0.15:
                return (0, 0)
            a = rng.randint(0, 60)
            return (a, a + rng.randint(1, 60))
        out.append((span(), span(), rng.randint(1, 5)))
    return out


@pytest.fixture(scope="module")
def harness(tmp_path_factory):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    exe = str(tmp_path_factory.mktemp("walk") / "walk_harness")
    subprocess.run([hipcc, "--offload-arch=gfx950", "-O1", "-std=c++17", "-x", "hip", "-I", CSRC,
                    "-I", os.path.join(os.path.dirname(HERE), "include"), os.path.join(HERE, "walk_harness.cpp"),
                    "-o", exe], check=True, capture_output=True)
    return exe


def test_closed_form_walk_equals_the_definition(harness):
    cs = cases()
    inp = "".join(f"{r0[0]} {r0[1]} {r1[0]} {r1[1]} {np_}\n" for r0, r1, np_ in cs)
    lines = subprocess.run([harness], input=inp, capture_output=True, text=True, check=True).stdout.split("\n")
    pos = 0
    for r0, r1, np_ in cs:
        want = walk_by_definition(r0, r1, np_)
        n = int(lines[pos]); pos += 1
        got = []
        for _ in range(n):
            q, s, hp, live = map(int, lines[pos].split()); pos += 1
            assert live == 1
            got.append((q, s, hp))
        assert got == want, (r0, r1, np_)
        past_end, before_start = map(int, lines[pos].split()); pos += 1
        assert past_end == 0 and before_start == 0
