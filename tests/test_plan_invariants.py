"""Invariants of the host planner on every configured weight set and on edge
sets: each GEMM tile list covers its output tiles exactly once (upper tiles
for the symmetric products, every tile for the P x Q update), the XCD-ordered
lists keep padding at the end of each XCD's queue and their longest tiles
first with loads within one job of each other, split-K parts partition
[0, Qp) in the order their reduce entry adds them, trace and norm slots are
contiguous per matrix, workspace regions and iterate buffers are aligned and
disjoint, the launch schedule chains x[xbuf(t)] -> x[xbuf(t + 1)] step by
step, and the plan's flop counts match its tile lists.

`tests/plan_check.cpp` is built with g++ against the planner's own sources
(no GPU, no HIP runtime); each case feeds it one set on stdin.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
from workloads import CONFIGS  # noqa: E402

CSRC = os.path.join(ROOT, "paper_2607_08754_amd", "csrc")
F32, BF16 = 0, 1
HOYER, NUCLEAR = 0, 1
ACCUMULATE, VALUES_ONLY, AUX, DEFER_GRAD = 0x1, 0x2, 0x8, 0x10


@pytest.fixture(scope="module")
def checker(tmp_path_factory):
    if shutil.which("g++") is None:
        pytest.skip("g++ not available")
    exe = str(tmp_path_factory.mktemp("plan_check") / "plan_check")
    cmd = ["g++", "-std=c++17", "-O1", "-I", CSRC, "-I", os.path.join(ROOT, "include"),
           os.path.join(ROOT, "tests", "plan_check.cpp"), os.path.join(CSRC, "plan.cpp"),
           os.path.join(CSRC, "pe_schedule.cpp"), "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    return exe


def run(checker, shapes, dtype=BF16, kind=HOYER, iters=6, flags=0, coeffs=None):
    head = f"{dtype} {kind} {iters} {flags} {1 if coeffs is not None else 0}\n"
    if coeffs is not None:
        assert len(coeffs) == 3 * iters
        head += " ".join(repr(float(c)) for c in coeffs) + "\n"
    body = f"{len(shapes)}\n" + "".join(f"{r} {c}\n" for r, c in shapes)
    r = subprocess.run([checker], input=head + body, capture_output=True, text=True, timeout=120)
    assert r.returncode == 0 and r.stdout.startswith("OK"), r.stdout[-4000:] + r.stderr[-2000:]
    return r.stdout


@pytest.mark.parametrize("name", sorted(CONFIGS))
@pytest.mark.parametrize("dtype", [F32, BF16])
def test_configured_sets(checker, name, dtype):
    cfg = CONFIGS[name]
    run(checker, cfg.shapes, dtype=dtype, iters=cfg.iters)


@pytest.mark.parametrize("flags", [VALUES_ONLY, DEFER_GRAD, ACCUMULATE | AUX])
def test_flags(checker, flags):
    run(checker, CONFIGS["vit_b16"].shapes, flags=flags)
    run(checker, CONFIGS["resnet18"].shapes, dtype=F32, kind=NUCLEAR, flags=flags)


RAGGED = [(7, 13), (13, 7), (130, 257), (257, 130), (1, 300), (300, 1), (128, 128), (129, 129),
          (64, 64), (200, 1000), (1000, 200), (1, 1), (255, 384)]


@pytest.mark.parametrize("dtype", [F32, BF16])
def test_edge_sets(checker, dtype):
    run(checker, RAGGED, dtype=dtype)
    run(checker, [(0, 5), (7, 13), (5, 0), (300, 1)], dtype=dtype)     # empty matrices among live ones
    run(checker, [(0, 5), (0, 0)], dtype=dtype)                        # no live matrix
    run(checker, [], dtype=dtype)                                      # empty set
    run(checker, [(128, 65536), (65536, 128)], dtype=dtype)            # split-K Gram (few, long tiles)
    run(checker, [(4096, 4096)] * 3 + [(256, 256)], dtype=dtype)       # few large matrices: jobs cut per XCD
    run(checker, RAGGED, dtype=dtype, iters=1)                         # the last update alone
    run(checker, [(16384, 65408)], dtype=BF16)                         # at the 2 GiB iterate limit


def test_cubic_and_mixed_tables(checker):
    """c_t = 0 steps: no poly launch, the update takes A (use_a); an all-cubic
    table leaves B aliased to A."""
    cubic = [1.5, -0.5, 0.0] * 4
    run(checker, CONFIGS["vit_b16"].shapes, iters=4, coeffs=cubic)
    run(checker, RAGGED, dtype=F32, iters=4, coeffs=cubic)
    mixed = [1.5, -0.5, 0.0] + [2.0, -1.5, 0.5] * 3
    run(checker, CONFIGS["vit_b16"].shapes, iters=4, coeffs=mixed)
    run(checker, CONFIGS["tiny"].shapes, dtype=F32, iters=4, coeffs=mixed)
