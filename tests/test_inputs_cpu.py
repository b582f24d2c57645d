"""CPU checks of the seeded input generators the parity tests use and of the
algorithmic byte counts `bench.py` reports for the memory-bound kernels."""
import numpy as np
import pytest

from workloads import CONFIGS, widen, with_spectrum


@pytest.mark.parametrize("shape", [(50, 120), (120, 50), (64, 64)])
def test_with_spectrum_has_the_prescribed_singular_values(shape):
    k = min(shape)
    sv = 0.05 * np.logspace(0, -3, k)
    a = with_spectrum(shape, sv, seed=3, dtype="f32", index=1)
    s = np.linalg.svd(a.astype(np.float64), compute_uv=False)
    assert np.allclose(s, sv, rtol=1e-5, atol=1e-9)
    # same seed and index: the same matrix; another index: another one
    assert np.array_equal(a, with_spectrum(shape, sv, seed=3, dtype="f32", index=1))
    assert not np.array_equal(a, with_spectrum(shape, sv, seed=3, dtype="f32", index=2))


def test_with_spectrum_rank_deficient_and_bf16():
    sv = np.linspace(1.0, 0.5, 8)
    a32 = with_spectrum((40, 90), sv, seed=5, dtype="f32")
    s = np.linalg.svd(a32.astype(np.float64), compute_uv=False)
    assert np.allclose(s[:8], sv, rtol=1e-5) and s[8] < 1e-5
    a16 = with_spectrum((40, 90), sv, seed=5, dtype="bf16")
    assert a16.dtype == np.uint16
    # bf16 storage: the same matrix to bf16 rounding (relative 2^-8 per entry)
    w = widen(a16, "bf16").astype(np.float64)
    assert np.all(np.abs(w - a32) <= 2.0 ** -8 * np.abs(a32) + 1e-30)


def test_bench_alg_bytes_vit_b16():
    import bench
    cfg = CONFIGS["vit_b16"]
    pq = sum(m * n for m, n in cfg.shapes)
    assert pq == 84934656
    assert bench._alg_bytes_per_launch(cfg.shapes, "bf16", "sumsq") == 2 * pq
    assert bench._alg_bytes_per_launch(cfg.shapes, "bf16", "prep") == 4 * pq
    # W and X_T read, fp32 gradient written, every matrix
    assert bench._alg_bytes_per_launch(cfg.shapes, "bf16", "grad") == 8 * pq
