"""GPU parity on the scaling workloads: the ViT sweep of App. D (ViT-T ...
ViT-H, embed dims 192 ... 1280, padded shapes for dims that are not multiples
of 128) and the paper's Llama-like 135M / 560M block shapes (App. F). The
whole set runs on the GPU in the benchmarked configuration (graph replay);
the oracle checks the first block and the last matrix.
"""
import numpy as np
import pytest

from parity_util import compare, run_gpu, run_oracle
from workloads import CONFIGS, VIT_SWEEP, make_set

pytestmark = pytest.mark.gpu

SMALL = ["vit_ti", "vit_256", "vit_s", "vit_512", "llm135_paper"]
LARGE = ["vit_b24", "vit_960_24", "vit_1152_28", "vit_h", "llm560_paper"]
assert set(SMALL + LARGE) | {"vit_b16", "vit_l16"} == set(VIT_SWEEP) | {"llm135_paper", "llm560_paper"}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    import paper_2607_08754_amd._lib as L
    L.lib()


def _check(name):
    cfg = CONFIGS[name]
    arrs = make_set(name, 0)
    print(f"[scaling] {name}: {cfg.n} matrices, {cfg.params() / 1e6:.1f} M parameters", flush=True)
    vals, grads, plan = run_gpu(arrs, cfg.dtype, "hoyer", cfg.iters)
    plan.close()
    idx = list(range(cfg.block)) + [cfg.n - 1]
    refs = run_oracle([arrs[i] for i in idx], cfg.dtype, "hoyer", cfg.iters)
    compare(np.array([vals[i] for i in idx] + [0.0]), [grads[i] for i in idx], refs, "hoyer", cfg.dtype,
            label=f"{name} sample", check_total=False)
    assert np.isfinite(vals[cfg.n]) and vals[cfg.n] == pytest.approx(float(np.sum(vals[: cfg.n], dtype=np.float64)),
                                                                     rel=1e-5)


@pytest.mark.parametrize("name", SMALL)
def test_scaling_small(name):
    _check(name)


@pytest.mark.slow
@pytest.mark.parametrize("name", LARGE)
def test_scaling_large(name):
    _check(name)
