"""Seeded synthetic weight sets shaped like the paper's models.

This module only draws random inputs; it holds none of the regularizer's
arithmetic, so the CPU oracle and the HIP path can both take their inputs from
it. The paper trains on ImageNet / FineWeb-Edu with timm, TorchVision and
OLMo-style models; those weights are not available, so each set is a seeded
synthetic stand-in with the same matrix shapes (conv kernels reshaped to
(C_out, C_in * k_h * k_w), App. C.1) and a stated value distribution.

Storage types
  * "f32":  numpy float32 arrays
  * "bf16": numpy uint16 arrays holding bfloat16 bit patterns (numpy has no
            bfloat16); `widen` converts them exactly to float32 / float64.

Every matrix i of a set is drawn from numpy's PCG64 generator seeded with
(base_seed, i), in float64, then rounded to float32 (round to nearest even)
and, for bf16 sets, from float32 to bfloat16 (round to nearest even).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Callable, List, Sequence, Tuple

import numpy as np

__all__ = ["WeightSet", "CONFIGS", "VIT_SWEEP", "make_set", "widen", "f32_to_bf16_bits",
           "bf16_bits_to_f32", "gaussian", "config_shapes"]

Shape = Tuple[int, int]


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns, round to nearest even (finite input)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def widen(arr: np.ndarray, dtype: str) -> np.ndarray:
    """Exact float64 value of a stored matrix."""
    if dtype == "bf16":
        return bf16_bits_to_f32(arr).astype(np.float64)
    return np.asarray(arr, dtype=np.float32).astype(np.float64)


def _store(x64: np.ndarray, dtype: str) -> np.ndarray:
    x32 = x64.astype(np.float32)
    return f32_to_bf16_bits(x32) if dtype == "bf16" else x32


def _rng(base_seed: int, i: int) -> np.random.Generator:
    return np.random.default_rng([int(base_seed), int(i)])


def gaussian(shape: Shape, seed: int, std: float, dtype: str = "f32", index: int = 0) -> np.ndarray:
    """i.i.d. N(0, std^2) matrix, stored as `dtype`."""
    return _store(_rng(seed, index).standard_normal(shape) * std, dtype)


def with_spectrum(shape: Shape, svals, seed: int, dtype: str = "f32", index: int = 0) -> np.ndarray:
    """U diag(svals) V^T with Haar-random orthonormal U (rows x k) and V
    (cols x k), k = len(svals) <= min(shape): a matrix of prescribed singular
    values (rank k when k < min(shape)), stored as `dtype`."""
    rng = _rng(seed, index)
    s = np.asarray(svals, dtype=np.float64)
    U = _haar_cols(rng, shape[0], len(s))
    V = _haar_cols(rng, shape[1], len(s))
    return _store((U * s[None, :]) @ V.T, dtype)


# ---------------------------------------------------------------- generators

def _gen_gauss(std_of: Callable[[Shape], float]):
    def gen(shape: Shape, rng: np.random.Generator) -> np.ndarray:
        return rng.standard_normal(shape) * std_of(shape)
    return gen


def _gen_vit_b(shape: Shape, rng: np.random.Generator) -> np.ndarray:
    # G ~ N(0, 0.02^2) plus a rank-16 term of Frobenius norm 0.3 ||G||_F
    M, N = shape
    G = rng.standard_normal(shape) * 0.02
    A = rng.standard_normal((M, 16))
    B = rng.standard_normal((N, 16))
    L = A @ B.T
    L *= 0.3 * np.linalg.norm(G) / np.linalg.norm(L)
    return G + L


def _haar_cols(rng: np.random.Generator, rows: int, cols: int) -> np.ndarray:
    Z = rng.standard_normal((rows, cols))
    Q, R = np.linalg.qr(Z)
    return Q * np.sign(np.diag(R))[None, :]


def _gen_vit_l(shape: Shape, rng: np.random.Generator) -> np.ndarray:
    # W = U diag(i^-1/2) V^T with Haar U, V, scaled to RMS entry 0.02
    M, N = shape
    P = min(M, N)
    U = _haar_cols(rng, M, P)
    V = _haar_cols(rng, N, P)
    s = np.arange(1, P + 1, dtype=np.float64) ** -0.5
    W = (U * s[None, :]) @ V.T
    W *= 0.02 * np.sqrt(M * N) / np.linalg.norm(W)
    return W


@dataclass
class WeightSet:
    name: str
    dtype: str                    # "f32" or "bf16"
    iters: int                    # Polar Express steps T
    kinds: Tuple[str, ...]        # regularizers exercised on this set
    shapes: List[Shape]
    gen: Callable = field(repr=False, default=None)
    note: str = ""
    block: int = 1                # matrices per repeated unit (transformer block / layer)

    @property
    def n(self) -> int:
        return len(self.shapes)

    def params(self) -> int:
        return int(sum(m * n for m, n in self.shapes))

    def flops(self) -> float:
        """Paper's matmul count T * sum(4 P^2 Q + 2 P^3) (Sec. 3)."""
        tot = 0.0
        for m, n in self.shapes:
            P, Q = min(m, n), max(m, n)
            tot += 4.0 * P * P * Q + 2.0 * P ** 3
        return self.iters * tot


def _tiny_shapes():
    return [(128, 256)] * 4


def _resnet18_shapes():
    return ([(64, 576)] * 4 + [(128, 1152)] * 3 + [(256, 2304)] * 3 + [(512, 4608)] * 3
            + [(128, 64), (256, 128), (512, 256), (1000, 512)])


def _vit_shapes(blocks: int, d: int):
    out = []
    for _ in range(blocks):
        out += [(3 * d, d), (d, d), (4 * d, d), (d, 4 * d)]
    return out


def _llm_shapes():
    out = []
    for _ in range(24):
        out += [(1536, 1536), (256, 1536), (256, 1536), (1536, 1536),
                (6144, 1536), (6144, 1536), (1536, 6144)]
    return out


def _llama_shapes(layers: int, hidden: int, inter: int):
    # Llama-like block with full multi-head attention (App. F table of model
    # sizes): q, k, v, o (hidden x hidden), SwiGLU gate and up (inter x hidden)
    # and down (hidden x inter); every linear layer of the block is regularized
    out = []
    for _ in range(layers):
        out += [(hidden, hidden)] * 4 + [(inter, hidden), (inter, hidden), (hidden, inter)]
    return out


# ViT scaling sweep (App. D, table of ViT configurations): name -> (embed dim,
# depth); patch 16 and MLP ratio 4 throughout. ViT-B and ViT-L are the
# vit_b16 / vit_l16 sets.
VIT_SWEEP = {"vit_ti": (192, 12), "vit_256": (256, 12), "vit_s": (384, 12), "vit_512": (512, 12),
             "vit_b16": (768, 12), "vit_b24": (768, 24), "vit_960_24": (960, 24), "vit_l16": (1024, 24),
             "vit_1152_28": (1152, 28), "vit_h": (1280, 32)}


CONFIGS = {
    "tiny": WeightSet("tiny", "f32", 5, ("hoyer", "nuclear"), _tiny_shapes(),
                      _gen_gauss(lambda s: 1.0 / 16.0),
                      "4 x 128x256, N(0, 1/256)"),
    "resnet18": WeightSet("resnet18", "f32", 6, ("hoyer", "nuclear"), _resnet18_shapes(),
                          _gen_gauss(lambda s: float(np.sqrt(2.0 / s[1]))),
                          "ResNet-18 convs reshaped (C_out, C_in k k) + downsample + fc; "
                          "Kaiming normal std sqrt(2 / fan_in)"),
    "vit_b16": WeightSet("vit_b16", "bf16", 6, ("hoyer", "nuclear"), _vit_shapes(12, 768),
                         _gen_vit_b,
                         "12 blocks qkv/proj/fc1/fc2; N(0, 0.02^2) + rank-16 term of "
                         "Frobenius norm 0.3 ||G||_F", block=4),
    "vit_l16": WeightSet("vit_l16", "bf16", 6, ("hoyer", "nuclear"), _vit_shapes(24, 1024),
                         _gen_vit_l,
                         "24 blocks qkv/proj/fc1/fc2; Haar U, V, sigma_i ~ i^-1/2, RMS 0.02", block=4),
    "llm560": WeightSet("llm560", "bf16", 6, ("hoyer",), _llm_shapes(),
                        _gen_gauss(lambda s: 0.02),
                        "24 layers GQA q/k/v/o + SwiGLU gate/up/down at hidden 1536; "
                        "N(0, 0.02^2)", block=7),
    "llm135_paper": WeightSet("llm135_paper", "bf16", 6, ("hoyer",), _llama_shapes(12, 768, 2048),
                              _gen_gauss(lambda s: 0.02),
                              "12 layers q/k/v/o 768^2 + SwiGLU gate/up 2048x768, down 768x2048; "
                              "N(0, 0.02^2)", block=7),
    "llm560_paper": WeightSet("llm560_paper", "bf16", 6, ("hoyer",), _llama_shapes(24, 1280, 3456),
                              _gen_gauss(lambda s: 0.02),
                              "24 layers q/k/v/o 1280^2 + SwiGLU gate/up 3456x1280, down 1280x3456; "
                              "N(0, 0.02^2)", block=7),
}
for _name, (_d, _depth) in VIT_SWEEP.items():
    if _name not in CONFIGS:
        CONFIGS[_name] = WeightSet(_name, "bf16", 6, ("hoyer",), _vit_shapes(_depth, _d), _gen_vit_b,
                                   f"{_depth} blocks qkv/proj/fc1/fc2 at embed dim {_d}; "
                                   "N(0, 0.02^2) + rank-16 term of Frobenius norm 0.3 ||G||_F", block=4)



def config_shapes(name: str) -> List[Shape]:
    return list(CONFIGS[name].shapes)


def make_set(name: str, seed: int = 0, indices: Sequence[int] = None) -> List[np.ndarray]:
    """The matrices of a configured set (all, or only `indices`)."""
    cfg = CONFIGS[name]
    idx = range(cfg.n) if indices is None else indices
    return [_store(cfg.gen(cfg.shapes[i], _rng(seed, i)), cfg.dtype) for i in idx]
