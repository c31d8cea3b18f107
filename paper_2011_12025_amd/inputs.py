"""Seeded synthetic inputs for SegBlocks block-conv layers.

This module only draws random numbers; it holds none of the method's
arithmetic.  Tests, the smoke check and the benchmark use it to feed the same
bits to the GPU path and to the CPU oracle.

Every tensor comes from its own generator ``numpy.random.default_rng([seed,
tag])`` (PCG64): tag 0 = mask, 1 = input map, 2 = weights, 3 = bias, 4+ =
extra tensors.  Values are drawn in float32 and rounded to the storage type
with torch's round-to-nearest-even cast.  The synthetic maps stand in for
Cityscapes-shaped feature maps (1024x2048 images, 128-pixel blocks giving an
8x16 block grid); no dataset content is used.
"""
from __future__ import annotations

import numpy as np
import torch

TORCH_DTYPES = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}

TAG_MASK, TAG_X, TAG_W, TAG_B = 0, 1, 2, 3


def rng(seed: int, tag: int) -> np.random.Generator:
    return np.random.default_rng([int(seed), int(tag)])


def to_storage(a: np.ndarray, dtype: str) -> torch.Tensor:
    """float32 numpy array -> CPU torch tensor of the storage dtype (RNE)."""
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(TORCH_DTYPES[dtype])


def normal(seed: int, tag: int, shape, std: float, dtype: str) -> torch.Tensor:
    a = rng(seed, tag).standard_normal(size=shape, dtype=np.float32) * np.float32(std)
    return to_storage(a, dtype)


def feature_map(seed: int, N: int, C: int, H: int, W: int, dtype: str, tag: int = TAG_X):
    """x ~ N(0, 1), logical shape [N, C, H, W] (contiguous NCHW CPU tensor)."""
    return normal(seed, tag, (N, C, H, W), 1.0, dtype)


def conv_weight(seed: int, C_out: int, C_in: int, k: int, dtype: str, tag: int = TAG_W):
    """w ~ N(0, 1/fan_in) with fan_in = k*k*C_in, OIHW."""
    return normal(seed, tag, (C_out, C_in, k, k), (1.0 / (k * k * C_in)) ** 0.5, dtype)


def conv_bias(seed: int, C_out: int, fan_in: int, dtype: str, tag: int = TAG_B):
    """b ~ N(0, 1/fan_in) (a folded batch-norm shift)."""
    return normal(seed, tag, (C_out,), (1.0 / fan_in) ** 0.5, dtype)


def mask_bernoulli(seed: int, N: int, GH: int, GW: int, p_low: float, tag: int = TAG_MASK):
    """Block k is low-resolution iff u_k < p_low, u drawn in block order.
    Returns uint8 [N, GH, GW], 1 = high resolution."""
    u = rng(seed, tag).random(size=(N, GH, GW))
    return (u >= p_low).astype(np.uint8)


def mask_exact_fraction(seed: int, N: int, GH: int, GW: int, f_low: float, tag: int = TAG_MASK):
    """Per image, one seeded permutation of the blocks; the first round(f*B)
    are low-resolution (the sets are nested across f for a fixed seed)."""
    B = GH * GW
    g = rng(seed, tag)
    out = np.ones((N, B), np.uint8)
    nlow = int(round(f_low * B))
    for n in range(N):
        perm = g.permutation(B)
        out[n, perm[:nlow]] = 0
    return out.reshape(N, GH, GW)


def _gauss_kernel(sigma: float) -> np.ndarray:
    r = int(np.ceil(4.0 * sigma))
    t = np.arange(-r, r + 1, dtype=np.float64)
    k = np.exp(-0.5 * (t / sigma) ** 2)
    return k / k.sum()


def _smooth_axis(a: np.ndarray, k: np.ndarray, axis: int) -> np.ndarray:
    r = (k.size - 1) // 2
    pad = [(0, 0)] * a.ndim
    pad[axis] = (r, r)
    p = np.pad(a, pad, mode="symmetric")
    out = np.zeros_like(a)
    n = a.shape[axis]
    for i in range(k.size):
        sl = [slice(None)] * a.ndim
        sl[axis] = slice(i, i + n)
        out += k[i] * p[tuple(sl)]
    return out


def mask_correlated(seed: int, N: int, GH: int, GW: int, q_low: float, sigma: float = 2.0,
                    tag: int = TAG_MASK):
    """Spatially correlated mask: N(0,1) noise on the block grid, separable
    Gaussian blur (sigma in blocks, reflected border), then per image the
    round(q*B) blocks with the smallest smoothed value are low-resolution
    (ties broken by block id)."""
    z = rng(seed, tag).standard_normal(size=(N, GH, GW))
    k = _gauss_kernel(sigma)
    s = _smooth_axis(_smooth_axis(z, k, 1), k, 2)
    B = GH * GW
    nlow = int(round(q_low * B))
    out = np.ones((N, B), np.uint8)
    for n in range(N):
        order = np.lexsort((np.arange(B), s[n].reshape(-1)))
        out[n, order[:nlow]] = 0
    return out.reshape(N, GH, GW)


ENCODER_WIDTHS = (64, 128, 256, 512)
ENCODER_STRIDES = (1, 2, 2, 2)


def encoder_weights(seed: int, dtype: str, C_in: int = 3) -> dict:
    """Random-init weights of the ResNet-18 encoder (folded batch norm = a
    per-channel bias): stem 7x7 C_in->64, four stages of two basic blocks of
    two 3x3 convolutions, a 1x1 shortcut where a block changes stride or
    width.  Every tensor has its own tag (100 + its index), OIHW, N(0, 1/fan_in)."""
    specs = [("stem", 64, C_in, 7)]
    cin = 64
    for si, (width, stride) in enumerate(zip(ENCODER_WIDTHS, ENCODER_STRIDES)):
        for bi in range(2):
            st = stride if bi == 0 else 1
            p = f"s{si + 1}.b{bi}."
            specs.append((p + "c1", width, cin, 3))
            if st != 1 or cin != width:
                specs.append((p + "sc", width, cin, 1))
            specs.append((p + "c2", width, width, 3))
            cin = width
    out = {}
    for i, (name, co, ci, k) in enumerate(specs):
        out[name + ".w"] = conv_weight(seed, co, ci, k, dtype, tag=100 + 2 * i)
        out[name + ".b"] = conv_bias(seed, co, k * k * ci, dtype, tag=101 + 2 * i)
    return out
