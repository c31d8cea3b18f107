"""Independent closed forms of the SegBlocks block modules, written with numpy
and torch library operations (no loops over blocks or pixels), used only to
pin the CPU oracle.

They follow from the definitions in the paper's "Block modules" section:

* BlockCombine writes a high block unchanged and a low block nearest-upsampled,
  so the combined map is Z = M*x + (1-M)*up2(pool(x)) after BlockSample.
* BlockPad copies neighbours at the same resolution, nearest-upsamples a low
  neighbour into a high block's halo and 2x2-averages a high neighbour into a
  low block's halo, with zeros outside the image.  Because the 2x2 average of
  a nearest-upsampled value is the value itself, a padded high block is a
  window of zeropad1(Z) and a padded low block a window of zeropad1(pool(Z)).
* A layer is therefore M*conv_pad1(Z) + (1-M)*up2(conv_pad1(pool(Z))).
"""
from __future__ import annotations

import numpy as np
import torch
import torch.nn.functional as F


def to_type(a: np.ndarray, dtype: str) -> np.ndarray:
    """Round float32 values to the storage type with library casts (RNE)."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    if dtype == "f32":
        return a.copy()
    if dtype == "f16":
        return a.astype(np.float16).astype(np.float32)
    return torch.from_numpy(a).to(torch.bfloat16).float().numpy()


def pool_f32(z: np.ndarray, dtype: str) -> np.ndarray:
    """2x2 mean of every cell with the fp32 association ((a+b)+(c+d))*0.25,
    vectorised over the whole map, then rounded to the storage type."""
    z = z.astype(np.float32)
    s = (z[..., 0::2, 0::2] + z[..., 0::2, 1::2]) + (z[..., 1::2, 0::2] + z[..., 1::2, 1::2])
    return to_type(s * np.float32(0.25), dtype)


def up2(z: np.ndarray) -> np.ndarray:
    return np.repeat(np.repeat(z, 2, axis=-2), 2, axis=-1)


def pixel_mask(mask: np.ndarray, bs: int) -> np.ndarray:
    """[N, GH, GW] block mask -> [N, 1, H, W] pixel mask (1 = high)."""
    m = (np.asarray(mask) != 0).astype(np.float32)
    return np.repeat(np.repeat(m, bs, axis=1), bs, axis=2)[:, None]


def windows(zp: np.ndarray, e: int) -> np.ndarray:
    """All (e+2)x(e+2) windows at stride e of a 1-px zero-padded map
    [N, C, GH*e+2, GW*e+2] -> [N, GH, GW, C, e+2, e+2]."""
    v = np.lib.stride_tricks.sliding_window_view(zp, (e + 2, e + 2), axis=(2, 3))
    v = v[:, :, ::e, ::e]                           # [N, C, GH, GW, e+2, e+2]
    return np.ascontiguousarray(v.transpose(0, 2, 3, 1, 4, 5))


def pad_closed_form(Z: np.ndarray, mask: np.ndarray, bs: int, dtype: str):
    """Padded stacks from the combined map Z (see module docstring)."""
    m = np.asarray(mask) != 0
    zp = np.pad(Z, ((0, 0), (0, 0), (1, 1), (1, 1)))
    pp = np.pad(pool_f32(Z, dtype), ((0, 0), (0, 0), (1, 1), (1, 1)))
    hw = windows(zp, bs)
    lw = windows(pp, bs // 2)
    return hw[m], lw[~m]          # boolean indexing keeps row-major (n, gy, gx) order


def conv_pad1_f64(z: np.ndarray, w: np.ndarray, b) -> np.ndarray:
    """Ordinary zero-padded 3x3 convolution in float64 (torch library op)."""
    zt = torch.from_numpy(np.asarray(z, np.float64))
    wt = torch.from_numpy(np.asarray(w, np.float64))
    bt = None if b is None else torch.from_numpy(np.asarray(b, np.float64))
    return F.conv2d(zt, wt, bt, padding=1).numpy()


def layer_closed_form(x: np.ndarray, mask: np.ndarray, bs: int, w, b, dtype: str) -> np.ndarray:
    """float64 closed form of one block-conv layer (before output rounding)."""
    M = pixel_mask(mask, bs)
    px = pool_f32(x, dtype)
    Z = M * x + (1 - M) * up2(px)
    hi_part = conv_pad1_f64(Z, w, b)
    lo_part = up2(conv_pad1_f64(pool_f32(Z, dtype), w, b))
    return M * hi_part + (1 - M) * lo_part
