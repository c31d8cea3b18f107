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
* With strided subsampling in place of the 2x2 average, a low block's halo
  from a high neighbour is the top-left pixel of the cell, which is the
  phase-(0,0) subsampled map S = Z[::2, ::2] there (and the low blocks' own
  values elsewhere): a padded low block is a window of zeropad1(S), and a
  layer is M*conv_pad1(Z) + (1-M)*up2(conv_pad1(S)).
* With zero padding instead of BlockPad every block is convolved on its
  own: high blocks conv_pad1(block), low blocks up2(conv_pad1(pool(block))).
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


def pad_closed_form_strided(Z: np.ndarray, mask: np.ndarray, bs: int):
    """Padded stacks under strided sampling: windows of zeropad1(Z) for the
    high blocks and of zeropad1(Z[::2, ::2]) for the low blocks."""
    m = np.asarray(mask) != 0
    zp = np.pad(Z, ((0, 0), (0, 0), (1, 1), (1, 1)))
    sp = np.pad(Z[..., ::2, ::2], ((0, 0), (0, 0), (1, 1), (1, 1)))
    return windows(zp, bs)[m], windows(sp, bs // 2)[~m]


def blocks_of(z: np.ndarray, e: int) -> np.ndarray:
    """[N, C, GH*e, GW*e] -> [N, GH, GW, C, e, e] (the blocks, without halo)."""
    N, C, H, W = z.shape
    return np.ascontiguousarray(z.reshape(N, C, H // e, e, W // e, e).transpose(0, 2, 4, 1, 3, 5))


def unblock(t: np.ndarray) -> np.ndarray:
    """Inverse of blocks_of."""
    N, GH, GW, C, e, _ = t.shape
    return np.ascontiguousarray(t.transpose(0, 3, 1, 4, 2, 5).reshape(N, C, GH * e, GW * e))


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


def layer_closed_form_strided(x: np.ndarray, mask: np.ndarray, bs: int, w, b, dtype: str) -> np.ndarray:
    """float64 closed form of a layer whose BlockPad samples strided."""
    M = pixel_mask(mask, bs)
    Z = M * x + (1 - M) * up2(pool_f32(x, dtype))
    return M * conv_pad1_f64(Z, w, b) + (1 - M) * up2(conv_pad1_f64(Z[..., ::2, ::2], w, b))


def layer_closed_form_zero(x: np.ndarray, mask: np.ndarray, bs: int, w, b, dtype: str) -> np.ndarray:
    """float64 closed form of a layer that zero-pads every block: each block
    (pooled for a low block) convolved on its own with zero padding."""
    M = pixel_mask(mask, bs)
    N, C, H, W = x.shape
    GH, GW = H // bs, W // bs
    hb = blocks_of(x, bs).reshape(N * GH * GW, C, bs, bs)
    lb = blocks_of(pool_f32(x, dtype), bs // 2).reshape(N * GH * GW, C, bs // 2, bs // 2)
    Co = w.shape[0]
    yh = unblock(conv_pad1_f64(hb, w, b).reshape(N, GH, GW, Co, bs, bs))
    yl = unblock(conv_pad1_f64(lb, w, b).reshape(N, GH, GW, Co, bs // 2, bs // 2))
    return M * yh + (1 - M) * up2(yl)
