"""SegBlocks CPU oracle -- TEST INFRASTRUCTURE ONLY.

Plain, slow CPU implementation of the SegBlocks block modules (arXiv
2011.12025, Method section "Block modules": BlockSample, BlockPad,
BlockCombine), of the block convolution that runs the same filters on the
high- and the low-resolution block stacks, and of the ResNet-18 encoder
built from them (dense stem and max-pool, block stages, strided block
convolutions whose blocks shrink with the feature map).  The arithmetic lives in
``segblocks_oracle.c`` (plain C, built with gcc ``-O2 -ffp-contract=off``);
this module only marshals numpy arrays.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It shares no code with the GPU path
(``paper_2011_12025_amd``) and neither imports the other.

All arrays are float32 in logical N,C,H,W order and hold values exactly
representable in the storage type ``dtype`` ("f32", "f16" or "bf16").
``mask[n, gy, gx] != 0`` marks a high-resolution block.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "segblocks_oracle.c")
_LIB = os.path.join(_HERE, "_liboracle.so")
_DT = {"f32": 0, "f16": 1, "bf16": 2}

_fp = ctypes.POINTER(ctypes.c_float)
_dp = ctypes.POINTER(ctypes.c_double)
_u8p = ctypes.POINTER(ctypes.c_uint8)
_i32p = ctypes.POINTER(ctypes.c_int32)


def build(force: bool = False) -> str:
    """Compile the oracle's C source into ``_liboracle.so`` (gcc, no fast-math)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
                               "-fPIC", "-shared", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _L():
    global _lib
    if _lib is None:
        lib = ctypes.CDLL(build())
        lib.orc_set_threads.argtypes = [ctypes.c_int]
        lib.orc_get_threads.restype = ctypes.c_int
        lib.orc_round.restype = ctypes.c_double
        lib.orc_round.argtypes = [ctypes.c_double, ctypes.c_int]
        lib.orc_round_array.argtypes = [_dp, _fp, ctypes.c_long, ctypes.c_int]
        lib.orc_avg4.restype = ctypes.c_float
        lib.orc_avg4.argtypes = [ctypes.c_float] * 4 + [ctypes.c_int]
        lib.orc_plan.argtypes = [_u8p, ctypes.c_long, _i32p, _i32p, _i32p, _i32p]
        lib.orc_split.argtypes = [_fp] + [ctypes.c_int] * 4 + [_u8p, ctypes.c_int, ctypes.c_int, _fp, _fp]
        lib.orc_pad.argtypes = [_fp, _fp] + [ctypes.c_int] * 4 + [_u8p, ctypes.c_int, ctypes.c_int, _fp, _fp]
        lib.orc_pad_ex.argtypes = [_fp, _fp] + [ctypes.c_int] * 4 + [_u8p] + [ctypes.c_int] * 3 + [_fp, _fp]
        lib.orc_conv3x3_valid.argtypes = [_fp, ctypes.c_long, ctypes.c_int, ctypes.c_int, _fp, _fp,
                                          ctypes.c_int, _dp]
        lib.orc_combine.argtypes = [_fp, _fp] + [ctypes.c_int] * 4 + [_u8p, ctypes.c_int, _fp]
        lib.orc_conv_block.argtypes = [_fp, ctypes.c_long, ctypes.c_int, ctypes.c_int, _fp, ctypes.c_int,
                                       ctypes.c_int, _fp, ctypes.c_int, _dp]
        lib.orc_conv_dense.argtypes = [_fp] + [ctypes.c_int] * 4 + [_fp] + [ctypes.c_int] * 3 + [_fp, ctypes.c_int, _dp]
        lib.orc_maxpool.argtypes = [_fp] + [ctypes.c_int] * 7 + [_fp]
        lib.orc_combine_bwd.argtypes = [_fp] + [ctypes.c_int] * 4 + [_u8p, ctypes.c_int, ctypes.c_int, _fp, _fp]
        lib.orc_split_bwd.argtypes = [_fp, _fp] + [ctypes.c_int] * 4 + [_u8p, ctypes.c_int, ctypes.c_int, _fp]
        lib.orc_pad_bwd.argtypes = [_fp, _fp] + [ctypes.c_int] * 4 + [_u8p] + [ctypes.c_int] * 3 + [_fp, _fp]
        lib.orc_conv3x3_bwd_data.argtypes = [_fp, ctypes.c_long, ctypes.c_int, ctypes.c_int, _fp, ctypes.c_int, _dp]
        lib.orc_conv3x3_bwd_weight.argtypes = [_fp, _fp, ctypes.c_long, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                               _dp, _dp]
        lib.orc_pad_halo.argtypes = [_fp, _fp] + [ctypes.c_int] * 4 + [_u8p] + [ctypes.c_int] * 4 + [_fp, _fp]
        lib.orc_conv_block_general.argtypes = [_fp, ctypes.c_long] + [ctypes.c_int] * 3 + [_fp] + \
            [ctypes.c_int] * 3 + [_fp, ctypes.c_int, _dp]
        lib.orc_maxpool_block.argtypes = [_fp, ctypes.c_long] + [ctypes.c_int] * 5 + [_fp]
        lib.orc_policy_scores.argtypes = [_fp] + [ctypes.c_int] * 6 + [_dp]
        lib.orc_policy_select.argtypes = [_dp, ctypes.c_int, ctypes.c_int, ctypes.c_int, _u8p]
        _lib = lib
    return _lib


def set_threads(n: int) -> None:
    """Host threads the convolutions use (n <= 0: all that OpenMP offers)."""
    _L().orc_set_threads(int(n))


def threads() -> int:
    return int(_L().orc_get_threads())


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def _ptr(a, t):
    return a.ctypes.data_as(t)


def _check_shape(mask, N, H, W, bs):
    if bs < 2 or bs % 2 or H % bs or W % bs:
        raise ValueError("block size must be even and divide H and W")
    if mask.shape != (N, H // bs, W // bs):
        raise ValueError("mask must have shape [N, H/bs, W/bs]")


# --------------------------------------------------------------------------
# rounding and the 2x2 average
# --------------------------------------------------------------------------

def round_to(a, dtype: str) -> np.ndarray:
    """Round float64 values to the storage type (round-to-nearest-even), as float32."""
    a = np.ascontiguousarray(a, dtype=np.float64)
    out = np.empty(a.shape, np.float32)
    _L().orc_round_array(_ptr(a, _dp), _ptr(out, _fp), a.size, _DT[dtype])
    return out


def round_scalar(v: float, dtype: str) -> float:
    return _L().orc_round(float(v), _DT[dtype])


def avg4(a: float, b: float, c: float, d: float, dtype: str) -> float:
    return _L().orc_avg4(a, b, c, d, _DT[dtype])


# --------------------------------------------------------------------------
# the block modules
# --------------------------------------------------------------------------

def plan(mask):
    """Slot of each block within its class, plus the inverse tables and counts."""
    m = np.ascontiguousarray(mask, dtype=np.uint8).reshape(-1)
    B = m.size
    slot = np.empty(max(B, 1), np.int32)
    inv_hi = np.empty(max(B, 1), np.int32)
    inv_lo = np.empty(max(B, 1), np.int32)
    counts = np.zeros(2, np.int32)
    _L().orc_plan(_ptr(m, _u8p), B, _ptr(slot, _i32p), _ptr(inv_hi, _i32p), _ptr(inv_lo, _i32p),
                  _ptr(counts, _i32p))
    nh, nl = int(counts[0]), int(counts[1])
    return slot[:B], inv_hi[:nh], inv_lo[:nl], nh, nl


def split(x, mask, bs: int, dtype: str):
    """BlockSample: x[N,C,H,W] -> (hi[nh,C,bs,bs], lo[nl,C,bs/2,bs/2])."""
    x = _f32(x)
    N, C, H, W = x.shape
    mask = np.ascontiguousarray(mask, dtype=np.uint8)
    _check_shape(mask, N, H, W, bs)
    _, _, _, nh, nl = plan(mask)
    hi = np.zeros((nh, C, bs, bs), np.float32)
    lo = np.zeros((nl, C, bs // 2, bs // 2), np.float32)
    _L().orc_split(_ptr(x, _fp), N, C, H, W, _ptr(mask, _u8p), bs, _DT[dtype],
                   _ptr(hi, _fp), _ptr(lo, _fp))
    return hi, lo


SAMPLING = {"avg": 0, "strided": 1, "zero": 2}


def pad(hi, lo, mask, bs: int, H: int, W: int, dtype: str, sampling: str = "avg"):
    """BlockPad: (hi, lo) -> (hi_pad[nh,C,bs+2,bs+2], lo_pad[nl,C,bs/2+2,bs/2+2]).

    sampling: how a low block's halo samples a high neighbour, "avg" (2x2
    average, the paper's choice) or "strided" (top-left pixel of the cell);
    "zero" pads every block with zeros instead (no BlockPad)."""
    hi, lo = _f32(hi), _f32(lo)
    mask = np.ascontiguousarray(mask, dtype=np.uint8)
    N = mask.shape[0]
    _check_shape(mask, N, H, W, bs)
    C = hi.shape[1] if hi.shape[0] else lo.shape[1]
    nh, nl = hi.shape[0], lo.shape[0]
    hp = np.zeros((nh, C, bs + 2, bs + 2), np.float32)
    lp = np.zeros((nl, C, bs // 2 + 2, bs // 2 + 2), np.float32)
    _L().orc_pad_ex(_ptr(hi, _fp), _ptr(lo, _fp), N, C, H, W, _ptr(mask, _u8p), bs, _DT[dtype],
                    SAMPLING[sampling], _ptr(hp, _fp), _ptr(lp, _fp))
    return hp, lp


def conv3x3_valid(P, w, b=None):
    """3x3 valid convolution of a stack of padded blocks, fp64 result (unrounded)."""
    P, w = _f32(P), _f32(w)
    S, Cin, pe, pe2 = P.shape
    assert pe == pe2 and pe >= 3
    Cout = w.shape[0]
    assert w.shape == (Cout, Cin, 3, 3)
    E = pe - 2
    out = np.zeros((S, Cout, E, E), np.float64)
    bp = None
    if b is not None:
        b = _f32(b)
        assert b.shape == (Cout,)
        bp = _ptr(b, _fp)
    if S:
        _L().orc_conv3x3_valid(_ptr(P, _fp), S, Cin, E, _ptr(w, _fp), bp, Cout, _ptr(out, _dp))
    return out


def conv3x3(hp, lp, w, b, dtype: str):
    """Block convolution of both padded stacks, rounded to the storage type."""
    return (round_to(conv3x3_valid(hp, w, b), dtype),
            round_to(conv3x3_valid(lp, w, b), dtype))


def combine(hi, lo, mask, bs: int, H: int, W: int):
    """BlockCombine: (hi, lo) -> y[N,C,H,W], low blocks nearest-upsampled."""
    hi, lo = _f32(hi), _f32(lo)
    mask = np.ascontiguousarray(mask, dtype=np.uint8)
    N = mask.shape[0]
    _check_shape(mask, N, H, W, bs)
    C = hi.shape[1] if hi.shape[0] else lo.shape[1]
    y = np.zeros((N, C, H, W), np.float32)
    _L().orc_combine(_ptr(hi, _fp), _ptr(lo, _fp), N, C, H, W, _ptr(mask, _u8p), bs, _ptr(y, _fp))
    return y


def layer(x, mask, bs: int, w, b, dtype: str, sampling: str = "avg"):
    """One block-conv layer: combine(conv3x3(pad(split(x)))), rounding to the
    storage type wherever a stage stores its result."""
    x = _f32(x)
    N, C, H, W = x.shape
    hi, lo = split(x, mask, bs, dtype)
    hp, lp = pad(hi, lo, mask, bs, H, W, dtype, sampling)
    ho, lo_o = conv3x3(hp, lp, w, b, dtype)
    return combine(ho, lo_o, mask, bs, H, W)


# ---------------------------------------------------------------------------
# Encoder: strided block convolutions and the dense stem (test infrastructure)
# ---------------------------------------------------------------------------

def conv_block(P, w, stride: int, b=None):
    """K x K convolution (K = 1 or 3) at `stride` of a stack of padded blocks,
    centred on block pixel (stride*i, stride*j); fp64 result (unrounded)."""
    P, w = _f32(P), _f32(w)
    S, Cin, pe, pe2 = P.shape
    Cout, Cin2, K, K2 = w.shape
    assert pe == pe2 and Cin2 == Cin and K == K2 and K in (1, 3) and stride in (1, 2)
    E = pe - 2
    assert E % stride == 0
    Eo = E // stride
    out = np.zeros((S, Cout, Eo, Eo), np.float64)
    bp = None
    if b is not None:
        b = _f32(b)
        assert b.shape == (Cout,)
        bp = _ptr(b, _fp)
    if S:
        _L().orc_conv_block(_ptr(P, _fp), S, Cin, E, _ptr(w, _fp), K, stride, bp, Cout, _ptr(out, _dp))
    return out


def _epilogue(acc, dtype: str, relu: bool, residual=None):
    """Bias is already in acc; adds the residual, applies ReLU, rounds once."""
    if residual is not None:
        acc = acc + _f32(residual).astype(np.float64)
    if relu:
        acc = np.maximum(acc, 0.0)
    return round_to(acc, dtype)


def block_conv_ex(hi, lo, mask, bs: int, H: int, W: int, w, b, stride: int, dtype: str, relu: bool = False,
                  residual=None, sampling: str = "avg"):
    """Block convolution of both stacks (K = w.shape[2]) at `stride`, BlockPad
    halo for 3x3, with the epilogue of the encoder's convolutions: bias,
    optional residual (a (hi, lo) pair of the output's shape), optional ReLU,
    one rounding.  Output stacks have extents bs/stride and bs/(2 stride)."""
    hp, lp = pad(hi, lo, mask, bs, H, W, dtype, sampling)
    rh, rl = (None, None) if residual is None else residual
    return (_epilogue(conv_block(hp, w, stride, b), dtype, relu, rh),
            _epilogue(conv_block(lp, w, stride, b), dtype, relu, rl))


def dense_conv(x, w, b, stride: int, padding: int, dtype: str, relu: bool = False):
    """Dense K x K convolution with zero padding, bias, optional ReLU, rounded."""
    x, w = _f32(x), _f32(w)
    N, Cin, H, W = x.shape
    Cout, Cin2, K, K2 = w.shape
    assert Cin2 == Cin and K == K2
    Ho, Wo = (H + 2 * padding - K) // stride + 1, (W + 2 * padding - K) // stride + 1
    out = np.zeros((N, Cout, Ho, Wo), np.float64)
    bp = None
    if b is not None:
        b = _f32(b)
        bp = _ptr(b, _fp)
    _L().orc_conv_dense(_ptr(x, _fp), N, Cin, H, W, _ptr(w, _fp), K, stride, padding, bp, Cout, _ptr(out, _dp))
    return _epilogue(out, dtype, relu)


def maxpool(x, k: int, stride: int, padding: int):
    """k x k max-pooling at `stride` with `padding` (padded positions never win)."""
    x = _f32(x)
    N, C, H, W = x.shape
    Ho, Wo = (H + 2 * padding - k) // stride + 1, (W + 2 * padding - k) // stride + 1
    y = np.zeros((N, C, Ho, Wo), np.float32)
    _L().orc_maxpool(_ptr(x, _fp), N, C, H, W, k, stride, padding, _ptr(y, _fp))
    return y


ENCODER_WIDTHS = (64, 128, 256, 512)
ENCODER_STRIDES = (1, 2, 2, 2)


def encoder(x, mask, image_block: int, weights: dict, dtype: str):
    """ResNet-18 encoder on block stacks: 7x7/2 stem + ReLU and 3x3/2 max-pool
    run dense, the map is split at stride 4 (block side image_block / 4), four
    stages of two basic blocks run on the stacks (a stage's first block may
    have stride 2, with a 1x1/2 shortcut), and the stacks are combined at
    stride 32.  Every convolution's result is rounded where it is stored.
    weights: as drawn by paper_2011_12025_amd.inputs.encoder_weights."""
    h = dense_conv(x, weights["stem.w"], weights["stem.b"], 2, 3, dtype, relu=True)
    h = maxpool(h, 3, 2, 1)
    N, C, H, W = h.shape
    bs = image_block // 4
    hi, lo = split(h, mask, bs, dtype)
    return _stages(hi, lo, mask, bs, H, W, weights, dtype)


def _stages(hi, lo, mask, bs: int, H: int, W: int, weights: dict, dtype: str):
    """The four stages of two basic blocks on the stacks, then BlockCombine."""
    for si, (width, stride) in enumerate(zip(ENCODER_WIDTHS, ENCODER_STRIDES)):
        for bi in range(2):
            st = stride if bi == 0 else 1
            p = f"s{si + 1}.b{bi}."
            h1 = block_conv_ex(hi, lo, mask, bs, H, W, weights[p + "c1.w"], weights[p + "c1.b"], st, dtype, relu=True)
            if p + "sc.w" in weights:
                sc = block_conv_ex(hi, lo, mask, bs, H, W, weights[p + "sc.w"], weights[p + "sc.b"], st, dtype)
            else:
                sc = (hi, lo)
            bs, H, W = bs // st, H // st, W // st
            hi, lo = block_conv_ex(h1[0], h1[1], mask, bs, H, W, weights[p + "c2.w"], weights[p + "c2.b"], 1, dtype,
                                   relu=True, residual=sc)
    return combine(hi, lo, mask, bs, H, W)


# ---------------------------------------------------------------------------
# Heuristic downsampling policy (test infrastructure)
# ---------------------------------------------------------------------------

def policy_scores(x, bs: int, dtype: str):
    """Per-block detail score [N, H/bs, W/bs] (fp64): the block's pixels'
    Euclidean distance over channels to its low-resolution version, averaged."""
    x = _f32(x)
    N, C, H, W = x.shape
    if bs < 2 or bs % 2 or H % bs or W % bs:
        raise ValueError("block size must be even and divide H and W")
    out = np.zeros((N, H // bs, W // bs), np.float64)
    _L().orc_policy_scores(_ptr(x, _fp), N, C, H, W, bs, _DT[dtype], _ptr(out, _dp))
    return out


def policy_k(tau_high: float, blocks_per_image: int) -> int:
    """High-resolution blocks per image for a target fraction tau."""
    return int(np.floor(tau_high * blocks_per_image + 0.5))


def policy_select(scores, tau_high: float):
    """Mask [N, GH, GW] (1 = high): per image the round(tau * GH * GW) blocks
    with the highest scores, equal scores ranked by block id."""
    sc = np.ascontiguousarray(scores, dtype=np.float64)
    N, GH, GW = sc.shape
    mask = np.zeros((N, GH, GW), np.uint8)
    _L().orc_policy_select(_ptr(sc, _dp), N, GH * GW, policy_k(tau_high, GH * GW), _ptr(mask, _u8p))
    return mask


def policy(x, bs: int, tau_high: float, dtype: str):
    """The heuristic policy: (mask, scores)."""
    sc = policy_scores(x, bs, dtype)
    return policy_select(sc, tau_high), sc


# ---------------------------------------------------------------------------
# Backward pass of the block modules and the block convolution
# ---------------------------------------------------------------------------

def _counts(mask):
    m = np.asarray(mask) != 0
    return int(m.sum()), int(m.size - m.sum())


def combine_backward(dy, mask, bs: int, dtype: str):
    """BlockCombine transposed: dy[N,C,H,W] -> (dhi, dlo); a low pixel gets the
    fp32 sum of its 2x2 cell's gradients, rounded."""
    dy = _f32(dy)
    N, C, H, W = dy.shape
    mask = np.ascontiguousarray(mask, dtype=np.uint8)
    _check_shape(mask, N, H, W, bs)
    nh, nl = _counts(mask)
    dhi = np.zeros((nh, C, bs, bs), np.float32)
    dlo = np.zeros((nl, C, bs // 2, bs // 2), np.float32)
    _L().orc_combine_bwd(_ptr(dy, _fp), N, C, H, W, _ptr(mask, _u8p), bs, _DT[dtype], _ptr(dhi, _fp),
                         _ptr(dlo, _fp))
    return dhi, dlo


def split_backward(dhi, dlo, mask, bs: int, H: int, W: int, dtype: str):
    """BlockSample transposed: (dhi, dlo) -> dx[N,C,H,W]."""
    dhi, dlo = _f32(dhi), _f32(dlo)
    mask = np.ascontiguousarray(mask, dtype=np.uint8)
    N = mask.shape[0]
    _check_shape(mask, N, H, W, bs)
    C = dhi.shape[1] if dhi.shape[0] else dlo.shape[1]
    dx = np.zeros((N, C, H, W), np.float32)
    _L().orc_split_bwd(_ptr(dhi, _fp), _ptr(dlo, _fp), N, C, H, W, _ptr(mask, _u8p), bs, _DT[dtype], _ptr(dx, _fp))
    return dx


def pad_backward(dhp, dlp, mask, bs: int, H: int, W: int, dtype: str, sampling: str = "avg"):
    """BlockPad transposed: (dhp, dlp) -> (dhi, dlo), accumulated in fp64, rounded."""
    dhp, dlp = _f32(dhp), _f32(dlp)
    mask = np.ascontiguousarray(mask, dtype=np.uint8)
    N = mask.shape[0]
    _check_shape(mask, N, H, W, bs)
    C = dhp.shape[1] if dhp.shape[0] else dlp.shape[1]
    nh, nl = dhp.shape[0], dlp.shape[0]
    dhi = np.zeros((nh, C, bs, bs), np.float32)
    dlo = np.zeros((nl, C, bs // 2, bs // 2), np.float32)
    _L().orc_pad_bwd(_ptr(dhp, _fp), _ptr(dlp, _fp), N, C, H, W, _ptr(mask, _u8p), bs, _DT[dtype],
                     SAMPLING[sampling], _ptr(dhi, _fp), _ptr(dlo, _fp))
    return dhi, dlo


def conv3x3_backward_data(dO, w):
    """Gradient of conv3x3_valid with respect to the padded input (fp64, unrounded)."""
    dO, w = _f32(dO), _f32(w)
    S, Cout, E, E2 = dO.shape
    Cout2, Cin, k1, k2 = w.shape
    assert E == E2 and Cout2 == Cout and (k1, k2) == (3, 3)
    dP = np.zeros((S, Cin, E + 2, E + 2), np.float64)
    if S:
        _L().orc_conv3x3_bwd_data(_ptr(dO, _fp), S, Cout, E, _ptr(w, _fp), Cin, _ptr(dP, _dp))
    return dP


def conv3x3_backward_weight(stacks, with_bias: bool = True):
    """Gradient with respect to weight and bias over several (P, dO) stacks
    (padded input, output gradient): (dw [Cout,Cin,3,3], db [Cout]) in fp64."""
    dw = db = None
    for P, dO in stacks:
        P, dO = _f32(P), _f32(dO)
        S, Cin, pe, _ = P.shape
        S2, Cout, E, _ = dO.shape
        assert S2 == S and pe == E + 2
        if dw is None:
            dw = np.zeros((Cout, Cin, 3, 3), np.float64)
            db = np.zeros(Cout, np.float64)
        if S:
            _L().orc_conv3x3_bwd_weight(_ptr(P, _fp), _ptr(dO, _fp), S, Cin, Cout, E, _ptr(dw, _dp),
                                        _ptr(db, _dp) if with_bias else None)
    return dw, (db if with_bias else None)


def layer_backward(x, mask, bs: int, w, b, dy, dtype: str, sampling: str = "avg"):
    """Gradients of one block-conv layer y = combine(conv3x3(pad(split(x)))):
    (dx, dw, db).  Every stored gradient is rounded to the storage type where
    the GPU stores it (output-block gradients, padded-stack gradients, block
    gradients, dx); dw and db are returned unrounded (fp64)."""
    x = _f32(x)
    N, C, H, W = x.shape
    hi, lo = split(x, mask, bs, dtype)
    hp, lp = pad(hi, lo, mask, bs, H, W, dtype, sampling)
    dho, dlo_o = combine_backward(dy, mask, bs, dtype)
    dw, db = conv3x3_backward_weight([(hp, dho), (lp, dlo_o)], with_bias=b is not None)
    dhp = round_to(conv3x3_backward_data(dho, w), dtype)
    dlp = round_to(conv3x3_backward_data(dlo_o, w), dtype)
    dhi, dlo = pad_backward(dhp, dlp, mask, bs, H, W, dtype, sampling)
    return split_backward(dhi, dlo, mask, bs, H, W, dtype), dw, db


# ---------------------------------------------------------------------------
# Wider halos: blockwise layers beyond 3x3 (test infrastructure)
# ---------------------------------------------------------------------------

def pad_halo(hi, lo, mask, bs: int, H: int, W: int, dtype: str, halo: int, sampling: str = "avg"):
    """BlockPad with a halo of `halo` pixels (1 <= halo <= bs/2):
    (hp [nh,C,bs+2h,bs+2h], lp [nl,C,bs/2+2h,bs/2+2h])."""
    hi, lo = _f32(hi), _f32(lo)
    mask = np.ascontiguousarray(mask, dtype=np.uint8)
    N = mask.shape[0]
    _check_shape(mask, N, H, W, bs)
    if not 1 <= halo <= bs // 2:
        raise ValueError("halo must be between 1 and bs/2")
    C = hi.shape[1] if hi.shape[0] else lo.shape[1]
    hp = np.zeros((hi.shape[0], C, bs + 2 * halo, bs + 2 * halo), np.float32)
    lp = np.zeros((lo.shape[0], C, bs // 2 + 2 * halo, bs // 2 + 2 * halo), np.float32)
    _L().orc_pad_halo(_ptr(hi, _fp), _ptr(lo, _fp), N, C, H, W, _ptr(mask, _u8p), bs, _DT[dtype],
                      SAMPLING[sampling], halo, _ptr(hp, _fp), _ptr(lp, _fp))
    return hp, lp


def conv_block_general(P, halo: int, w, stride: int = 1, dilation: int = 1, b=None):
    """K x K (odd K) convolution at `stride` and `dilation` of a stack padded
    by `halo`, centred on block pixel (stride*i, stride*j); fp64, unrounded."""
    P, w = _f32(P), _f32(w)
    S, Cin, pe, _ = P.shape
    Cout, Cin2, K, _ = w.shape
    E = pe - 2 * halo
    assert Cin2 == Cin and K % 2 == 1 and dilation * (K - 1) // 2 <= halo and E % stride == 0
    out = np.zeros((S, Cout, E // stride, E // stride), np.float64)
    bp = None
    if b is not None:
        b = _f32(b)
        bp = _ptr(b, _fp)
    if S:
        _L().orc_conv_block_general(_ptr(P, _fp), S, Cin, E, halo, _ptr(w, _fp), K, stride, dilation, bp, Cout,
                                    _ptr(out, _dp))
    return out


def maxpool_block(P, halo: int, k: int, stride: int):
    """k x k max-pooling at `stride` of a stack padded by `halo` (halo values
    take part)."""
    P = _f32(P)
    S, C, pe, _ = P.shape
    E = pe - 2 * halo
    assert k % 2 == 1 and (k - 1) // 2 <= halo and E % stride == 0
    out = np.zeros((S, C, E // stride, E // stride), np.float32)
    if S:
        _L().orc_maxpool_block(_ptr(P, _fp), S, C, E, halo, k, stride, _ptr(out, _fp))
    return out


def blockwise_stem(x, mask, image_block: int, w, b, dtype: str):
    """The encoder's stem on image blocks: 7x7/2 convolution with a 3-pixel
    BlockPad, bias, ReLU (rounded), then 3x3/2 max-pooling with a 1-pixel
    BlockPad: (hi, lo) stacks at stride 4 (block side image_block / 4)."""
    x = _f32(x)
    N, C, H, W = x.shape
    hi, lo = split(x, mask, image_block, dtype)
    hp, lp = pad_halo(hi, lo, mask, image_block, H, W, dtype, 3)
    sh = round_to(np.maximum(conv_block_general(hp, 3, w, 2, 1, b), 0.0), dtype)
    sl = round_to(np.maximum(conv_block_general(lp, 3, w, 2, 1, b), 0.0), dtype)
    bs2, H2, W2 = image_block // 2, H // 2, W // 2
    ph, pl = pad_halo(sh, sl, mask, bs2, H2, W2, dtype, 1)
    return maxpool_block(ph, 1, 3, 2), maxpool_block(pl, 1, 3, 2)


def encoder_blockwise(x, mask, image_block: int, weights: dict, dtype: str):
    """The ResNet-18 encoder with the blocks kept from the image on: the
    stem and its max-pool run blockwise (blockwise_stem), then the stages as
    in encoder()."""
    N, C, H, W = np.asarray(x).shape
    hi, lo = blockwise_stem(x, mask, image_block, weights["stem.w"], weights["stem.b"], dtype)
    return _stages(hi, lo, mask, image_block // 4, H // 4, W // 4, weights, dtype)
