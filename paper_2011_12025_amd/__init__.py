"""SegBlocks block-based dynamic-resolution convolution on MI355X (gfx950).

Python face of ``libsegblocks.so``.  Tensors are torch CUDA(HIP) tensors with
logical shape [N, C, H, W] (stacks: [S, C, e, e]) in either the default
contiguous (NCHW) or the channels_last (NHWC) memory format; all tensors of
one call share the dtype (float32, float16 or bfloat16) and the memory format.
``mask`` is a uint8 [N, H/bs, W/bs] tensor, non-zero = high resolution.

Paper: Verelst & Tuytelaars, SegBlocks (arXiv 2011.12025), Method section,
"Block modules" (BlockSample, BlockPad, BlockCombine) and the block
convolution that applies the same filters to both block stacks.
"""
from __future__ import annotations

import ctypes

import torch

from . import _binding as _b

__all__ = ["count", "split", "pad", "conv3x3", "combine", "block_conv3x3", "block_conv_ex", "layer", "conv2d",
           "maxpool", "layout_of", "block_conv3x3_workspace_size", "block_conv_ex_workspace_size",
           "layer_workspace_size", "policy_heuristic", "combine_backward", "split_backward", "pad_backward",
           "conv3x3_backward_data", "conv3x3_backward_weight", "layer_backward", "pad_halo", "conv_halo",
           "maxpool_halo", "block_conv_chain", "block_conv_chain_workspace_size", "block_conv_chain_reads_half"]

_DT = {torch.float32: _b.SB_F32, torch.float16: _b.SB_F16, torch.bfloat16: _b.SB_BF16}


def layout_of(t: torch.Tensor) -> int:
    """SB_NCHW for a contiguous tensor, SB_NHWC for a channels_last one."""
    if t.dim() != 4:
        raise ValueError("expected a 4-d tensor")
    if t.is_contiguous():
        return _b.SB_NCHW
    if t.is_contiguous(memory_format=torch.channels_last):
        return _b.SB_NHWC
    raise ValueError("tensor must be contiguous or channels_last")


def _fmt(layout: int):
    return torch.channels_last if layout == _b.SB_NHWC else torch.contiguous_format


def _empty(shape, like: torch.Tensor, layout: int) -> torch.Tensor:
    return torch.empty(shape, dtype=like.dtype, device=like.device, memory_format=_fmt(layout))


def _check_layout(layout: int, *ts):
    for t in ts:
        if t is None or t.numel() == 0:
            continue
        ok = t.is_contiguous(memory_format=_fmt(layout))
        if not ok:
            raise ValueError("all feature tensors of a call must share the memory format")


def _dt(t: torch.Tensor) -> int:
    try:
        return _DT[t.dtype]
    except KeyError:
        raise TypeError(f"unsupported dtype {t.dtype}") from None


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(t: torch.Tensor):
    return ctypes.c_void_p(torch.cuda.current_stream(t.device).cuda_stream)


def _weight(weight: torch.Tensor, layout: int, k: int = 3) -> torch.Tensor:
    """The weight in the call's memory format (OHWI memory for channels_last)."""
    if weight.dim() != 4 or tuple(weight.shape[2:]) != (k, k):
        raise ValueError(f"weight must be [C_out, C_in, {k}, {k}]")
    return weight.contiguous(memory_format=_fmt(layout))


_SAMPLING = {"avg": 0, "strided": 1, "zero": 2}


def _flags(relu: bool, sampling: str) -> int:
    """Convolution flags: ReLU and the BlockPad alternative ("avg" = BlockPad
    with average sampling, "strided" = strided subsampling, "zero" = plain
    zero padding of every block)."""
    if sampling not in _SAMPLING:
        raise ValueError(f"sampling must be one of {sorted(_SAMPLING)}")
    return (_b.SB_FLAG_RELU if relu else 0) | {0: 0, 1: _b.SB_FLAG_PAD_STRIDED, 2: _b.SB_FLAG_PAD_ZERO}[
        _SAMPLING[sampling]]


def _mask(mask: torch.Tensor) -> torch.Tensor:
    if mask.dtype != torch.uint8 or mask.dim() != 3 or not mask.is_contiguous():
        raise ValueError("mask must be a contiguous uint8 tensor [N, GH, GW]")
    return mask


def _query(fn: str, *args) -> int:
    n = ctypes.c_size_t(0)
    _b.call(fn, *args, ctypes.byref(n))
    return int(n.value)


def block_conv3x3_workspace_size(dtype: torch.dtype, layout: int, N: int, C_in: int, H: int, W: int, bs: int,
                                 C_out: int, hi_cap: int, lo_cap: int) -> int:
    """Bytes of workspace that block_conv3x3 needs for these shapes (0 = none)."""
    return _query("segblocks_block_conv3x3_workspace_size", _DT[dtype], layout, N, C_in, H, W, bs, C_out, hi_cap,
                  lo_cap)


def block_conv_ex_workspace_size(dtype: torch.dtype, N: int, C_in: int, H: int, W: int, bs: int, C_out: int,
                                 k: int, stride: int, hi_cap: int, lo_cap: int) -> int:
    """Bytes of workspace that block_conv_ex needs for these shapes (0 = none)."""
    return _query("segblocks_block_conv_ex_workspace_size", _DT[dtype], _b.SB_NHWC, N, C_in, H, W, bs, C_out, k,
                  stride, hi_cap, lo_cap)


def block_conv_chain_workspace_size(dtype: torch.dtype, N: int, C_in: int, H: int, W: int, bs: int, C_out: int,
                                    k: int, stride: int, hi_cap: int, lo_cap: int) -> int:
    """Bytes of workspace that block_conv_chain needs for these shapes (0 = none)."""
    return _query("segblocks_block_conv_chain_workspace_size", _DT[dtype], _b.SB_NHWC, N, C_in, H, W, bs, C_out, k,
                  stride, hi_cap, lo_cap)


def layer_workspace_size(dtype: torch.dtype, layout: int, N: int, C_in: int, H: int, W: int, bs: int,
                         C_out: int) -> int:
    """Bytes of workspace that layer needs for these shapes (0 = none)."""
    return _query("segblocks_layer_workspace_size", _DT[dtype], layout, N, C_in, H, W, bs, C_out)


def _ws(nbytes: int, device, workspace):
    """(pointer, size) of the workspace of a call: the caller's uint8 tensor, or
    a new one from torch's allocator.  The pointer is 256-byte aligned."""
    if nbytes == 0:
        return None, 0, None
    if workspace is None:
        workspace = torch.empty(nbytes + 256, dtype=torch.uint8, device=device)
    if workspace.dtype != torch.uint8 or not workspace.is_contiguous():
        raise ValueError("workspace must be a contiguous uint8 tensor")
    p = workspace.data_ptr()
    off = (-p) % 256
    if workspace.numel() - off < nbytes:
        raise ValueError(f"workspace too small: need {nbytes} bytes (256-byte aligned)")
    return ctypes.c_void_p(p + off), workspace.numel() - off, workspace


def count(mask: torch.Tensor):
    """(n_high, n_low) of a device mask.  Blocks on the current stream."""
    mask = _mask(mask)
    nh, nl = ctypes.c_int(0), ctypes.c_int(0)
    N, GH, GW = mask.shape
    _b.call("segblocks_count", _ptr(mask), N, GH, GW, ctypes.byref(nh), ctypes.byref(nl), _stream(mask))
    return nh.value, nl.value


def split(x: torch.Tensor, mask: torch.Tensor, bs: int, counts=None, layout=None, out=None):
    """BlockSample: returns (hi [nh,C,bs,bs], lo [nl,C,bs/2,bs/2]).

    ``counts`` = (n_high, n_low) sizes the stacks; without it (and without
    ``out``) they are counted (one host synchronisation)."""
    mask = _mask(mask)
    layout = layout_of(x) if layout is None else layout
    _check_layout(layout, x)
    N, C, H, W = x.shape
    if out is not None:
        hi, lo = out
        nh, nl = hi.shape[0], lo.shape[0]
    else:
        nh, nl = counts if counts is not None else count(mask)
        hi = _empty((nh, C, bs, bs), x, layout)
        lo = _empty((nl, C, bs // 2, bs // 2), x, layout)
    _b.call("segblocks_split", _ptr(x), _dt(x), layout, N, C, H, W, _ptr(mask), bs, _ptr(hi), nh, _ptr(lo), nl,
            _stream(x))
    return hi, lo


def pad(hi: torch.Tensor, lo: torch.Tensor, mask: torch.Tensor, bs: int, H: int, W: int, layout=None,
        sampling: str = "avg"):
    """BlockPad: returns (hi_pad [nh,C,bs+2,bs+2], lo_pad [nl,C,bs/2+2,bs/2+2]).
    sampling: "avg" (BlockPad's average sampling), "strided" or "zero"."""
    mask = _mask(mask)
    ref = hi if hi.shape[0] else lo
    layout = layout_of(ref) if layout is None else layout
    _check_layout(layout, hi, lo)
    C = ref.shape[1]
    N = mask.shape[0]
    hp = _empty((hi.shape[0], C, bs + 2, bs + 2), ref, layout)
    lp = _empty((lo.shape[0], C, bs // 2 + 2, bs // 2 + 2), ref, layout)
    if sampling not in _SAMPLING:
        raise ValueError(f"sampling must be one of {sorted(_SAMPLING)}")
    _b.call("segblocks_pad_ex", _ptr(hi), _ptr(lo), _dt(ref), layout, N, C, H, W, _ptr(mask), bs, _ptr(hp),
            _ptr(lp), hi.shape[0], lo.shape[0], _SAMPLING[sampling], _stream(ref))
    return hp, lp


def conv3x3(hp: torch.Tensor, lp: torch.Tensor, mask: torch.Tensor, bs: int, H: int, W: int,
            weight: torch.Tensor, bias=None, layout=None):
    """3x3 valid convolution of both padded stacks: returns (hi_out, lo_out)."""
    mask = _mask(mask)
    ref = hp if hp.shape[0] else lp
    layout = layout_of(ref) if layout is None else layout
    _check_layout(layout, hp, lp)
    C_in = ref.shape[1]
    C_out = weight.shape[0]
    N = mask.shape[0]
    weight = _weight(weight, layout)
    bias = None if bias is None else bias.contiguous()
    ho = _empty((hp.shape[0], C_out, bs, bs), ref, layout)
    lo = _empty((lp.shape[0], C_out, bs // 2, bs // 2), ref, layout)
    _b.call("segblocks_conv3x3", _ptr(hp), _ptr(lp), _dt(ref), layout, N, C_in, H, W, _ptr(mask), bs,
            _ptr(weight), _ptr(bias), C_out, _ptr(ho), _ptr(lo), hp.shape[0], lp.shape[0], _stream(ref))
    return ho, lo


def combine(hi: torch.Tensor, lo: torch.Tensor, mask: torch.Tensor, bs: int, H: int, W: int, layout=None,
            out=None):
    """BlockCombine: returns y [N,C,H,W] with the low blocks nearest-upsampled."""
    mask = _mask(mask)
    ref = hi if hi.shape[0] else lo
    layout = layout_of(ref) if layout is None else layout
    _check_layout(layout, hi, lo)
    N, C = mask.shape[0], ref.shape[1]
    y = _empty((N, C, H, W), ref, layout) if out is None else out
    _b.call("segblocks_combine", _ptr(hi), _ptr(lo), _dt(ref), layout, N, C, H, W, _ptr(mask), bs, hi.shape[0],
            lo.shape[0], _ptr(y), _stream(ref))
    return y


def block_conv3x3(hi: torch.Tensor, lo: torch.Tensor, mask: torch.Tensor, bs: int, H: int, W: int,
                  weight: torch.Tensor, bias=None, relu: bool = False, residual=None, layout=None, out=None,
                  workspace=None, sampling: str = "avg"):
    """3x3 block convolution with BlockPad fused into the tile load (packed in,
    packed out); optional epilogue act(conv + bias + residual).  ``workspace``:
    a uint8 tensor of at least block_conv3x3_workspace_size() + 256 bytes, or
    None (one is taken from torch's allocator when the call needs one)."""
    mask = _mask(mask)
    ref = hi if hi.shape[0] else lo
    layout = layout_of(ref) if layout is None else layout
    _check_layout(layout, hi, lo)
    C_in, C_out, N = ref.shape[1], weight.shape[0], mask.shape[0]
    weight = _weight(weight, layout)
    bias = None if bias is None else bias.contiguous()
    if out is None:
        ho = _empty((hi.shape[0], C_out, bs, bs), ref, layout)
        lo_o = _empty((lo.shape[0], C_out, bs // 2, bs // 2), ref, layout)
    else:
        ho, lo_o = out
    rh, rl = (None, None) if residual is None else residual
    need = block_conv3x3_workspace_size(ref.dtype, layout, N, C_in, H, W, bs, C_out, hi.shape[0], lo.shape[0])
    wp, wn, _keep = _ws(need, ref.device, workspace)
    _b.call("segblocks_block_conv3x3", _ptr(hi), _ptr(lo), _dt(ref), layout, N, C_in, H, W, _ptr(mask), bs,
            _ptr(weight), _ptr(bias), C_out, _flags(relu, sampling), _ptr(rh), _ptr(rl), _ptr(ho),
            _ptr(lo_o), hi.shape[0], lo.shape[0], wp, wn, _stream(ref))
    return ho, lo_o


def layer(x: torch.Tensor, mask: torch.Tensor, bs: int, weight: torch.Tensor, bias=None, layout=None, out=None,
          workspace=None, relu: bool = False, sampling: str = "avg"):
    """One block-conv layer: combine(conv3x3(pad(split(x)))), fused (see
    segblocks_layer for the routes).  ``workspace`` as in block_conv3x3, sized
    by layer_workspace_size()."""
    mask = _mask(mask)
    layout = layout_of(x) if layout is None else layout
    _check_layout(layout, x)
    N, C_in, H, W = x.shape
    C_out = weight.shape[0]
    weight = _weight(weight, layout)
    bias = None if bias is None else bias.contiguous()
    y = _empty((N, C_out, H, W), x, layout) if out is None else out
    need = layer_workspace_size(x.dtype, layout, N, C_in, H, W, bs, C_out)
    wp, wn, _keep = _ws(need, x.device, workspace)
    _b.call("segblocks_layer", _ptr(x), _dt(x), layout, N, C_in, H, W, _ptr(mask), bs, _ptr(weight), _ptr(bias),
            C_out, _flags(relu, sampling), _ptr(y), wp, wn, _stream(x))
    return y


def block_conv_ex(hi: torch.Tensor, lo: torch.Tensor, mask: torch.Tensor, bs: int, H: int, W: int,
                  weight: torch.Tensor, bias=None, stride: int = 1, relu: bool = False, residual=None, out=None,
                  workspace=None, sampling: str = "avg"):
    """K x K block convolution (K = weight.shape[2], 1 or 3) at `stride` (1 or
    2) of channels-last packed stacks, BlockPad fused, epilogue
    act(conv + bias + residual); outputs have block sides bs/stride and
    bs/(2 stride).  H, W, bs describe the input map.  ``workspace`` as in
    block_conv3x3, sized by block_conv_ex_workspace_size()."""
    mask = _mask(mask)
    ref = hi if hi.shape[0] else lo
    layout = _b.SB_NHWC
    _check_layout(layout, hi, lo)
    k = weight.shape[2]
    C_in, C_out, N = ref.shape[1], weight.shape[0], mask.shape[0]
    weight = _weight(weight, layout, k)
    bias = None if bias is None else bias.contiguous()
    bo, lo_e = bs // stride, bs // 2 // stride
    if out is None:
        ho = _empty((hi.shape[0], C_out, bo, bo), ref, layout)
        lo_o = _empty((lo.shape[0], C_out, lo_e, lo_e), ref, layout)
    else:
        ho, lo_o = out
    rh, rl = (None, None) if residual is None else residual
    need = block_conv_ex_workspace_size(ref.dtype, N, C_in, H, W, bs, C_out, k, stride, hi.shape[0], lo.shape[0])
    wp, wn, _keep = _ws(need, ref.device, workspace)
    _b.call("segblocks_block_conv_ex", _ptr(hi), _ptr(lo), _dt(ref), layout, N, C_in, H, W, _ptr(mask), bs,
            _ptr(weight), _ptr(bias), C_out, k, stride, _flags(relu, sampling), _ptr(rh), _ptr(rl),
            _ptr(ho), _ptr(lo_o), hi.shape[0], lo.shape[0], wp, wn, _stream(ref))
    return ho, lo_o


def block_conv_chain_reads_half(dtype: torch.dtype, N: int, C_in: int, H: int, W: int, bs: int, C_out: int, k: int,
                                stride: int, hi_cap: int, lo_cap: int, sampling: str = "avg") -> bool:
    """Whether block_conv_chain with these shapes reads ``hi_half`` (so that
    the call producing its input knows whether to ask for it)."""
    r = ctypes.c_int(0)
    _b.call("segblocks_block_conv_chain_reads_half", _DT[dtype], _b.SB_NHWC, N, C_in, H, W, bs, C_out, k, stride,
            _flags(False, sampling), hi_cap, lo_cap, ctypes.byref(r))
    return bool(r.value)


def block_conv_chain(hi: torch.Tensor, lo: torch.Tensor, mask: torch.Tensor, bs: int, H: int, W: int,
                     weight: torch.Tensor, bias=None, stride: int = 1, relu: bool = False, residual=None,
                     hi_half=None, want_half: bool = False, out=None, workspace=None, sampling: str = "avg"):
    """block_conv_ex for chains of block convolutions: ``hi_half`` (or None)
    is ``hi`` at half resolution (each block's 2x2 averages, as a previous
    call's third result), from which the implicit GEMM takes a low block's
    halo cells beside a high neighbour instead of padding the low stack in a
    launch of its own; with ``want_half`` the call also returns the high
    output at half resolution.  3x3 at stride 1 takes the routes of
    block_conv3x3.  Returns (hi_out, lo_out, hi_out_half or None)."""
    mask = _mask(mask)
    ref = hi if hi.shape[0] else lo
    layout = _b.SB_NHWC
    _check_layout(layout, hi, lo)
    k = weight.shape[2]
    C_in, C_out, N = ref.shape[1], weight.shape[0], mask.shape[0]
    weight = _weight(weight, layout, k)
    bias = None if bias is None else bias.contiguous()
    bo, lo_e = bs // stride, bs // 2 // stride
    if out is None:
        ho = _empty((hi.shape[0], C_out, bo, bo), ref, layout)
        lo_o = _empty((lo.shape[0], C_out, lo_e, lo_e), ref, layout)
        hh = _empty((hi.shape[0], C_out, bo // 2, bo // 2), ref, layout) if want_half else None
    else:
        ho, lo_o, hh = out
    rh, rl = (None, None) if residual is None else residual
    need = block_conv_chain_workspace_size(ref.dtype, N, C_in, H, W, bs, C_out, k, stride, hi.shape[0], lo.shape[0])
    wp, wn, _keep = _ws(need, ref.device, workspace)
    _b.call("segblocks_block_conv_chain", _ptr(hi), _ptr(lo), _ptr(hi_half), _dt(ref), layout, N, C_in, H, W,
            _ptr(mask), bs, _ptr(weight), _ptr(bias), C_out, k, stride, _flags(relu, sampling), _ptr(rh), _ptr(rl),
            _ptr(ho), _ptr(lo_o), _ptr(hh), hi.shape[0], lo.shape[0], wp, wn, _stream(ref))
    return ho, lo_o, hh


def conv2d(x: torch.Tensor, weight: torch.Tensor, bias=None, stride: int = 1, padding: int = 0,
           relu: bool = False, out=None):
    """Dense K x K convolution of a channels-last map with zero padding (the
    encoder's stem), bias and optional ReLU."""
    layout = _b.SB_NHWC
    _check_layout(layout, x)
    N, C_in, H, W = x.shape
    k = weight.shape[2]
    weight = _weight(weight, layout, k)
    bias = None if bias is None else bias.contiguous()
    C_out = weight.shape[0]
    Ho, Wo = (H + 2 * padding - k) // stride + 1, (W + 2 * padding - k) // stride + 1
    y = _empty((N, C_out, Ho, Wo), x, layout) if out is None else out
    _b.call("segblocks_conv2d", _ptr(x), _dt(x), layout, N, C_in, H, W, _ptr(weight), _ptr(bias), C_out, k,
            stride, padding, _b.SB_FLAG_RELU if relu else 0, _ptr(y), _stream(x))
    return y


def maxpool(x: torch.Tensor, k: int = 3, stride: int = 2, padding: int = 1, out=None):
    """k x k max-pooling of a channels-last map at `stride` with `padding`."""
    layout = _b.SB_NHWC
    _check_layout(layout, x)
    N, C, H, W = x.shape
    Ho, Wo = (H + 2 * padding - k) // stride + 1, (W + 2 * padding - k) // stride + 1
    y = _empty((N, C, Ho, Wo), x, layout) if out is None else out
    _b.call("segblocks_maxpool", _ptr(x), _dt(x), layout, N, C, H, W, k, stride, padding, _ptr(y), _stream(x))
    return y


def policy_heuristic(x: torch.Tensor, bs: int, tau_high: float, layout=None, out=None):
    """Heuristic downsampling policy: returns (mask [N, H/bs, W/bs] uint8,
    1 = high resolution, score [N, H/bs, W/bs] float32).  Per image the
    round(tau_high * blocks) blocks whose low-resolution version loses the
    most detail are high resolution."""
    layout = layout_of(x) if layout is None else layout
    _check_layout(layout, x)
    N, C, H, W = x.shape
    if H % bs or W % bs:
        raise ValueError("bs must divide H and W")
    if out is None:
        mask = torch.empty((N, H // bs, W // bs), dtype=torch.uint8, device=x.device)
        score = torch.empty((N, H // bs, W // bs), dtype=torch.float32, device=x.device)
    else:
        mask, score = out
    _b.call("segblocks_policy_heuristic", _ptr(x), _dt(x), layout, N, C, H, W, bs, float(tau_high), _ptr(score),
            _ptr(mask), _stream(x))
    return mask, score


# ---------------------------------------------------------------------------
# Backward pass
# ---------------------------------------------------------------------------

def combine_backward(dy: torch.Tensor, mask: torch.Tensor, bs: int, counts=None, layout=None):
    """BlockCombine transposed: dy [N,C,H,W] -> (dhi, dlo)."""
    mask = _mask(mask)
    layout = layout_of(dy) if layout is None else layout
    _check_layout(layout, dy)
    N, C, H, W = dy.shape
    nh, nl = counts if counts is not None else count(mask)
    dhi = _empty((nh, C, bs, bs), dy, layout)
    dlo = _empty((nl, C, bs // 2, bs // 2), dy, layout)
    _b.call("segblocks_combine_backward", _ptr(dy), _dt(dy), layout, N, C, H, W, _ptr(mask), bs, _ptr(dhi), nh,
            _ptr(dlo), nl, _stream(dy))
    return dhi, dlo


def split_backward(dhi: torch.Tensor, dlo: torch.Tensor, mask: torch.Tensor, bs: int, H: int, W: int, layout=None):
    """BlockSample transposed: (dhi, dlo) -> dx [N,C,H,W]."""
    mask = _mask(mask)
    ref = dhi if dhi.shape[0] else dlo
    layout = layout_of(ref) if layout is None else layout
    _check_layout(layout, dhi, dlo)
    N, C = mask.shape[0], ref.shape[1]
    dx = _empty((N, C, H, W), ref, layout)
    _b.call("segblocks_split_backward", _ptr(dhi), _ptr(dlo), _dt(ref), layout, N, C, H, W, _ptr(mask), bs,
            dhi.shape[0], dlo.shape[0], _ptr(dx), _stream(ref))
    return dx


def pad_backward(dhp: torch.Tensor, dlp: torch.Tensor, mask: torch.Tensor, bs: int, H: int, W: int, layout=None,
                 sampling: str = "avg"):
    """BlockPad transposed: (dhp, dlp) -> (dhi, dlo)."""
    mask = _mask(mask)
    ref = dhp if dhp.shape[0] else dlp
    layout = layout_of(ref) if layout is None else layout
    _check_layout(layout, dhp, dlp)
    N, C = mask.shape[0], ref.shape[1]
    dhi = _empty((dhp.shape[0], C, bs, bs), ref, layout)
    dlo = _empty((dlp.shape[0], C, bs // 2, bs // 2), ref, layout)
    _b.call("segblocks_pad_backward", _ptr(dhp), _ptr(dlp), _dt(ref), layout, N, C, H, W, _ptr(mask), bs,
            _SAMPLING[sampling], _ptr(dhi), _ptr(dlo), dhp.shape[0], dlp.shape[0], _stream(ref))
    return dhi, dlo


def conv3x3_backward_data(dho: torch.Tensor, dlo: torch.Tensor, mask: torch.Tensor, bs: int, H: int, W: int,
                          weight: torch.Tensor, layout=None, workspace=None):
    """Gradient of the padded-stack convolution with respect to its input: (dhp, dlp)."""
    mask = _mask(mask)
    ref = dho if dho.shape[0] else dlo
    layout = layout_of(ref) if layout is None else layout
    _check_layout(layout, dho, dlo)
    C_out, C_in = weight.shape[0], weight.shape[1]
    N = mask.shape[0]
    weight = _weight(weight, layout)
    dhp = _empty((dho.shape[0], C_in, bs + 2, bs + 2), ref, layout)
    dlp = _empty((dlo.shape[0], C_in, bs // 2 + 2, bs // 2 + 2), ref, layout)
    need = _query("segblocks_conv3x3_backward_data_workspace_size", _DT[ref.dtype], layout, N, C_in, H, W, bs, C_out,
                  dho.shape[0], dlo.shape[0])
    wp, wn, _keep = _ws(need, ref.device, workspace)
    _b.call("segblocks_conv3x3_backward_data", _ptr(dho), _ptr(dlo), _dt(ref), layout, N, C_in, H, W, _ptr(mask), bs,
            _ptr(weight), C_out, _ptr(dhp), _ptr(dlp), dho.shape[0], dlo.shape[0], wp, wn, _stream(ref))
    return dhp, dlp


def conv3x3_backward_weight(hp: torch.Tensor, lp: torch.Tensor, dho: torch.Tensor, dlo: torch.Tensor,
                            mask: torch.Tensor, bs: int, H: int, W: int, bias: bool = True, layout=None,
                            workspace=None):
    """Gradients of the padded-stack convolution with respect to its weight
    (OIHW logical shape, in the call's memory format) and bias: (dw, db)."""
    mask = _mask(mask)
    ref = dho if dho.shape[0] else dlo
    pref = hp if hp.shape[0] else lp
    layout = layout_of(ref) if layout is None else layout
    _check_layout(layout, hp, lp, dho, dlo)
    C_out, C_in, N = ref.shape[1], pref.shape[1], mask.shape[0]
    dw = torch.empty((C_out, C_in, 3, 3), dtype=ref.dtype, device=ref.device, memory_format=_fmt(layout))
    db = torch.empty((C_out,), dtype=ref.dtype, device=ref.device) if bias else None
    need = _query("segblocks_conv3x3_backward_weight_workspace_size", _DT[ref.dtype], layout, N, C_in, H, W, bs,
                  C_out, hp.shape[0], lp.shape[0], 1 if bias else 0)
    wp, wn, _keep = _ws(need, ref.device, workspace)
    _b.call("segblocks_conv3x3_backward_weight", _ptr(hp), _ptr(lp), _ptr(dho), _ptr(dlo), _dt(ref), layout, N, C_in,
            H, W, _ptr(mask), bs, C_out, _ptr(dw), _ptr(db), hp.shape[0], lp.shape[0], wp, wn, _stream(ref))
    return dw, db


def layer_backward(x: torch.Tensor, mask: torch.Tensor, bs: int, weight: torch.Tensor, dy: torch.Tensor,
                   bias: bool = True, sampling: str = "avg"):
    """Gradients (dx, dw, db) of y = layer(x) for an output gradient dy: the
    forward stacks are recomputed (split, pad), then combine, convolution,
    pad and split are run transposed.  Every step is a library call."""
    layout = layout_of(x)
    N, C, H, W = x.shape
    nh, nl = count(mask)
    hi, lo = split(x, mask, bs, counts=(nh, nl))
    hp, lp = pad(hi, lo, mask, bs, H, W, sampling=sampling)
    dho, dlo_o = combine_backward(dy, mask, bs, counts=(nh, nl), layout=layout)
    dw, db = conv3x3_backward_weight(hp, lp, dho, dlo_o, mask, bs, H, W, bias=bias, layout=layout)
    dhp, dlp = conv3x3_backward_data(dho, dlo_o, mask, bs, H, W, weight, layout=layout)
    dhi, dlo = pad_backward(dhp, dlp, mask, bs, H, W, layout=layout, sampling=sampling)
    return split_backward(dhi, dlo, mask, bs, H, W, layout=layout), dw, db


# ---------------------------------------------------------------------------
# Wider halos: layers beyond 3x3 on block stacks
# ---------------------------------------------------------------------------

def pad_halo(hi: torch.Tensor, lo: torch.Tensor, mask: torch.Tensor, bs: int, H: int, W: int, halo: int,
             layout=None, sampling: str = "avg"):
    """BlockPad with a halo of `halo` pixels: (hi_pad, lo_pad)."""
    mask = _mask(mask)
    ref = hi if hi.shape[0] else lo
    layout = layout_of(ref) if layout is None else layout
    _check_layout(layout, hi, lo)
    C, N = ref.shape[1], mask.shape[0]
    hp = _empty((hi.shape[0], C, bs + 2 * halo, bs + 2 * halo), ref, layout)
    lp = _empty((lo.shape[0], C, bs // 2 + 2 * halo, bs // 2 + 2 * halo), ref, layout)
    _b.call("segblocks_pad_halo", _ptr(hi), _ptr(lo), _dt(ref), layout, N, C, H, W, _ptr(mask), bs, halo,
            _SAMPLING[sampling], _ptr(hp), _ptr(lp), hi.shape[0], lo.shape[0], _stream(ref))
    return hp, lp


def conv_halo(hp: torch.Tensor, lp: torch.Tensor, mask: torch.Tensor, bs: int, H: int, W: int, halo: int,
              weight: torch.Tensor, bias=None, stride: int = 1, dilation: int = 1, relu: bool = False, layout=None):
    """K x K (K = weight.shape[2], odd) convolution at `stride` / `dilation` of
    stacks padded by `halo`: (hi_out, lo_out) with sides bs/stride, bs/(2 stride)."""
    mask = _mask(mask)
    ref = hp if hp.shape[0] else lp
    layout = layout_of(ref) if layout is None else layout
    _check_layout(layout, hp, lp)
    k = weight.shape[2]
    C_in, C_out, N = ref.shape[1], weight.shape[0], mask.shape[0]
    weight = _weight(weight, layout, k)
    bias = None if bias is None else bias.contiguous()
    ho = _empty((hp.shape[0], C_out, bs // stride, bs // stride), ref, layout)
    lo = _empty((lp.shape[0], C_out, bs // 2 // stride, bs // 2 // stride), ref, layout)
    _b.call("segblocks_conv_halo", _ptr(hp), _ptr(lp), _dt(ref), layout, N, C_in, H, W, _ptr(mask), bs, halo,
            _ptr(weight), _ptr(bias), C_out, k, stride, dilation, _b.SB_FLAG_RELU if relu else 0, _ptr(ho), _ptr(lo),
            hp.shape[0], lp.shape[0], _stream(ref))
    return ho, lo


def maxpool_halo(hp: torch.Tensor, lp: torch.Tensor, mask: torch.Tensor, bs: int, H: int, W: int, halo: int,
                 k: int = 3, stride: int = 2, layout=None):
    """k x k max-pooling at `stride` of stacks padded by `halo`: (hi_out, lo_out)."""
    mask = _mask(mask)
    ref = hp if hp.shape[0] else lp
    layout = layout_of(ref) if layout is None else layout
    _check_layout(layout, hp, lp)
    C, N = ref.shape[1], mask.shape[0]
    ho = _empty((hp.shape[0], C, bs // stride, bs // stride), ref, layout)
    lo = _empty((lp.shape[0], C, bs // 2 // stride, bs // 2 // stride), ref, layout)
    _b.call("segblocks_maxpool_halo", _ptr(hp), _ptr(lp), _dt(ref), layout, N, C, H, W, _ptr(mask), bs, halo, k,
            stride, _ptr(ho), _ptr(lo), hp.shape[0], lp.shape[0], _stream(ref))
    return ho, lo
