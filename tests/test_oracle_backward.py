"""Pins of the oracle's backward pass: every transposed module, the
convolution's data and weight gradients and the whole layer's gradients
against torch.autograd of independent float64 library forms (the combined
map, windows of the zero-padded map and of its pool, F.conv2d, and the
layer's closed form), plus the adjoint identity <A u, v> = <u, A^T v> for
BlockPad."""
from __future__ import annotations

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from paper_2011_12025_amd import inputs

DTYPES = ["f32", "f16", "bf16"]
ULP = {"f32": 2.0 ** -23, "f16": 2.0 ** -10, "bf16": 2.0 ** -7}


def _t(a):
    return torch.tensor(np.asarray(a, np.float64), requires_grad=True)


def _x(seed, shape, dtype):
    return inputs.normal(seed, 7, shape, 1.0, dtype).float().numpy()


def combine_t(hi, lo, mask, bs, H, W):
    """Differentiable BlockCombine: high blocks copied, low blocks nearest-upsampled."""
    N, GH, GW = mask.shape
    m = torch.from_numpy(mask.reshape(-1) != 0)
    C = hi.shape[1] if hi.shape[0] else lo.shape[1]
    idx_h = torch.nonzero(m).reshape(-1)
    idx_l = torch.nonzero(~m).reshape(-1)
    blocks = torch.zeros((N * GH * GW, C, bs, bs), dtype=torch.float64)
    blocks = blocks.index_add(0, idx_h, hi)
    blocks = blocks.index_add(0, idx_l, lo.repeat_interleave(2, -2).repeat_interleave(2, -1))
    return blocks.view(N, GH, GW, C, bs, bs).permute(0, 3, 1, 4, 2, 5).reshape(N, C, H, W)


def windows_t(zp, e, GH, GW):
    """(e+2)x(e+2) windows at stride e of a 1-px zero-padded map -> [N*GH*GW, C, e+2, e+2]."""
    N, C = zp.shape[:2]
    rows = [zp[:, :, gy * e:gy * e + e + 2, :] for gy in range(GH)]
    out = []
    for gy in range(GH):
        for gx in range(GW):
            out.append(rows[gy][:, :, :, gx * e:gx * e + e + 2])
    return torch.stack(out, 1).reshape(N * GH * GW, C, e + 2, e + 2)


def pad_t(hi, lo, mask, bs, H, W, sampling):
    N, GH, GW = mask.shape
    m = torch.from_numpy(mask.reshape(-1) != 0)
    if sampling == "zero":
        return F.pad(hi, (1, 1, 1, 1)), F.pad(lo, (1, 1, 1, 1))
    Z = combine_t(hi, lo, mask, bs, H, W)
    small = F.avg_pool2d(Z, 2) if sampling == "avg" else Z[..., ::2, ::2]
    hw = windows_t(F.pad(Z, (1, 1, 1, 1)), bs, GH, GW)
    lw = windows_t(F.pad(small, (1, 1, 1, 1)), bs // 2, GH, GW)
    return hw[m], lw[~m]


def _stacks(seed, N, C, GH, GW, bs, dtype, p=0.5):
    mask = inputs.mask_bernoulli(seed, N, GH, GW, p)
    nh = int(mask.sum())
    nl = mask.size - nh
    hi = _x(seed + 1, (nh, C, bs, bs), dtype)
    lo = _x(seed + 2, (nl, C, bs // 2, bs // 2), dtype)
    return mask, hi, lo


def _within_ulps(got, ref, dtype, n=1):
    return np.all(np.abs(got - ref) <= n * ULP[dtype] * np.abs(ref) + 1e-30)


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("bs", [2, 4, 6])
def test_combine_backward_is_autograd_of_combine(dtype, bs):
    N, C, GH, GW = 2, 3, 3, 4
    mask, hi, lo = _stacks(70, N, C, GH, GW, bs, dtype)
    dy = _x(71, (N, C, GH * bs, GW * bs), dtype)
    th, tl = _t(hi), _t(lo)
    combine_t(th, tl, mask, bs, GH * bs, GW * bs).backward(torch.from_numpy(dy.astype(np.float64)))
    ah, al = _t(hi), _t(lo)                       # the same map of |dy|: the scale of the fp32 sums
    combine_t(ah, al, mask, bs, GH * bs, GW * bs).backward(torch.from_numpy(np.abs(dy).astype(np.float64)))
    dhi, dlo = oracle.combine_backward(dy, mask, bs, dtype)
    np.testing.assert_array_equal(dhi, th.grad.numpy())
    ref = tl.grad.numpy()
    # fp32 sum of four terms (two roundings of the partial sums at most), then one rounding to the storage type
    assert np.all(np.abs(dlo - ref) <= ULP[dtype] * np.abs(ref) + 3 * 2.0 ** -24 * al.grad.numpy() + 1e-30)
    if dtype == "f32":
        assert np.mean(dlo == ref.astype(np.float32)) > 0.5


@pytest.mark.parametrize("dtype", DTYPES)
def test_split_backward_is_autograd_of_split(dtype):
    N, C, GH, GW, bs = 2, 3, 3, 4, 4
    mask = inputs.mask_bernoulli(72, N, GH, GW, 0.5)
    x = _x(73, (N, C, GH * bs, GW * bs), dtype)
    tx = _t(x)
    blocks = tx.view(N, C, GH, bs, GW, bs).permute(0, 2, 4, 1, 3, 5).reshape(N * GH * GW, C, bs, bs)
    m = torch.from_numpy(mask.reshape(-1) != 0)
    hi, lo = blocks[m], F.avg_pool2d(blocks[~m], 2)
    dhi = _x(74, tuple(hi.shape), dtype)
    dlo = _x(75, tuple(lo.shape), dtype)
    torch.autograd.backward([hi, lo], [torch.from_numpy(dhi.astype(np.float64)),
                                       torch.from_numpy(dlo.astype(np.float64))])
    got = oracle.split_backward(dhi, dlo, mask, bs, GH * bs, GW * bs, dtype)
    np.testing.assert_array_equal(got, tx.grad.numpy().astype(np.float32))


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("sampling", ["avg", "strided", "zero"])
@pytest.mark.parametrize("bs", [2, 4, 8])
def test_pad_backward_is_autograd_of_pad(dtype, sampling, bs):
    N, C, GH, GW = 2, 3, 3, 5
    H, W = GH * bs, GW * bs
    for p in [0.0, 0.4, 1.0]:
        mask, hi, lo = _stacks(76, N, C, GH, GW, bs, dtype, p)
        th, tl = _t(hi), _t(lo)
        hp, lp = pad_t(th, tl, mask, bs, H, W, sampling)
        dhp = _x(77, tuple(hp.shape), dtype)
        dlp = _x(78, tuple(lp.shape), dtype)
        torch.autograd.backward([hp, lp], [torch.from_numpy(dhp.astype(np.float64)),
                                           torch.from_numpy(dlp.astype(np.float64))])
        dhi, dlo = oracle.pad_backward(dhp, dlp, mask, bs, H, W, dtype, sampling)
        rh = th.grad.numpy() if th.grad is not None else np.zeros(hi.shape)
        rl = tl.grad.numpy() if tl.grad is not None else np.zeros(lo.shape)
        # the oracle rounds its fp64 sums once: within half an ulp of the storage type
        assert _within_ulps(dhi, rh, dtype), (sampling, p)
        assert _within_ulps(dlo, rl, dtype), (sampling, p)


def test_pad_backward_adjoint_identity():
    """<pad(u), v> = <u, pad^T(v)> for random u, v (fp32 storage, the 2x2
    average's rounding aside)."""
    N, C, GH, GW, bs = 1, 2, 4, 4, 4
    mask, hi, lo = _stacks(79, N, C, GH, GW, bs, "f32")
    hp, lp = oracle.pad(hi, lo, mask, bs, GH * bs, GW * bs, "f32")
    vh = _x(80, hp.shape, "f32")
    vl = _x(81, lp.shape, "f32")
    dhi, dlo = oracle.pad_backward(vh, vl, mask, bs, GH * bs, GW * bs, "f32")
    lhs = np.sum(hp.astype(np.float64) * vh) + np.sum(lp.astype(np.float64) * vl)
    rhs = np.sum(hi.astype(np.float64) * dhi) + np.sum(lo.astype(np.float64) * dlo)
    assert abs(lhs - rhs) <= 1e-5 * (abs(lhs) + 1.0)


def test_conv_backward_matches_autograd():
    g = np.random.default_rng(82)
    P = g.standard_normal((3, 5, 8, 8)).astype(np.float32)
    w = g.standard_normal((4, 5, 3, 3)).astype(np.float32)
    dO = g.standard_normal((3, 4, 6, 6)).astype(np.float32)
    tP, tw, tb = _t(P), _t(w), _t(np.zeros(4))
    F.conv2d(tP, tw, tb).backward(torch.from_numpy(dO.astype(np.float64)))
    np.testing.assert_allclose(oracle.conv3x3_backward_data(dO, w), tP.grad.numpy(), rtol=1e-12, atol=1e-12)
    dw, db = oracle.conv3x3_backward_weight([(P[:2], dO[:2]), (P[2:], dO[2:])])
    np.testing.assert_allclose(dw, tw.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(db, tb.grad.numpy(), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("sampling", ["avg", "strided", "zero"])
def test_layer_backward_is_autograd_of_closed_form(dtype, sampling):
    """The whole layer: autograd of the float64 library form (split as
    crops and avg_pool2d, BlockPad as windows of the padded combined map,
    F.conv2d per stack, BlockCombine) against the oracle's chain, which
    rounds every stored gradient."""
    N, C, Co, GH, GW, bs = 2, 4, 3, 3, 4, 6
    H, W = GH * bs, GW * bs
    mask = inputs.mask_bernoulli(83, N, GH, GW, 0.5)
    x = _x(84, (N, C, H, W), dtype)
    w = _x(85, (Co, C, 3, 3), dtype) * np.float32(1 / 6)
    w = oracle.round_to(w, dtype)
    b = _x(86, (Co,), dtype)
    dy = _x(87, (N, Co, H, W), dtype)
    tx, tw, tb = _t(x), _t(w), _t(b)
    blocks = tx.view(N, C, GH, bs, GW, bs).permute(0, 2, 4, 1, 3, 5).reshape(N * GH * GW, C, bs, bs)
    m = torch.from_numpy(mask.reshape(-1) != 0)
    hi, lo = blocks[m], F.avg_pool2d(blocks[~m], 2)
    hp, lp = pad_t(hi, lo, mask, bs, H, W, sampling)
    y = combine_t(F.conv2d(hp, tw, tb), F.conv2d(lp, tw, tb), mask, bs, H, W)
    y.backward(torch.from_numpy(dy.astype(np.float64)))
    dx, dw, db = oracle.layer_backward(x, mask, bs, w, b, dy, dtype, sampling)
    tol = {"f32": 1e-5, "f16": 1e-2, "bf16": 6e-2}[dtype]
    for got, ref in [(dx, tx.grad.numpy()), (dw, tw.grad.numpy()), (db, tb.grad.numpy())]:
        assert np.max(np.abs(got - ref)) <= tol * np.max(np.abs(ref))
