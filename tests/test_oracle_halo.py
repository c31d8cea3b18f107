"""Pins of the oracle's wider halos and blockwise layers beyond 3x3: BlockPad
with a p-pixel halo against windows of the p-pixel zero-padded combined map
(and its pool), K x K strided / dilated block convolution and block
max-pooling against F.conv2d / F.max_pool2d, and the blockwise stem, which
with every block at high resolution is the ordinary stem bit for bit and
with every block at low resolution the stem of the pooled image."""
from __future__ import annotations

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from oracle_closed_forms import pool_f32, up2
from paper_2011_12025_amd import inputs

DTYPES = ["f32", "f16", "bf16"]


def windows_p(zp, e, p):
    v = np.lib.stride_tricks.sliding_window_view(zp, (e + 2 * p, e + 2 * p), axis=(2, 3))[:, :, ::e, ::e]
    return np.ascontiguousarray(v.transpose(0, 2, 3, 1, 4, 5))


def pad_halo_closed(Z, mask, bs, p, sampling, hi=None, lo=None):
    m = np.asarray(mask) != 0
    if sampling == "zero":
        pw = ((0, 0), (0, 0), (p, p), (p, p))
        return np.pad(hi, pw), np.pad(lo, pw)
    small = pool_f32(Z, "f32") if sampling == "avg" else Z[..., ::2, ::2]
    pw = ((0, 0), (0, 0), (p, p), (p, p))
    return windows_p(np.pad(Z, pw), bs, p)[m], windows_p(np.pad(small, pw), bs // 2, p)[~m]


@pytest.mark.parametrize("sampling", ["avg", "strided", "zero"])
@pytest.mark.parametrize("bs,p", [(4, 1), (4, 2), (6, 2), (8, 3), (8, 4)])
def test_pad_halo_closed_form(bs, p, sampling):
    N, C, GH, GW = 2, 3, 3, 4
    H, W = GH * bs, GW * bs
    x = inputs.feature_map(90, N, C, H, W, "f32").numpy()
    for q in [0.0, 0.5, 1.0]:
        mask = inputs.mask_bernoulli(91, N, GH, GW, q)
        hi, lo = oracle.split(x, mask, bs, "f32")
        hp, lp = oracle.pad_halo(hi, lo, mask, bs, H, W, "f32", p, sampling)
        Z = oracle.combine(hi, lo, mask, bs, H, W)
        rhp, rlp = pad_halo_closed(Z, mask, bs, p, sampling, hi, lo)
        np.testing.assert_array_equal(hp, rhp)
        np.testing.assert_array_equal(lp, rlp)
        if p == 1:
            ahp, alp = oracle.pad(hi, lo, mask, bs, H, W, "f32", sampling)
            np.testing.assert_array_equal(hp, ahp)
            np.testing.assert_array_equal(lp, alp)


@pytest.mark.parametrize("K,st,dl,p", [(7, 2, 1, 3), (3, 1, 2, 2), (5, 1, 1, 2), (3, 2, 1, 1), (1, 2, 1, 1),
                                       (3, 1, 3, 4)])
def test_conv_block_general_matches_library(K, st, dl, p):
    g = np.random.default_rng(92)
    E = 8
    P = g.standard_normal((3, 4, E + 2 * p, E + 2 * p)).astype(np.float32)
    w = g.standard_normal((5, 4, K, K)).astype(np.float32)
    b = g.standard_normal(5).astype(np.float32)
    got = oracle.conv_block_general(P, p, w, st, dl, b)
    o = p - dl * (K - 1) // 2
    ref = F.conv2d(torch.from_numpy(P[:, :, o:, o:]).double(), torch.from_numpy(w).double(),
                   torch.from_numpy(b).double(), stride=st, dilation=dl).numpy()[:, :, :E // st, :E // st]
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("k,st,p", [(3, 2, 1), (3, 1, 1), (5, 2, 2), (3, 2, 2)])
def test_maxpool_block_matches_library(k, st, p):
    g = np.random.default_rng(93)
    P = g.standard_normal((2, 3, 8 + 2 * p, 8 + 2 * p)).astype(np.float32)
    o = p - (k - 1) // 2
    ref = F.max_pool2d(torch.from_numpy(P[:, :, o:, o:]), k, st).numpy()[:, :, :8 // st, :8 // st]
    np.testing.assert_array_equal(oracle.maxpool_block(P, p, k, st), ref)


@pytest.mark.parametrize("dtype", DTYPES)
def test_blockwise_stem_all_high_is_the_dense_stem(dtype):
    """Every block high: BlockPad's halos are the neighbours' pixels (zeros at
    the border), so the blockwise 7x7/2 stem and 3x3/2 max-pool equal the
    dense ones bit for bit (post-ReLU zeros never exceed the window maximum)."""
    N, H, W, blk = 2, 64, 128, 32
    x = inputs.feature_map(94, N, 3, H, W, dtype).float().numpy()
    Wt = {k: v.float().numpy() for k, v in inputs.encoder_weights(94, dtype).items()}
    mask = np.ones((N, H // blk, W // blk), np.uint8)
    hi, lo = oracle.blockwise_stem(x, mask, blk, Wt["stem.w"], Wt["stem.b"], dtype)
    got = oracle.combine(hi, lo, mask, blk // 4, H // 4, W // 4)
    ref = oracle.maxpool(oracle.dense_conv(x, Wt["stem.w"], Wt["stem.b"], 2, 3, dtype, relu=True), 3, 2, 1)
    np.testing.assert_array_equal(got, ref)


def test_blockwise_stem_all_low_is_the_stem_of_the_pooled_image():
    N, H, W, blk = 1, 64, 64, 32
    x = inputs.feature_map(95, N, 3, H, W, "f32").float().numpy()
    Wt = {k: v.float().numpy() for k, v in inputs.encoder_weights(95, "f32").items()}
    mask = np.zeros((N, H // blk, W // blk), np.uint8)
    hi, lo = oracle.blockwise_stem(x, mask, blk, Wt["stem.w"], Wt["stem.b"], "f32")
    got = oracle.combine(hi, lo, mask, blk // 4, H // 4, W // 4)
    small = oracle.maxpool(oracle.dense_conv(pool_f32(x, "f32"), Wt["stem.w"], Wt["stem.b"], 2, 3, "f32", relu=True),
                           3, 2, 1)
    np.testing.assert_array_equal(got, up2(small))


def test_blockwise_encoder_all_high_is_the_dense_stem_encoder():
    N, H, W, blk = 1, 128, 256, 64
    x = inputs.feature_map(96, N, 3, H, W, "f16").float().numpy()
    Wt = {k: v.float().numpy() for k, v in inputs.encoder_weights(96, "f16").items()}
    mask = np.ones((N, H // blk, W // blk), np.uint8)
    np.testing.assert_array_equal(oracle.encoder_blockwise(x, mask, blk, Wt, "f16"),
                                  oracle.encoder(x, mask, blk, Wt, "f16"))
