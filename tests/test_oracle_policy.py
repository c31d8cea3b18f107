"""Pins of the oracle's heuristic downsampling policy (a block's score is the
average, over its pixels, of the Euclidean distance across channels between
the block and its low-resolution version; per image the highest-scoring
fraction tau of the blocks is processed at high resolution) against numpy
library operations, exact special cases and a sort-based selection."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from oracle_closed_forms import pool_f32, up2
from paper_2011_12025_amd import inputs

DTYPES = ["f32", "f16", "bf16"]


def closed_scores(x: np.ndarray, bs: int, dtype: str) -> np.ndarray:
    """Vectorised library form: up2(pool(x)) with the BlockSample average, the
    channel norm of the difference, block means."""
    d = x.astype(np.float64) - up2(pool_f32(x, dtype)).astype(np.float64)
    dist = np.sqrt(np.sum(d * d, axis=1))                 # [N, H, W]
    N, H, W = dist.shape
    return dist.reshape(N, H // bs, bs, W // bs, bs).mean(axis=(2, 4))


def sort_select(scores: np.ndarray, k: int) -> np.ndarray:
    N, GH, GW = scores.shape
    out = np.zeros((N, GH * GW), np.uint8)
    for n in range(N):
        s = scores[n].reshape(-1)
        order = np.lexsort((np.arange(s.size), -s))      # highest first, then lower block id
        out[n, order[:k]] = 1
    return out.reshape(N, GH, GW)


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("bs", [2, 4, 8])
def test_scores_match_library_form(dtype, bs):
    x = inputs.feature_map(60, 2, 3, 4 * bs, 6 * bs, dtype).float().numpy()
    got = oracle.policy_scores(x, bs, dtype)
    ref = closed_scores(x, bs, dtype)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-14)


def test_scores_zero_exactly_when_nothing_is_lost():
    """A map constant on every 2x2 cell loses nothing at half resolution."""
    g = np.random.default_rng(61)
    small = g.standard_normal((1, 4, 8, 12)).astype(np.float32)
    x = up2(small)
    np.testing.assert_array_equal(oracle.policy_scores(x, 4, "f32"), np.zeros((1, 4, 6)))


def test_detail_raises_the_score():
    """Fine texture added to one block makes it the top-ranked block."""
    g = np.random.default_rng(62)
    x = up2(g.standard_normal((1, 3, 8, 8)).astype(np.float32))     # smooth: every score 0
    x[0, :, 4:8, 8:12] += np.where((np.add.outer(np.arange(4), np.arange(4)) % 2) == 0, 1.0, -1.0)
    sc = oracle.policy_scores(x, 4, "f32")
    assert np.unravel_index(np.argmax(sc), sc.shape) == (0, 1, 2)
    np.testing.assert_array_equal(oracle.policy_select(sc, 1 / 16), (sc > 0).astype(np.uint8))


def test_selection_matches_sort_with_ties():
    g = np.random.default_rng(63)
    sc = np.round(g.random((3, 5, 7)) * 4) / 4                       # many exact ties
    for tau in [0.0, 0.2, 0.4, 0.5, 0.77, 1.0]:
        k = oracle.policy_k(tau, 35)
        np.testing.assert_array_equal(oracle.policy_select(sc, tau), sort_select(sc, k))
        assert np.all(oracle.policy_select(sc, tau).reshape(3, -1).sum(1) == k)


def test_selection_nests_over_tau():
    sc = oracle.policy_scores(inputs.feature_map(64, 2, 3, 32, 64, "f16").float().numpy(), 8, "f16")
    prev = np.zeros(sc.shape, np.uint8)
    for tau in np.linspace(0, 1, 9):
        m = oracle.policy_select(sc, tau)
        assert np.all(m >= prev)
        prev = m
    assert np.all(prev == 1)


@pytest.mark.parametrize("dtype", DTYPES)
def test_policy_on_a_random_image(dtype):
    x = inputs.feature_map(65, 2, 3, 64, 128, dtype).float().numpy()
    mask, sc = oracle.policy(x, 16, 0.4, dtype)
    np.testing.assert_array_equal(mask, sort_select(closed_scores(x, 16, dtype), oracle.policy_k(0.4, 32)))
    assert mask.dtype == np.uint8 and mask.shape == (2, 4, 8)
