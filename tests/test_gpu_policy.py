"""GPU parity of the heuristic downsampling policy against the CPU oracle.

The score of a block is floating point (fp32 sums on the GPU, fp64 in the
oracle): it must lie within a relative 1e-4 of the oracle's.  The selection
is an integer decision taken from those scores, so it is checked in two
parts: the GPU mask must be exactly the selection rule applied to the GPU's
own scores (the rule: per image the round(tau * blocks) highest scores, ties
by block id), and it must equal the oracle's mask wherever the oracle's
score is not within the score tolerance of the selection threshold (only
blocks that near-tie at the threshold may differ)."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from parity_util import log
from paper_2011_12025_amd import inputs

pytestmark = pytest.mark.gpu

SCORE_RTOL = 1e-4


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2011_12025_amd._binding as b
    b.lib()


def _check(x_cpu: torch.Tensor, bs: int, tau: float, dtype: str, layout: str, name: str):
    import paper_2011_12025_amd as sb
    log(f"[policy] {name}: oracle ...")
    ref_mask, ref_sc = oracle.policy(x_cpu.float().numpy(), bs, tau, dtype)
    log(f"[policy] {name}: gpu")
    xd = x_cpu.cuda()
    xd = xd.contiguous(memory_format=torch.channels_last) if layout == "nhwc" else xd.contiguous()
    mask, sc = sb.policy_heuristic(xd, bs, tau)
    torch.cuda.synchronize()
    g_sc = sc.cpu().numpy().astype(np.float64)
    g_mask = mask.cpu().numpy()
    assert np.all(np.isfinite(g_sc))
    tol = SCORE_RTOL * np.abs(ref_sc) + 1e-6
    bad = np.abs(g_sc - ref_sc) > tol
    assert not bad.any(), f"{name}: score off at {np.argwhere(bad)[0]}: {g_sc[bad][0]} vs {ref_sc[bad][0]}"
    # (a) the GPU's mask is the selection rule applied to its own scores
    np.testing.assert_array_equal(g_mask, oracle.policy_select(g_sc, tau))
    # (b) it equals the oracle's mask except for near-ties at the threshold
    N = ref_sc.shape[0]
    k = oracle.policy_k(tau, ref_sc[0].size)
    for n in range(N):
        s = np.sort(ref_sc[n].reshape(-1))[::-1]
        if 0 < k < s.size:
            # the last selected and the first unselected score, widened by twice the score tolerance
            t = 2 * (SCORE_RTOL * s[k - 1] + 1e-6)
            near = (ref_sc[n] >= s[k] - t) & (ref_sc[n] <= s[k - 1] + t)
        else:
            near = np.zeros(ref_sc[n].shape, bool)
        diff = g_mask[n] != ref_mask[n]
        assert not np.any(diff & ~near), f"{name}: image {n} selection differs at {np.argwhere(diff & ~near)[0]}"
    assert np.all(g_mask.reshape(N, -1).sum(1) == k)


@pytest.mark.parametrize("dtype,layout,N,C,H,W,bs,tau,seed", [
    ("f16", "nhwc", 2, 3, 256, 512, 64, 0.4, 150),
    ("bf16", "nhwc", 1, 3, 256, 512, 128, 0.25, 151),
    ("f32", "nchw", 2, 16, 64, 96, 16, 0.5, 152),
    ("f16", "nchw", 1, 64, 64, 128, 8, 0.6, 153),
    ("f16", "nhwc", 3, 8, 32, 48, 2, 0.3, 154),          # 1x1 low pixels
    ("bf16", "nhwc", 1, 3, 128, 128, 16, 0.0, 155),     # nothing high
    ("f16", "nhwc", 1, 3, 128, 128, 16, 1.0, 156),      # everything high
])
def test_policy_matches_oracle(dtype, layout, N, C, H, W, bs, tau, seed):
    x = inputs.feature_map(seed, N, C, H, W, dtype)
    _check(x, bs, tau, dtype, layout, f"{dtype} {layout} {N}x{C}x{H}x{W} bs{bs} tau{tau}")


def test_policy_full_size_image():
    """The paper's setting: a 1024x2048 RGB image, 128-pixel blocks (8x16
    grid), tau = 0.4."""
    x = inputs.feature_map(157, 1, 3, 1024, 2048, "f16")
    _check(x, 128, 0.4, "f16", "nhwc", "full-size 1024x2048 block 128")


def test_policy_ties_rank_by_block_id():
    """A map constant on 2x2 cells scores 0 everywhere: every block ties, so
    the first k blocks in id order are high."""
    import paper_2011_12025_amd as sb
    g = np.random.default_rng(158)
    small = torch.from_numpy(g.standard_normal((1, 4, 16, 32)).astype(np.float32)).half()
    x = small.repeat_interleave(2, 2).repeat_interleave(2, 3).cuda().contiguous(memory_format=torch.channels_last)
    mask, sc = sb.policy_heuristic(x, 8, 0.3)
    torch.cuda.synchronize()
    assert torch.all(sc == 0)
    k = oracle.policy_k(0.3, 32)
    want = np.zeros(32, np.uint8)
    want[:k] = 1
    np.testing.assert_array_equal(mask.cpu().numpy().reshape(-1), want)
