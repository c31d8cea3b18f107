"""GPU parity: every entry point of libsegblocks.so against the CPU oracle on
the same seeded inputs.  split / pad / combine must be bit-exact; the
convolutions must meet the tolerance of the block-conv contract (1e-4 for
fp32, 2e-2 for fp16/bf16, max-norm relative) and an element-wise bound.

Cases span several tiles and ragged tails (channel counts that are not
multiples of the K chunk or of the 64-channel output tile, block sizes that
are not powers of two, bs = 2 where low blocks are single pixels, bs = 256,
all-high and all-low masks, batches of several images) in both memory
formats."""
from __future__ import annotations

import numpy as np
import pytest
import torch

from parity_util import (Case, assert_bitexact, assert_conv_close, log, make_inputs, oracle_stages, to_dev,
                         y64_from_stacks)

pytestmark = pytest.mark.gpu

CASES = [
    Case("cfg_fp32_64x64_bs16", "f32", 1, 16, 16, 64, 64, 16),     # the small fp32 parity configuration
    Case("c64_f16", "f16", 1, 64, 64, 64, 128, 32),
    Case("c64_bf16", "bf16", 1, 64, 64, 64, 128, 32),
    Case("ragged_f16", "f16", 2, 24, 40, 18, 30, 6, p_low=0.4, seed=1),
    Case("ragged_f32_nobias", "f32", 2, 20, 36, 24, 16, 8, p_low=0.6, bias=False, seed=2),
    Case("deep_bf16", "bf16", 1, 96, 136, 32, 32, 8, seed=3),
    Case("tiny_bs2_f16", "f16", 2, 8, 8, 8, 12, 2, seed=4),
    Case("bs64_f16", "f16", 1, 32, 32, 128, 128, 64, seed=5),
    Case("bs256_bf16", "bf16", 1, 16, 24, 256, 512, 256, p_low=0.5, seed=6),
    Case("allhigh_f16", "f16", 1, 16, 16, 32, 64, 16, mask_kind="high", seed=7),
    Case("alllow_bf16", "bf16", 1, 16, 16, 32, 64, 16, mask_kind="low", seed=8),
    Case("bs64_c64_bf16", "bf16", 1, 64, 64, 128, 192, 64, seed=14),
    Case("blocks1056_f16", "f16", 1, 8, 8, 1024, 1056, 32, seed=12),  # more than 1024 blocks
]
LAYOUTS = ["nchw", "nhwc"]
TDT = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}

_cache = {}


def prepared(c: Case):
    if c.name not in _cache:
        mask, x, w, b = make_inputs(c)
        _cache[c.name] = (mask, x, w, b, oracle_stages(c, mask, x, w, b))
    return _cache[c.name]


def up(a: np.ndarray, dtype: str, layout: str) -> torch.Tensor:
    return to_dev(torch.from_numpy(np.ascontiguousarray(a)).to(TDT[dtype]), layout)


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2011_12025_amd._binding as b
    b.lib()  # fails loudly if the library is missing


def _ids(cs):
    return [c.name for c in cs]


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("c", CASES, ids=_ids(CASES))
def test_split_pad_combine_bitexact(c, layout):
    import paper_2011_12025_amd as sb
    mask, x, w, b, ref = prepared(c)
    log(f"[split/pad/combine] {c.name} {layout} N={c.N} C={c.C} {c.H}x{c.W} bs={c.bs}")
    md = torch.from_numpy(mask).cuda()
    nh, nl = sb.count(md)
    assert (nh, nl) == (int(mask.sum()), int(mask.size - mask.sum()))
    hi, lo = sb.split(to_dev(x, layout), md, c.bs, counts=(nh, nl))
    assert_bitexact(hi, ref["hi"], "split hi")
    assert_bitexact(lo, ref["lo"], "split lo")
    hp, lp = sb.pad(hi, lo, md, c.bs, c.H, c.W)
    assert_bitexact(hp, ref["hp"], "pad hi")
    assert_bitexact(lp, ref["lp"], "pad lo")
    y = sb.combine(up(ref["ho"], c.dtype, layout), up(ref["lo_o"], c.dtype, layout), md, c.bs, c.H, c.W)
    assert_bitexact(y, ref["y"], "combine")
    torch.cuda.synchronize()


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("c", CASES, ids=_ids(CASES))
def test_convolutions_match_oracle(c, layout):
    import paper_2011_12025_amd as sb
    mask, x, w, b, ref = prepared(c)
    log(f"[conv] {c.name} {layout} N={c.N} C={c.C}->{c.Co} {c.H}x{c.W} bs={c.bs}")
    md = torch.from_numpy(mask).cuda()
    wd = w.cuda()
    bd = None if b is None else b.cuda()
    K = 9 * c.C
    # 3x3 conv on the oracle's padded stacks
    ho, lo = sb.conv3x3(up(ref["hp"], c.dtype, layout), up(ref["lp"], c.dtype, layout), md, c.bs, c.H, c.W, wd, bd)
    assert_conv_close(ho, ref["ho64"], c.dtype, K, "conv3x3 hi")
    assert_conv_close(lo, ref["lo64"], c.dtype, K, "conv3x3 lo")
    # BlockPad fused into the convolution (packed stacks in and out)
    fho, flo = sb.block_conv3x3(up(ref["hi"], c.dtype, layout), up(ref["lo"], c.dtype, layout), md, c.bs, c.H,
                                c.W, wd, bd)
    assert_conv_close(fho, ref["ho64"], c.dtype, K, "block_conv3x3 hi")
    assert_conv_close(flo, ref["lo64"], c.dtype, K, "block_conv3x3 lo")
    # the whole layer in one kernel
    y = sb.layer(to_dev(x, layout), md, c.bs, wd, bd)
    assert_conv_close(y, y64_from_stacks(c, mask, ref["ho64"], ref["lo64"]), c.dtype, K, "layer")
    # the three paths share one MFMA schedule, so they agree bit for bit
    assert torch.equal(fho, ho) and torch.equal(flo, lo)
    ych = sb.combine(ho, lo, md, c.bs, c.H, c.W)
    assert torch.equal(ych, y)
    torch.cuda.synchronize()


EPI_CASES = [Case("epilogue_f16", "f16", 2, 40, 72, 32, 48, 16, seed=11),
             Case("epilogue_bs32_f16", "f16", 2, 40, 72, 64, 96, 32, seed=13)]


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("c", EPI_CASES, ids=_ids(EPI_CASES))
def test_block_conv_epilogue_relu_residual(c, layout):
    import paper_2011_12025_amd as sb
    mask, x, w, b, ref = prepared(c)
    log(f"[epilogue] {c.name} {layout}")
    g = np.random.default_rng(99)
    rh = torch.from_numpy(g.standard_normal(ref["ho64"].shape).astype(np.float32)).to(torch.float16)
    rl = torch.from_numpy(g.standard_normal(ref["lo64"].shape).astype(np.float32)).to(torch.float16)
    md = torch.from_numpy(mask).cuda()
    ho, lo = sb.block_conv3x3(up(ref["hi"], c.dtype, layout), up(ref["lo"], c.dtype, layout), md, c.bs, c.H, c.W,
                              w.cuda(), b.cuda(), relu=True, residual=(to_dev(rh, layout), to_dev(rl, layout)))
    K = 9 * c.C
    assert_conv_close(ho, np.maximum(ref["ho64"] + rh.float().numpy(), 0), c.dtype, K, "relu(conv+res) hi")
    assert_conv_close(lo, np.maximum(ref["lo64"] + rl.float().numpy(), 0), c.dtype, K, "relu(conv+res) lo")


def test_stack_capacity_skips_blocks():
    """A stack smaller than the number of blocks of its class: the blocks past
    the capacity are neither read nor written, and BlockCombine writes zeros."""
    import paper_2011_12025_amd as sb
    c = CASES[1]
    mask, x, w, b, ref = prepared(c)
    log(f"[capacity] {c.name}")
    md = torch.from_numpy(mask).cuda()
    nh, nl = int(mask.sum()), int(mask.size - mask.sum())
    assert nh >= 2 and nl >= 2
    hi, lo = sb.split(to_dev(x, "nhwc"), md, c.bs, counts=(nh - 1, nl - 1))
    assert_bitexact(hi, ref["hi"][:nh - 1], "split hi (capacity)")
    assert_bitexact(lo, ref["lo"][:nl - 1], "split lo (capacity)")
    y = sb.combine(up(ref["ho"][:nh - 1], c.dtype, "nhwc"), up(ref["lo_o"][:nl - 1], c.dtype, "nhwc"), md, c.bs,
                   c.H, c.W)
    yr = ref["y"].copy()
    m = mask.reshape(-1)
    last_hi, last_lo = np.flatnonzero(m)[-1], np.flatnonzero(m == 0)[-1]
    GW = c.W // c.bs
    for k in (last_hi, last_lo):
        gy, gx = (k // GW) % (c.H // c.bs), k % GW
        yr[k // ((c.H // c.bs) * GW), :, gy * c.bs:(gy + 1) * c.bs, gx * c.bs:(gx + 1) * c.bs] = 0
    assert_bitexact(y, yr, "combine (capacity)")


def test_full_size_layer_stage1_config():
    """The benchmark's workload at full size (fp16, C=64, 256x512, bs 32, 8x16
    block grid, Bernoulli(0.5) low-resolution mask), in the launch
    configuration the benchmark times (channels_last, fused layer and the
    four-call chain), against the full oracle."""
    import paper_2011_12025_amd as sb
    c = Case("stage1_full", "f16", 1, 64, 64, 256, 512, 32, seed=0)
    log(f"[full-size] {c.name}: oracle ...")
    mask, x, w, b, ref = prepared(c)
    log(f"[full-size] {c.name}: gpu")
    md = torch.from_numpy(mask).cuda()
    xd = to_dev(x, "nhwc")
    y = sb.layer(xd, md, c.bs, w.cuda(), b.cuda())
    y64 = y64_from_stacks(c, mask, ref["ho64"], ref["lo64"])
    assert_conv_close(y, y64, c.dtype, 9 * c.C, "full-size layer")
    hi, lo = sb.split(xd, md, c.bs)
    assert_bitexact(hi, ref["hi"], "full-size split hi")
    hp, lp = sb.pad(hi, lo, md, c.bs, c.H, c.W)
    assert_bitexact(lp, ref["lp"], "full-size pad lo")
    ho, lo_o = sb.conv3x3(hp, lp, md, c.bs, c.H, c.W, w.cuda(), b.cuda())
    assert torch.equal(sb.combine(ho, lo_o, md, c.bs, c.H, c.W), y)


# Fused layers on the resident-weight kernel over several images: tile lists
# of more than two rounds of workgroups, blocks of 32 and 64, one class only,
# fewer output channels than a workgroup's 64, and more than 1024 blocks (the
# mask is then read in strides of 1024 blocks).
ROUNDS_CASES = [Case("res_n3_bs32_f16", "f16", 3, 64, 64, 256, 512, 32, seed=60),
                Case("res_n2_bs64_bf16", "bf16", 2, 64, 64, 256, 512, 64, p_low=0.6, seed=61),
                Case("res_n2_bs32_alllow_f16", "f16", 2, 64, 64, 256, 512, 32, mask_kind="low", seed=62),
                Case("res_n2_bs32_co48_bf16", "bf16", 2, 64, 48, 256, 512, 32, p_low=0.3, seed=63),
                # more than 1024 blocks
                Case("res_n9_c16_f16", "f16", 9, 16, 16, 256, 512, 32, seed=64)]


@pytest.mark.parametrize("c", ROUNDS_CASES, ids=_ids(ROUNDS_CASES))
def test_resident_layer_many_rounds(c):
    import paper_2011_12025_amd as sb
    log(f"[layer, many rounds] {c.name}: oracle ...")
    mask, x, w, b, ref = prepared(c)
    log(f"[layer, many rounds] {c.name}: gpu")
    md = torch.from_numpy(mask).cuda()
    xd = to_dev(x, "nhwc")
    y = sb.layer(xd, md, c.bs, w.cuda(), None if b is None else b.cuda())
    assert_conv_close(y, y64_from_stacks(c, mask, ref["ho64"], ref["lo64"]), c.dtype, 9 * c.C, "layer")
    # the unfused chain computes every output pixel with the same MFMA schedule
    hi, lo = sb.split(xd, md, c.bs)
    hp, lp = sb.pad(hi, lo, md, c.bs, c.H, c.W)
    ho, lo_o = sb.conv3x3(hp, lp, md, c.bs, c.H, c.W, w.cuda(), None if b is None else b.cuda())
    assert torch.equal(sb.combine(ho, lo_o, md, c.bs, c.H, c.W), y)
    torch.cuda.synchronize()


# Fused layers with 128 or more than 256 input channels, and with 129-256
# above 8192 pixels, run as split, the implicit GEMM's block convolution and
# combine over library workspace stacks.
DEEP_CASES = [Case("deep512_f16", "f16", 1, 512, 64, 32, 64, 8, seed=21),
              Case("c256_n2_packed_route_f16", "f16", 2, 256, 64, 48, 96, 8, p_low=0.5, seed=26),
              Case("c192_n3_packed_route_bf16", "bf16", 3, 192, 64, 32, 96, 4, p_low=0.3, seed=27),
              Case("c128_layer_f16", "f16", 2, 128, 128, 32, 64, 8, seed=24),
              # a larger dense-route layer: more workgroups than CUs
              Case("c128_layer_2rounds_f16", "f16", 2, 128, 128, 128, 256, 16, seed=28),
              Case("c128_layer_alllow_bf16", "bf16", 1, 128, 64, 32, 32, 16, mask_kind="low", seed=25),
              Case("deep384_bf16", "bf16", 2, 384, 128, 16, 32, 4, p_low=0.6, seed=22),
              Case("deep512_allhigh_f16", "f16", 1, 512, 32, 16, 32, 4, mask_kind="high", seed=23)]


@pytest.mark.parametrize("c", DEEP_CASES, ids=_ids(DEEP_CASES))
def test_deep_layer_matches_oracle(c):
    import paper_2011_12025_amd as sb
    mask, x, w, b, ref = prepared(c)
    log(f"[deep layer] {c.name} N={c.N} C={c.C}->{c.Co} {c.H}x{c.W} bs={c.bs}")
    md = torch.from_numpy(mask).cuda()
    y = sb.layer(to_dev(x, "nhwc"), md, c.bs, w.cuda(), None if b is None else b.cuda())
    assert_conv_close(y, y64_from_stacks(c, mask, ref["ho64"], ref["lo64"]), c.dtype, 9 * c.C, "layer")
    # a second call reuses the workspace
    y2 = sb.layer(to_dev(x, "nhwc"), md, c.bs, w.cuda(), None if b is None else b.cuda())
    assert torch.equal(y, y2)
    torch.cuda.synchronize()
