"""GPU parity at the benchmarked configurations' own kernel routes.

The deeper stage shapes of a 1024x2048 image run kernels that the small
parity cases do not reach: the fused layer at 256 and 512 input channels
(blocks of 8 and 4 pixels, exact-fraction masks), stride-2 block
convolutions whose 128-pixel tiles lie inside one block (input blocks of 32
and 64), the encoder with 128- and 256-pixel image blocks (stage 1 on the
resident-weight kernel), four images with spatially correlated masks in
fp16 and bf16, and one whole encoder forward at 1024x2048.  Every result is
compared with the CPU oracle on the same seeded inputs: convolutions by the
max-norm relative bound (2e-2 for fp16 / bf16) plus the element-wise bound,
the composed encoder by the max-norm bound."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from parity_util import NORM_TOL, Case, assert_bitexact, assert_conv_close, f32, log, to_dev, y64_from_stacks
from paper_2011_12025_amd import inputs

pytestmark = pytest.mark.gpu

TDT = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2011_12025_amd._binding as b
    b.lib()
    oracle.set_threads(0)


def _cl(t: torch.Tensor) -> torch.Tensor:
    return t.cuda().contiguous(memory_format=torch.channels_last)


# (C, H, W, bs): the stage shapes of a 1024x2048 image with 128-pixel blocks
STAGES = {2: (128, 128, 256, 16), 3: (256, 64, 128, 8), 4: (512, 32, 64, 4)}


@pytest.mark.parametrize("stage,f_low,dtype", [(3, 0.25, "f16"), (3, 0.75, "f16"), (4, 0.25, "f16"),
                                               (4, 0.75, "bf16"), (2, 0.5, "f16"), (4, 0.0, "f16")])
def test_layer_at_stage_shapes(stage, f_low, dtype):
    """segblocks_layer at the sweep's stage shapes with exact-fraction masks."""
    import paper_2011_12025_amd as sb
    C, H, W, bs = STAGES[stage]
    c = Case(f"stage{stage}_f{f_low}", dtype, 1, C, C, H, W, bs, seed=30 + stage)
    mask = inputs.mask_exact_fraction(c.seed, 1, H // bs, W // bs, f_low)
    x = inputs.feature_map(c.seed, 1, C, H, W, dtype)
    w = inputs.conv_weight(c.seed, C, C, 3, dtype)
    b = inputs.conv_bias(c.seed, C, 9 * C, dtype)
    log(f"[stage layer] {c.name} {dtype}: oracle ...")
    hi, lo = oracle.split(x.float().numpy(), mask, bs, dtype)
    hp, lp = oracle.pad(hi, lo, mask, bs, H, W, dtype)
    ho64 = oracle.conv3x3_valid(hp, w.float().numpy(), b.float().numpy())
    lo64 = oracle.conv3x3_valid(lp, w.float().numpy(), b.float().numpy())
    log(f"[stage layer] {c.name} {dtype}: gpu")
    md = torch.from_numpy(mask).cuda()
    y = sb.layer(to_dev(x, "nhwc"), md, bs, w.cuda(), b.cuda())
    torch.cuda.synchronize()
    assert_conv_close(y, y64_from_stacks(c, mask, ho64, lo64), dtype, 9 * C, c.name)
    # the packed convolution of the same stacks, as the sweep times it
    t = TDT[dtype]
    fho, flo = sb.block_conv3x3(_cl(torch.from_numpy(hi).to(t)), _cl(torch.from_numpy(lo).to(t)), md, bs, H, W,
                                w.cuda(), b.cuda())
    torch.cuda.synchronize()
    assert_conv_close(fho, ho64, dtype, 9 * C, c.name + " block_conv3x3 hi")
    assert_conv_close(flo, lo64, dtype, 9 * C, c.name + " block_conv3x3 lo")


@pytest.mark.parametrize("bs,f_low,dtype,relu", [(32, 0.5, "f16", False), (64, 0.5, "bf16", True),
                                                 (32, 0.55, "f16", False), (32, 0.75, "bf16", True)])
def test_resident_conv_low_tile_sizes(bs, f_low, dtype, relu):
    """The resident-weight convolutions at the stage-1 shape (C=64, 256x512)
    with exact-fraction masks: at 0.5 and 0.55 low the high tiles fit in one
    round of workgroups and the low blocks are cut into quarter-block tiles
    spread over every workgroup in the second; at 0.75 the whole low tiles
    fit beside the high ones in one round and stay whole.  Padded and packed
    sources against the oracle, and bit for bit against each other and the
    fused layer (one MFMA schedule per output pixel)."""
    import paper_2011_12025_amd as sb
    C, H, W = 64, 256, 512
    c = Case(f"res_bs{bs}_f{f_low}", dtype, 1, C, C, H, W, bs, seed=70)
    mask = inputs.mask_exact_fraction(c.seed, 1, H // bs, W // bs, f_low)
    x = inputs.feature_map(c.seed, 1, C, H, W, dtype)
    w = inputs.conv_weight(c.seed, C, C, 3, dtype)
    b = inputs.conv_bias(c.seed, C, 9 * C, dtype)
    log(f"[resident low tiles] {c.name}: oracle ...")
    hi, lo = oracle.split(x.float().numpy(), mask, bs, dtype)
    hp, lp = oracle.pad(hi, lo, mask, bs, H, W, dtype)
    ho64 = oracle.conv3x3_valid(hp, w.float().numpy(), b.float().numpy())
    lo64 = oracle.conv3x3_valid(lp, w.float().numpy(), b.float().numpy())
    if relu:
        ho64, lo64 = np.maximum(ho64, 0), np.maximum(lo64, 0)
    log(f"[resident low tiles] {c.name}: gpu")
    t = TDT[dtype]
    md = torch.from_numpy(mask).cuda()
    wd, bd = w.cuda(), b.cuda()
    fho, flo = sb.block_conv3x3(_cl(torch.from_numpy(hi).to(t)), _cl(torch.from_numpy(lo).to(t)), md, bs, H, W,
                                wd, bd, relu=relu)
    pho, plo = sb.conv3x3(_cl(torch.from_numpy(hp).to(t)), _cl(torch.from_numpy(lp).to(t)), md, bs, H, W, wd, bd)
    if relu:  # rounding and ReLU commute
        pho, plo = pho.clamp(min=0), plo.clamp(min=0)
    y = sb.layer(to_dev(x, "nhwc"), md, bs, wd, bd, relu=relu)
    torch.cuda.synchronize()
    assert_conv_close(fho, ho64, dtype, 9 * C, c.name + " block_conv3x3 hi")
    assert_conv_close(flo, lo64, dtype, 9 * C, c.name + " block_conv3x3 lo")
    assert torch.equal(fho, pho) and torch.equal(flo, plo)
    assert torch.equal(sb.combine(fho, flo, md, bs, H, W), y)


# stride-2 block convolutions with input blocks of 32 and 64 pixels: the
# implicit GEMM's 128-pixel tiles lie inside one output block
@pytest.mark.parametrize("name,dtype,N,C,Co,H,W,bs,k,p_low,seed", [
    ("k3s2_bs32_c64_co128_f16", "f16", 1, 64, 128, 128, 256, 32, 3, 0.5, 40),
    ("k3s2_bs64_c128_co256_bf16", "bf16", 1, 128, 256, 128, 256, 64, 3, 0.5, 41),
    ("k1s2_bs32_c64_co128_f16", "f16", 1, 64, 128, 128, 256, 32, 1, 0.5, 42),
    ("k1s2_bs64_c128_co256_bf16", "bf16", 2, 128, 256, 128, 128, 64, 1, 0.25, 43),
    ("k3s2_bs64_c64_co128_alllow_f16", "f16", 1, 64, 128, 128, 128, 64, 3, 1.0, 44),
])
def test_stride2_tiles_inside_one_block(name, dtype, N, C, Co, H, W, bs, k, p_low, seed):
    import paper_2011_12025_amd as sb
    mask = inputs.mask_bernoulli(seed, N, H // bs, W // bs, p_low)
    x = inputs.feature_map(seed, N, C, H, W, dtype)
    w = inputs.conv_weight(seed, Co, C, k, dtype)
    b = inputs.conv_bias(seed, Co, k * k * C, dtype)
    log(f"[stride-2 in-block] {name}: oracle ...")
    hi, lo = oracle.split(x.float().numpy(), mask, bs, dtype)
    hp, lp = oracle.pad(hi, lo, mask, bs, H, W, dtype)
    wf, bf = w.float().numpy(), b.float().numpy()
    ref = [np.maximum(oracle.conv_block(P, wf, 2, bf), 0.0) for P in (hp, lp)]
    log(f"[stride-2 in-block] {name}: gpu")
    t = TDT[dtype]
    ho, lo_o = sb.block_conv_ex(_cl(torch.from_numpy(hi).to(t)), _cl(torch.from_numpy(lo).to(t)),
                                torch.from_numpy(mask).cuda(), bs, H, W, _cl(w), b.cuda(), stride=2, relu=True)
    torch.cuda.synchronize()
    assert_conv_close(ho, ref[0], dtype, k * k * C, name + " high")
    assert_conv_close(lo_o, ref[1], dtype, k * k * C, name + " low")


def _encoder_case(dtype, N, H, W, blk, mask_np, seed):
    import paper_2011_12025_amd as sb  # noqa: F401
    from paper_2011_12025_amd.encoder import BlockEncoder
    x = inputs.feature_map(seed, N, 3, H, W, dtype)
    Wt = inputs.encoder_weights(seed, dtype)
    log(f"[encoder] {dtype} N={N} {H}x{W} block {blk} high={int(mask_np.sum())}/{mask_np.size}: oracle ...")
    ref = oracle.encoder(x.float().numpy(), mask_np, blk, {k: v.float().numpy() for k, v in Wt.items()}, dtype)
    log(f"[encoder] {dtype} N={N} {H}x{W} block {blk}: gpu")
    enc = BlockEncoder(Wt, blk)
    y = enc(_cl(x), torch.from_numpy(mask_np).cuda())
    torch.cuda.synchronize()
    g = f32(y).astype(np.float64)
    assert g.shape == ref.shape == (N, 512, H // 32, W // 32)
    assert np.all(np.isfinite(g))
    rel = float(np.max(np.abs(g - ref)) / np.max(np.abs(ref)))
    log(f"[encoder] max-norm relative error {rel:.3e}")
    assert rel <= NORM_TOL[dtype]


@pytest.mark.parametrize("dtype,blk,H,W,q", [("f16", 128, 256, 512, 0.5), ("bf16", 128, 256, 512, 0.25),
                                             ("f16", 256, 512, 512, 0.75), ("bf16", 256, 512, 512, 0.5)])
def test_encoder_batched_correlated(dtype, blk, H, W, q):
    """Four images, spatially correlated masks at quantile q, image blocks of
    128 / 256 pixels (stage-1 blocks of 32 / 64 on the resident-weight
    kernel, stage 4 blocks of 4 / 8), fp16 and bf16 through 17 chained
    convolutions."""
    N = 4
    mask = inputs.mask_correlated(50, N, H // blk, W // blk, q)
    _encoder_case(dtype, N, H, W, blk, mask, seed=51)


def test_encoder_full_size_1024x2048():
    """One whole encoder forward at 1024x2048, 128-pixel blocks (8x16 grid),
    Bernoulli(0.5) low-resolution mask, fp16: the benchmarked encoder."""
    mask = inputs.mask_bernoulli(0, 1, 8, 16, 0.5)
    _encoder_case("f16", 1, 1024, 2048, 128, mask, seed=0)


def test_full_size_stage1_every_stack_bitexact():
    """Split and pad at the benchmark's layer shape (fp16, C=64, 256x512,
    blocks of 32, Bernoulli(0.5)): every stack bit for bit."""
    import paper_2011_12025_amd as sb
    c = Case("stage1_full", "f16", 1, 64, 64, 256, 512, 32, seed=0)
    mask = inputs.mask_bernoulli(0, 1, 8, 16, 0.5)
    x = inputs.feature_map(0, 1, 64, 256, 512, "f16")
    log("[full-size stacks] oracle ...")
    hi, lo = oracle.split(x.float().numpy(), mask, 32, "f16")
    hp, lp = oracle.pad(hi, lo, mask, 32, 256, 512, "f16")
    log("[full-size stacks] gpu")
    md = torch.from_numpy(mask).cuda()
    dhi, dlo = sb.split(to_dev(x, "nhwc"), md, 32)
    dhp, dlp = sb.pad(dhi, dlo, md, 32, 256, 512)
    torch.cuda.synchronize()
    assert_bitexact(dhi, hi, "split hi")
    assert_bitexact(dlo, lo, "split lo")
    assert_bitexact(dhp, hp, "pad hi")
    assert_bitexact(dlp, lp, "pad lo")
    assert c.grid == (1, 8, 16)
