"""GPU parity of the BlockPad alternatives: strided subsampling (a low
block's halo takes the top-left pixel of a high neighbour's cell) and plain
zero padding of every block, against the CPU oracle's branches for them.
segblocks_pad_ex is bit-exact; the convolutions that fuse the pad (packed
block convolution, strided block convolution, fused layer) meet the
convolution tolerance on every kernel route: the resident-weight kernel
(64 channels, blocks of 32), the multi-block implicit GEMM (C_in % 64 = 0),
the general kernel (other channel counts, NCHW) and the fused layer's packed
route (128 channels)."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from parity_util import Case, assert_bitexact, assert_conv_close, log, make_inputs, to_dev, y64_from_stacks

pytestmark = pytest.mark.gpu

TDT = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}
SAMPLINGS = ["strided", "zero"]

CASES = [
    Case("res_c64_bs32_f16", "f16", 1, 64, 64, 64, 128, 32, seed=130),        # resident-weight kernel
    Case("res_c64_bs64_bf16", "bf16", 1, 64, 64, 128, 128, 64, seed=131),
    Case("ig_c128_bs8_f16", "f16", 2, 128, 128, 32, 48, 8, seed=132),          # implicit GEMM / packed layer
    Case("gen_c24_bs6_f16", "f16", 2, 24, 40, 18, 30, 6, p_low=0.4, seed=133),  # general kernel
    Case("gen_f32_bs8", "f32", 1, 20, 16, 24, 32, 8, p_low=0.6, seed=134),
    Case("tiny_bs2_bf16", "bf16", 1, 8, 8, 8, 12, 2, seed=135),
]


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2011_12025_amd._binding as b
    b.lib()


def up(a, dtype, layout):
    return to_dev(torch.from_numpy(np.ascontiguousarray(a)).to(TDT[dtype]), layout)


@pytest.mark.parametrize("sampling", SAMPLINGS)
@pytest.mark.parametrize("layout", ["nchw", "nhwc"])
@pytest.mark.parametrize("c", CASES, ids=lambda c: c.name)
def test_pad_variants(c, layout, sampling):
    import paper_2011_12025_amd as sb
    mask, x, w, b = make_inputs(c)
    log(f"[pad {sampling}] {c.name} {layout}")
    hi, lo = oracle.split(x.float().numpy(), mask, c.bs, c.dtype)
    hp, lp = oracle.pad(hi, lo, mask, c.bs, c.H, c.W, c.dtype, sampling)
    md = torch.from_numpy(mask).cuda()
    dhp, dlp = sb.pad(up(hi, c.dtype, layout), up(lo, c.dtype, layout), md, c.bs, c.H, c.W, sampling=sampling)
    torch.cuda.synchronize()
    assert_bitexact(dhp, hp, f"pad {sampling} hi")
    assert_bitexact(dlp, lp, f"pad {sampling} lo")
    # the fused-pad convolutions and the layer on the same inputs
    wf, bf = w.float().numpy(), b.float().numpy()
    ho64, lo64 = oracle.conv3x3_valid(hp, wf, bf), oracle.conv3x3_valid(lp, wf, bf)
    K = 9 * c.C
    fho, flo = sb.block_conv3x3(up(hi, c.dtype, layout), up(lo, c.dtype, layout), md, c.bs, c.H, c.W, w.cuda(),
                                b.cuda(), sampling=sampling)
    torch.cuda.synchronize()
    assert_conv_close(fho, ho64, c.dtype, K, f"block_conv3x3 {sampling} hi")
    assert_conv_close(flo, lo64, c.dtype, K, f"block_conv3x3 {sampling} lo")
    y = sb.layer(to_dev(x, layout), md, c.bs, w.cuda(), b.cuda(), sampling=sampling)
    torch.cuda.synchronize()
    assert_conv_close(y, y64_from_stacks(c, mask, ho64, lo64), c.dtype, K, f"layer {sampling}")


@pytest.mark.parametrize("sampling", SAMPLINGS)
@pytest.mark.parametrize("C,Co,bs,k", [(64, 128, 16, 3), (128, 128, 8, 3), (32, 64, 8, 3), (64, 64, 4, 1)])
def test_strided_block_conv_pad_variants(C, Co, bs, k, sampling):
    """Stride-2 block convolutions with the alternatives (implicit GEMM for
    C_in % 64 = 0, the fallback block convolution otherwise)."""
    import paper_2011_12025_amd as sb
    from paper_2011_12025_amd import inputs
    N, H, W, seed = 2, 4 * bs, 6 * bs, 140 + C + bs
    mask = inputs.mask_bernoulli(seed, N, H // bs, W // bs, 0.5)
    x = inputs.feature_map(seed, N, C, H, W, "f16")
    w = inputs.conv_weight(seed, Co, C, k, "f16")
    b = inputs.conv_bias(seed, Co, k * k * C, "f16")
    log(f"[strided conv {sampling}] C={C}->{Co} bs={bs} k={k}")
    hi, lo = oracle.split(x.float().numpy(), mask, bs, "f16")
    hp, lp = oracle.pad(hi, lo, mask, bs, H, W, "f16", sampling)
    wf, bf = w.float().numpy(), b.float().numpy()
    ref = [np.maximum(oracle.conv_block(P, wf, 2, bf), 0.0) for P in (hp, lp)]
    cl = torch.channels_last
    ho, lo_o = sb.block_conv_ex(torch.from_numpy(hi).half().cuda().contiguous(memory_format=cl),
                                torch.from_numpy(lo).half().cuda().contiguous(memory_format=cl),
                                torch.from_numpy(mask).cuda(), bs, H, W, w.cuda().contiguous(memory_format=cl),
                                b.cuda(), stride=2, relu=True, sampling=sampling)
    torch.cuda.synchronize()
    assert_conv_close(ho, ref[0], "f16", k * k * C, f"strided {sampling} hi")
    assert_conv_close(lo_o, ref[1], "f16", k * k * C, f"strided {sampling} lo")
