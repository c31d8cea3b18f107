"""GPU tests of segblocks_block_conv_chain: a block convolution that reads
its input's high stack at half resolution (the 2x2 averages that BlockPad
with average sampling gives a low block's halo beside a high neighbour) and
writes its own output's, so that a chain of convolutions needs no launch
that pads the low stack.

The results must equal those of segblocks_block_conv_ex /
segblocks_block_conv3x3 on the same stacks bit for bit (the same sums, the
halo cells only come from another buffer), and the half-resolution output
must equal the 2x2 averages of the high output computed on the CPU in the
library's association ((a + b) + (c + d)) * 0.25 in fp32, rounded once.
Those two calls are compared with the oracle in test_gpu_encoder.py and
test_gpu_parity.py."""
from __future__ import annotations

import dataclasses

import numpy as np
import pytest
import torch

import oracle
from parity_util import assert_bitexact, f32, log
from paper_2011_12025_amd import inputs

pytestmark = pytest.mark.gpu

TDT = {"f16": torch.float16, "bf16": torch.bfloat16}


def _cl(t: torch.Tensor) -> torch.Tensor:
    return t.cuda().contiguous(memory_format=torch.channels_last)


def half_res(st: torch.Tensor) -> torch.Tensor:
    """2x2 averages of a [S, C, e, e] stack on the CPU: top-left, top-right,
    bottom-left, bottom-right summed as ((a + b) + (c + d)) in fp32, times
    0.25, rounded to the stack's dtype."""
    x = st.detach().cpu().float()
    a, b = x[:, :, 0::2, 0::2], x[:, :, 0::2, 1::2]
    c, d = x[:, :, 1::2, 0::2], x[:, :, 1::2, 1::2]
    return (((a + b) + (c + d)) * 0.25).to(st.dtype)


@dataclasses.dataclass
class CCase:
    name: str
    dtype: str
    N: int
    C: int
    Co: int
    H: int
    W: int
    bs: int
    k: int = 3
    stride: int = 1
    relu: bool = True
    residual: bool = False
    mask_kind: str = "bernoulli"
    p_low: float = 0.5
    seed: int = 0


CASES = [
    # output block extent 16: the row below a pixel is the next fragment of its lane
    CCase("eo16_c128_f16", "f16", 2, 128, 128, 64, 96, 16, seed=300),
    # extent 8 and 4 on the 128 x 256 tile with split K (the reduction pass writes the averages)
    CCase("eo8_c256_split_f16", "f16", 1, 256, 256, 64, 128, 8, residual=True, seed=301),
    CCase("eo4_c512_split_bf16", "bf16", 1, 512, 512, 32, 64, 4, p_low=0.75, residual=True, seed=302),
    # extent 2: a 16-lane group holds four 2x2 blocks
    CCase("eo2_c64_bf16", "bf16", 1, 64, 64, 16, 32, 2, p_low=0.6, seed=303),
    # extent 32 on the 128-row tiles of four fragments (the row below: two fragments on)
    CCase("eo32_c128_f16", "f16", 1, 128, 128, 64, 96, 32, seed=304),
    # extent 32 on the 128 x 64 tile (two fragments): averages from the extra launch
    CCase("eo32_tn64_fallback_bf16", "bf16", 1, 128, 64, 64, 96, 32, seed=305),
    # extent 64 and a non-power-of-two extent: the extra launch
    CCase("eo64_fallback_f16", "f16", 1, 128, 128, 128, 128, 64, seed=306),
    CCase("eo12_fallback_f16", "f16", 1, 128, 64, 48, 72, 12, seed=307),
    # stride 2 (a stage transition) and 1x1 at stride 2
    CCase("k3s2_c128_co256_f16", "f16", 2, 128, 256, 64, 96, 16, stride=2, seed=308),
    CCase("k1s2_c128_co256_bf16", "bf16", 1, 128, 256, 64, 64, 16, k=1, stride=2, relu=False, seed=309),
    # the resident kernel's route (64 channels, blocks of 32 and 64): averages from the extra launch
    CCase("resident_c64_bs32_f16", "f16", 1, 64, 64, 64, 128, 32, residual=True, seed=310),
    CCase("resident_c64_bs64_bf16", "bf16", 2, 64, 64, 128, 256, 64, p_low=0.4, seed=314),
    # 48 output channels on the resident kernel
    CCase("resident_c64_co48_f16", "f16", 1, 64, 48, 64, 128, 32, seed=315),
    # one class only, and more than 1024 blocks
    CCase("allhigh_eo8_f16", "f16", 1, 128, 128, 32, 64, 8, mask_kind="high", seed=311),
    CCase("alllow_eo8_bf16", "bf16", 1, 128, 128, 32, 64, 8, mask_kind="low", seed=312),
    CCase("blocks1200_eo4_f16", "f16", 1, 64, 64, 120, 160, 4, seed=313),
]


def _mask(c):
    GH, GW = c.H // c.bs, c.W // c.bs
    if c.mask_kind == "high":
        return np.ones((c.N, GH, GW), np.uint8)
    if c.mask_kind == "low":
        return np.zeros((c.N, GH, GW), np.uint8)
    return inputs.mask_bernoulli(c.seed, c.N, GH, GW, c.p_low)


@pytest.mark.parametrize("c", CASES, ids=lambda c: c.name)
def test_chain_matches_block_conv(c):
    import paper_2011_12025_amd as sb
    log(f"[block_conv_chain] {c}")
    mask = _mask(c)
    x = inputs.feature_map(c.seed, c.N, c.C, c.H, c.W, c.dtype)
    w = inputs.conv_weight(c.seed, c.Co, c.C, c.k, c.dtype)
    b = inputs.conv_bias(c.seed, c.Co, c.k * c.k * c.C, c.dtype)
    hi, lo = oracle.split(x.float().numpy(), mask, c.bs, c.dtype)
    t = TDT[c.dtype]
    dhi, dlo = _cl(torch.from_numpy(hi).to(t)), _cl(torch.from_numpy(lo).to(t))
    bo = c.bs // c.stride
    dres = None
    if c.residual:
        r = inputs.feature_map(c.seed + 1000, c.N, c.Co, c.H // c.stride, c.W // c.stride, c.dtype).float().numpy()
        dres = tuple(_cl(torch.from_numpy(a).to(t)) for a in oracle.split(r, mask, bo, c.dtype))
    dmask, dw, db = torch.from_numpy(mask).cuda(), _cl(w), b.cuda()
    if c.k == 3 and c.stride == 1:
        ref = sb.block_conv3x3(dhi, dlo, dmask, c.bs, c.H, c.W, dw, db, relu=c.relu, residual=dres)
    else:
        ref = sb.block_conv_ex(dhi, dlo, dmask, c.bs, c.H, c.W, dw, db, stride=c.stride, relu=c.relu, residual=dres)
    hh_in = _cl(half_res(dhi))
    got = sb.block_conv_chain(dhi, dlo, dmask, c.bs, c.H, c.W, dw, db, stride=c.stride, relu=c.relu, residual=dres,
                              hi_half=hh_in, want_half=True)
    plain = sb.block_conv_chain(dhi, dlo, dmask, c.bs, c.H, c.W, dw, db, stride=c.stride, relu=c.relu,
                                residual=dres, want_half=False)
    torch.cuda.synchronize()
    assert plain[2] is None
    for k, nm in ((0, "high"), (1, "low")):
        assert_bitexact(got[k], f32(ref[k]), f"{c.name} {nm} (with the half stack)")
        assert_bitexact(plain[k], f32(ref[k]), f"{c.name} {nm} (without)")
    assert got[2].shape == (hi.shape[0], c.Co, bo // 2, bo // 2)
    assert_bitexact(got[2], f32(half_res(ref[0])), f"{c.name} high output at half resolution")


@pytest.mark.parametrize("dtype,blk,H,W,N,mask_kind,seed", [
    ("f16", 128, 256, 512, 1, "bernoulli", 320),   # stage-1 blocks of 32 (resident kernel), extents 16 / 8 / 4 after
    ("bf16", 64, 256, 512, 1, "bernoulli", 321),   # stage-1 blocks of 16 (the GEMM), extents 8 / 4 / 2 after
    ("f16", 64, 128, 256, 2, "correlated", 322),
])
def test_encoder_half_stacks_bitexact(dtype, blk, H, W, N, mask_kind, seed):
    """The encoder with half stacks chained between its convolutions equals
    the encoder that pads each low stack in a launch of its own, bit for bit."""
    from paper_2011_12025_amd.encoder import BlockEncoder
    import paper_2011_12025_amd as sb
    log(f"[encoder half stacks] {dtype} blk={blk} {N}x3x{H}x{W} {mask_kind} seed={seed}")
    t = TDT[dtype]
    Wt = inputs.encoder_weights(seed, dtype)
    x = _cl(inputs.feature_map(seed, N, 3, H, W, dtype))
    GH, GW = H // blk, W // blk
    m = (inputs.mask_bernoulli(seed, N, GH, GW, 0.5) if mask_kind == "bernoulli"
         else inputs.mask_correlated(seed, N, GH, GW, 0.5))
    dmask = torch.from_numpy(m).cuda()
    counts = sb.count(dmask)
    assert counts[0] > 0 and counts[1] > 0, "the case needs blocks of both classes"
    y1 = BlockEncoder(Wt, blk, half_stacks=True)(x, dmask, counts)
    y0 = BlockEncoder(Wt, blk, half_stacks=False)(x, dmask, counts)
    torch.cuda.synchronize()
    assert y1.dtype == t
    assert_bitexact(y1, f32(y0), f"encoder {dtype} blk={blk}")
