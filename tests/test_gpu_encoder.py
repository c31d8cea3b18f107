"""GPU parity of the encoder's entry points against the CPU oracle: strided
block convolutions (3x3 and 1x1 at stride 1 and 2, BlockPad fused, bias /
residual / ReLU epilogue), the dense stem convolution, max-pooling, and the
whole ResNet-18 encoder on block stacks.

Comparison rules are those of the block convolutions (max-norm relative 2e-2
for fp16 / bf16 plus an element-wise bound against the oracle's unrounded
fp64 result); max-pooling only selects stored values and must be bit-exact.
The composed encoder is compared by the max-norm rule alone: both sides
round every stored map, and one-ulp differences in early layers move later
ones by more than one ulp element-wise."""
from __future__ import annotations

import dataclasses

import numpy as np
import pytest
import torch

import oracle
from parity_util import NORM_TOL, assert_bitexact, assert_conv_close, f32, log
from paper_2011_12025_amd import inputs

pytestmark = pytest.mark.gpu

TDT = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}


def _cl(t: torch.Tensor) -> torch.Tensor:
    return t.cuda().contiguous(memory_format=torch.channels_last)


@dataclasses.dataclass
class BCase:
    name: str
    dtype: str
    N: int
    C: int
    Co: int
    H: int
    W: int
    bs: int
    k: int
    stride: int
    relu: bool = False
    residual: bool = False
    bias: bool = True
    mask_kind: str = "bernoulli"
    p_low: float = 0.5
    seed: int = 0


BCASES = [
    BCase("k3s2_f16", "f16", 1, 64, 128, 64, 96, 16, 3, 2, relu=True, seed=60),
    BCase("k1s2_bf16", "bf16", 2, 64, 128, 32, 48, 8, 1, 2, seed=61),
    BCase("k3s1_res_relu_f16", "f16", 1, 128, 128, 32, 64, 8, 3, 1, relu=True, residual=True, seed=62),
    BCase("k3s2_bs4_bf16", "bf16", 2, 32, 64, 16, 24, 4, 3, 2, relu=True, seed=63),
    BCase("k3s1_ragged_co_bf16", "bf16", 1, 72, 40, 24, 40, 8, 3, 1, seed=64),
    BCase("k3s2_allhigh_f16", "f16", 1, 16, 32, 32, 32, 16, 3, 2, mask_kind="high", seed=65),
    BCase("k1s2_alllow_f16", "f16", 1, 16, 32, 32, 32, 16, 1, 2, mask_kind="low", seed=66),
    BCase("k3s2_res_nobias_f16", "f16", 1, 64, 64, 32, 32, 8, 3, 2, residual=True, relu=True, bias=False, seed=67),
    BCase("k3s2_blocks1120_f16", "f16", 1, 16, 16, 128, 140, 4, 3, 2, seed=68),   # more than 1024 blocks
    BCase("k1s1_f16", "f16", 1, 24, 24, 16, 16, 8, 1, 1, seed=69),
    # multi-block implicit GEMM (C_in % 64 == 0): tiles spanning many blocks
    BCase("ig_k3s1_c128_bs4_res_f16", "f16", 1, 128, 128, 32, 48, 4, 3, 1, relu=True, residual=True, seed=75),
    BCase("ig_k3s2_c256_co512_bf16", "bf16", 1, 256, 512, 32, 64, 8, 3, 2, relu=True, seed=76),
    BCase("ig_k3s1_c64_co64_bs16_f16", "f16", 2, 64, 64, 64, 64, 16, 3, 1, seed=77),
    BCase("ig_k1s2_c128_co256_f16", "f16", 1, 128, 256, 32, 32, 8, 1, 2, seed=78),
    BCase("ig_k3s1_bs2_bf16", "bf16", 1, 64, 64, 16, 32, 2, 3, 1, p_low=0.6, seed=79),
    BCase("ig_blocks1200_f16", "f16", 1, 64, 64, 120, 160, 4, 3, 1, seed=80),
    BCase("ig_alllow_k3s2_f16", "f16", 1, 64, 128, 32, 32, 8, 3, 2, mask_kind="low", seed=81),
    BCase("ig_allhigh_k3s1_bf16", "bf16", 1, 128, 64, 16, 32, 8, 3, 1, mask_kind="high", seed=82),
    # 128 input channels with both classes: the low stack is padded once before the GEMM
    BCase("ig_lowpad_k3s2_c128_bf16", "bf16", 2, 128, 128, 32, 64, 8, 3, 2, relu=True, seed=83),
    BCase("ig_lowpad_k3s1_c128_bs16_f16", "f16", 2, 128, 64, 64, 96, 16, 3, 1, p_low=0.75, residual=True, seed=84),
    # 256 and more output channels: the 128x256 workgroup tile (split K, and a
    # partial second N tile at 320 channels), padded low stack at 256 / 512 channels
    BCase("ig_tn256_k3s1_c256_bs8_f16", "f16", 1, 256, 256, 64, 128, 8, 3, 1, relu=True, residual=True, seed=85),
    BCase("ig_tn256_k3s1_c64_co320_bf16", "bf16", 1, 64, 320, 32, 64, 8, 3, 1, seed=86),
    BCase("ig_tn256_k3s2_c256_co256_f16", "f16", 2, 256, 256, 32, 64, 8, 3, 2, p_low=0.25, seed=87),
    BCase("ig_tn256_k3s1_c512_bs4_bf16", "bf16", 1, 512, 512, 32, 64, 4, 3, 1, p_low=0.75, residual=True, seed=88),
    # enough pixel rows for the 256 x 128 workgroup tile (eight 64 x 64 wave tiles)
    BCase("ig_tm256_k3s1_c64_co128_f16", "f16", 1, 64, 128, 256, 256, 16, 3, 1, relu=True, residual=True, seed=89),
    BCase("ig_tm256_k3s1_c64_co128_bs8_bf16", "bf16", 2, 64, 128, 128, 256, 8, 3, 1, p_low=0.3, seed=90),
]


def _mask(c):
    GH, GW = c.H // c.bs, c.W // c.bs
    if c.mask_kind == "high":
        return np.ones((c.N, GH, GW), np.uint8)
    if c.mask_kind == "low":
        return np.zeros((c.N, GH, GW), np.uint8)
    return inputs.mask_bernoulli(c.seed, c.N, GH, GW, c.p_low)


@pytest.mark.parametrize("c", BCASES, ids=lambda c: c.name)
def test_block_conv_ex(c):
    import paper_2011_12025_amd as sb
    log(f"[block_conv_ex] {c}")
    mask = _mask(c)
    x = inputs.feature_map(c.seed, c.N, c.C, c.H, c.W, c.dtype)
    w = inputs.conv_weight(c.seed, c.Co, c.C, c.k, c.dtype)
    b = inputs.conv_bias(c.seed, c.Co, c.k * c.k * c.C, c.dtype) if c.bias else None
    xf, wf, bf = x.float().numpy(), w.float().numpy(), None if b is None else b.float().numpy()
    hi, lo = oracle.split(xf, mask, c.bs, c.dtype)
    bo, Ho, Wo = c.bs // c.stride, c.H // c.stride, c.W // c.stride
    res = None
    if c.residual:
        r = inputs.feature_map(c.seed + 1000, c.N, c.Co, Ho, Wo, c.dtype).float().numpy()
        res = oracle.split(r, mask, bo, c.dtype)
    # oracle: padded stacks, unrounded convolution + residual + ReLU in fp64
    hp, lp = oracle.pad(hi, lo, mask, c.bs, c.H, c.W, c.dtype)
    ref64 = []
    for P, R in zip((hp, lp), (None, None) if res is None else res):
        a = oracle.conv_block(P, wf, c.stride, bf)
        if R is not None:
            a = a + R.astype(np.float64)
        ref64.append(np.maximum(a, 0.0) if c.relu else a)

    t = TDT[c.dtype]
    dhi, dlo = _cl(torch.from_numpy(hi).to(t)), _cl(torch.from_numpy(lo).to(t))
    dres = None if res is None else tuple(_cl(torch.from_numpy(a).to(t)) for a in res)
    dmask = torch.from_numpy(mask).cuda()
    ho, lo_o = sb.block_conv_ex(dhi, dlo, dmask, c.bs, c.H, c.W, _cl(w), None if b is None else b.cuda(),
                                stride=c.stride, relu=c.relu, residual=dres)
    torch.cuda.synchronize()
    assert ho.shape == (hi.shape[0], c.Co, bo, bo) and lo_o.shape == (lo.shape[0], c.Co, bo // 2, bo // 2)
    K = c.k * c.k * c.C
    assert_conv_close(ho, ref64[0], c.dtype, K, f"{c.name} high")
    assert_conv_close(lo_o, ref64[1], c.dtype, K, f"{c.name} low")


@dataclasses.dataclass
class DCase:
    name: str
    dtype: str
    N: int
    C: int
    Co: int
    H: int
    W: int
    k: int
    stride: int
    pad: int
    relu: bool = True
    bias: bool = True
    seed: int = 0


DCASES = [
    DCase("stem_f16", "f16", 1, 3, 64, 64, 96, 7, 2, 3, seed=70),
    DCase("stem_bf16_ragged", "bf16", 2, 3, 64, 50, 70, 7, 2, 3, seed=71),
    DCase("k3s1_c16_nobias_f16", "f16", 1, 16, 24, 20, 130, 3, 1, 1, relu=False, bias=False, seed=72),
    DCase("k3s1_c64_bf16", "bf16", 1, 64, 96, 16, 64, 3, 1, 1, seed=73),
    DCase("k1s2_f16", "f16", 1, 8, 8, 17, 33, 1, 2, 0, seed=74),
]


@pytest.mark.parametrize("c", DCASES, ids=lambda c: c.name)
def test_conv2d(c):
    import paper_2011_12025_amd as sb
    log(f"[conv2d] {c}")
    x = inputs.feature_map(c.seed, c.N, c.C, c.H, c.W, c.dtype)
    w = inputs.conv_weight(c.seed, c.Co, c.C, c.k, c.dtype)
    b = inputs.conv_bias(c.seed, c.Co, c.k * c.k * c.C, c.dtype) if c.bias else None
    xf, wf = x.float().numpy(), w.float().numpy()
    t64 = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    ref = torch.nn.functional.conv2d(t64(xf), t64(wf), None if b is None else t64(b.float().numpy()),
                                     stride=c.stride, padding=c.pad).numpy()
    if c.relu:
        ref = np.maximum(ref, 0.0)
    y = sb.conv2d(_cl(x), _cl(w), None if b is None else b.cuda(), stride=c.stride, padding=c.pad, relu=c.relu)
    torch.cuda.synchronize()
    assert_conv_close(y, ref, c.dtype, c.k * c.k * c.C, c.name)
    # the oracle's own dense convolution rounds the same fp64 values
    assert np.array_equal(oracle.dense_conv(xf, wf, None if b is None else b.float().numpy(), c.stride, c.pad,
                                            c.dtype, relu=c.relu), oracle.round_to(ref, c.dtype))


@pytest.mark.parametrize("dtype,shape,k,s,p", [("f16", (2, 64, 31, 47), 3, 2, 1), ("bf16", (1, 24, 64, 64), 3, 2, 1),
                                               ("f32", (1, 8, 9, 14), 3, 2, 1), ("f16", (1, 16, 10, 12), 2, 2, 0)])
def test_maxpool_bitexact(dtype, shape, k, s, p):
    import paper_2011_12025_amd as sb
    log(f"[maxpool] {dtype} {shape} k{k} s{s} p{p}")
    x = inputs.feature_map(80, *shape, dtype)
    ref = oracle.maxpool(x.float().numpy(), k, s, p)
    y = sb.maxpool(_cl(x), k, s, p)
    torch.cuda.synchronize()
    assert_bitexact(y, ref, f"maxpool {dtype} {shape}")


@pytest.mark.parametrize("dtype,mask_kind,seed", [("f16", "bernoulli", 90), ("bf16", "bernoulli", 91),
                                                  ("f16", "high", 92)])
def test_encoder(dtype, mask_kind, seed):
    """ResNet-18 encoder on block stacks, 3 x 128 x 256 input, image blocks of
    64 pixels (block side 16 at stride 4, 2 at stride 32)."""
    import paper_2011_12025_amd as sb
    from paper_2011_12025_amd.encoder import BlockEncoder
    log(f"[encoder] {dtype} {mask_kind} seed {seed}")
    N, H, W, blk = 1, 128, 256, 64
    x = inputs.feature_map(seed, N, 3, H, W, dtype)
    Wt = inputs.encoder_weights(seed, dtype)
    GH, GW = H // blk, W // blk
    mask = np.ones((N, GH, GW), np.uint8) if mask_kind == "high" else inputs.mask_bernoulli(seed, N, GH, GW, 0.5)
    ref = oracle.encoder(x.float().numpy(), mask, blk, {k: v.float().numpy() for k, v in Wt.items()}, dtype)
    enc = BlockEncoder(Wt, blk)
    y = enc(_cl(x), torch.from_numpy(mask).cuda())
    torch.cuda.synchronize()
    g = f32(y).astype(np.float64)
    assert g.shape == ref.shape == (N, 512, H // 32, W // 32)
    assert np.all(np.isfinite(g))
    rel = float(np.max(np.abs(g - ref)) / np.max(np.abs(ref)))
    log(f"[encoder] max-norm relative error {rel:.3e}")
    assert rel <= NORM_TOL[dtype]
    assert sb is not None


def test_encoder_graph_replays_match_eager():
    """The encoder captured as one HIP graph before any eager call: every
    replay, with eager work of the program between replays and new data
    written into the static input, equals the eager forward bit for bit (the
    kernels are deterministic).  Blocks of 64 image pixels at 512 x 512 give
    the deep stages split-K partials in the workspace."""
    from paper_2011_12025_amd.encoder import BlockEncoder
    log("[encoder graph] f16 3x512x512 block 64")
    N, H, W, blk = 1, 512, 512, 64
    Wt = inputs.encoder_weights(93, "f16")
    mask_np = inputs.mask_bernoulli(93, N, H // blk, W // blk, 0.5)
    nh = int(mask_np.sum())
    counts = (nh, mask_np.size - nh)
    mask = torch.from_numpy(mask_np).cuda()
    xa = _cl(inputs.feature_map(93, N, 3, H, W, "f16"))
    xb = _cl(inputs.feature_map(94, N, 3, H, W, "f16"))
    enc = BlockEncoder(Wt, blk)
    x = xa.clone(memory_format=torch.channels_last)
    g, y = enc.capture(x, mask, counts)       # no call before the capture: nothing is allocated by the library
    ws = enc.workspace_bytes(N, H // 4, W // 4, torch.float16, counts)
    log(f"[encoder graph] captured; workspace {ws} bytes")
    assert ws > 0
    ya, yb = enc(xa, mask, counts).clone(), enc(xb, mask, counts).clone()
    for r, (src, ref) in enumerate([(xa, ya), (xb, yb), (xa, ya), (xb, yb)]):
        enc(xb if r % 2 == 0 else xa, mask, counts)       # eager work between replays
        torch.cuda.synchronize()
        x.copy_(src)
        y.zero_()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, ref), f"replay {r} differs from the eager forward"
