"""Stored hand-worked values (tests/golden/): the oracle on the CPU, and the
GPU kernels through the C ABI, must reproduce them bit for bit.

blockpad_two_blocks.json: the configuration of the paper's BlockPad sampling
figure (a 4x4 high block beside a low block of 2x2 pixels), every value
derived by hand from the definitions in Method, Block modules (see the
file's "source").  All values are exact in fp16 and fp32, so no rounding
decides anything.  The GPU case adds 16 c to channel c of a replicated input
(C = 8, whole 16-byte pixels): copies and averages move by the same 16 c,
exactly, while halo zeros stay zero."""
from __future__ import annotations

import json
import os

import numpy as np
import pytest

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))


def load(name):
    with open(os.path.join(HERE, "golden", name)) as f:
        d = json.load(f)
    return {k: (np.array(v, dtype=np.float64) if isinstance(v, list) else v) for k, v in d.items()}


G = load("blockpad_two_blocks.json")
MASK = G["mask"].astype(np.uint8)


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
def test_oracle_reproduces_hand_worked_blockpad(dtype):
    bs, H, W = G["bs"], G["H"], G["W"]
    hi, lo = oracle.split(G["x"].astype(np.float32), MASK, bs, dtype)
    assert np.array_equal(hi, G["split_hi"]) and np.array_equal(lo, G["split_lo"])
    for sampling, ref_lo, ref_hi in [("avg", "pad_lo_avg", "pad_hi"), ("strided", "pad_lo_strided", "pad_hi"),
                                      ("zero", "pad_lo_zero", "pad_hi_zero")]:
        hp, lp = oracle.pad(hi, lo, MASK, bs, H, W, dtype, sampling)
        assert np.array_equal(hp, G[ref_hi]), sampling
        assert np.array_equal(lp, G[ref_lo]), sampling
    assert np.array_equal(oracle.combine(hi, lo, MASK, bs, H, W), G["combine"])


def _with_channels(a, C):
    """Channel c = a + 16 c where a is non-zero (data), 0 where a is 0 (halo)."""
    out = np.repeat(a, C, axis=1)
    for c in range(C):
        out[:, c] = np.where(a[:, 0] != 0, a[:, 0] + 16 * c, 0)
    return out


@pytest.mark.gpu
@pytest.mark.parametrize("layout", ["nchw", "nhwc"])
@pytest.mark.parametrize("dtype", ["f32", "f16"])
def test_gpu_reproduces_hand_worked_blockpad(dtype, layout):
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2011_12025_amd as sb
    td = {"f32": torch.float32, "f16": torch.float16}[dtype]
    bs, H, W, C = G["bs"], G["H"], G["W"], 8
    cl = torch.channels_last if layout == "nhwc" else torch.contiguous_format

    def dev(a):
        return torch.from_numpy(np.ascontiguousarray(a)).to(td).cuda().contiguous(memory_format=cl)

    def host(t):
        return t.float().cpu().numpy()

    md = torch.from_numpy(MASK).cuda()
    hi, lo = sb.split(dev(_with_channels(G["x"], C)), md, bs, counts=(1, 1))
    torch.cuda.synchronize()
    assert np.array_equal(host(hi), _with_channels(G["split_hi"], C))
    assert np.array_equal(host(lo), _with_channels(G["split_lo"], C))
    for sampling, ref_lo, ref_hi in [("avg", "pad_lo_avg", "pad_hi"), ("strided", "pad_lo_strided", "pad_hi"),
                                      ("zero", "pad_lo_zero", "pad_hi_zero")]:
        hp, lp = sb.pad(hi, lo, md, bs, H, W, sampling=sampling)
        torch.cuda.synchronize()
        assert np.array_equal(host(hp), _with_channels(G[ref_hi], C)), sampling
        assert np.array_equal(host(lp), _with_channels(G[ref_lo], C)), sampling
    y = sb.combine(hi, lo, md, bs, H, W)
    torch.cuda.synchronize()
    assert np.array_equal(host(y), _with_channels(G["combine"], C))
