"""segblocks_block_conv_ex_noalloc: the block convolution without a
workspace argument, its scratch space taken from the library's fixed
per-device buffer.  Called through the C ABI and compared with
segblocks_block_conv_ex (caller's workspace) on the same inputs, two calls in
a row with the second on a smaller input, both with scratch in use (split-K
partials, the padded low stack).  The kernels are the same, so the outputs
must agree bit for bit."""
from __future__ import annotations

import ctypes

import pytest
import torch

import paper_2011_12025_amd._binding as B
from paper_2011_12025_amd import inputs


def _cl(t):
    return t.cuda().contiguous(memory_format=torch.channels_last)


def _P(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


# (N, C_in, C_out, H, W, bs, k, stride, p_low, seed)
CALLS = [(1, 128, 128, 64, 128, 8, 3, 2, 0.5, 120),    # padded low stack + split partials
         (1, 256, 256, 16, 32, 4, 3, 1, 0.4, 121)]     # a smaller input: split partials only


def _need(c):
    N, Ci, Co, H, W, bs, k, st, p, seed = c
    m = inputs.mask_bernoulli(seed, N, H // bs, W // bs, p)
    nh = int(m.sum())
    n = ctypes.c_size_t(0)
    rc = B.lib().segblocks_block_conv_ex_workspace_size(B.SB_F16, B.SB_NHWC, N, Ci, H, W, bs, Co, k, st, nh,
                                                       m.size - nh, ctypes.byref(n))
    assert rc == 0
    return m, nh, int(n.value)


def test_noalloc_rejects_needs_beyond_the_fixed_scratch():
    """Host check (no GPU needed): a shape whose scratch exceeds the fixed
    buffer is rejected with SB_ENOMEM before anything is launched."""
    lib = B.lib()
    n = ctypes.c_size_t(0)
    # 128 channels, 4095 low blocks of 8x8 around one high block: the padded
    # low stack alone takes about 105 MB
    rc = lib.segblocks_block_conv_ex_workspace_size(B.SB_F16, B.SB_NHWC, 1, 128, 1024, 1024, 16, 128, 3, 1, 1, 4095,
                                                    ctypes.byref(n))
    assert rc == 0 and n.value > 16 << 20
    P = ctypes.c_void_p
    base = 0x100000000
    rc = lib.segblocks_block_conv_ex_noalloc(P(base), P(base + 0x10000000), B.SB_F16, B.SB_NHWC, 1, 128, 1024, 1024,
                                             P(base + 0x20000000), 16, P(base + 0x30000000), None, 128, 3, 1, 0, None,
                                             None, P(base + 0x40000000), P(base + 0x50000000), 1, 4095, None)
    assert rc == B.SB_ENOMEM
    assert "fixed" in lib.segblocks_last_error().decode()


@pytest.mark.gpu
def test_noalloc_matches_workspace_entry_point():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lib = B.lib()
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    for i, c in enumerate(CALLS):
        N, Ci, Co, H, W, bs, k, st, p, seed = c
        m, nh, need = _need(c)
        nl = m.size - nh
        assert 0 < need <= 16 << 20 and nh > 0 and nl > 0
        print(f"[no-alloc] call {i}: N={N} C={Ci}->{Co} {H}x{W} bs={bs} k{k}s{st} nh={nh} nl={nl} "
              f"scratch {need} B", flush=True)
        x = inputs.feature_map(seed, N, Ci, H, W, "f16")
        hi_np = [x[0, :, (kk // (W // bs)) * bs:(kk // (W // bs) + 1) * bs,
                   (kk % (W // bs)) * bs:(kk % (W // bs) + 1) * bs] for kk in range(m.size) if m.reshape(-1)[kk]]
        lo_np = [torch.nn.functional.avg_pool2d(
            x[0:1, :, (kk // (W // bs)) * bs:(kk // (W // bs) + 1) * bs,
              (kk % (W // bs)) * bs:(kk % (W // bs) + 1) * bs].float(), 2)[0].half()
            for kk in range(m.size) if not m.reshape(-1)[kk]]
        hi, lo = _cl(torch.stack(hi_np)), _cl(torch.stack(lo_np))
        w = _cl(inputs.conv_weight(seed, Co, Ci, k, "f16"))
        b = inputs.conv_bias(seed, Co, k * k * Ci, "f16").cuda()
        md = torch.from_numpy(m).cuda()
        bo, lo_e = bs // st, bs // 2 // st

        def outs():
            return (torch.full((nh, Co, bo, bo), float("nan"), dtype=torch.float16, device="cuda").contiguous(
                        memory_format=torch.channels_last),
                    torch.full((nl, Co, lo_e, lo_e), float("nan"), dtype=torch.float16, device="cuda").contiguous(
                        memory_format=torch.channels_last))
        ref_h, ref_l = outs()
        ws = torch.empty(need + 256, dtype=torch.uint8, device="cuda")
        wp = ws.data_ptr() + (-ws.data_ptr()) % 256
        rc = lib.segblocks_block_conv_ex(_P(hi), _P(lo), B.SB_F16, B.SB_NHWC, N, Ci, H, W, _P(md), bs, _P(w), _P(b), Co,
                                         k, st, 1, None, None, _P(ref_h), _P(ref_l), nh, nl, ctypes.c_void_p(wp),
                                         need, stream)
        assert rc == 0, lib.segblocks_last_error().decode()
        got_h, got_l = outs()
        rc = lib.segblocks_block_conv_ex_noalloc(_P(hi), _P(lo), B.SB_F16, B.SB_NHWC, N, Ci, H, W, _P(md), bs, _P(w),
                                                 _P(b), Co, k, st, 1, None, None, _P(got_h), _P(got_l), nh, nl, stream)
        assert rc == 0, lib.segblocks_last_error().decode()
        torch.cuda.synchronize()
        assert torch.isfinite(ref_h).all() and torch.isfinite(ref_l).all()
        assert torch.equal(got_h, ref_h), f"call {i}: high stack differs"
        assert torch.equal(got_l, ref_l), f"call {i}: low stack differs"
