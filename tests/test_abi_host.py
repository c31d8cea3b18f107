"""Host-only checks of the C ABI: the library loads, exports every entry point
that include/segblocks.h declares, and rejects bad arguments on the host
before anything reaches the GPU (no compute call is made here)."""
from __future__ import annotations

import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "segblocks.h")

b = pytest.importorskip("paper_2011_12025_amd._binding")

FAKE = ctypes.c_void_p(0x10000)      # never dereferenced: validation fails first
FAKE2 = ctypes.c_void_p(0x20000000)
NULL = None


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(segblocks_\w+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(b.LIB_PATH):
        pytest.fail("libsegblocks.so is not built (run __graft_entry__.build())")
    return b.lib()


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert set(names) >= {"segblocks_split", "segblocks_pad", "segblocks_conv3x3", "segblocks_combine",
                          "segblocks_layer", "segblocks_count", "segblocks_last_error",
                          "segblocks_block_conv3x3"}
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(b.EXPORTS)


def _split(lib, **kw):
    a = dict(x=FAKE, dtype=1, layout=1, N=1, C=8, H=32, W=32, mask=FAKE2, bs=16, hi=ctypes.c_void_p(0x30000000),
             hi_cap=4, lo=ctypes.c_void_p(0x40000000), lo_cap=4)
    a.update(kw)
    return lib.segblocks_split(a["x"], a["dtype"], a["layout"], a["N"], a["C"], a["H"], a["W"], a["mask"], a["bs"],
                               a["hi"], a["hi_cap"], a["lo"], a["lo_cap"], None)


@pytest.mark.parametrize("kw,code,msg", [
    (dict(dtype=3), -1, "dtype"),
    (dict(layout=2), -1, "layout"),
    (dict(N=0), -1, "positive"),
    (dict(C=-1), -1, "positive"),
    (dict(mask=NULL), -1, "mask"),
    (dict(x=NULL), -1, "x is NULL"),
    (dict(bs=3), -2, "even"),
    (dict(bs=0), -2, "even"),
    (dict(bs=12), -2, "divide"),
    (dict(H=48, bs=32), -2, "divide"),
    (dict(hi=NULL), -1, "hi is NULL"),
    (dict(hi_cap=-1), -1, "capacities"),
    (dict(hi=FAKE), -1, "overlap"),
    (dict(lo=ctypes.c_void_p(0x30000000 + 100)), -1, "overlap"),
])
def test_split_rejects_bad_arguments(lib, kw, code, msg):
    assert _split(lib, **kw) == code
    assert msg in lib.segblocks_last_error().decode()


def test_null_stack_allowed_with_zero_capacity_is_not_an_error_path(lib):
    # only the validation result matters here: a NULL stack with capacity 0 passes
    # validation, so use an invalid dtype to stop before any launch
    assert _split(lib, hi=NULL, hi_cap=0, dtype=9) == -1
    assert "dtype" in lib.segblocks_last_error().decode()


def test_conv_and_layer_validation(lib):
    # conv3x3: bs above the supported maximum
    r = lib.segblocks_conv3x3(FAKE, FAKE2, 1, 1, 1, 8, 512, 512, ctypes.c_void_p(0x50000000), 512,
                              ctypes.c_void_p(0x60000000), NULL, 8, ctypes.c_void_p(0x70000000),
                              ctypes.c_void_p(0x78000000), 1, 0, None)
    assert r == -2 and "256" in lib.segblocks_last_error().decode()
    # missing weight
    r = lib.segblocks_layer(FAKE, 1, 1, 1, 8, 32, 32, FAKE2, 16, NULL, NULL, 8, 0, ctypes.c_void_p(0x50000000), NULL,
                            0, None)
    assert r == -1 and "weight" in lib.segblocks_last_error().decode()
    # output aliasing the input
    r = lib.segblocks_layer(FAKE, 1, 1, 1, 8, 32, 32, FAKE2, 16, ctypes.c_void_p(0x60000000), NULL, 8, 0, FAKE, NULL,
                            0, None)
    assert r == -1 and "overlap" in lib.segblocks_last_error().decode()
    # unknown flag on the fused-pad convolution
    for flags, msg in [(8, "unknown flags"), (6, "exclude each other")]:
        r = lib.segblocks_block_conv3x3(FAKE, FAKE2, 1, 1, 1, 8, 32, 32, ctypes.c_void_p(0x30000000), 16,
                                        ctypes.c_void_p(0x60000000), NULL, 8, flags, NULL, NULL,
                                        ctypes.c_void_p(0x70000000), ctypes.c_void_p(0x78000000), 1, 3, NULL, 0, None)
        assert r == -1 and msg in lib.segblocks_last_error().decode()
        r = lib.segblocks_layer(FAKE, 1, 1, 1, 8, 32, 32, FAKE2, 16, ctypes.c_void_p(0x60000000), NULL, 8, flags,
                                ctypes.c_void_p(0x50000000), NULL, 0, None)
        assert r == -1 and msg in lib.segblocks_last_error().decode()
    # pad_ex: sampling outside the three choices
    r = lib.segblocks_pad_ex(FAKE, FAKE2, 1, 1, 1, 8, 32, 32, ctypes.c_void_p(0x30000000), 16,
                             ctypes.c_void_p(0x40000000), ctypes.c_void_p(0x48000000), 1, 3, 3, None)
    assert r == -1 and "sampling" in lib.segblocks_last_error().decode()


def test_pad_combine_count_validation(lib):
    r = lib.segblocks_pad(FAKE, FAKE2, 1, 0, 1, 4, 16, 16, ctypes.c_void_p(0x30000000), 5,
                          ctypes.c_void_p(0x40000000), ctypes.c_void_p(0x48000000), 1, 1, None)
    assert r == -2
    r = lib.segblocks_combine(FAKE, FAKE2, 1, 0, 1, 4, 16, 16, ctypes.c_void_p(0x30000000), 8, 2, 2, NULL, None)
    assert r == -1 and "y is NULL" in lib.segblocks_last_error().decode()
    nh, nl = ctypes.c_int(), ctypes.c_int()
    r = lib.segblocks_count(NULL, 1, 2, 2, ctypes.byref(nh), ctypes.byref(nl), None)
    assert r == -1


def _ws_query(lib, fn, *args):
    n = ctypes.c_size_t(12345)
    r = getattr(lib, fn)(*args, ctypes.byref(n))
    return r, n.value


def test_workspace_size_queries(lib):
    """The sizes depend on the route the shapes take: none for a fused layer
    on the resident convolution (64 channels, blocks of 32), split-K partials
    for the deep stages, the packed stacks for a fused layer with 512
    channels."""
    r, n = _ws_query(lib, "segblocks_layer_workspace_size", 1, 1, 1, 64, 256, 512, 32, 64)
    assert r == 0 and n == 0
    r, n = _ws_query(lib, "segblocks_block_conv_ex_workspace_size", 1, 1, 1, 512, 32, 64, 4, 512, 3, 1, 128, 128)
    assert r == 0 and n > 0 and n % 256 == 0
    r, n = _ws_query(lib, "segblocks_layer_workspace_size", 1, 1, 1, 512, 32, 64, 4, 512)
    # at least the packed input and output stacks of both classes
    assert r == 0 and n >= 2 * 128 * (16 + 4) * 512 * 2
    r, n = _ws_query(lib, "segblocks_layer_workspace_size", 0, 0, 1, 16, 64, 64, 16, 16)
    assert r == 0 and n == 0        # fp32 NCHW: the general kernel, no scratch
    # bad arguments are rejected like the calls themselves
    r, _ = _ws_query(lib, "segblocks_block_conv_ex_workspace_size", 1, 1, 1, 512, 32, 64, 4, 512, 5, 1, 128, 128)
    assert r == -1 and "ksize" in lib.segblocks_last_error().decode()
    r, _ = _ws_query(lib, "segblocks_layer_workspace_size", 1, 1, 1, 64, 30, 64, 4, 64)
    assert r == -2
    r = lib.segblocks_layer_workspace_size(1, 1, 1, 64, 32, 64, 4, 64, None)
    assert r == -1 and "bytes is NULL" in lib.segblocks_last_error().decode()


def test_calls_reject_missing_or_small_workspace(lib):
    """SB_ENOMEM before anything is launched when the workspace is NULL or
    smaller than the query's size; SB_EINVAL when it is misaligned or
    overlaps an argument (fake device addresses: nothing is dereferenced)."""
    _, need = _ws_query(lib, "segblocks_block_conv_ex_workspace_size", 1, 1, 1, 512, 32, 64, 4, 512, 3, 1, 128, 128)
    P = ctypes.c_void_p
    base = 0x100000000
    args = [P(base), P(base + 0x1000000), 1, 1, 1, 512, 32, 64, P(base + 0x2000000), 4, P(base + 0x3000000), NULL,
            512, 3, 1, 0, NULL, NULL, P(base + 0x4000000), P(base + 0x5000000), 128, 128]
    ws = base + 0x10000000
    assert lib.segblocks_block_conv_ex(*args, NULL, 0, None) == b.SB_ENOMEM
    assert "workspace" in lib.segblocks_last_error().decode()
    assert lib.segblocks_block_conv_ex(*args, P(ws), need - 1, None) == b.SB_ENOMEM
    assert lib.segblocks_block_conv_ex(*args, P(ws + 16), need, None) == b.SB_EINVAL
    assert "aligned" in lib.segblocks_last_error().decode()
    assert lib.segblocks_block_conv_ex(*args, P(base + 0x4000000), need, None) == b.SB_EINVAL   # = hi_out
    assert "overlap" in lib.segblocks_last_error().decode()
    # the fused layer with 512 channels takes its packed stacks from the workspace
    _, lneed = _ws_query(lib, "segblocks_layer_workspace_size", 1, 1, 1, 512, 32, 64, 4, 512)
    largs = [P(base), 1, 1, 1, 512, 32, 64, P(base + 0x2000000), 4, P(base + 0x3000000), NULL, 512, 0,
             P(base + 0x4000000)]
    assert lib.segblocks_layer(*largs, P(ws), lneed // 2, None) == b.SB_ENOMEM
    # block_conv3x3 at a deep-stage shape
    _, bneed = _ws_query(lib, "segblocks_block_conv3x3_workspace_size", 1, 1, 1, 512, 32, 64, 4, 512, 128, 128)
    assert bneed > 0
    bargs = [P(base), P(base + 0x1000000), 1, 1, 1, 512, 32, 64, P(base + 0x2000000), 4, P(base + 0x3000000), NULL,
             512, 0, NULL, NULL, P(base + 0x4000000), P(base + 0x5000000), 128, 128]
    assert lib.segblocks_block_conv3x3(*bargs, NULL, 0, None) == b.SB_ENOMEM


def test_chain_queries_and_validation(lib):
    """segblocks_block_conv_chain: its workspace is what block_conv_ex /
    block_conv3x3 need for the same shapes; the host query tells whether a
    call reads hi_half (the implicit GEMM with average sampling and blocks of
    both classes); a channel count the half-resolution output cannot be
    stored in, or misaligned half stacks, are rejected before anything is launched."""
    _, ex = _ws_query(lib, "segblocks_block_conv_ex_workspace_size", 1, 1, 1, 512, 32, 64, 4, 512, 3, 2, 128, 128)
    r, ch = _ws_query(lib, "segblocks_block_conv_chain_workspace_size", 1, 1, 1, 512, 32, 64, 4, 512, 3, 2, 128, 128)
    assert r == 0 and ch == ex
    _, b3 = _ws_query(lib, "segblocks_block_conv3x3_workspace_size", 1, 1, 1, 512, 32, 64, 4, 512, 128, 128)
    r, ch = _ws_query(lib, "segblocks_block_conv_chain_workspace_size", 1, 1, 1, 512, 32, 64, 4, 512, 3, 1, 128, 128)
    assert r == 0 and ch == b3

    def reads(*a):
        v = ctypes.c_int(7)
        assert lib.segblocks_block_conv_chain_reads_half(*a, ctypes.byref(v)) == 0
        return v.value

    # dtype, layout, N, C_in, H, W, bs, C_out, k, stride, flags, hi_cap, lo_cap
    assert reads(1, 1, 1, 128, 64, 128, 16, 128, 3, 1, 0, 10, 22) == 1
    assert reads(1, 1, 1, 64, 256, 512, 32, 128, 3, 2, 0, 70, 58) == 1      # stride 2: the GEMM
    assert reads(1, 1, 1, 64, 256, 512, 32, 64, 3, 1, 0, 70, 58) == 0       # the resident kernel pads itself
    assert reads(1, 1, 1, 128, 64, 128, 16, 128, 3, 1, 0, 32, 0) == 0       # no low blocks
    assert reads(1, 1, 1, 128, 64, 128, 16, 128, 3, 1, b.SB_FLAG_PAD_STRIDED, 10, 22) == 0
    assert reads(1, 1, 1, 128, 64, 128, 16, 256, 1, 2, 0, 10, 22) == 0      # 1x1: no halo
    v = ctypes.c_int(0)
    assert lib.segblocks_block_conv_chain_reads_half(1, 1, 1, 128, 64, 128, 16, 128, 5, 1, 0, 10, 22,
                                                     ctypes.byref(v)) == b.SB_EINVAL

    P = ctypes.c_void_p
    base = 0x100000000

    _, need = _ws_query(lib, "segblocks_block_conv_chain_workspace_size", 1, 1, 1, 128, 64, 128, 16, 128, 3, 1, 16,
                        16)

    def call(hi_half, hi_out_half, bs=16, stride=1, C_out=128):
        return lib.segblocks_block_conv_chain(P(base), P(base + 0x1000000), hi_half, 1, 1, 1, 128, 64, 128,
                                              P(base + 0x2000000), bs, P(base + 0x3000000), NULL, C_out, 3, stride, 0,
                                              NULL, NULL, P(base + 0x4000000), P(base + 0x5000000), hi_out_half,
                                              16, 16, P(base + 0x10000000), need, None)
    # the half-resolution output is stored 8 channels at a time
    assert call(NULL, P(base + 0x6000000), C_out=12) == b.SB_ESHAPE
    assert "C_out % 8" in lib.segblocks_last_error().decode()
    assert call(P(base + 0x6000008), NULL) == b.SB_EINVAL
    assert "aligned" in lib.segblocks_last_error().decode()
    assert call(NULL, P(base + 0x4000000)) == b.SB_EINVAL        # hi_out_half = hi_out
    assert "overlap" in lib.segblocks_last_error().decode()


def test_bench_runs_on_one_gpu_only():
    """bench.py measures one GPU; asked for more it exits with a message, before
    anything touches a device."""
    import subprocess
    import sys
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=600, cwd=ROOT)
    assert r.returncode != 0
    assert "one GPU only" in r.stdout + r.stderr
