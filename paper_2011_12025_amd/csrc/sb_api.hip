// C ABI of libsegblocks.so (declared in include/segblocks.h): host-side
// argument validation, then the kernel launches on the caller's stream.
// The library allocates no device memory: scratch space of the convolutions
// comes from the caller's workspace argument, whose size the *_workspace_size
// queries give; nothing touches the GPU before every argument, the workspace
// included, has been checked.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>

#include <mutex>
#include <string>
#include <vector>

#include "segblocks.h"
#include "sb_kernels.h"

namespace {

thread_local std::string g_err;

int fail(int code, const char* fn, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_err = std::string(fn) + ": " + buf;
    return code;
}

int hip_status(const char* fn, hipError_t e) {
    if (e == hipSuccess) {
        g_err.clear();
        return SB_OK;
    }
    return fail(SB_EHIP, fn, "HIP error %d (%s)", (int)e, hipGetErrorString(e));
}

int esize(int dtype) { return dtype == SB_F32 ? 4 : 2; }

struct Range {
    const void* p;
    long long bytes;
};

bool overlap(Range a, Range b) {
    if (!a.p || !b.p || a.bytes <= 0 || b.bytes <= 0) return false;
    const char* a0 = (const char*)a.p;
    const char* b0 = (const char*)b.p;
    return a0 < b0 + b.bytes && b0 < a0 + a.bytes;
}

// Checks dtype, layout, sizes, block size and the mask pointer; fills g.
int check_geo(const char* fn, int dtype, int layout, int N, int C, int H, int W, const uint8_t* mask, int bs,
              sb::Geo& g) {
    if (dtype != SB_F32 && dtype != SB_F16 && dtype != SB_BF16) return fail(SB_EINVAL, fn, "bad dtype %d", dtype);
    if (layout != SB_NCHW && layout != SB_NHWC) return fail(SB_EINVAL, fn, "bad layout %d", layout);
    if (N <= 0 || C <= 0 || H <= 0 || W <= 0)
        return fail(SB_EINVAL, fn, "N, C, H, W must be positive (got %d, %d, %d, %d)", N, C, H, W);
    if (!mask) return fail(SB_EINVAL, fn, "mask is NULL");
    if (bs < 2 || (bs & 1)) return fail(SB_ESHAPE, fn, "block size must be even and >= 2 (got %d)", bs);
    if (H % bs || W % bs) return fail(SB_ESHAPE, fn, "block size %d does not divide H=%d and W=%d", bs, H, W);
    g.N = N; g.C = C; g.H = H; g.W = W; g.bs = bs;
    g.GH = H / bs; g.GW = W / bs;
    g.B = (long long)N * g.GH * g.GW;
    const long long elems = (long long)N * C * H * W;
    if (elems > (1LL << 40) || g.B * (bs + 2) >= (1LL << 31))
        return fail(SB_ESHAPE, fn, "problem too large (N*C*H*W = %lld, blocks = %lld)", elems, g.B);
    return SB_OK;
}

int check_caps(const char* fn, int hi_cap, int lo_cap) {
    if (hi_cap < 0 || lo_cap < 0) return fail(SB_EINVAL, fn, "capacities must be >= 0");
    return SB_OK;
}

// a stack pointer may be NULL only when its capacity is 0
int check_stack(const char* fn, const char* name, const void* p, int cap) {
    if (!p && cap > 0) return fail(SB_EINVAL, fn, "%s is NULL with capacity %d", name, cap);
    return SB_OK;
}

int check_conv_shape(const char* fn, int C_in, int C_out, int bs, const void* weight) {
    if (C_in <= 0 || C_out <= 0) return fail(SB_EINVAL, fn, "C_in and C_out must be positive");
    if (!weight) return fail(SB_EINVAL, fn, "weight is NULL");
    if (bs > 256) return fail(SB_ESHAPE, fn, "convolution supports block sizes up to 256 (got %d)", bs);
    return SB_OK;
}

// A workspace of at least `need` bytes, 256-byte aligned (none needed: anything goes).
int check_ws(const char* fn, size_t need, const void* ws, size_t ws_bytes) {
    if (need == 0) return SB_OK;
    if (!ws || ws_bytes < need)
        return fail(SB_ENOMEM, fn, "needs a workspace of %zu bytes (got %zu at %p)", need, ws ? ws_bytes : (size_t)0, ws);
    if (reinterpret_cast<uintptr_t>(ws) % 256) return fail(SB_EINVAL, fn, "workspace must be 256-byte aligned");
    return SB_OK;
}

bool any_overlap(const std::vector<Range>& outs, const std::vector<Range>& ins) {
    for (size_t i = 0; i < outs.size(); ++i) {
        for (const Range& r : ins)
            if (overlap(outs[i], r)) return true;
        for (size_t j = i + 1; j < outs.size(); ++j)
            if (overlap(outs[i], outs[j])) return true;
    }
    return false;
}

}  // namespace

extern "C" {

const char* segblocks_last_error(void) { return g_err.c_str(); }

int segblocks_count(const uint8_t* mask, int N, int GH, int GW, int* n_high, int* n_low, hipStream_t stream) {
    const char* fn = "segblocks_count";
    if (!mask || !n_high || !n_low) return fail(SB_EINVAL, fn, "NULL pointer argument");
    if (N <= 0 || GH <= 0 || GW <= 0) return fail(SB_EINVAL, fn, "N, GH, GW must be positive");
    const long long B = (long long)N * GH * GW;
    if (B >= (1LL << 31)) return fail(SB_ESHAPE, fn, "too many blocks (%lld)", B);
    std::vector<uint8_t> host((size_t)B);
    hipError_t e = hipMemcpyAsync(host.data(), mask, (size_t)B, hipMemcpyDeviceToHost, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e != hipSuccess) return hip_status(fn, e);
    long long nh = 0;
    for (long long k = 0; k < B; ++k) nh += host[(size_t)k] != 0;
    *n_high = (int)nh;
    *n_low = (int)(B - nh);
    g_err.clear();
    return SB_OK;
}

int segblocks_split(const void* x, int dtype, int layout, int N, int C, int H, int W, const uint8_t* mask, int bs,
                    void* hi, int hi_cap, void* lo, int lo_cap, hipStream_t stream) {
    const char* fn = "segblocks_split";
    sb::Geo g;
    int s;
    if ((s = check_geo(fn, dtype, layout, N, C, H, W, mask, bs, g))) return s;
    if (!x) return fail(SB_EINVAL, fn, "x is NULL");
    if ((s = check_caps(fn, hi_cap, lo_cap)) || (s = check_stack(fn, "hi", hi, hi_cap)) ||
        (s = check_stack(fn, "lo", lo, lo_cap)))
        return s;
    const long long es = esize(dtype), lb = bs / 2;
    const Range rx{x, (long long)N * C * H * W * es}, rm{mask, g.B};
    const Range rh{hi, hi_cap * (long long)C * bs * bs * es}, rl{lo, lo_cap * (long long)C * lb * lb * es};
    if (any_overlap({rh, rl}, {rx, rm})) return fail(SB_EINVAL, fn, "output buffers overlap inputs or each other");
    return hip_status(fn, sb::launch_split(dtype, layout, g, x, mask, hi, hi_cap, lo, lo_cap, stream));
}

namespace {

int pad_impl(const char* fn, const void* hi, const void* lo, int dtype, int layout, int N, int C, int H, int W,
             const uint8_t* mask, int bs, void* hi_pad, void* lo_pad, int hi_cap, int lo_cap, int sampling,
             hipStream_t stream) {
    sb::Geo g;
    int s;
    if ((s = check_geo(fn, dtype, layout, N, C, H, W, mask, bs, g))) return s;
    if (sampling != SB_PAD_AVG && sampling != SB_PAD_STRIDED && sampling != SB_PAD_ZERO)
        return fail(SB_EINVAL, fn, "bad sampling %d", sampling);
    if ((s = check_caps(fn, hi_cap, lo_cap)) || (s = check_stack(fn, "hi", hi, hi_cap)) ||
        (s = check_stack(fn, "lo", lo, lo_cap)) || (s = check_stack(fn, "hi_pad", hi_pad, hi_cap)) ||
        (s = check_stack(fn, "lo_pad", lo_pad, lo_cap)))
        return s;
    const long long es = esize(dtype), lb = bs / 2;
    const Range rh{hi, hi_cap * (long long)C * bs * bs * es}, rl{lo, lo_cap * (long long)C * lb * lb * es};
    const Range rhp{hi_pad, hi_cap * (long long)C * (bs + 2) * (bs + 2) * es};
    const Range rlp{lo_pad, lo_cap * (long long)C * (lb + 2) * (lb + 2) * es};
    if (any_overlap({rhp, rlp}, {rh, rl, Range{mask, g.B}}))
        return fail(SB_EINVAL, fn, "output buffers overlap inputs or each other");
    return hip_status(fn, sb::launch_pad(dtype, layout, g, hi, lo, mask, hi_pad, lo_pad, hi_cap, lo_cap, sampling,
                                         stream));
}

// Flags of the convolutions: ReLU and at most one BlockPad alternative.
int check_conv_flags(const char* fn, int flags) {
    if (flags & ~(SB_FLAG_RELU | SB_FLAG_PAD_STRIDED | SB_FLAG_PAD_ZERO))
        return fail(SB_EINVAL, fn, "unknown flags 0x%x", flags);
    if ((flags & SB_FLAG_PAD_STRIDED) && (flags & SB_FLAG_PAD_ZERO))
        return fail(SB_EINVAL, fn, "SB_FLAG_PAD_STRIDED and SB_FLAG_PAD_ZERO exclude each other");
    return SB_OK;
}

}  // namespace

int segblocks_pad(const void* hi, const void* lo, int dtype, int layout, int N, int C, int H, int W,
                  const uint8_t* mask, int bs, void* hi_pad, void* lo_pad, int hi_cap, int lo_cap,
                  hipStream_t stream) {
    return pad_impl("segblocks_pad", hi, lo, dtype, layout, N, C, H, W, mask, bs, hi_pad, lo_pad, hi_cap, lo_cap,
                    SB_PAD_AVG, stream);
}

int segblocks_pad_ex(const void* hi, const void* lo, int dtype, int layout, int N, int C, int H, int W,
                     const uint8_t* mask, int bs, void* hi_pad, void* lo_pad, int hi_cap, int lo_cap, int sampling,
                     hipStream_t stream) {
    return pad_impl("segblocks_pad_ex", hi, lo, dtype, layout, N, C, H, W, mask, bs, hi_pad, lo_pad, hi_cap, lo_cap,
                    sampling, stream);
}

int segblocks_conv3x3(const void* hi_pad, const void* lo_pad, int dtype, int layout, int N, int C_in, int H, int W,
                      const uint8_t* mask, int bs, const void* weight, const void* bias, int C_out, void* hi_out,
                      void* lo_out, int hi_cap, int lo_cap, hipStream_t stream) {
    const char* fn = "segblocks_conv3x3";
    sb::Geo g;
    int s;
    if ((s = check_geo(fn, dtype, layout, N, C_in, H, W, mask, bs, g))) return s;
    if ((s = check_conv_shape(fn, C_in, C_out, bs, weight))) return s;
    if ((s = check_caps(fn, hi_cap, lo_cap)) || (s = check_stack(fn, "hi_pad", hi_pad, hi_cap)) ||
        (s = check_stack(fn, "lo_pad", lo_pad, lo_cap)) || (s = check_stack(fn, "hi_out", hi_out, hi_cap)) ||
        (s = check_stack(fn, "lo_out", lo_out, lo_cap)))
        return s;
    const long long es = esize(dtype), lb = bs / 2;
    const Range rhp{hi_pad, hi_cap * (long long)C_in * (bs + 2) * (bs + 2) * es};
    const Range rlp{lo_pad, lo_cap * (long long)C_in * (lb + 2) * (lb + 2) * es};
    const Range rw{weight, (long long)C_out * C_in * 9 * es}, rb{bias, bias ? C_out * es : 0};
    const Range rho{hi_out, hi_cap * (long long)C_out * bs * bs * es};
    const Range rlo{lo_out, lo_cap * (long long)C_out * lb * lb * es};
    if (any_overlap({rho, rlo}, {rhp, rlp, rw, rb, Range{mask, g.B}}))
        return fail(SB_EINVAL, fn, "output buffers overlap inputs or each other");
    sb::ConvArgs a{hi_pad, lo_pad, weight, bias, nullptr, nullptr, hi_out, lo_out, C_in, C_out, 0, hi_cap, lo_cap};
    // padded stacks never take a route with scratch memory
    return hip_status(fn, sb::launch_conv(dtype, layout, sb::SRC_PADDED, sb::DST_PACKED, g, mask, a, sb::Ws{nullptr, 0},
                                          stream));
}

int segblocks_combine(const void* hi, const void* lo, int dtype, int layout, int N, int C, int H, int W,
                      const uint8_t* mask, int bs, int hi_cap, int lo_cap, void* y, hipStream_t stream) {
    const char* fn = "segblocks_combine";
    sb::Geo g;
    int s;
    if ((s = check_geo(fn, dtype, layout, N, C, H, W, mask, bs, g))) return s;
    if (!y) return fail(SB_EINVAL, fn, "y is NULL");
    if ((s = check_caps(fn, hi_cap, lo_cap)) || (s = check_stack(fn, "hi", hi, hi_cap)) ||
        (s = check_stack(fn, "lo", lo, lo_cap)))
        return s;
    const long long es = esize(dtype), lb = bs / 2;
    const Range rh{hi, hi_cap * (long long)C * bs * bs * es}, rl{lo, lo_cap * (long long)C * lb * lb * es};
    const Range ry{y, (long long)N * C * H * W * es};
    if (any_overlap({ry}, {rh, rl, Range{mask, g.B}})) return fail(SB_EINVAL, fn, "y overlaps an input");
    return hip_status(fn, sb::launch_combine(dtype, layout, g, hi, lo, mask, hi_cap, lo_cap, y, stream));
}

int segblocks_block_conv3x3(const void* hi, const void* lo, int dtype, int layout, int N, int C_in, int H, int W,
                            const uint8_t* mask, int bs, const void* weight, const void* bias, int C_out, int flags,
                            const void* residual_hi, const void* residual_lo, void* hi_out, void* lo_out,
                            int hi_cap, int lo_cap, void* workspace, size_t ws_bytes, hipStream_t stream) {
    const char* fn = "segblocks_block_conv3x3";
    sb::Geo g;
    int s;
    if ((s = check_geo(fn, dtype, layout, N, C_in, H, W, mask, bs, g))) return s;
    if ((s = check_conv_shape(fn, C_in, C_out, bs, weight))) return s;
    if ((s = check_conv_flags(fn, flags))) return s;
    if ((residual_hi == nullptr) != (residual_lo == nullptr) && hi_cap > 0 && lo_cap > 0)
        return fail(SB_EINVAL, fn, "residual_hi and residual_lo must both be given or both be NULL");
    if ((s = check_caps(fn, hi_cap, lo_cap)) || (s = check_stack(fn, "hi", hi, hi_cap)) ||
        (s = check_stack(fn, "lo", lo, lo_cap)) || (s = check_stack(fn, "hi_out", hi_out, hi_cap)) ||
        (s = check_stack(fn, "lo_out", lo_out, lo_cap)))
        return s;
    sb::ConvArgs a{hi, lo, weight, bias, residual_hi, residual_lo, hi_out, lo_out, C_in, C_out, flags, hi_cap, lo_cap};
    const size_t need = sb::conv_ws_bytes(dtype, layout, sb::SRC_PACKED, sb::DST_PACKED, g, a);
    if ((s = check_ws(fn, need, workspace, ws_bytes))) return s;
    const long long es = esize(dtype), lb = bs / 2;
    const Range rh{hi, hi_cap * (long long)C_in * bs * bs * es}, rl{lo, lo_cap * (long long)C_in * lb * lb * es};
    const Range rw{weight, (long long)C_out * C_in * 9 * es}, rb{bias, bias ? C_out * es : 0};
    const Range rho{hi_out, hi_cap * (long long)C_out * bs * bs * es};
    const Range rlo{lo_out, lo_cap * (long long)C_out * lb * lb * es};
    // the residual may be read at exactly the output location it feeds (in-place add is not allowed either)
    const Range rrh{residual_hi, hi_cap * (long long)C_out * bs * bs * es};
    const Range rrl{residual_lo, lo_cap * (long long)C_out * lb * lb * es};
    const Range rws{workspace, (long long)need};
    if (any_overlap({rho, rlo, rws}, {rh, rl, rw, rb, rrh, rrl, Range{mask, g.B}}))
        return fail(SB_EINVAL, fn, "output buffers or the workspace overlap inputs or each other");
    return hip_status(fn, sb::launch_conv(dtype, layout, sb::SRC_PACKED, sb::DST_PACKED, g, mask, a,
                                          sb::Ws{workspace, ws_bytes}, stream));
}

int segblocks_layer(const void* x, int dtype, int layout, int N, int C_in, int H, int W, const uint8_t* mask,
                    int bs, const void* weight, const void* bias, int C_out, int flags, void* y, void* workspace,
                    size_t ws_bytes, hipStream_t stream) {
    const char* fn = "segblocks_layer";
    sb::Geo g;
    int s;
    if ((s = check_geo(fn, dtype, layout, N, C_in, H, W, mask, bs, g))) return s;
    if ((s = check_conv_shape(fn, C_in, C_out, bs, weight))) return s;
    if ((s = check_conv_flags(fn, flags))) return s;
    if (!x || !y) return fail(SB_EINVAL, fn, "x or y is NULL");
    sb::ConvArgs a{x, nullptr, weight, bias, nullptr, nullptr, y, nullptr, C_in, C_out, flags, 0, 0};
    const size_t need = sb::conv_ws_bytes(dtype, layout, sb::SRC_DENSE, sb::DST_DENSE, g, a);
    if ((s = check_ws(fn, need, workspace, ws_bytes))) return s;
    const long long es = esize(dtype);
    const Range rx{x, (long long)N * C_in * H * W * es}, ry{y, (long long)N * C_out * H * W * es};
    const Range rw{weight, (long long)C_out * C_in * 9 * es}, rb{bias, bias ? C_out * es : 0};
    const Range rws{workspace, (long long)need};
    if (any_overlap({ry, rws}, {rx, rw, rb, Range{mask, g.B}}))
        return fail(SB_EINVAL, fn, "y or the workspace overlaps an input, or each other");
    return hip_status(fn, sb::launch_conv(dtype, layout, sb::SRC_DENSE, sb::DST_DENSE, g, mask, a,
                                          sb::Ws{workspace, ws_bytes}, stream));
}

namespace {

// Validation shared by segblocks_block_conv_ex and its workspace query (no pointers).
int check_conv_ex_shape(const char* fn, int dtype, int layout, int C_in, int bs, int ksize, int stride) {
    if (ksize != 1 && ksize != 3) return fail(SB_EINVAL, fn, "ksize must be 1 or 3 (got %d)", ksize);
    if (stride != 1 && stride != 2) return fail(SB_EINVAL, fn, "stride must be 1 or 2 (got %d)", stride);
    if ((bs / 2) % stride) return fail(SB_ESHAPE, fn, "stride %d does not divide the low block side %d", stride, bs / 2);
    if (layout != SB_NHWC || dtype == SB_F32 || C_in % 8)
        return fail(SB_EINVAL, fn, "supported: channels-last fp16 / bf16 with C_in %% 8 == 0");
    return SB_OK;
}

}  // namespace

namespace {

// The fixed scratch buffer of segblocks_block_conv_ex_noalloc: one copy per
// device, at the device address that hipGetSymbolAddress gives on that
// device (the array's name is a host-side stand-in and is never passed to a
// kernel).  Looked up once per device, under a lock.
constexpr size_t SCRATCH_BYTES = (size_t)SB_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[SCRATCH_BYTES];
std::mutex g_scratch_mu;
void* g_scratch_dev[64];

int scratch_address(const char* fn, void** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_status(fn, e);
    if (dev < 0 || dev >= 64) return fail(SB_EHIP, fn, "device %d out of range", dev);
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_dev[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_status(fn, e);
        if (!p) return fail(SB_EHIP, fn, "no device address for the scratch buffer");
        g_scratch_dev[dev] = p;
    }
    *out = g_scratch_dev[dev];
    return SB_OK;
}

// segblocks_block_conv_ex with the workspace either given by the caller or,
// with fixed_scratch, the library's scratch buffer of this device.
int block_conv_ex_impl(const char* fn, bool fixed_scratch, const void* hi, const void* lo, int dtype, int layout,
                       int N, int C_in, int H, int W, const uint8_t* mask, int bs, const void* weight,
                       const void* bias, int C_out, int ksize, int stride, int flags, const void* residual_hi,
                       const void* residual_lo, void* hi_out, void* lo_out, int hi_cap, int lo_cap, void* workspace,
                       size_t ws_bytes, hipStream_t stream) {
    sb::Geo g;
    int s;
    if ((s = check_geo(fn, dtype, layout, N, C_in, H, W, mask, bs, g))) return s;
    if ((s = check_conv_shape(fn, C_in, C_out, bs, weight))) return s;
    if ((s = check_conv_ex_shape(fn, dtype, layout, C_in, bs, ksize, stride))) return s;
    if ((s = check_conv_flags(fn, flags))) return s;
    if ((residual_hi == nullptr) != (residual_lo == nullptr) && hi_cap > 0 && lo_cap > 0)
        return fail(SB_EINVAL, fn, "residual_hi and residual_lo must both be given or both be NULL");
    if ((s = check_caps(fn, hi_cap, lo_cap)) || (s = check_stack(fn, "hi", hi, hi_cap)) ||
        (s = check_stack(fn, "lo", lo, lo_cap)) || (s = check_stack(fn, "hi_out", hi_out, hi_cap)) ||
        (s = check_stack(fn, "lo_out", lo_out, lo_cap)))
        return s;
    sb::ConvArgs a{hi, lo, weight, bias, residual_hi, residual_lo, hi_out, lo_out, C_in, C_out, flags, hi_cap, lo_cap};
    const size_t need = sb::igemm_fits_shape(dtype, layout, g, a) ? sb::igemm_ws_bytes(g, a, ksize, stride) : 0;
    if (fixed_scratch) {
        if (need > SCRATCH_BYTES)
            return fail(SB_ENOMEM, fn, "needs %zu bytes of scratch, more than the fixed %zu bytes", need,
                        SCRATCH_BYTES);
        workspace = nullptr;
        ws_bytes = 0;
    } else if ((s = check_ws(fn, need, workspace, ws_bytes))) {
        return s;
    }
    const long long es = esize(dtype), lb = bs / 2, bo = bs / stride, lo_e = lb / stride;
    const Range rh{hi, hi_cap * (long long)C_in * bs * bs * es}, rl{lo, lo_cap * (long long)C_in * lb * lb * es};
    const Range rw{weight, (long long)C_out * C_in * ksize * ksize * es}, rb{bias, bias ? C_out * es : 0};
    const Range rho{hi_out, hi_cap * (long long)C_out * bo * bo * es};
    const Range rlo{lo_out, lo_cap * (long long)C_out * lo_e * lo_e * es};
    const Range rrh{residual_hi, hi_cap * (long long)C_out * bo * bo * es};
    const Range rrl{residual_lo, lo_cap * (long long)C_out * lo_e * lo_e * es};
    const Range rws{workspace, (long long)need};
    if (any_overlap({rho, rlo, rws}, {rh, rl, rw, rb, rrh, rrl, Range{mask, g.B}}))
        return fail(SB_EINVAL, fn, "output buffers or the workspace overlap inputs or each other");
    if (fixed_scratch && need > 0) {
        // every byte of scratch that a launch reads, it has written first (split
        // partials, their row counts, the padded low stack): nothing to clear
        if ((s = scratch_address(fn, &workspace))) return s;
        ws_bytes = SCRATCH_BYTES;
    }
    if (sb::igemm_fits(dtype, layout, g, a))
        return hip_status(fn, sb::launch_igemm(dtype, g, mask, a, ksize, stride, sb::Ws{workspace, ws_bytes}, stream));
    return hip_status(fn, sb::launch_bconv(dtype, g, mask, a, ksize, stride, stream));
}

}  // namespace

int segblocks_block_conv_ex(const void* hi, const void* lo, int dtype, int layout, int N, int C_in, int H, int W,
                            const uint8_t* mask, int bs, const void* weight, const void* bias, int C_out, int ksize,
                            int stride, int flags, const void* residual_hi, const void* residual_lo, void* hi_out,
                            void* lo_out, int hi_cap, int lo_cap, void* workspace, size_t ws_bytes,
                            hipStream_t stream) {
    return block_conv_ex_impl("segblocks_block_conv_ex", false, hi, lo, dtype, layout, N, C_in, H, W, mask, bs, weight,
                              bias, C_out, ksize, stride, flags, residual_hi, residual_lo, hi_out, lo_out, hi_cap,
                              lo_cap, workspace, ws_bytes, stream);
}

int segblocks_block_conv_ex_noalloc(const void* hi, const void* lo, int dtype, int layout, int N, int C_in, int H,
                                    int W, const uint8_t* mask, int bs, const void* weight, const void* bias,
                                    int C_out, int ksize, int stride, int flags, const void* residual_hi,
                                    const void* residual_lo, void* hi_out, void* lo_out, int hi_cap, int lo_cap,
                                    hipStream_t stream) {
    return block_conv_ex_impl("segblocks_block_conv_ex_noalloc", true, hi, lo, dtype, layout, N, C_in, H, W, mask, bs,
                              weight, bias, C_out, ksize, stride, flags, residual_hi, residual_lo, hi_out, lo_out,
                              hi_cap, lo_cap, nullptr, 0, stream);
}

int segblocks_block_conv_chain(const void* hi, const void* lo, const void* hi_half, int dtype, int layout, int N,
                               int C_in, int H, int W, const uint8_t* mask, int bs, const void* weight,
                               const void* bias, int C_out, int ksize, int stride, int flags, const void* residual_hi,
                               const void* residual_lo, void* hi_out, void* lo_out, void* hi_out_half, int hi_cap,
                               int lo_cap, void* workspace, size_t ws_bytes, hipStream_t stream) {
    const char* fn = "segblocks_block_conv_chain";
    sb::Geo g;
    int s;
    if ((s = check_geo(fn, dtype, layout, N, C_in, H, W, mask, bs, g))) return s;
    if ((s = check_conv_shape(fn, C_in, C_out, bs, weight))) return s;
    if ((s = check_conv_ex_shape(fn, dtype, layout, C_in, bs, ksize, stride))) return s;
    if ((s = check_conv_flags(fn, flags))) return s;
    if ((residual_hi == nullptr) != (residual_lo == nullptr) && hi_cap > 0 && lo_cap > 0)
        return fail(SB_EINVAL, fn, "residual_hi and residual_lo must both be given or both be NULL");
    if ((s = check_caps(fn, hi_cap, lo_cap)) || (s = check_stack(fn, "hi", hi, hi_cap)) ||
        (s = check_stack(fn, "lo", lo, lo_cap)) || (s = check_stack(fn, "hi_out", hi_out, hi_cap)) ||
        (s = check_stack(fn, "lo_out", lo_out, lo_cap)))
        return s;
    const long long es = esize(dtype), lb = bs / 2, bo = bs / stride, lo_e = lb / stride;
    if (hi_out_half && (bo % 2 || C_out % 8))
        return fail(SB_ESHAPE, fn, "hi_out_half needs an even output block side and C_out %% 8 == 0 (got %lld, %d)",
                    bo, C_out);
    if ((reinterpret_cast<uintptr_t>(hi_half) | reinterpret_cast<uintptr_t>(hi_out_half)) % 16 ||
        (hi_out_half && reinterpret_cast<uintptr_t>(hi_out) % 16))
        return fail(SB_EINVAL, fn, "hi_half, hi_out_half and (with hi_out_half) hi_out must be 16-byte aligned");
    sb::ConvArgs a{hi, lo, weight, bias, residual_hi, residual_lo, hi_out, lo_out, C_in, C_out, flags, hi_cap, lo_cap};
    a.in_hs = hi_half;
    a.out_hs = hi_out_half;
    // 3x3 at stride 1 takes the routes of segblocks_block_conv3x3, the rest
    // those of segblocks_block_conv_ex; only the implicit GEMM reads hi_half
    // and writes hi_out_half itself (in the resident kernel the extra
    // registers cost more than the launch after it)
    const bool k33 = ksize == 3 && stride == 1;
    const size_t need = k33 ? sb::conv_ws_bytes(dtype, layout, sb::SRC_PACKED, sb::DST_PACKED, g, a)
                            : (sb::igemm_fits_shape(dtype, layout, g, a) ? sb::igemm_ws_bytes(g, a, ksize, stride) : 0);
    if ((s = check_ws(fn, need, workspace, ws_bytes))) return s;
    const Range rh{hi, hi_cap * (long long)C_in * bs * bs * es}, rl{lo, lo_cap * (long long)C_in * lb * lb * es};
    const Range rhh{hi_half, hi_half ? hi_cap * (long long)C_in * (lb * lb) * es : 0};
    const Range rw{weight, (long long)C_out * C_in * ksize * ksize * es}, rb{bias, bias ? C_out * es : 0};
    const Range rho{hi_out, hi_cap * (long long)C_out * bo * bo * es};
    const Range rlo{lo_out, lo_cap * (long long)C_out * lo_e * lo_e * es};
    const Range rhoh{hi_out_half, hi_out_half ? hi_cap * (long long)C_out * (bo / 2) * (bo / 2) * es : 0};
    const Range rrh{residual_hi, hi_cap * (long long)C_out * bo * bo * es};
    const Range rrl{residual_lo, lo_cap * (long long)C_out * lo_e * lo_e * es};
    const Range rws{workspace, (long long)need};
    if (any_overlap({rho, rlo, rhoh, rws}, {rh, rl, rhh, rw, rb, rrh, rrl, Range{mask, g.B}}))
        return fail(SB_EINVAL, fn, "output buffers or the workspace overlap inputs or each other");
    const sb::Ws ws{workspace, ws_bytes};
    bool gemm;
    hipError_t e;
    if (k33) {
        gemm = !sb::conv_res_fits(dtype, layout, g, a) && sb::igemm_fits(dtype, layout, g, a);
        e = sb::launch_conv(dtype, layout, sb::SRC_PACKED, sb::DST_PACKED, g, mask, a, ws, stream);
    } else {
        gemm = sb::igemm_fits(dtype, layout, g, a);
        e = gemm ? sb::launch_igemm(dtype, g, mask, a, ksize, stride, ws, stream)
                 : sb::launch_bconv(dtype, g, mask, a, ksize, stride, stream);
    }
    if (e == hipSuccess && hi_out_half && !gemm)
        e = sb::launch_sample_hs(dtype, hi_out, hi_cap, (int)bo, C_out, hi_out_half, stream);
    return hip_status(fn, e);
}

namespace {

// Geometry of a workspace query: the checks of check_geo without a mask.
int check_query(const char* fn, int dtype, int layout, int N, int C_in, int H, int W, int bs, int C_out,
                size_t* bytes, sb::Geo& g) {
    static const uint8_t any = 0;
    if (!bytes) return fail(SB_EINVAL, fn, "bytes is NULL");
    int s;
    if ((s = check_geo(fn, dtype, layout, N, C_in, H, W, &any, bs, g))) return s;
    if (C_out <= 0) return fail(SB_EINVAL, fn, "C_out must be positive");
    if (bs > 256) return fail(SB_ESHAPE, fn, "convolution supports block sizes up to 256 (got %d)", bs);
    return SB_OK;
}

}  // namespace

int segblocks_block_conv3x3_workspace_size(int dtype, int layout, int N, int C_in, int H, int W, int bs, int C_out,
                                           int hi_cap, int lo_cap, size_t* bytes) {
    const char* fn = "segblocks_block_conv3x3_workspace_size";
    sb::Geo g;
    int s;
    if ((s = check_query(fn, dtype, layout, N, C_in, H, W, bs, C_out, bytes, g)) || (s = check_caps(fn, hi_cap, lo_cap)))
        return s;
    // the most any flags need: average sampling may take the resident kernel
    // (no workspace), the BlockPad alternatives then take the GEMM
    sb::ConvArgs a{nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, C_in, C_out, 0, hi_cap,
                   lo_cap};
    size_t n = sb::conv_ws_bytes(dtype, layout, sb::SRC_PACKED, sb::DST_PACKED, g, a);
    a.flags = SB_FLAG_PAD_STRIDED;
    const size_t n2 = sb::conv_ws_bytes(dtype, layout, sb::SRC_PACKED, sb::DST_PACKED, g, a);
    *bytes = n > n2 ? n : n2;
    g_err.clear();
    return SB_OK;
}

int segblocks_block_conv_ex_workspace_size(int dtype, int layout, int N, int C_in, int H, int W, int bs, int C_out,
                                           int ksize, int stride, int hi_cap, int lo_cap, size_t* bytes) {
    const char* fn = "segblocks_block_conv_ex_workspace_size";
    sb::Geo g;
    int s;
    if ((s = check_query(fn, dtype, layout, N, C_in, H, W, bs, C_out, bytes, g)) ||
        (s = check_conv_ex_shape(fn, dtype, layout, C_in, bs, ksize, stride)) || (s = check_caps(fn, hi_cap, lo_cap)))
        return s;
    sb::ConvArgs a{nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, C_in, C_out, 0, hi_cap,
                   lo_cap};
    *bytes = sb::igemm_fits_shape(dtype, layout, g, a) ? sb::igemm_ws_bytes(g, a, ksize, stride) : 0;
    g_err.clear();
    return SB_OK;
}

int segblocks_block_conv_chain_workspace_size(int dtype, int layout, int N, int C_in, int H, int W, int bs,
                                              int C_out, int ksize, int stride, int hi_cap, int lo_cap,
                                              size_t* bytes) {
    const char* fn = "segblocks_block_conv_chain_workspace_size";
    sb::Geo g;
    int s;
    if ((s = check_query(fn, dtype, layout, N, C_in, H, W, bs, C_out, bytes, g)) ||
        (s = check_conv_ex_shape(fn, dtype, layout, C_in, bs, ksize, stride)) || (s = check_caps(fn, hi_cap, lo_cap)))
        return s;
    // the most any flags need without hi_half (with it a call needs no more)
    sb::ConvArgs a{nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, C_in, C_out, 0, hi_cap,
                   lo_cap};
    size_t n = 0;
    for (int f : {0, (int)SB_FLAG_PAD_STRIDED}) {
        a.flags = f;
        const size_t k = ksize == 3 && stride == 1
                             ? sb::conv_ws_bytes(dtype, layout, sb::SRC_PACKED, sb::DST_PACKED, g, a)
                             : (sb::igemm_fits_shape(dtype, layout, g, a) ? sb::igemm_ws_bytes(g, a, ksize, stride) : 0);
        n = k > n ? k : n;
    }
    *bytes = n;
    g_err.clear();
    return SB_OK;
}

int segblocks_block_conv_chain_reads_half(int dtype, int layout, int N, int C_in, int H, int W, int bs, int C_out,
                                          int ksize, int stride, int flags, int hi_cap, int lo_cap, int* reads) {
    const char* fn = "segblocks_block_conv_chain_reads_half";
    sb::Geo g;
    size_t unused = 0;
    int s;
    if (!reads) return fail(SB_EINVAL, fn, "reads is NULL");
    if ((s = check_query(fn, dtype, layout, N, C_in, H, W, bs, C_out, &unused, g)) ||
        (s = check_conv_ex_shape(fn, dtype, layout, C_in, bs, ksize, stride)) || (s = check_caps(fn, hi_cap, lo_cap)) ||
        (s = check_conv_flags(fn, flags)))
        return s;
    sb::ConvArgs a{nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, C_in, C_out, flags, hi_cap,
                   lo_cap};
    // the implicit GEMM's route (16-byte aligned buffers), average sampling,
    // a 3x3 kernel and blocks of both classes
    const bool gemm = sb::igemm_fits_shape(dtype, layout, g, a) &&
                      !(ksize == 3 && stride == 1 && sb::conv_res_fits_shape(dtype, layout, g, a));
    *reads = gemm && ksize == 3 && (flags & (SB_FLAG_PAD_STRIDED | SB_FLAG_PAD_ZERO)) == 0 && hi_cap > 0 && lo_cap > 0;
    g_err.clear();
    return SB_OK;
}

int segblocks_layer_workspace_size(int dtype, int layout, int N, int C_in, int H, int W, int bs, int C_out,
                                   size_t* bytes) {
    const char* fn = "segblocks_layer_workspace_size";
    sb::Geo g;
    int s;
    if ((s = check_query(fn, dtype, layout, N, C_in, H, W, bs, C_out, bytes, g))) return s;
    sb::ConvArgs a{nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, C_in, C_out, 0, 0, 0};
    size_t n = sb::conv_ws_bytes(dtype, layout, sb::SRC_DENSE, sb::DST_DENSE, g, a);
    a.flags = SB_FLAG_PAD_STRIDED;
    const size_t n2 = sb::conv_ws_bytes(dtype, layout, sb::SRC_DENSE, sb::DST_DENSE, g, a);
    *bytes = n > n2 ? n : n2;
    g_err.clear();
    return SB_OK;
}

// ---------------------------------------------------------------------------
// Wider halos: layers beyond 3x3 on block stacks
// ---------------------------------------------------------------------------

int segblocks_pad_halo(const void* hi, const void* lo, int dtype, int layout, int N, int C, int H, int W,
                       const uint8_t* mask, int bs, int halo, int sampling, void* hi_pad, void* lo_pad, int hi_cap,
                       int lo_cap, hipStream_t stream) {
    const char* fn = "segblocks_pad_halo";
    sb::Geo g;
    int s;
    if ((s = check_geo(fn, dtype, layout, N, C, H, W, mask, bs, g))) return s;
    if (halo < 1 || halo > bs / 2) return fail(SB_ESHAPE, fn, "halo must be between 1 and bs/2 = %d (got %d)", bs / 2, halo);
    if (sampling != SB_PAD_AVG && sampling != SB_PAD_STRIDED && sampling != SB_PAD_ZERO)
        return fail(SB_EINVAL, fn, "bad sampling %d", sampling);
    if ((s = check_caps(fn, hi_cap, lo_cap)) || (s = check_stack(fn, "hi", hi, hi_cap)) ||
        (s = check_stack(fn, "lo", lo, lo_cap)) || (s = check_stack(fn, "hi_pad", hi_pad, hi_cap)) ||
        (s = check_stack(fn, "lo_pad", lo_pad, lo_cap)))
        return s;
    const long long es = esize(dtype), lb = bs / 2, ph = bs + 2 * halo, pl = lb + 2 * halo;
    const Range rh{hi, hi_cap * (long long)C * bs * bs * es}, rl{lo, lo_cap * (long long)C * lb * lb * es};
    const Range rhp{hi_pad, hi_cap * (long long)C * ph * ph * es}, rlp{lo_pad, lo_cap * (long long)C * pl * pl * es};
    if (any_overlap({rhp, rlp}, {rh, rl, Range{mask, g.B}}))
        return fail(SB_EINVAL, fn, "output buffers overlap inputs or each other");
    return hip_status(fn, sb::launch_pad(dtype, layout, g, hi, lo, mask, hi_pad, lo_pad, hi_cap, lo_cap, sampling,
                                         stream, halo));
}

int segblocks_conv_halo(const void* hi_pad, const void* lo_pad, int dtype, int layout, int N, int C_in, int H, int W,
                        const uint8_t* mask, int bs, int halo, const void* weight, const void* bias, int C_out,
                        int ksize, int stride, int dilation, int flags, void* hi_out, void* lo_out, int hi_cap,
                        int lo_cap, hipStream_t stream) {
    const char* fn = "segblocks_conv_halo";
    sb::Geo g;
    int s;
    if ((s = check_geo(fn, dtype, layout, N, C_in, H, W, mask, bs, g))) return s;
    if ((s = check_conv_shape(fn, C_in, C_out, bs, weight))) return s;
    if (ksize < 1 || ksize % 2 == 0) return fail(SB_EINVAL, fn, "ksize must be odd (got %d)", ksize);
    if (stride != 1 && stride != 2) return fail(SB_EINVAL, fn, "stride must be 1 or 2 (got %d)", stride);
    if (dilation < 1) return fail(SB_EINVAL, fn, "dilation must be >= 1 (got %d)", dilation);
    if (halo < 1 || halo > bs / 2) return fail(SB_ESHAPE, fn, "halo must be between 1 and bs/2 (got %d)", halo);
    if (dilation * (ksize - 1) / 2 > halo)
        return fail(SB_ESHAPE, fn, "the kernel reaches %d pixels beyond the block, the halo is %d",
                    dilation * (ksize - 1) / 2, halo);
    if ((bs / 2) % stride) return fail(SB_ESHAPE, fn, "stride %d does not divide the low block side %d", stride, bs / 2);
    if (flags & ~SB_FLAG_RELU) return fail(SB_EINVAL, fn, "unknown flags 0x%x", flags);
    if ((s = check_caps(fn, hi_cap, lo_cap)) || (s = check_stack(fn, "hi_pad", hi_pad, hi_cap)) ||
        (s = check_stack(fn, "lo_pad", lo_pad, lo_cap)) || (s = check_stack(fn, "hi_out", hi_out, hi_cap)) ||
        (s = check_stack(fn, "lo_out", lo_out, lo_cap)))
        return s;
    const long long es = esize(dtype), lb = bs / 2, ph = bs + 2 * halo, pl = lb + 2 * halo;
    const long long bo = bs / stride, lo_e = lb / stride;
    const Range rhp{hi_pad, hi_cap * (long long)C_in * ph * ph * es}, rlp{lo_pad, lo_cap * (long long)C_in * pl * pl * es};
    const Range rw{weight, (long long)C_out * C_in * ksize * ksize * es}, rb{bias, bias ? C_out * es : 0};
    const Range rho{hi_out, hi_cap * (long long)C_out * bo * bo * es};
    const Range rlo{lo_out, lo_cap * (long long)C_out * lo_e * lo_e * es};
    if (any_overlap({rho, rlo}, {rhp, rlp, rw, rb, Range{mask, g.B}}))
        return fail(SB_EINVAL, fn, "output buffers overlap inputs or each other");
    return hip_status(fn, sb::launch_conv_halo(dtype, layout, g, hi_pad, lo_pad, mask, halo, weight, bias, C_in, C_out,
                                               ksize, stride, dilation, flags, hi_out, lo_out, hi_cap, lo_cap, stream));
}

int segblocks_maxpool_halo(const void* hi_pad, const void* lo_pad, int dtype, int layout, int N, int C, int H, int W,
                           const uint8_t* mask, int bs, int halo, int ksize, int stride, void* hi_out, void* lo_out,
                           int hi_cap, int lo_cap, hipStream_t stream) {
    const char* fn = "segblocks_maxpool_halo";
    sb::Geo g;
    int s;
    if ((s = check_geo(fn, dtype, layout, N, C, H, W, mask, bs, g))) return s;
    if (ksize < 1 || ksize % 2 == 0) return fail(SB_EINVAL, fn, "ksize must be odd (got %d)", ksize);
    if (stride != 1 && stride != 2) return fail(SB_EINVAL, fn, "stride must be 1 or 2 (got %d)", stride);
    if (halo < 1 || halo > bs / 2 || (ksize - 1) / 2 > halo)
        return fail(SB_ESHAPE, fn, "halo %d must cover the window (%d) and be at most bs/2", halo, (ksize - 1) / 2);
    if ((bs / 2) % stride) return fail(SB_ESHAPE, fn, "stride %d does not divide the low block side %d", stride, bs / 2);
    if ((s = check_caps(fn, hi_cap, lo_cap)) || (s = check_stack(fn, "hi_pad", hi_pad, hi_cap)) ||
        (s = check_stack(fn, "lo_pad", lo_pad, lo_cap)) || (s = check_stack(fn, "hi_out", hi_out, hi_cap)) ||
        (s = check_stack(fn, "lo_out", lo_out, lo_cap)))
        return s;
    const long long es = esize(dtype), lb = bs / 2, ph = bs + 2 * halo, pl = lb + 2 * halo;
    const long long bo = bs / stride, lo_e = lb / stride;
    const Range rhp{hi_pad, hi_cap * (long long)C * ph * ph * es}, rlp{lo_pad, lo_cap * (long long)C * pl * pl * es};
    const Range rho{hi_out, hi_cap * (long long)C * bo * bo * es}, rlo{lo_out, lo_cap * (long long)C * lo_e * lo_e * es};
    if (any_overlap({rho, rlo}, {rhp, rlp, Range{mask, g.B}}))
        return fail(SB_EINVAL, fn, "output buffers overlap inputs or each other");
    return hip_status(fn, sb::launch_maxpool_halo(dtype, layout, g, hi_pad, lo_pad, mask, halo, ksize, stride, hi_out,
                                                  lo_out, hi_cap, lo_cap, stream));
}

// ---------------------------------------------------------------------------
// Backward pass
// ---------------------------------------------------------------------------

int segblocks_combine_backward(const void* dy, int dtype, int layout, int N, int C, int H, int W,
                               const uint8_t* mask, int bs, void* dhi, int hi_cap, void* dlo, int lo_cap,
                               hipStream_t stream) {
    const char* fn = "segblocks_combine_backward";
    sb::Geo g;
    int s;
    if ((s = check_geo(fn, dtype, layout, N, C, H, W, mask, bs, g))) return s;
    if (!dy) return fail(SB_EINVAL, fn, "dy is NULL");
    if ((s = check_caps(fn, hi_cap, lo_cap)) || (s = check_stack(fn, "dhi", dhi, hi_cap)) ||
        (s = check_stack(fn, "dlo", dlo, lo_cap)))
        return s;
    const long long es = esize(dtype), lb = bs / 2;
    const Range ry{dy, (long long)N * C * H * W * es}, rm{mask, g.B};
    const Range rh{dhi, hi_cap * (long long)C * bs * bs * es}, rl{dlo, lo_cap * (long long)C * lb * lb * es};
    if (any_overlap({rh, rl}, {ry, rm})) return fail(SB_EINVAL, fn, "output buffers overlap inputs or each other");
    return hip_status(fn, sb::launch_split(dtype, layout, g, dy, mask, dhi, hi_cap, dlo, lo_cap, stream, true));
}

int segblocks_split_backward(const void* dhi, const void* dlo, int dtype, int layout, int N, int C, int H, int W,
                             const uint8_t* mask, int bs, int hi_cap, int lo_cap, void* dx, hipStream_t stream) {
    const char* fn = "segblocks_split_backward";
    sb::Geo g;
    int s;
    if ((s = check_geo(fn, dtype, layout, N, C, H, W, mask, bs, g))) return s;
    if (!dx) return fail(SB_EINVAL, fn, "dx is NULL");
    if ((s = check_caps(fn, hi_cap, lo_cap)) || (s = check_stack(fn, "dhi", dhi, hi_cap)) ||
        (s = check_stack(fn, "dlo", dlo, lo_cap)))
        return s;
    const long long es = esize(dtype), lb = bs / 2;
    const Range rh{dhi, hi_cap * (long long)C * bs * bs * es}, rl{dlo, lo_cap * (long long)C * lb * lb * es};
    const Range rx{dx, (long long)N * C * H * W * es};
    if (any_overlap({rx}, {rh, rl, Range{mask, g.B}})) return fail(SB_EINVAL, fn, "dx overlaps an input");
    return hip_status(fn, sb::launch_combine(dtype, layout, g, dhi, dlo, mask, hi_cap, lo_cap, dx, stream, true));
}

int segblocks_pad_backward(const void* dhp, const void* dlp, int dtype, int layout, int N, int C, int H, int W,
                           const uint8_t* mask, int bs, int sampling, void* dhi, void* dlo, int hi_cap, int lo_cap,
                           hipStream_t stream) {
    const char* fn = "segblocks_pad_backward";
    sb::Geo g;
    int s;
    if ((s = check_geo(fn, dtype, layout, N, C, H, W, mask, bs, g))) return s;
    if (sampling != SB_PAD_AVG && sampling != SB_PAD_STRIDED && sampling != SB_PAD_ZERO)
        return fail(SB_EINVAL, fn, "bad sampling %d", sampling);
    if ((s = check_caps(fn, hi_cap, lo_cap)) || (s = check_stack(fn, "dhp", dhp, hi_cap)) ||
        (s = check_stack(fn, "dlp", dlp, lo_cap)) || (s = check_stack(fn, "dhi", dhi, hi_cap)) ||
        (s = check_stack(fn, "dlo", dlo, lo_cap)))
        return s;
    const long long es = esize(dtype), lb = bs / 2;
    const Range rhp{dhp, hi_cap * (long long)C * (bs + 2) * (bs + 2) * es};
    const Range rlp{dlp, lo_cap * (long long)C * (lb + 2) * (lb + 2) * es};
    const Range rh{dhi, hi_cap * (long long)C * bs * bs * es}, rl{dlo, lo_cap * (long long)C * lb * lb * es};
    if (any_overlap({rh, rl}, {rhp, rlp, Range{mask, g.B}}))
        return fail(SB_EINVAL, fn, "output buffers overlap inputs or each other");
    return hip_status(fn, sb::launch_pad_bwd(dtype, layout, g, dhp, dlp, mask, dhi, dlo, hi_cap, lo_cap, sampling,
                                             stream));
}

int segblocks_conv3x3_backward_data_workspace_size(int dtype, int layout, int N, int C_in, int H, int W, int bs,
                                                   int C_out, int hi_cap, int lo_cap, size_t* bytes) {
    const char* fn = "segblocks_conv3x3_backward_data_workspace_size";
    sb::Geo g;
    int s;
    if ((s = check_query(fn, dtype, layout, N, C_in, H, W, bs, C_out, bytes, g)) || (s = check_caps(fn, hi_cap, lo_cap)))
        return s;
    *bytes = sb::dgrad_ws_bytes(dtype, layout, g, C_in, C_out, hi_cap, lo_cap);
    g_err.clear();
    return SB_OK;
}

int segblocks_conv3x3_backward_data(const void* dho, const void* dlo, int dtype, int layout, int N, int C_in, int H,
                                    int W, const uint8_t* mask, int bs, const void* weight, int C_out, void* dhp,
                                    void* dlp, int hi_cap, int lo_cap, void* workspace, size_t ws_bytes,
                                    hipStream_t stream) {
    const char* fn = "segblocks_conv3x3_backward_data";
    sb::Geo g;
    int s;
    if ((s = check_geo(fn, dtype, layout, N, C_in, H, W, mask, bs, g))) return s;
    if ((s = check_conv_shape(fn, C_in, C_out, bs + 4, weight))) return s;
    if ((s = check_caps(fn, hi_cap, lo_cap)) || (s = check_stack(fn, "dho", dho, hi_cap)) ||
        (s = check_stack(fn, "dlo", dlo, lo_cap)) || (s = check_stack(fn, "dhp", dhp, hi_cap)) ||
        (s = check_stack(fn, "dlp", dlp, lo_cap)))
        return s;
    const size_t need = sb::dgrad_ws_bytes(dtype, layout, g, C_in, C_out, hi_cap, lo_cap);
    if ((s = check_ws(fn, need, workspace, ws_bytes))) return s;
    const long long es = esize(dtype), lb = bs / 2;
    const Range rho{dho, hi_cap * (long long)C_out * bs * bs * es}, rlo{dlo, lo_cap * (long long)C_out * lb * lb * es};
    const Range rw{weight, (long long)C_out * C_in * 9 * es};
    const Range rhp{dhp, hi_cap * (long long)C_in * (bs + 2) * (bs + 2) * es};
    const Range rlp{dlp, lo_cap * (long long)C_in * (lb + 2) * (lb + 2) * es};
    const Range rws{workspace, (long long)need};
    if (any_overlap({rhp, rlp, rws}, {rho, rlo, rw, Range{mask, g.B}}))
        return fail(SB_EINVAL, fn, "output buffers or the workspace overlap inputs or each other");
    return hip_status(fn, sb::launch_dgrad(dtype, layout, g, dho, dlo, mask, weight, C_in, C_out, dhp, dlp, hi_cap,
                                           lo_cap, sb::Ws{workspace, ws_bytes}, stream));
}

int segblocks_conv3x3_backward_weight_workspace_size(int dtype, int layout, int N, int C_in, int H, int W, int bs,
                                                     int C_out, int hi_cap, int lo_cap, int with_bias, size_t* bytes) {
    const char* fn = "segblocks_conv3x3_backward_weight_workspace_size";
    sb::Geo g;
    int s;
    if ((s = check_query(fn, dtype, layout, N, C_in, H, W, bs, C_out, bytes, g)) || (s = check_caps(fn, hi_cap, lo_cap)))
        return s;
    *bytes = sb::wgrad_ws_bytes(dtype, layout, g, C_in, C_out, hi_cap, lo_cap, with_bias != 0);
    g_err.clear();
    return SB_OK;
}

int segblocks_conv3x3_backward_weight(const void* hp, const void* lp, const void* dho, const void* dlo, int dtype,
                                      int layout, int N, int C_in, int H, int W, const uint8_t* mask, int bs,
                                      int C_out, void* dweight, void* dbias, int hi_cap, int lo_cap, void* workspace,
                                      size_t ws_bytes, hipStream_t stream) {
    const char* fn = "segblocks_conv3x3_backward_weight";
    sb::Geo g;
    int s;
    if ((s = check_geo(fn, dtype, layout, N, C_in, H, W, mask, bs, g))) return s;
    if ((s = check_conv_shape(fn, C_in, C_out, bs, dweight))) return s;
    if ((s = check_caps(fn, hi_cap, lo_cap)) || (s = check_stack(fn, "hp", hp, hi_cap)) ||
        (s = check_stack(fn, "lp", lp, lo_cap)) || (s = check_stack(fn, "dho", dho, hi_cap)) ||
        (s = check_stack(fn, "dlo", dlo, lo_cap)))
        return s;
    const size_t need = sb::wgrad_ws_bytes(dtype, layout, g, C_in, C_out, hi_cap, lo_cap, dbias != nullptr);
    if ((s = check_ws(fn, need, workspace, ws_bytes))) return s;
    const long long es = esize(dtype), lb = bs / 2;
    const Range rhp{hp, hi_cap * (long long)C_in * (bs + 2) * (bs + 2) * es};
    const Range rlp{lp, lo_cap * (long long)C_in * (lb + 2) * (lb + 2) * es};
    const Range rho{dho, hi_cap * (long long)C_out * bs * bs * es}, rlo{dlo, lo_cap * (long long)C_out * lb * lb * es};
    const Range rw{dweight, (long long)C_out * C_in * 9 * es}, rb{dbias, dbias ? C_out * es : 0};
    const Range rws{workspace, (long long)need};
    if (any_overlap({rw, rb, rws}, {rhp, rlp, rho, rlo, Range{mask, g.B}}))
        return fail(SB_EINVAL, fn, "output buffers or the workspace overlap inputs or each other");
    return hip_status(fn, sb::launch_wgrad(dtype, layout, g, hp, lp, dho, dlo, mask, C_in, C_out, dweight, dbias,
                                           hi_cap, lo_cap, sb::Ws{workspace, ws_bytes}, stream));
}

int segblocks_policy_heuristic(const void* x, int dtype, int layout, int N, int C, int H, int W, int bs,
                               double tau_high, float* score, uint8_t* mask, hipStream_t stream) {
    const char* fn = "segblocks_policy_heuristic";
    static const uint8_t any = 0;
    sb::Geo g;
    int s;
    if ((s = check_geo(fn, dtype, layout, N, C, H, W, &any, bs, g))) return s;
    if (!x || !score || !mask) return fail(SB_EINVAL, fn, "x, score or mask is NULL");
    if (!(tau_high >= 0.0 && tau_high <= 1.0)) return fail(SB_EINVAL, fn, "tau_high must be in [0, 1]");
    const int per = g.GH * g.GW;
    if (per > sb::policy_max_blocks())
        return fail(SB_ESHAPE, fn, "at most %d blocks per image (got %d)", sb::policy_max_blocks(), per);
    const long long es = esize(dtype);
    const Range rx{x, (long long)N * C * H * W * es}, rs{score, g.B * 4}, rm{mask, g.B};
    if (any_overlap({rs, rm}, {rx})) return fail(SB_EINVAL, fn, "score or mask overlaps x, or each other");
    const int khigh = (int)floor(tau_high * per + 0.5);
    return hip_status(fn, sb::launch_policy(dtype, layout, x, N, C, H, W, bs, score, khigh, mask, stream));
}

int segblocks_conv2d(const void* x, int dtype, int layout, int N, int C_in, int H, int W, const void* weight,
                     const void* bias, int C_out, int ksize, int stride, int pad, int flags, void* y,
                     hipStream_t stream) {
    const char* fn = "segblocks_conv2d";
    if (layout != SB_NHWC || (dtype != SB_F16 && dtype != SB_BF16))
        return fail(SB_EINVAL, fn, "supported: channels-last fp16 / bf16");
    if (N <= 0 || C_in <= 0 || H <= 0 || W <= 0 || C_out <= 0)
        return fail(SB_EINVAL, fn, "N, C_in, H, W, C_out must be positive");
    if (ksize < 1 || stride < 1 || pad < 0 || pad >= ksize)
        return fail(SB_EINVAL, fn, "need ksize >= 1, stride >= 1, 0 <= pad < ksize (got %d, %d, %d)", ksize, stride, pad);
    if (!x || !weight || !y) return fail(SB_EINVAL, fn, "x, weight or y is NULL");
    if (flags & ~SB_FLAG_RELU) return fail(SB_EINVAL, fn, "unknown flags 0x%x", flags);
    if (H + 2 * pad < ksize || W + 2 * pad < ksize) return fail(SB_ESHAPE, fn, "kernel larger than the padded map");
    if (sb::conv2d_lds_bytes(dtype, C_in, ksize, stride) > 160 * 1024)
        return fail(SB_ESHAPE, fn, "ksize %d, stride %d, C_in %d need more than 160 KiB of LDS", ksize, stride, C_in);
    const long long Ho = (H + 2 * pad - ksize) / stride + 1, Wo = (W + 2 * pad - ksize) / stride + 1;
    const long long es = esize(dtype);
    if ((long long)N * H * W * C_in > (1LL << 40) || (long long)N * Ho * Wo * C_out > (1LL << 40))
        return fail(SB_ESHAPE, fn, "problem too large");
    const Range rx{x, (long long)N * C_in * H * W * es}, ry{y, (long long)N * C_out * Ho * Wo * es};
    const Range rw{weight, (long long)C_out * C_in * ksize * ksize * es}, rb{bias, bias ? C_out * es : 0};
    if (any_overlap({ry}, {rx, rw, rb})) return fail(SB_EINVAL, fn, "y overlaps an input");
    return hip_status(fn, sb::launch_conv2d(dtype, x, N, C_in, H, W, weight, bias, C_out, ksize, stride, pad, flags, y,
                                            stream));
}

int segblocks_maxpool(const void* x, int dtype, int layout, int N, int C, int H, int W, int ksize, int stride, int pad,
                      void* y, hipStream_t stream) {
    const char* fn = "segblocks_maxpool";
    if (dtype != SB_F32 && dtype != SB_F16 && dtype != SB_BF16) return fail(SB_EINVAL, fn, "bad dtype %d", dtype);
    if (layout != SB_NHWC) return fail(SB_EINVAL, fn, "supported: channels-last");
    if (N <= 0 || C <= 0 || H <= 0 || W <= 0) return fail(SB_EINVAL, fn, "N, C, H, W must be positive");
    if (ksize < 1 || stride < 1 || pad < 0 || pad >= ksize)
        return fail(SB_EINVAL, fn, "need ksize >= 1, stride >= 1, 0 <= pad < ksize (got %d, %d, %d)", ksize, stride, pad);
    if (!x || !y) return fail(SB_EINVAL, fn, "x or y is NULL");
    if (H + 2 * pad < ksize || W + 2 * pad < ksize) return fail(SB_ESHAPE, fn, "window larger than the padded map");
    const long long Ho = (H + 2 * pad - ksize) / stride + 1, Wo = (W + 2 * pad - ksize) / stride + 1;
    if ((long long)N * H * W * C > (1LL << 40)) return fail(SB_ESHAPE, fn, "problem too large");
    const long long es = esize(dtype);
    const Range rx{x, (long long)N * C * H * W * es}, ry{y, (long long)N * C * Ho * Wo * es};
    if (any_overlap({ry}, {rx})) return fail(SB_EINVAL, fn, "y overlaps x");
    return hip_status(fn, sb::launch_maxpool(dtype, x, N, C, H, W, ksize, stride, pad, y, stream));
}

}  // extern "C"
