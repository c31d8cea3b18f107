// Layers beyond 3x3 on padded block stacks, so that blocks can persist from
// the image to the last stage (the stem and its max-pool included): a K x K
// convolution (K odd) at stride 1 or 2 with dilation, and K x K max-pooling,
// on stacks padded by BlockPad with a halo of `halo` pixels (segblocks_pad
// with a wider halo).  Output pixel (i, j) of a block is the window centred
// on block pixel (stride * i, stride * j).
//
// Direct kernels: a thread computes four consecutive output channels of one
// output pixel (the convolution, fp32 sums in the order tap, input channel)
// or one channel vector (the max-pooling).  Only blocks inside the true class
// counts (from the mask) are read or written.
#include "sb_common.h"
#include "sb_kernels.h"

namespace sb {

namespace {

// Number of high blocks of the mask (every thread of the workgroup gets it).
__device__ __forceinline__ int hcount(const uint8_t* __restrict__ mask, int B, int* s_red) {
    int c = 0;
    for (int i = (int)threadIdx.x; i < B; i += WG) c += mask[i] != 0;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) c += __shfl_xor(c, o, 64);
    if ((threadIdx.x & 63) == 0) s_red[threadIdx.x >> 6] = c;
    __syncthreads();
    int t = 0;
#pragma unroll
    for (int w = 0; w < WG / 64; ++w) t += s_red[w];
    return t;
}

template <typename T, int L>
__device__ __forceinline__ size_t sidx(int s, int C, int ext, int y, int x, int c) {
    if constexpr (L == NHWC) return (((size_t)s * ext + y) * ext + x) * C + c;
    else                     return (((size_t)s * C + c) * ext + y) * ext + x;
}

// Items: [high: hi_cap * Eo_h^2 * COG][low: lo_cap * Eo_l^2 * COG], COG = groups of 4 output channels.
template <typename T, int L>
__global__ __launch_bounds__(WG) void k_conv_halo(const T* __restrict__ hp, const T* __restrict__ lp,
                                                  const uint8_t* __restrict__ mask, int B, int bs, int halo, int C_in,
                                                  int C_out, const T* __restrict__ w, const T* __restrict__ bias,
                                                  int K, int st, int dl, int flags, T* __restrict__ ho,
                                                  T* __restrict__ lo, int hi_cap, int lo_cap) {
    __shared__ int s_red[WG / 64];
    const int nh_all = hcount(mask, B, s_red);
    const int lb = bs >> 1, COG = (C_out + 3) / 4;
    const int eo_h = bs / st, eo_l = lb / st;
    const long long items_h = (long long)hi_cap * eo_h * eo_h * COG;
    const long long items_l = (long long)lo_cap * eo_l * eo_l * COG;
    const long long it = (long long)blockIdx.x * WG + threadIdx.x;
    if (it >= items_h + items_l) return;
    const bool high = it < items_h;
    const long long q = high ? it : it - items_h;
    const int eo = high ? eo_h : eo_l, e = high ? bs : lb, pe = e + 2 * halo;
    const int cg = (int)(q % COG);
    const long long pix = q / COG;
    const int j = (int)(pix % eo), i = (int)((pix / eo) % eo), s = (int)(pix / ((long long)eo * eo));
    if (s >= (high ? min(nh_all, hi_cap) : min(B - nh_all, lo_cap))) return;
    const T* P = high ? hp : lp;
    const int o = halo - dl * (K - 1) / 2;
    const int co0 = cg * 4;
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    for (int ky = 0; ky < K; ++ky) {
        const int y = st * i + dl * ky + o;
        for (int kx = 0; kx < K; ++kx) {
            const int x = st * j + dl * kx + o;
            for (int ci = 0; ci < C_in; ++ci) {
                const float pv = to_f32(P[sidx<T, L>(s, C_in, pe, y, x, ci)]);
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int co = co0 + r;
                    if (co < C_out) {
                        size_t wi;
                        if constexpr (L == NHWC) wi = (((size_t)co * K + ky) * K + kx) * C_in + ci;  // OHWI
                        else                     wi = (((size_t)co * C_in + ci) * K + ky) * K + kx;  // OIHW
                        acc[r] += pv * to_f32(w[wi]);
                    }
                }
            }
        }
    }
    T* out = high ? ho : lo;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int co = co0 + r;
        if (co >= C_out) break;
        float v = acc[r] + (bias ? to_f32(bias[co]) : 0.0f);
        if (flags & 1) v = fmaxf(v, 0.0f);
        out[sidx<T, L>(s, C_out, eo, i, j, co)] = from_f32<T>(v);
    }
}

template <typename T, int L>
__global__ __launch_bounds__(WG) void k_maxpool_halo(const T* __restrict__ hp, const T* __restrict__ lp,
                                                     const uint8_t* __restrict__ mask, int B, int bs, int halo, int C,
                                                     int K, int st, T* __restrict__ ho, T* __restrict__ lo, int hi_cap,
                                                     int lo_cap) {
    __shared__ int s_red[WG / 64];
    const int nh_all = hcount(mask, B, s_red);
    const int lb = bs >> 1;
    const int eo_h = bs / st, eo_l = lb / st;
    const long long items_h = (long long)hi_cap * eo_h * eo_h * C;
    const long long items_l = (long long)lo_cap * eo_l * eo_l * C;
    const long long it = (long long)blockIdx.x * WG + threadIdx.x;
    if (it >= items_h + items_l) return;
    const bool high = it < items_h;
    const long long q = high ? it : it - items_h;
    const int eo = high ? eo_h : eo_l, e = high ? bs : lb, pe = e + 2 * halo;
    int s, i, j, c;
    if constexpr (L == NHWC) {
        c = (int)(q % C);
        const long long pix = q / C;
        j = (int)(pix % eo);
        i = (int)((pix / eo) % eo);
        s = (int)(pix / ((long long)eo * eo));
    } else {
        j = (int)(q % eo);
        i = (int)((q / eo) % eo);
        c = (int)((q / ((long long)eo * eo)) % C);
        s = (int)(q / ((long long)eo * eo * C));
    }
    if (s >= (high ? min(nh_all, hi_cap) : min(B - nh_all, lo_cap))) return;
    const T* P = high ? hp : lp;
    const int o = halo - (K - 1) / 2;
    float m = -INFINITY;
    for (int ky = 0; ky < K; ++ky)
        for (int kx = 0; kx < K; ++kx) m = fmaxf(m, to_f32(P[sidx<T, L>(s, C, pe, st * i + ky + o, st * j + kx + o, c)]));
    (high ? ho : lo)[sidx<T, L>(s, C, eo, i, j, c)] = from_f32<T>(m);
}

template <typename T, int L>
hipError_t conv_halo_t(const Geo& g, const void* hp, const void* lp, const uint8_t* mask, int halo, const void* w,
                       const void* bias, int C_in, int C_out, int K, int st, int dl, int flags, void* ho, void* lo,
                       int hi_cap, int lo_cap, hipStream_t s) {
    const int lb = g.bs / 2, COG = (C_out + 3) / 4;
    const long long items = (long long)hi_cap * (g.bs / st) * (g.bs / st) * COG +
                            (long long)lo_cap * (lb / st) * (lb / st) * COG;
    if (items == 0) return hipSuccess;
    hipLaunchKernelGGL((k_conv_halo<T, L>), dim3((unsigned)((items + WG - 1) / WG)), dim3(WG), 0, s, (const T*)hp,
                       (const T*)lp, mask, (int)g.B, g.bs, halo, C_in, C_out, (const T*)w, (const T*)bias, K, st, dl,
                       flags, (T*)ho, (T*)lo, hi_cap, lo_cap);
    return hipGetLastError();
}

template <typename T, int L>
hipError_t maxpool_halo_t(const Geo& g, const void* hp, const void* lp, const uint8_t* mask, int halo, int K, int st,
                          void* ho, void* lo, int hi_cap, int lo_cap, hipStream_t s) {
    const int lb = g.bs / 2;
    const long long items = ((long long)hi_cap * (g.bs / st) * (g.bs / st) + (long long)lo_cap * (lb / st) * (lb / st)) *
                            g.C;
    if (items == 0) return hipSuccess;
    hipLaunchKernelGGL((k_maxpool_halo<T, L>), dim3((unsigned)((items + WG - 1) / WG)), dim3(WG), 0, s,
                       (const T*)hp, (const T*)lp, mask, (int)g.B, g.bs, halo, g.C, K, st, (T*)ho, (T*)lo, hi_cap,
                       lo_cap);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_conv_halo(int dtype, int layout, const Geo& g, const void* hp, const void* lp, const uint8_t* mask,
                            int halo, const void* w, const void* bias, int C_in, int C_out, int K, int st, int dl,
                            int flags, void* ho, void* lo, int hi_cap, int lo_cap, hipStream_t s) {
#define SB_CH(T, L) conv_halo_t<T, L>(g, hp, lp, mask, halo, w, bias, C_in, C_out, K, st, dl, flags, ho, lo, hi_cap, lo_cap, s)
    if (layout == NHWC) {
        switch (dtype) {
        case 0: return SB_CH(float, NHWC);
        case 1: return SB_CH(f16, NHWC);
        default: return SB_CH(bf16, NHWC);
        }
    }
    switch (dtype) {
    case 0: return SB_CH(float, NCHW);
    case 1: return SB_CH(f16, NCHW);
    default: return SB_CH(bf16, NCHW);
    }
#undef SB_CH
}

hipError_t launch_maxpool_halo(int dtype, int layout, const Geo& g, const void* hp, const void* lp,
                               const uint8_t* mask, int halo, int K, int st, void* ho, void* lo, int hi_cap,
                               int lo_cap, hipStream_t s) {
#define SB_MH(T, L) maxpool_halo_t<T, L>(g, hp, lp, mask, halo, K, st, ho, lo, hi_cap, lo_cap, s)
    if (layout == NHWC) {
        switch (dtype) {
        case 0: return SB_MH(float, NHWC);
        case 1: return SB_MH(f16, NHWC);
        default: return SB_MH(bf16, NHWC);
        }
    }
    switch (dtype) {
    case 0: return SB_MH(float, NCHW);
    case 1: return SB_MH(f16, NCHW);
    default: return SB_MH(bf16, NCHW);
    }
#undef SB_MH
}

}  // namespace sb
