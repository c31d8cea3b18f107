// The encoder's kernels around and between the block stages, channels-last
// fp16/bf16:
//
//   k_bconv   : K x K block convolution (K = 1 or 3) at stride 1 or 2 on the
//               packed stacks, BlockPad fused (a 3x3 stride-2 output reads
//               only the top and left halo), epilogue bias + residual + ReLU,
//               packed stacks of extent e / stride out.  MFMA
//               v_mfma_f32_16x16x32 with weights as A (16 output channels)
//               and 16 output pixels as B; both operands are read straight
//               from the L1/L2-resident inputs (the deep stages' blocks are
//               small, so an LDS tile would be mostly halo).
//   k_conv2d  : dense K x K convolution with zero padding at a stride (the
//               7x7/2 stem), bias, optional ReLU.  The input patch of a
//               4 x 64 output tile and the weights (K*K*C_in padded to a
//               multiple of 32) are staged in LDS; each lane gathers its 8
//               K values through a table of patch offsets.
//   k_stem    : the same for at most 4 input channels and K <= 8 (the stem):
//               K is ordered (ky, kx padded to 8, channel padded to 4), so the
//               8 K values of an MFMA operand lane are two adjacent input
//               pixels of the LDS tile (16 bytes) instead of a gather; the
//               weight rows are permuted so that a lane stores 8 consecutive
//               output channels (16 bytes) of a pixel.
//   k_maxpool : dense K x K max-pooling at a stride with padding that never
//               wins; k_maxpool_v does 16 bytes of channels per thread.
#include "sb_common.h"
#include "sb_kernels.h"
#include "sb_pixel.h"

namespace sb {

namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef _Float16 halfx8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

template <typename T> struct EMF;
template <> struct EMF<f16> {
    typedef halfx8 frag;
    static __device__ __forceinline__ floatx4 mma(frag a, frag b, floatx4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
    }
};
template <> struct EMF<bf16> {
    typedef bf16x8 frag;
    static __device__ __forceinline__ floatx4 mma(frag a, frag b, floatx4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
    }
};

template <typename T>
__device__ __forceinline__ typename EMF<T>::frag as_frag(uint4 v) {
    return __builtin_bit_cast(typename EMF<T>::frag, v);
}

template <typename T>
__device__ __forceinline__ uint4 avg_raw16(uint4 a, uint4 b, uint4 c, uint4 d) {
    Vec<T, 8> va, vb, vc, vd;
    va.raw = a;
    vb.raw = b;
    vc.raw = c;
    vd.raw = d;
    return vavg4<T, 8>(va, vb, vc, vd).raw;
}

// Epilogue of one lane: 4 consecutive output channels co..co+3 of one pixel
// at element offset `off` of the output (and of the residual).
template <typename T>
__device__ __forceinline__ void store4(T* out, const T* res, const T* bias, size_t off, int co, int C_out,
                                       floatx4 acc, bool relu) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        if (co + r >= C_out) break;
        float f = acc[r] + (bias ? to_f32(bias[co + r]) : 0.0f);
        if (res) f += to_f32(res[off + co + r]);
        out[off + co + r] = from_f32<T>(relu ? fmaxf(f, 0.0f) : f);
    }
}

// ---------------------------------------------------------------------------
// block convolution at a stride
// ---------------------------------------------------------------------------
constexpr int BC_PX = 32;  // output pixels per wave (two 16-pixel sub-tiles)

template <typename T, int KS, int ST, bool ONE>
__global__ __launch_bounds__(WG) void k_bconv(Geo g, const uint8_t* __restrict__ mask, ConvArgs a, int G) {
    typedef EMF<T> mf;
    typedef typename mf::frag frag;
    __shared__ __align__(16) uint8_t s_mask[1024];
    __shared__ __align__(16) PlanTable s_pt;
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    if (wave == 0) {
        stage_mask(mask, (int)g.B, s_mask);
        if (ONE) build_plan_table(s_mask, &s_pt);
    }
    __syncthreads();

    const int k = (int)blockIdx.x / G, grp = (int)blockIdx.x - k * G;
    const int per = g.GH * g.GW;
    const int n = k / per, rem = k - n * per, gy = rem / g.GW, gx = rem - gy * g.GW;
    Neigh nb;
    if constexpr (ONE) {
        nb = table_neighbourhood(&s_pt, g.GH, g.GW, n, gy, gx);
    } else {
        WaveMaskT<ONE> wm;
        wm.init_staged(mask, (int)g.B, s_mask);
        nb = wave_neighbourhood<true>(wm, g.GH, g.GW, n, gy, gx);
    }
    const int high = (nb.high >> 4) & 1, slot = nb.slot[4];
    if (slot >= (high ? a.hi_cap : a.lo_cap)) return;
    const int e = high ? g.bs : (g.bs >> 1), Eo = e / ST, npx = Eo * Eo;
    const int p0 = grp * (BC_PX * (WG / 64)) + wave * BC_PX;
    if (p0 >= npx) return;

    const int lane = lane_id(), l16 = lane & 15, kg = lane >> 4;
    const int co0 = blockIdx.y * 64;
    const int C = a.C_in, Co = a.C_out;
    const T* __restrict__ hi = (const T*)a.in_hi;
    const T* __restrict__ lo = (const T*)a.in_lo;
    const T* __restrict__ wgt = (const T*)a.weight;

    int oy[2], ox[2];
    bool pv[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
        const int p = p0 + t * 16 + l16;
        pv[t] = p < npx;
        oy[t] = pv[t] ? p / Eo : 0;
        ox[t] = pv[t] ? p - oy[t] * Eo : 0;
    }
    floatx4 acc[2][4];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int ns = 0; ns < 4; ++ns) acc[t][ns] = floatx4{0.f, 0.f, 0.f, 0.f};

    const int nks = (C + 31) / 32;
    for (int tap = 0; tap < KS * KS; ++tap) {
        const int ky = tap / KS, kx = tap - ky * KS;
        Src<T> src[2];
#pragma unroll
        for (int t = 0; t < 2; ++t)
            src[t] = pv[t] ? packed_src<T, NHWC>(hi, lo, C, g.bs, nb, a.hi_cap, a.lo_cap, ST * oy[t] + ky - KS / 2,
                                                 ST * ox[t] + kx - KS / 2, 0, pad_mode(a.flags))
                           : src_zero<T>();
        for (int ks = 0; ks < nks; ++ks) {
            const int c = ks * 32 + kg * 8;
            const bool cin = c < C;
            frag wf[4], bf[2];
#pragma unroll
            for (int ns = 0; ns < 4; ++ns) {
                const int co = co0 + ns * 16 + l16;
                uint4 v = uint4{0u, 0u, 0u, 0u};
                if (cin && co < Co) v = *reinterpret_cast<const uint4*>(wgt + ((size_t)co * KS * KS + tap) * C + c);
                wf[ns] = as_frag<T>(v);
            }
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                uint4 v = uint4{0u, 0u, 0u, 0u};
                if (cin && src[t].p) {
                    const T* q = src[t].p + c;
                    v = *reinterpret_cast<const uint4*>(q);
                    if (src[t].avg)
                        v = avg_raw16<T>(v, *reinterpret_cast<const uint4*>(q + src[t].d1),
                                         *reinterpret_cast<const uint4*>(q + src[t].d2),
                                         *reinterpret_cast<const uint4*>(q + src[t].d2 + src[t].d1));
                }
                bf[t] = as_frag<T>(v);
            }
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
                for (int ns = 0; ns < 4; ++ns) acc[t][ns] = mf::mma(wf[ns], bf[t], acc[t][ns]);
        }
    }

    // epilogue: lane holds channels co0 + ns*16 + kg*4 + {0..3} of pixel l16 of sub-tile t
    const size_t blk = (size_t)slot * Eo * Eo * Co;
    T* out = (T*)(high ? a.out_hi : a.out_lo) + blk;
    const T* rb = (const T*)(high ? a.res_hi : a.res_lo);
    const T* res = rb ? rb + blk : nullptr;
    const bool relu = (a.flags & 1) != 0;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
        if (!pv[t]) continue;
        const size_t off = ((size_t)oy[t] * Eo + ox[t]) * Co;
#pragma unroll
        for (int ns = 0; ns < 4; ++ns) {
            const int co = co0 + ns * 16 + kg * 4;
            if (co < Co) store4<T>(out, res, (const T*)a.bias, off, co, Co, acc[t][ns], relu);
        }
    }
}

// ---------------------------------------------------------------------------
// dense convolution (the stem)
// ---------------------------------------------------------------------------
constexpr int DC_TH = 4, DC_TW = 64;  // output tile rows x columns (one row per wave)

template <typename T>
__global__ __launch_bounds__(WG) void k_conv2d(const T* __restrict__ x, int C_in, int H, int W,
                                               const T* __restrict__ w, const T* __restrict__ bias, int C_out, int K,
                                               int S, int P, int flags, T* __restrict__ y, int Ho, int Wo, int TY,
                                               int TX, int KP) {
    typedef EMF<T> mf;
    typedef typename mf::frag frag;
    extern __shared__ __align__(16) unsigned char smem[];
    const int KKC = K * K * C_in;
    const int PH = S * (DC_TH - 1) + K, PW = S * (DC_TW - 1) + K;
    T* s_w = reinterpret_cast<T*>(smem);                       // [64][KP]
    int* s_koff = reinterpret_cast<int*>(smem + 64 * KP * (int)sizeof(T));  // [KP]
    T* s_in = reinterpret_cast<T*>(s_koff + KP);               // [PH][PW][C_in]

    const int tile = (int)blockIdx.x;
    const int n = tile / (TY * TX), tr = tile - n * TY * TX, ty = tr / TX, tx = tr - ty * TX;
    const int oy0 = ty * DC_TH, ox0 = tx * DC_TW, co0 = blockIdx.y * 64;
    const int Y0 = oy0 * S - P, X0 = ox0 * S - P;
    const int tid = threadIdx.x;

    for (int i = tid; i < 64 * KP; i += WG) {
        const int co = i / KP, kk = i - co * KP;
        s_w[i] = (co0 + co < C_out && kk < KKC) ? w[(size_t)(co0 + co) * KKC + kk] : from_f32<T>(0.0f);
    }
    for (int kk = tid; kk < KP; kk += WG) {
        int off = -1;
        if (kk < KKC) {
            const int tap = kk / C_in, ci = kk - tap * C_in, ky = tap / K, kx = tap - ky * K;
            off = (ky * PW + kx) * C_in + ci;
        }
        s_koff[kk] = off;
    }
    const T* __restrict__ img = x + (size_t)n * H * W * C_in;
    for (int i = tid; i < PH * PW * C_in; i += WG) {
        const int pix = i / C_in, ci = i - pix * C_in, r = pix / PW, c = pix - r * PW;
        const int yy = Y0 + r, xx = X0 + c;
        s_in[i] = (yy >= 0 && yy < H && xx >= 0 && xx < W) ? img[((size_t)yy * W + xx) * C_in + ci] : from_f32<T>(0.0f);
    }
    __syncthreads();

    const int wave = tid >> 6, lane = tid & 63, l16 = lane & 15, kg = lane >> 4;
    floatx4 acc[4][4];
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int ns = 0; ns < 4; ++ns) acc[t][ns] = floatx4{0.f, 0.f, 0.f, 0.f};
    int base[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) base[t] = ((wave * S) * PW + (t * 16 + l16) * S) * C_in;

    for (int kc = 0; kc < KP; kc += 32) {
        const int k0 = kc + kg * 8;
        frag wf[4], bf[4];
#pragma unroll
        for (int ns = 0; ns < 4; ++ns) wf[ns] = *reinterpret_cast<const frag*>(s_w + (ns * 16 + l16) * KP + k0);
        int off[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) off[e] = s_koff[k0 + e];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            Vec<T, 8> v;
#pragma unroll
            for (int e = 0; e < 8; ++e) v.e[e] = off[e] >= 0 ? s_in[base[t] + off[e]] : from_f32<T>(0.0f);
            bf[t] = as_frag<T>(v.raw);
        }
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
            for (int ns = 0; ns < 4; ++ns) acc[t][ns] = mf::mma(wf[ns], bf[t], acc[t][ns]);
    }

    const int oy = oy0 + wave;
    if (oy >= Ho) return;
    const bool relu = (flags & 1) != 0;
    T* yrow = y + ((size_t)n * Ho + oy) * Wo * C_out;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        const int ox = ox0 + t * 16 + l16;
        if (ox >= Wo) continue;
#pragma unroll
        for (int ns = 0; ns < 4; ++ns) {
            const int co = co0 + ns * 16 + kg * 4;
            if (co < C_out) store4<T>(yrow, nullptr, bias, (size_t)ox * C_out, co, C_out, acc[t][ns], relu);
        }
    }
}

// ---------------------------------------------------------------------------
// max-pooling
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(WG) void k_maxpool(const T* __restrict__ x, int N, int C, int H, int W, int K, int S,
                                                int P, T* __restrict__ y, int Ho, int Wo) {
    const long long total = (long long)N * Ho * Wo * C;
    const long long i = (long long)blockIdx.x * WG + threadIdx.x;
    if (i >= total) return;
    const int c = (int)(i % C);
    const long long pix = i / C;
    const int ox = (int)(pix % Wo), oy = (int)((pix / Wo) % Ho), n = (int)(pix / ((long long)Wo * Ho));
    float m = -INFINITY;
    T best = from_f32<T>(0.0f);
    for (int ky = 0; ky < K; ++ky) {
        const int yy = oy * S + ky - P;
        if (yy < 0 || yy >= H) continue;
        for (int kx = 0; kx < K; ++kx) {
            const int xx = ox * S + kx - P;
            if (xx < 0 || xx >= W) continue;
            const T v = x[(((size_t)n * H + yy) * W + xx) * C + c];
            if (to_f32(v) > m) {
                m = to_f32(v);
                best = v;
            }
        }
    }
    y[i] = best;
}

template <typename T, int KS, int ST>
hipError_t run_bconv(const Geo& g, const uint8_t* mask, const ConvArgs& a, hipStream_t st) {
    const int Eo = g.bs / ST;
    const int G = (Eo * Eo + BC_PX * (WG / 64) - 1) / (BC_PX * (WG / 64));
    const dim3 grid((unsigned)(g.B * G), (unsigned)((a.C_out + 63) / 64));
    if (g.B <= 1024) hipLaunchKernelGGL((k_bconv<T, KS, ST, true>), grid, dim3(WG), 0, st, g, mask, a, G);
    else hipLaunchKernelGGL((k_bconv<T, KS, ST, false>), grid, dim3(WG), 0, st, g, mask, a, G);
    return hipGetLastError();
}

template <typename T>
hipError_t bconv_t(const Geo& g, const uint8_t* mask, const ConvArgs& a, int ksize, int stride, hipStream_t st) {
    if (ksize == 3) return stride == 1 ? run_bconv<T, 3, 1>(g, mask, a, st) : run_bconv<T, 3, 2>(g, mask, a, st);
    return stride == 1 ? run_bconv<T, 1, 1>(g, mask, a, st) : run_bconv<T, 1, 2>(g, mask, a, st);
}

// ---------------------------------------------------------------------------
// stem: dense convolution of a map with at most 4 channels
// ---------------------------------------------------------------------------
constexpr int ST_WG = 1024, ST_WAVES = ST_WG / 64;  // sixteen waves, one workgroup per CU
constexpr int ST_TH = 32, ST_TW = 64;  // output tile: 32 rows (two per wave) x 64 columns x 64 channels

// output channel of LDS weight row r (within a 32-row group, row 16h + 4kg + i
// holds channel 8kg + 4h + i), so that a lane's two fragments of a group
// hold 8 consecutive channels
__device__ __forceinline__ int stem_perm(int r) {
    const int l = r & 15;
    return (r & ~31) + (l >> 2) * 8 + ((r >> 4) & 1) * 4 + (l & 3);
}

template <typename T>
__global__ __launch_bounds__(ST_WG) void k_stem(const T* __restrict__ x, int C_in, int H, int W,
                                             const T* __restrict__ w, const T* __restrict__ bias, int C_out, int K,
                                             int S, int P, int flags, T* __restrict__ y, int Ho, int Wo, int TY,
                                             int TX) {
    typedef EMF<T> mf;
    typedef typename mf::frag frag;
    extern __shared__ __align__(16) unsigned char smem[];
    const int WROW = K * 32 + 8;                          // elements per LDS weight row (padded: no bank conflicts)
    const int IH = S * (ST_TH - 1) + K, IW = S * (ST_TW - 1) + 8;
    T* s_w = reinterpret_cast<T*>(smem);                  // [64][WROW]: (ky, kx8, ci4)
    T* s_in = s_w + 64 * WROW;                            // [IH][IW][4]

    const int tile = (int)blockIdx.x;
    const int n = tile / (TY * TX), tr = tile - n * TY * TX, ty = tr / TX, tx = tr - ty * TX;
    const int oy0 = ty * ST_TH, ox0 = tx * ST_TW, co0 = blockIdx.y * 64;
    const int Y0 = oy0 * S - P, X0 = ox0 * S - P;
    const int tid = threadIdx.x;

    // Staging in batches: every thread issues a batch of loads before it
    // writes any of them to LDS, so the loads of a batch are in flight
    // together.  The batches cover the whole weight slice (7 x 7 taps: one
    // batch) and the whole input tile (one batch): each further batch is one
    // more memory round trip at kernel start, about 3 us each.
    // Element i of a staged array is (row, column) = (i / width, i % width);
    // a thread's elements are ST_WG apart, so both advance by constants (no
    // division per element).
    constexpr int SBW = 14, SBI = 10;
    const int KW = K * 32, nw = 64 * KW;
    const int dwq = ST_WG / KW, dwr = ST_WG - dwq * KW;
    for (int base = tid; base < nw; base += ST_WG * SBW) {
        T v[SBW];
        int r = base / KW, rem = base - r * KW;
#pragma unroll
        for (int u = 0; u < SBW; ++u) {
            const int i = base + u * ST_WG;
            v[u] = from_f32<T>(0.0f);
            if (i < nw) {
                const int ky = rem >> 5, kx = (rem & 31) >> 2, ci = rem & 3;
                const int co = co0 + stem_perm(r);
                if (co < C_out && kx < K && ci < C_in) v[u] = w[(((size_t)co * K + ky) * K + kx) * C_in + ci];
            }
            r += dwq;
            rem += dwr;
            if (rem >= KW) { rem -= KW; ++r; }
        }
        r = base / KW;
        rem = base - r * KW;
#pragma unroll
        for (int u = 0; u < SBW; ++u) {
            const int i = base + u * ST_WG;
            if (i < nw) s_w[r * WROW + rem] = v[u];
            r += dwq;
            rem += dwr;
            if (rem >= KW) { rem -= KW; ++r; }
        }
    }
    const T* __restrict__ img = x + (size_t)n * H * W * C_in;
    const int np = IH * IW;
    const int diq = ST_WG / IW, dir = ST_WG - diq * IW;
    for (int base = tid; base < np; base += ST_WG * SBI) {
        Vec<T, 4> v[SBI];
        int r = base / IW, c = base - r * IW;
#pragma unroll
        for (int u = 0; u < SBI; ++u) {
            const int i = base + u * ST_WG;
            v[u] = vzero<T, 4>();
            const int yy = Y0 + r, xx = X0 + c;
            r += diq;
            c += dir;
            if (c >= IW) { c -= IW; ++r; }
            if (i < np) {
                if (yy >= 0 && yy < H && xx >= 0 && xx < W) {
                    const T* p = img + ((size_t)yy * W + xx) * C_in;
#pragma unroll
                    for (int ci = 0; ci < 4; ++ci)
                        if (ci < C_in) v[u].e[ci] = p[ci];
                }
            }
        }
#pragma unroll
        for (int u = 0; u < SBI; ++u) {
            const int i = base + u * ST_WG;
            if (i < np) *reinterpret_cast<uint2*>(s_in + (size_t)i * 4) = v[u].raw;
        }
    }
    __syncthreads();

    const int wave = tid >> 6, lane = tid & 63, l16 = lane & 15, kg = lane >> 4;
    const bool relu = (flags & 1) != 0;
    float bv[2][8];
#pragma unroll
    for (int jj = 0; jj < 2; ++jj)
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int co = co0 + jj * 32 + kg * 8 + i;
            bv[jj][i] = (bias && co < C_out) ? to_f32(bias[co]) : 0.0f;
        }
    for (int rr = 0; rr < ST_TH / ST_WAVES; ++rr) {
        const int ol = wave * (ST_TH / ST_WAVES) + rr;  // output row within the tile
        floatx4 acc[4][4];
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
            for (int ns = 0; ns < 4; ++ns) acc[t][ns] = floatx4{0.f, 0.f, 0.f, 0.f};
        for (int ky = 0; ky < K; ++ky) {
            frag wf[4], bf[4];
#pragma unroll
            for (int ns = 0; ns < 4; ++ns)
                wf[ns] = *reinterpret_cast<const frag*>(s_w + (ns * 16 + l16) * WROW + ky * 32 + kg * 8);
            const T* row = s_in + (size_t)((S * ol + ky) * IW) * 4;
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const T* p = row + (size_t)(S * (t * 16 + l16) + 2 * kg) * 4;
                const uint2 lo = *reinterpret_cast<const uint2*>(p), hi = *reinterpret_cast<const uint2*>(p + 4);
                bf[t] = as_frag<T>(uint4{lo.x, lo.y, hi.x, hi.y});
            }
#pragma unroll
            for (int t = 0; t < 4; ++t)
#pragma unroll
                for (int ns = 0; ns < 4; ++ns) acc[t][ns] = mf::mma(wf[ns], bf[t], acc[t][ns]);
        }
        const int oy = oy0 + ol;
        if (oy >= Ho) continue;
        T* yrow = y + ((size_t)n * Ho + oy) * Wo * C_out;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const int ox = ox0 + t * 16 + l16;
            if (ox >= Wo) continue;
#pragma unroll
            for (int jj = 0; jj < 2; ++jj) {
                const int co = co0 + jj * 32 + kg * 8;
                if (co >= C_out) continue;
                Vec<T, 8> o;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float f0 = acc[t][2 * jj][i] + bv[jj][i], f1 = acc[t][2 * jj + 1][i] + bv[jj][4 + i];
                    o.e[i] = from_f32<T>(relu ? fmaxf(f0, 0.0f) : f0);
                    o.e[4 + i] = from_f32<T>(relu ? fmaxf(f1, 0.0f) : f1);
                }
                *reinterpret_cast<uint4*>(yrow + (size_t)ox * C_out + co) = o.raw;
            }
        }
    }
}

// Max-pooling, 16 bytes of channels per thread (C a multiple of 16 / sizeof(T)).
template <typename T>
__global__ __launch_bounds__(WG) void k_maxpool_v(const T* __restrict__ x, int N, int C, int H, int W, int K, int S,
                                                  int P, T* __restrict__ y, int Ho, int Wo) {
    constexpr int V = 16 / (int)sizeof(T);
    const int CV = C / V;
    const long long total = (long long)N * Ho * Wo * CV;
    const long long i = (long long)blockIdx.x * WG + threadIdx.x;
    if (i >= total) return;
    const int cv = (int)(i % CV);
    const long long pix = i / CV;
    const int ox = (int)(pix % Wo), oy = (int)((pix / Wo) % Ho), n = (int)(pix / ((long long)Wo * Ho));
    float m[V];
    Vec<T, V> best = vzero<T, V>();
#pragma unroll
    for (int e = 0; e < V; ++e) m[e] = -INFINITY;
    for (int ky = 0; ky < K; ++ky) {
        const int yy = oy * S + ky - P;
        if (yy < 0 || yy >= H) continue;
        for (int kx = 0; kx < K; ++kx) {
            const int xx = ox * S + kx - P;
            if (xx < 0 || xx >= W) continue;
            Vec<T, V> v;
            v.raw = *reinterpret_cast<const uint4*>(x + (((size_t)n * H + yy) * W + xx) * C + cv * V);
#pragma unroll
            for (int e = 0; e < V; ++e)
                if (to_f32(v.e[e]) > m[e]) {
                    m[e] = to_f32(v.e[e]);
                    best.e[e] = v.e[e];
                }
        }
    }
    *reinterpret_cast<uint4*>(y + pix * C + cv * V) = best.raw;
}

}  // namespace

int conv2d_lds_bytes(int dtype, int C_in, int K, int S) {
    const int es = dtype == 0 ? 4 : 2;
    const int KP = (K * K * C_in + 31) / 32 * 32;
    const int PH = S * (DC_TH - 1) + K, PW = S * (DC_TW - 1) + K;
    return 64 * KP * es + KP * 4 + PH * PW * C_in * es;
}

hipError_t launch_bconv(int dtype, const Geo& g, const uint8_t* mask, const ConvArgs& a, int ksize, int stride,
                        hipStream_t st) {
    if (dtype == 1) return bconv_t<f16>(g, mask, a, ksize, stride, st);
    return bconv_t<bf16>(g, mask, a, ksize, stride, st);
}

namespace {
template <typename T>
hipError_t stem_t(const void* x, int N, int C_in, int H, int W, const void* w, const void* bias, int C_out, int K,
                  int S, int P, int flags, void* y, int Ho, int Wo, hipStream_t st) {
    const int TY = (Ho + ST_TH - 1) / ST_TH, TX = (Wo + ST_TW - 1) / ST_TW;
    const int smem = stem_lds_bytes(K, S);
    hipError_t e = ensure_dyn_lds((const void*)k_stem<T>, smem);
    if (e != hipSuccess) return e;
    const dim3 grid((unsigned)(N * TY * TX), (unsigned)((C_out + 63) / 64));
    hipLaunchKernelGGL(k_stem<T>, grid, dim3(ST_WG), smem, st, (const T*)x, C_in, H, W, (const T*)w, (const T*)bias,
                       C_out, K, S, P, flags, (T*)y, Ho, Wo, TY, TX);
    return hipGetLastError();
}
}  // namespace

int stem_lds_bytes(int K, int S) {
    const int IH = S * (ST_TH - 1) + K, IW = S * (ST_TW - 1) + 8;
    return (64 * (K * 32 + 8) + IH * IW * 4) * 2;
}

hipError_t launch_conv2d(int dtype, const void* x, int N, int C_in, int H, int W, const void* w, const void* bias,
                         int C_out, int K, int S, int P, int flags, void* y, hipStream_t st) {
    const int Ho = (H + 2 * P - K) / S + 1, Wo = (W + 2 * P - K) / S + 1;
    // the stem path: few input channels, 16-byte channel groups of the output
    if (C_in <= 4 && K <= 8 && C_out % 8 == 0 && (reinterpret_cast<uintptr_t>(y) & 15) == 0 &&
        stem_lds_bytes(K, S) <= 160 * 1024) {
        if (dtype == 1) return stem_t<f16>(x, N, C_in, H, W, w, bias, C_out, K, S, P, flags, y, Ho, Wo, st);
        return stem_t<bf16>(x, N, C_in, H, W, w, bias, C_out, K, S, P, flags, y, Ho, Wo, st);
    }
    const int TY = (Ho + DC_TH - 1) / DC_TH, TX = (Wo + DC_TW - 1) / DC_TW;
    const int KP = (K * K * C_in + 31) / 32 * 32;
    const int smem = conv2d_lds_bytes(dtype, C_in, K, S);
    const dim3 grid((unsigned)(N * TY * TX), (unsigned)((C_out + 63) / 64));
    if (dtype == 1) {
        hipError_t e = ensure_dyn_lds((const void*)k_conv2d<f16>, smem);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(k_conv2d<f16>, grid, dim3(WG), smem, st, (const f16*)x, C_in, H, W, (const f16*)w,
                           (const f16*)bias, C_out, K, S, P, flags, (f16*)y, Ho, Wo, TY, TX, KP);
    } else {
        hipError_t e = ensure_dyn_lds((const void*)k_conv2d<bf16>, smem);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(k_conv2d<bf16>, grid, dim3(WG), smem, st, (const bf16*)x, C_in, H, W, (const bf16*)w,
                           (const bf16*)bias, C_out, K, S, P, flags, (bf16*)y, Ho, Wo, TY, TX, KP);
    }
    return hipGetLastError();
}

hipError_t launch_maxpool(int dtype, const void* x, int N, int C, int H, int W, int K, int S, int P, void* y,
                          hipStream_t st) {
    const int Ho = (H + 2 * P - K) / S + 1, Wo = (W + 2 * P - K) / S + 1;
    const long long total = (long long)N * Ho * Wo * C;
    const unsigned grid = (unsigned)((total + WG - 1) / WG);
    if (total == 0) return hipSuccess;
    const int es = dtype == 0 ? 4 : 2;
    if ((C * es) % 16 == 0 && (reinterpret_cast<uintptr_t>(x) & 15) == 0 && (reinterpret_cast<uintptr_t>(y) & 15) == 0) {
        const long long tv = total * es / 16;
        const unsigned gv = (unsigned)((tv + WG - 1) / WG);
        if (dtype == 0) hipLaunchKernelGGL(k_maxpool_v<float>, dim3(gv), dim3(WG), 0, st, (const float*)x, N, C, H, W, K, S, P, (float*)y, Ho, Wo);
        else if (dtype == 1) hipLaunchKernelGGL(k_maxpool_v<f16>, dim3(gv), dim3(WG), 0, st, (const f16*)x, N, C, H, W, K, S, P, (f16*)y, Ho, Wo);
        else hipLaunchKernelGGL(k_maxpool_v<bf16>, dim3(gv), dim3(WG), 0, st, (const bf16*)x, N, C, H, W, K, S, P, (bf16*)y, Ho, Wo);
        return hipGetLastError();
    }
    if (dtype == 0) hipLaunchKernelGGL(k_maxpool<float>, dim3(grid), dim3(WG), 0, st, (const float*)x, N, C, H, W, K, S, P, (float*)y, Ho, Wo);
    else if (dtype == 1) hipLaunchKernelGGL(k_maxpool<f16>, dim3(grid), dim3(WG), 0, st, (const f16*)x, N, C, H, W, K, S, P, (f16*)y, Ho, Wo);
    else hipLaunchKernelGGL(k_maxpool<bf16>, dim3(grid), dim3(WG), 0, st, (const bf16*)x, N, C, H, W, K, S, P, (bf16*)y, Ho, Wo);
    return hipGetLastError();
}

}  // namespace sb
