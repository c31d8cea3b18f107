// 3x3 block convolution as an MFMA implicit GEMM for gfx950.
//
// GEMM view per block: M = output pixels of the block (e x e), N = output
// channels, K = 9 taps x C_in.  One workgroup (4 waves) computes a tile of
// up to 256 output pixels (whole rows of one block) x 64 output channels.
// K is walked in chunks of 64 bytes of channels (32 fp16/bf16 or 16 fp32):
// the padded input rows of the tile and the chunk's weights are staged in
// LDS with an XOR swizzle of the 16-byte sub-chunks, then every tap reads
// its A fragments at a constant pixel offset from the same LDS tile.
// MFMA: v_mfma_f32_16x16x32_{f16,bf16} (8 K-values per lane) or
// v_mfma_f32_16x16x4_f32.  Each wave owns up to four 16-row M sub-tiles and
// all four 16-column N sub-tiles (64 fp32 accumulators per lane).
//
// The tile loader is where the block modules live:
//   SRC_PADDED : reads padded stacks (plain conv of segblocks_conv3x3)
//   SRC_PACKED : BlockPad fused (neighbour lookup into the packed stacks)
//   SRC_DENSE  : BlockSample + BlockPad fused (reads the dense input map)
// and the store is either a packed stack or BlockCombine into a dense map.
#include "sb_common.h"
#include "sb_kernels.h"
#include "sb_pixel.h"

namespace sb {

namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef _Float16 halfx8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

template <typename T> struct MF;
template <> struct MF<f16> {
    static constexpr int KS = 32, EL = 8;  // K per instruction, K values per lane
    typedef halfx8 frag;
    static __device__ __forceinline__ floatx4 mma(frag a, frag b, floatx4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
    }
};
template <> struct MF<bf16> {
    static constexpr int KS = 32, EL = 8;
    typedef bf16x8 frag;
    static __device__ __forceinline__ floatx4 mma(frag a, frag b, floatx4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
    }
};
template <> struct MF<float> {
    static constexpr int KS = 4, EL = 1;
    typedef float frag;
    static __device__ __forceinline__ floatx4 mma(frag a, frag b, floatx4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
    }
};

constexpr int NT = 64;     // output channels per workgroup
constexpr int ROWB = 64;   // LDS bytes per tile pixel / weight row (one K chunk)
constexpr int MT = 256;    // target output pixels per workgroup
constexpr int SROW = NT + 4;  // fp32 staging row (padded against bank conflicts)
constexpr int W_BYTES = 9 * NT * ROWB;

// byte offset of 16-byte sub-chunk q of LDS row `row`: sub-chunks are XOR-
// swizzled with bits 1..2 of the row so that 8 consecutive rows read at the
// same sub-chunk hit 8 distinct 16-byte bank groups.
__device__ __forceinline__ int swz(int row, int q) { return row * ROWB + ((q ^ ((row >> 1) & 3)) << 4); }

template <typename T, int L, int SRC, int V>
__device__ __forceinline__ Vec<T, V> tile_pixel(const Geo& g, const ConvArgs& a, const Neigh& nb, int n, int gy,
                                                int gx, int slot, bool high, int pe, int u, int v, int c) {
    if constexpr (SRC == SRC_PADDED) {
        const T* base = (const T*)(high ? a.in_hi : a.in_lo);
        return vload<T, V>(stack_at<T, L>(base, slot, a.C_in, pe, u, v, c));
    } else if constexpr (SRC == SRC_PACKED) {
        return packed_pixel<T, L, V>((const T*)a.in_hi, (const T*)a.in_lo, a.C_in, g.bs, nb, a.hi_cap, a.lo_cap,
                                     u - 1, v - 1, c);
    } else {
        return dense_pixel<T, L, V>((const T*)a.in_hi, n, a.C_in, g.H, g.W, g.bs, gy, gx, nb, u - 1, v - 1, c);
    }
}

template <typename T, int L, int SRC, int DST>
__global__ __launch_bounds__(WG) void k_conv(Geo g, const uint8_t* __restrict__ mask, ConvArgs a, int Rh, int Rl,
                                             int G, int w_off, int vec_in, int vec_out) {
    extern __shared__ __align__(16) unsigned char smem[];
    __shared__ Neigh s_nb;
    typedef MF<T> mf;
    constexpr int KC = ROWB / (int)sizeof(T);  // channels per K chunk
    constexpr int VQ = 16 / (int)sizeof(T);    // channels per 16-byte sub-chunk
    constexpr bool NEED_SLOTS = !(SRC == SRC_DENSE && DST == DST_DENSE);

    const long long k = blockIdx.x / G;
    const int grp = (int)(blockIdx.x - k * G);
    const int co0 = blockIdx.y * NT;
    const long long per = (long long)g.GH * g.GW;
    const int n = (int)(k / per);
    const int rem = (int)(k - (long long)n * per);
    const int gy = rem / g.GW, gx = rem - gy * g.GW;

    if (threadIdx.x < 64) block_neighbourhood<NEED_SLOTS>(mask, g.GH, g.GW, n, gy, gx, &s_nb);
    __syncthreads();
    const bool high = (s_nb.high >> 4) & 1;
    const int slot = s_nb.slot[4];
    if (NEED_SLOTS && slot >= (high ? a.hi_cap : a.lo_cap)) return;
    const int e = high ? g.bs : (g.bs >> 1);
    const int R = high ? Rh : Rl;
    const int r0 = grp * R;
    if (r0 >= e) return;
    const int rows = min(R, e - r0);
    const int M = rows * e;
    const int pe = e + 2;
    const int in_px = (rows + 2) * pe;

    unsigned char* s_in = smem;
    unsigned char* s_w = smem + w_off;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int l16 = lane & 15, kg = lane >> 4;

    const int nst = (M + 15) >> 4;  // 16-row M sub-tiles
    int pbase[4];
#pragma unroll
    for (int ms = 0; ms < 4; ++ms) {
        const int m = min((wave + 4 * ms) * 16 + l16, M - 1);
        const int i = m / e, j = m - i * e;
        pbase[ms] = i * pe + j;
    }
    floatx4 acc[4][4];
#pragma unroll
    for (int ms = 0; ms < 4; ++ms)
#pragma unroll
        for (int ns = 0; ns < 4; ++ns) acc[ms][ns] = floatx4{0.f, 0.f, 0.f, 0.f};

    const T* __restrict__ wgt = (const T*)a.weight;
    const int nchunks = (a.C_in + KC - 1) / KC;
    for (int kc = 0; kc < nchunks; ++kc) {
        // -- stage the padded input rows of the tile for channels [kc*KC, kc*KC + KC)
        for (int it = tid; it < in_px * 4; it += WG) {
            const int p = it >> 2, q = it & 3;
            const int pu = p / pe, pv = p - pu * pe;
            const int c0 = kc * KC + q * VQ;
            Vec<T, VQ> val;
            if (c0 >= a.C_in) {
                val = vzero<T, VQ>();
            } else if (L == NHWC && vec_in) {
                val = tile_pixel<T, L, SRC, VQ>(g, a, s_nb, n, gy, gx, slot, high, pe, r0 + pu, pv, c0);
            } else {
#pragma unroll
                for (int t = 0; t < VQ; ++t)
                    val.e[t] = (c0 + t < a.C_in)
                                   ? tile_pixel<T, L, SRC, 1>(g, a, s_nb, n, gy, gx, slot, high, pe, r0 + pu, pv,
                                                              c0 + t).e[0]
                                   : from_f32<T>(0.0f);
            }
            *reinterpret_cast<uint4*>(s_in + swz(p, q)) = val.raw;
        }
        // -- stage the chunk's weights as [tap][co][ci]
        for (int it = tid; it < NT * KC; it += WG) {
            const int col = it / KC, cil = it - col * KC;
            const int co = co0 + col, ci = kc * KC + cil;
            T wv[9];
            if (co < a.C_out && ci < a.C_in) {
                const T* src = wgt + ((size_t)co * a.C_in + ci) * 9;
#pragma unroll
                for (int t = 0; t < 9; ++t) wv[t] = src[t];
            } else {
#pragma unroll
                for (int t = 0; t < 9; ++t) wv[t] = from_f32<T>(0.0f);
            }
            const int byte = cil * (int)sizeof(T);
#pragma unroll
            for (int t = 0; t < 9; ++t) {
                const int row = t * NT + col;
                *reinterpret_cast<T*>(s_w + swz(row, byte >> 4) + (byte & 15)) = wv[t];
            }
        }
        __syncthreads();
        // -- MFMA over the 9 taps of this chunk
#pragma unroll
        for (int tap = 0; tap < 9; ++tap) {
            const int toff = (tap / 3) * pe + (tap % 3);
#pragma unroll
            for (int ks = 0; ks < KC / mf::KS; ++ks) {
                const int byte = (ks * mf::KS + kg * mf::EL) * (int)sizeof(T);
                typename mf::frag b[4];
#pragma unroll
                for (int ns = 0; ns < 4; ++ns) {
                    const int row = tap * NT + ns * 16 + l16;
                    b[ns] = *reinterpret_cast<const typename mf::frag*>(s_w + swz(row, byte >> 4) + (byte & 15));
                }
#pragma unroll
                for (int ms = 0; ms < 4; ++ms) {
                    if (wave + 4 * ms < nst) {
                        const int p = pbase[ms] + toff;
                        const typename mf::frag av =
                            *reinterpret_cast<const typename mf::frag*>(s_in + swz(p, byte >> 4) + (byte & 15));
#pragma unroll
                        for (int ns = 0; ns < 4; ++ns) acc[ms][ns] = mf::mma(av, b[ns], acc[ms][ns]);
                    }
                }
            }
        }
        __syncthreads();
    }

    // -- epilogue: stage fp32 accumulators as [m][co], then store vectors
    float* s_st = reinterpret_cast<float*>(smem);
#pragma unroll
    for (int ms = 0; ms < 4; ++ms) {
        if (wave + 4 * ms < nst) {
#pragma unroll
            for (int ns = 0; ns < 4; ++ns)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int m = (wave + 4 * ms) * 16 + kg * 4 + r;
                    if (m < M) s_st[m * SROW + ns * 16 + l16] = acc[ms][ns][r];
                }
        }
    }
    __syncthreads();

    const T* __restrict__ bias = (const T*)a.bias;
    const bool relu = (a.flags & 1) != 0;
    if constexpr (L == NHWC) {
        constexpr int VS = 16 / (int)sizeof(T);
        const int items = M * (NT / VS);
        for (int it = tid; it < items; it += WG) {
            const int m = it / (NT / VS), nq = (it - m * (NT / VS)) * VS;
            const int co = co0 + nq;
            if (co >= a.C_out) continue;
            const int i = r0 + m / e, j = m % e;
            float f[VS];
#pragma unroll
            for (int t = 0; t < VS; ++t) {
                f[t] = s_st[m * SROW + nq + t];
                if (bias && co + t < a.C_out) f[t] += to_f32(bias[co + t]);
            }
            size_t off = 0;
            T* out;
            if constexpr (DST == DST_PACKED) {
                off = (((size_t)slot * e + i) * e + j) * a.C_out + co;
                out = (T*)(high ? a.out_hi : a.out_lo);
                const T* res = (const T*)(high ? a.res_hi : a.res_lo);
                if (res) {
#pragma unroll
                    for (int t = 0; t < VS; ++t)
                        if (co + t < a.C_out) f[t] += to_f32(res[off + t]);
                }
            } else {
                out = (T*)a.out_hi;
            }
            Vec<T, VS> o;
#pragma unroll
            for (int t = 0; t < VS; ++t) o.e[t] = from_f32<T>(relu ? fmaxf(f[t], 0.0f) : f[t]);
            if constexpr (DST == DST_PACKED) {
                if (vec_out) {
                    vstore<T, VS>(out + off, o);
                } else {
#pragma unroll
                    for (int t = 0; t < VS; ++t)
                        if (co + t < a.C_out) out[off + t] = o.e[t];
                }
            } else {
                const int reps = high ? 1 : 2;
                for (int dy = 0; dy < reps; ++dy)
                    for (int dx = 0; dx < reps; ++dx) {
                        const int Y = gy * g.bs + (high ? i : 2 * i + dy);
                        const int X = gx * g.bs + (high ? j : 2 * j + dx);
                        const size_t doff = (((size_t)n * g.H + Y) * g.W + X) * a.C_out + co;
                        if (vec_out) {
                            vstore<T, VS>(out + doff, o);
                        } else {
#pragma unroll
                            for (int t = 0; t < VS; ++t)
                                if (co + t < a.C_out) out[doff + t] = o.e[t];
                        }
                    }
            }
        }
    } else {
        const int items = NT * M;
        for (int it = tid; it < items; it += WG) {
            const int nn = it / M, m = it - nn * M;
            const int co = co0 + nn;
            if (co >= a.C_out) continue;
            const int i = r0 + m / e, j = m % e;
            float f = s_st[m * SROW + nn];
            if (bias) f += to_f32(bias[co]);
            if constexpr (DST == DST_PACKED) {
                const size_t off = (((size_t)slot * a.C_out + co) * e + i) * e + j;
                const T* res = (const T*)(high ? a.res_hi : a.res_lo);
                if (res) f += to_f32(res[off]);
                T* out = (T*)(high ? a.out_hi : a.out_lo);
                out[off] = from_f32<T>(relu ? fmaxf(f, 0.0f) : f);
            } else {
                T* out = (T*)a.out_hi;
                const T o = from_f32<T>(relu ? fmaxf(f, 0.0f) : f);
                const int reps = high ? 1 : 2;
                for (int dy = 0; dy < reps; ++dy)
                    for (int dx = 0; dx < reps; ++dx) {
                        const int Y = gy * g.bs + (high ? i : 2 * i + dy);
                        const int X = gx * g.bs + (high ? j : 2 * j + dx);
                        out[(((size_t)n * a.C_out + co) * g.H + Y) * g.W + X] = o;
                    }
            }
        }
    }
}

inline int clampi(int v, int lo, int hi) { return v < lo ? lo : (v > hi ? hi : v); }
inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

template <typename T, int L, int SRC, int DST>
hipError_t run_conv(const Geo& g, const uint8_t* mask, const ConvArgs& a, hipStream_t st) {
    const int eh = g.bs, el = g.bs / 2;
    const int Rh = clampi(MT / eh, 1, eh), Rl = clampi(MT / el, 1, el);
    const int G = (((eh + Rh - 1) / Rh) > ((el + Rl - 1) / Rl)) ? (eh + Rh - 1) / Rh : (el + Rl - 1) / Rl;
    const int in_px = ((Rh + 2) * (eh + 2) > (Rl + 2) * (el + 2)) ? (Rh + 2) * (eh + 2) : (Rl + 2) * (el + 2);
    const int w_off = in_px * ROWB;
    const int m_max = (Rh * eh > Rl * el) ? Rh * eh : Rl * el;
    const int stage = m_max * SROW * 4;
    const int smem = (w_off + W_BYTES > stage) ? w_off + W_BYTES : stage;
    const int vec_in = (L == NHWC) && (a.C_in % (16 / (int)sizeof(T)) == 0) && aligned16(a.in_hi) &&
                       (SRC == SRC_DENSE || aligned16(a.in_lo));
    constexpr int VS = 16 / (int)sizeof(T);
    const int vec_out = (a.C_out % VS == 0) && aligned16(a.out_hi) && (DST == DST_DENSE || aligned16(a.out_lo)) &&
                        aligned16(a.res_hi) && aligned16(a.res_lo);
    // raise the kernel's dynamic-LDS limit to what this launch needs (kept per instantiation)
    static int attr_bytes = 0;
    if (smem > attr_bytes) {
        hipError_t e = hipFuncSetAttribute((const void*)k_conv<T, L, SRC, DST>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, smem);
        if (e != hipSuccess) return e;
        attr_bytes = smem;
    }
    const dim3 grid((unsigned)(g.B * G), (unsigned)((a.C_out + NT - 1) / NT));
    hipLaunchKernelGGL((k_conv<T, L, SRC, DST>), grid, dim3(WG), smem, st, g, mask, a, Rh, Rl, G, w_off, vec_in,
                       vec_out);
    return hipGetLastError();
}

template <typename T, int SRC, int DST>
hipError_t conv_l(int layout, const Geo& g, const uint8_t* mask, const ConvArgs& a, hipStream_t st) {
    if (layout == NHWC) return run_conv<T, NHWC, SRC, DST>(g, mask, a, st);
    return run_conv<T, NCHW, SRC, DST>(g, mask, a, st);
}

template <typename T>
hipError_t conv_t(int layout, ConvSrc src, ConvDst dst, const Geo& g, const uint8_t* mask, const ConvArgs& a,
                  hipStream_t st) {
    if (src == SRC_PADDED) return conv_l<T, SRC_PADDED, DST_PACKED>(layout, g, mask, a, st);
    if (src == SRC_PACKED) return conv_l<T, SRC_PACKED, DST_PACKED>(layout, g, mask, a, st);
    (void)dst;
    return conv_l<T, SRC_DENSE, DST_DENSE>(layout, g, mask, a, st);
}

}  // namespace

hipError_t launch_conv(int dtype, int layout, ConvSrc src, ConvDst dst, const Geo& g, const uint8_t* mask,
                       const ConvArgs& a, hipStream_t st) {
    switch (dtype) {
    case 0: return conv_t<float>(layout, src, dst, g, mask, a, st);
    case 1: return conv_t<f16>(layout, src, dst, g, mask, a, st);
    default: return conv_t<bf16>(layout, src, dst, g, mask, a, st);
    }
}

}  // namespace sb
