// 3x3 block convolution as an MFMA implicit GEMM for gfx950.
//
// GEMM view per block: output pixels x output channels, K = 9 taps x C_in.
// One workgroup (4 waves) computes a tile of up to 256 output pixels (whole
// rows of one block) x 64 output channels.  K is walked in chunks of 64
// bytes of input channels (32 fp16/bf16 or 16 fp32): the padded input rows
// of the tile and the chunk's weights are staged in LDS with an XOR swizzle
// of the 16-byte sub-chunks, and every tap reads its pixel fragments at a
// constant offset from the same LDS tile.
//
// MFMA: v_mfma_f32_16x16x32_{f16,bf16} (8 K values per lane) or
// v_mfma_f32_16x16x4_f32, with the weights as the A operand (16 output
// channels) and the pixels as the B operand (16 pixels).  A lane's result is
// then 4 consecutive output channels of one pixel, which the epilogue stores
// directly (8 bytes for fp16/bf16) without a trip through LDS.  Each wave
// owns up to four 16-pixel sub-tiles and all four 16-channel sub-tiles (64
// fp32 accumulators per lane).
//
// Staging is batched: every thread computes the sources of several 16-byte
// vectors, issues all their loads, then writes LDS.  While the MFMAs of
// chunk kc run, the weights and the first input batch of chunk kc+1 are
// already being loaded into registers.  LDS use (58.6 KiB for 32-pixel
// blocks) allows two workgroups per CU, so one workgroup's loads overlap
// the other's MFMAs.
//
// The tile loader is where the block modules live:
//   SRC_PADDED : reads padded stacks (plain conv of segblocks_conv3x3)
//   SRC_PACKED : BlockPad fused (neighbour lookup into the packed stacks)
//   SRC_DENSE  : BlockSample + BlockPad fused (reads the dense input map)
// and the store is either a packed stack or BlockCombine into a dense map.
//
// Weights: channels-last calls take OHWI memory ([C_out][3][3][C_in], the
// memory of a channels_last [C_out, C_in, 3, 3] tensor), NCHW calls OIHW.
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
constexpr int W_BYTES = 9 * NT * ROWB;
// Input-tile vectors per thread per batch (UI), and prefetched during the
// MFMAs (UP).  A fused-pad source may need four loads per vector (2x2
// average), so its batches are smaller and only its weights are prefetched,
// to stay within 256 VGPRs (the next chunk's input pixels share cache lines
// with the current chunk's and come from L2).
template <int SRC> struct Batches { static constexpr int UI = 2, UP = 0; };
template <> struct Batches<SRC_PADDED> { static constexpr int UI = 4, UP = 2; };
constexpr int UW = 9 * NT * (ROWB / 16) / WG;  // weight vectors per thread per chunk
static_assert(UW * WG == 9 * NT * (ROWB / 16), "weight staging covers the chunk exactly");

// byte offset of 16-byte sub-chunk q of LDS row `row`: sub-chunks are XOR-
// swizzled with bits 1..2 of the row so that 8 consecutive rows read at the
// same sub-chunk hit 8 distinct 16-byte bank groups.
__device__ __forceinline__ int swz(int row, int q) { return row * ROWB + ((q ^ ((row >> 1) & 3)) << 4); }

// Geometry of one workgroup's tile (uniform across the workgroup).
struct Tile {
    int n, gy, gx, slot, high, e, pe, r0, rows, M, in_px;
};

// Source of the tile pixel p (padded-tile coordinates, row-major over
// (rows + 2) x pe) for channels starting at c.
template <typename T, int L, int SRC>
__device__ __forceinline__ Src<T> tile_src(const Geo& g, const ConvArgs& a, const Neigh& nb, const Tile& t, int p,
                                           int c) {
    const int pu = p / t.pe, pv = p - pu * t.pe;
    const int u = t.r0 + pu;
    if constexpr (SRC == SRC_PADDED) {
        return src_copy<T>(stack_at<T, L>((const T*)(t.high ? a.in_hi : a.in_lo), t.slot, a.C_in, t.pe, u, pv, c));
    } else if constexpr (SRC == SRC_PACKED) {
        return packed_src<T, L>((const T*)a.in_hi, (const T*)a.in_lo, a.C_in, g.bs, nb, a.hi_cap, a.lo_cap, u - 1,
                                pv - 1, c, pad_mode(a.flags));
    } else {
        return dense_src<T, L>((const T*)a.in_hi, t.n, a.C_in, g.H, g.W, g.bs, t.gy, t.gx, nb, u - 1, pv - 1, c,
                               pad_mode(a.flags));
    }
}

// One batch of UI 16-byte input vectors (channels-last, C_in % 8 (fp16) or
// % 4 (fp32) == 0): item it -> pixel it/4, sub-chunk it%4.
template <typename T, int L, int SRC, int U>
struct InBatch {
    static constexpr int KC = ROWB / (int)sizeof(T);
    static constexpr int VQ = 16 / (int)sizeof(T);
    SrcBatch<T, VQ, U> b;

    __device__ __forceinline__ void issue(const Geo& g, const ConvArgs& a, const Neigh& nb, const Tile& t,
                                          int base, int kc) {
        const int items = t.in_px * 4;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int it = base + u * WG + (int)threadIdx.x;
            Src<T> s = src_zero<T>();
            if (it < items) {
                const int c0 = kc * KC + (it & 3) * VQ;
                if (c0 < a.C_in) s = tile_src<T, L, SRC>(g, a, nb, t, it >> 2, c0);
            }
            b.issue(u, s);
        }
    }
    __device__ __forceinline__ void commit(unsigned char* s_in, const Tile& t, int base) const {
        const int items = t.in_px * 4;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int it = base + u * WG + (int)threadIdx.x;
            if (it < items) *reinterpret_cast<uint4*>(s_in + swz(it >> 2, it & 3)) = b.value(u).raw;
        }
    }
};

// The weights of one K chunk as 16-byte vectors of OHWI memory, stored in LDS
// as rows [tap][co] of 64 bytes (the chunk's input channels).
template <typename T>
struct WBatch {
    static constexpr int KC = ROWB / (int)sizeof(T);
    static constexpr int VQ = 16 / (int)sizeof(T);
    Vec<T, VQ> w[UW];

    __device__ __forceinline__ void issue(const ConvArgs& a, int co0, int kc) {
        const T* __restrict__ wgt = (const T*)a.weight;
#pragma unroll
        for (int u = 0; u < UW; ++u) {
            const int v = u * WG + (int)threadIdx.x;
            const int col = v / 36, rem = v - col * 36;
            const int tap = rem >> 2, q = rem & 3;
            const int co = co0 + col, ci = kc * KC + q * VQ;
            if (co < a.C_out && ci < a.C_in) w[u] = vload<T, VQ>(wgt + ((size_t)co * 9 + tap) * a.C_in + ci);
            else                             w[u] = vzero<T, VQ>();
        }
    }
    __device__ __forceinline__ void commit(unsigned char* s_w) const {
#pragma unroll
        for (int u = 0; u < UW; ++u) {
            const int v = u * WG + (int)threadIdx.x;
            const int col = v / 36, rem = v - col * 36;
            const int tap = rem >> 2, q = rem & 3;
            *reinterpret_cast<uint4*>(s_w + swz(tap * NT + col, q)) = w[u].raw;
        }
    }
};

// Element-wise staging of one K chunk (any layout and channel count): the
// input tile and the weights (OIHW for NCHW calls, OHWI for NHWC calls).
template <typename T, int L, int SRC>
__device__ __forceinline__ void stage_scalar(const Geo& g, const ConvArgs& a, const Neigh& nb, const Tile& t,
                                             int co0, int kc, unsigned char* s_in, unsigned char* s_w) {
    constexpr int KC = ROWB / (int)sizeof(T);
    constexpr int VQ = 16 / (int)sizeof(T);
    const int tid = threadIdx.x;
    for (int it = tid; it < t.in_px * 4; it += WG) {
        const int p = it >> 2, q = it & 3;
        const int c0 = kc * KC + q * VQ;
        Vec<T, VQ> val;
#pragma unroll
        for (int e = 0; e < VQ; ++e) {
            const int c = c0 + e;
            T v = from_f32<T>(0.0f);
            if (c < a.C_in) {
                const Src<T> s = tile_src<T, L, SRC>(g, a, nb, t, p, c);
                if (s.p) v = s.avg ? avg4(s.p[0], s.p[s.d1], s.p[s.d2], s.p[s.d2 + s.d1]) : s.p[0];
            }
            val.e[e] = v;
        }
        *reinterpret_cast<uint4*>(s_in + swz(p, q)) = val.raw;
    }
    const T* __restrict__ wgt = (const T*)a.weight;
    for (int it = tid; it < NT * KC; it += WG) {
        const int col = it / KC, cil = it - col * KC;
        const int co = co0 + col, ci = kc * KC + cil;
        const bool ok = co < a.C_out && ci < a.C_in;
        const int byte = cil * (int)sizeof(T);
#pragma unroll
        for (int tap = 0; tap < 9; ++tap) {
            T wv = from_f32<T>(0.0f);
            if (ok) {
                if constexpr (L == NHWC) wv = wgt[((size_t)co * 9 + tap) * a.C_in + ci];
                else                     wv = wgt[((size_t)co * a.C_in + ci) * 9 + tap];
            }
            *reinterpret_cast<T*>(s_w + swz(tap * NT + col, byte >> 4) + (byte & 15)) = wv;
        }
    }
}

template <typename T, int L, int SRC, int DST, bool VEC>
__global__ __launch_bounds__(WG, 2) void k_conv(Geo g, const uint8_t* __restrict__ mask, ConvArgs a, int Rh,
                                                int Rl, int G, int w_off, int vec_out) {
    extern __shared__ __align__(16) unsigned char smem[];
    typedef MF<T> mf;
    constexpr int KC = ROWB / (int)sizeof(T);  // channels per K chunk
    constexpr bool NEED_SLOTS = !(SRC == SRC_DENSE && DST == DST_DENSE);

    const int k = (int)blockIdx.x / G;
    const int grp = (int)blockIdx.x - k * G;
    const int co0 = blockIdx.y * NT;
    Tile t;
    {
        const int per = g.GH * g.GW;
        t.n = k / per;
        const int rem = k - t.n * per;
        t.gy = rem / g.GW;
        t.gx = rem - t.gy * g.GW;
    }
    WaveMask wm;
    wm.init(mask, (int)g.B);
    const Neigh nb = wave_neighbourhood<NEED_SLOTS>(wm, g.GH, g.GW, t.n, t.gy, t.gx);
    t.high = (nb.high >> 4) & 1;
    t.slot = nb.slot[4];
    if (NEED_SLOTS && t.slot >= (t.high ? a.hi_cap : a.lo_cap)) return;
    t.e = t.high ? g.bs : (g.bs >> 1);
    const int R = t.high ? Rh : Rl;
    t.r0 = grp * R;
    if (t.r0 >= t.e) return;
    t.rows = min(R, t.e - t.r0);
    t.M = t.rows * t.e;
    t.pe = t.e + 2;
    t.in_px = (t.rows + 2) * t.pe;

    unsigned char* s_in = smem;
    unsigned char* s_w = smem + w_off;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int l16 = lane & 15, kg = lane >> 4;

    const int nst = (t.M + 15) >> 4;  // 16-pixel sub-tiles
    int pbase[4];
#pragma unroll
    for (int ms = 0; ms < 4; ++ms) {
        const int m = min((wave + 4 * ms) * 16 + l16, t.M - 1);
        const int i = m / t.e, j = m - i * t.e;
        pbase[ms] = i * t.pe + j;
    }
    const int nchunks = (a.C_in + KC - 1) / KC;
    const int in_items = t.in_px * 4;
    constexpr int UI = Batches<SRC>::UI, UP = Batches<SRC>::UP;

    // -- chunk 0
    if constexpr (VEC) {
        {
            WBatch<T> wb;
            InBatch<T, L, SRC, UI> ib;
            wb.issue(a, co0, 0);
            ib.issue(g, a, nb, t, 0, 0);
            wb.commit(s_w);
            ib.commit(s_in, t, 0);
        }
        for (int base = WG * UI; base < in_items; base += WG * UI) {
            InBatch<T, L, SRC, UI> ib;
            ib.issue(g, a, nb, t, base, 0);
            ib.commit(s_in, t, base);
        }
    } else {
        stage_scalar<T, L, SRC>(g, a, nb, t, co0, 0, s_in, s_w);
    }
    __syncthreads();

    floatx4 acc[4][4];
#pragma unroll
    for (int ms = 0; ms < 4; ++ms)
#pragma unroll
        for (int ns = 0; ns < 4; ++ns) acc[ms][ns] = floatx4{0.f, 0.f, 0.f, 0.f};

    for (int kc = 0; kc < nchunks; ++kc) {
        const bool more = kc + 1 < nchunks;
        // -- prefetch the next chunk's weights and first input batch
        WBatch<T> wb;
        InBatch<T, L, SRC, (UP > 0 ? UP : 1)> ib;
        if constexpr (VEC) {
            if (more) {
                wb.issue(a, co0, kc + 1);
                if constexpr (UP > 0) ib.issue(g, a, nb, t, 0, kc + 1);
            }
        }
        // -- MFMA over the 9 taps of this chunk
#pragma unroll 1
        for (int tap = 0; tap < 9; ++tap) {
            const int toff = (tap / 3) * t.pe + (tap % 3);
#pragma unroll
            for (int ks = 0; ks < KC / mf::KS; ++ks) {
                const int byte = (ks * mf::KS + kg * mf::EL) * (int)sizeof(T);
                typename mf::frag wf[4];
#pragma unroll
                for (int ns = 0; ns < 4; ++ns) {
                    const int row = tap * NT + ns * 16 + l16;
                    wf[ns] = *reinterpret_cast<const typename mf::frag*>(s_w + swz(row, byte >> 4) + (byte & 15));
                }
#pragma unroll
                for (int ms = 0; ms < 4; ++ms) {
                    if (wave + 4 * ms < nst) {
                        const int p = pbase[ms] + toff;
                        const typename mf::frag pf =
                            *reinterpret_cast<const typename mf::frag*>(s_in + swz(p, byte >> 4) + (byte & 15));
#pragma unroll
                        for (int ns = 0; ns < 4; ++ns) acc[ms][ns] = mf::mma(wf[ns], pf, acc[ms][ns]);
                    }
                }
            }
        }
        __syncthreads();
        if (more) {
            if constexpr (VEC) {
                wb.commit(s_w);
                if constexpr (UP > 0) ib.commit(s_in, t, 0);
                for (int base = WG * UP; base < in_items; base += WG * UI) {
                    InBatch<T, L, SRC, UI> ib2;
                    ib2.issue(g, a, nb, t, base, kc + 1);
                    ib2.commit(s_in, t, base);
                }
            } else {
                stage_scalar<T, L, SRC>(g, a, nb, t, co0, kc + 1, s_in, s_w);
            }
            __syncthreads();
        }
    }

    // -- epilogue: lane holds channels co0 + ns*16 + kg*4 + {0..3} of pixel (wave + 4*ms)*16 + l16
    const T* __restrict__ bias = (const T*)a.bias;
    const bool relu = (a.flags & 1) != 0;
    float bv[4][4];
#pragma unroll
    for (int ns = 0; ns < 4; ++ns)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int co = co0 + ns * 16 + kg * 4 + r;
            bv[ns][r] = (bias && co < a.C_out) ? to_f32(bias[co]) : 0.0f;
        }
    const T* res_base = (const T*)(t.high ? a.res_hi : a.res_lo);
    T* out_base = (T*)((DST == DST_DENSE || t.high) ? a.out_hi : a.out_lo);
#pragma unroll
    for (int ms = 0; ms < 4; ++ms) {
        if (wave + 4 * ms >= nst) continue;
        const int m = (wave + 4 * ms) * 16 + l16;
        if (m >= t.M) continue;
        const int i = t.r0 + m / t.e, j = m % t.e;
#pragma unroll
        for (int ns = 0; ns < 4; ++ns) {
            const int co = co0 + ns * 16 + kg * 4;
            if (co >= a.C_out) continue;
            float f[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) f[r] = acc[ms][ns][r] + bv[ns][r];
            const bool full = vec_out && co + 4 <= a.C_out;
            if constexpr (DST == DST_PACKED) {
                // packed stack element (slot, co + r, i, j)
                size_t off[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    if constexpr (L == NHWC) off[r] = (((size_t)t.slot * t.e + i) * t.e + j) * a.C_out + co + r;
                    else off[r] = (((size_t)t.slot * a.C_out + co + r) * t.e + i) * t.e + j;
                }
                if (res_base) {
                    if (L == NHWC && full) {
                        const Vec<T, 4> rv = vload<T, 4>(res_base + off[0]);
#pragma unroll
                        for (int r = 0; r < 4; ++r) f[r] += to_f32(rv.e[r]);
                    } else {
#pragma unroll
                        for (int r = 0; r < 4; ++r)
                            if (co + r < a.C_out) f[r] += to_f32(res_base[off[r]]);
                    }
                }
                Vec<T, 4> o;
#pragma unroll
                for (int r = 0; r < 4; ++r) o.e[r] = from_f32<T>(relu ? fmaxf(f[r], 0.0f) : f[r]);
                if (L == NHWC && full) {
                    vstore<T, 4>(out_base + off[0], o);
                } else {
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        if (co + r < a.C_out) out_base[off[r]] = o.e[r];
                }
            } else {
                Vec<T, 4> o;
#pragma unroll
                for (int r = 0; r < 4; ++r) o.e[r] = from_f32<T>(relu ? fmaxf(f[r], 0.0f) : f[r]);
                const int reps = t.high ? 1 : 2;
                for (int dy = 0; dy < reps; ++dy)
                    for (int dx = 0; dx < reps; ++dx) {
                        const int Y = t.gy * g.bs + (t.high ? i : 2 * i + dy);
                        const int X = t.gx * g.bs + (t.high ? j : 2 * j + dx);
                        if constexpr (L == NHWC) {
                            T* p = out_base + (((size_t)t.n * g.H + Y) * g.W + X) * a.C_out + co;
                            if (full) {
                                vstore<T, 4>(p, o);
                            } else {
#pragma unroll
                                for (int r = 0; r < 4; ++r)
                                    if (co + r < a.C_out) p[r] = o.e[r];
                            }
                        } else {
#pragma unroll
                            for (int r = 0; r < 4; ++r)
                                if (co + r < a.C_out)
                                    out_base[(((size_t)t.n * a.C_out + co + r) * g.H + Y) * g.W + X] = o.e[r];
                        }
                    }
            }
        }
    }
}

inline int clampi(int v, int lo, int hi) { return v < lo ? lo : (v > hi ? hi : v); }
inline bool aligned(const void* p, int bytes) { return (reinterpret_cast<uintptr_t>(p) & (bytes - 1)) == 0; }

template <typename T, int L, int SRC, int DST, bool VEC>
hipError_t run_conv(const Geo& g, const uint8_t* mask, const ConvArgs& a, hipStream_t st) {
    const int eh = g.bs, el = g.bs / 2;
    const int Rh = clampi(MT / eh, 1, eh), Rl = clampi(MT / el, 1, el);
    const int G = (((eh + Rh - 1) / Rh) > ((el + Rl - 1) / Rl)) ? (eh + Rh - 1) / Rh : (el + Rl - 1) / Rl;
    const int in_px = ((Rh + 2) * (eh + 2) > (Rl + 2) * (el + 2)) ? (Rh + 2) * (eh + 2) : (Rl + 2) * (el + 2);
    const int w_off = in_px * ROWB;
    const int smem = w_off + W_BYTES;
    const int ob = 4 * (int)sizeof(T);  // one epilogue vector: 4 channels
    const int vec_out = (a.C_out % 4 == 0) && aligned(a.out_hi, ob) && aligned(a.out_lo, ob) &&
                        aligned(a.res_hi, ob) && aligned(a.res_lo, ob);
    hipError_t e = ensure_dyn_lds((const void*)k_conv<T, L, SRC, DST, VEC>, smem);
    if (e != hipSuccess) return e;
    const dim3 grid((unsigned)(g.B * G), (unsigned)((a.C_out + NT - 1) / NT));
    hipLaunchKernelGGL((k_conv<T, L, SRC, DST, VEC>), grid, dim3(WG), smem, st, g, mask, a, Rh, Rl, G, w_off,
                       vec_out);
    return hipGetLastError();
}

template <typename T, int SRC, int DST>
hipError_t conv_l(int layout, const Geo& g, const uint8_t* mask, const ConvArgs& a, hipStream_t st) {
    constexpr int VQ = 16 / (int)sizeof(T);
    if (layout == NHWC) {
        const bool vec = (a.C_in % VQ == 0) && aligned(a.in_hi, 16) && aligned(a.in_lo, 16) &&
                         aligned(a.weight, 16);
        if (vec) return run_conv<T, NHWC, SRC, DST, true>(g, mask, a, st);
        return run_conv<T, NHWC, SRC, DST, false>(g, mask, a, st);
    }
    return run_conv<T, NCHW, SRC, DST, false>(g, mask, a, st);
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

// A fused layer (dense map in and out) with many channels runs on the GEMM:
// with average sampling and blocks that tile the map, as the padded low
// stack (straight from the map) and the GEMM reading the high blocks from
// the map and writing the dense output; otherwise as split, the GEMM's block
// convolution (BlockPad fused) and combine over packed stacks in the
// caller's workspace, with room for every block in either class (the counts
// are only known on the device).  The values equal the one-kernel layer's up
// to the order of the fp32 accumulation.
namespace {

inline size_t round256(size_t b) { return (b + 255) / 256 * 256; }

bool layer_packed_route(int dtype, int layout, const Geo& g, const ConvArgs& a) {
    // Measured on the stage shapes of a 1024x2048 image (8x16 blocks): at 128
    // channels 44-50 -> 38-43 us (all-low 29 -> 38), at 512 105-116 -> 37-62 us
    // with split + GEMM + combine; the dense GEMM route (the padded low stack
    // from the map, high pixels read from it, the output written to it) takes
    // 8-10 us more off (128 channels 34 / 37 -> 24 / 27 us at 0 / 50 % low,
    // 512 channels 41 -> 33 us) and beats the general kernel at 256 channels as
    // well (40 / 43 -> 34 / 35 us on one 64x128 map).  Without the dense route
    // the general kernel stays faster at 129-256 channels on up to 8192 pixels
    // (two maps: 77 / 82 against 56 / 57 us with split + GEMM + combine).
    if (a.C_in <= 64 || layout != NHWC || (dtype != 1 && dtype != 2)) return false;
    if (a.C_in > 128 && a.C_in <= 256 && (long long)g.N * g.H * g.W <= 8192 && !igemm_dense_fits(dtype, layout, g, a))
        return false;
    Geo gi = g, go = g;
    gi.C = a.C_in;
    go.C = a.C_out;
    ConvArgs p = a;
    p.hi_cap = p.lo_cap = (int)g.B;
    return igemm_fits_shape(dtype, layout, g, p) && rows_fit(dtype, layout, gi, {}) && rows_fit(dtype, layout, go, {});
}

// the packed stacks of the route: [hi in][lo in][hi out][lo out][GEMM workspace]
struct PackedLayout {
    size_t hi_in, lo_in, hi_out, lo_out, gemm, total;
};

PackedLayout packed_layout(const Geo& g, const ConvArgs& a) {
    const size_t es = 2, cap = (size_t)g.B, lb = (size_t)g.bs / 2;
    PackedLayout L;
    L.hi_in = round256(cap * g.bs * g.bs * a.C_in * es);
    L.lo_in = round256(cap * lb * lb * a.C_in * es);
    L.hi_out = round256(cap * g.bs * g.bs * a.C_out * es);
    L.lo_out = round256(cap * lb * lb * a.C_out * es);
    ConvArgs p = a;
    p.hi_cap = p.lo_cap = (int)cap;
    L.gemm = igemm_ws_bytes(g, p, 3, 1);
    L.total = L.hi_in + L.lo_in + L.hi_out + L.lo_out + L.gemm;
    return L;
}

hipError_t layer_via_packed(int dtype, const Geo& g, const uint8_t* mask, const ConvArgs& a, Ws ws, hipStream_t st) {
    const PackedLayout L = packed_layout(g, a);
    if (ws.bytes < L.total || !ws.p) return hipErrorInvalidValue;
    const int cap = (int)g.B;
    char* base = (char*)ws.p;
    void *hi = base, *lo = base + L.hi_in, *ho = base + L.hi_in + L.lo_in;
    void* lo_o = base + L.hi_in + L.lo_in + L.hi_out;
    const Ws gws{base + L.hi_in + L.lo_in + L.hi_out + L.lo_out, L.gemm};
    Geo gi = g, go = g;
    gi.C = a.C_in;
    go.C = a.C_out;
    hipError_t e = launch_split_rows(dtype, gi, a.in_hi, mask, hi, cap, lo, cap, st);
    if (e != hipSuccess) return e;
    const ConvArgs p{hi, lo, a.weight, a.bias, nullptr, nullptr, ho, lo_o, a.C_in, a.C_out, a.flags, cap, cap};
    if ((e = launch_igemm(dtype, g, mask, p, 3, 1, gws, st)) != hipSuccess) return e;
    return launch_combine_rows(dtype, go, ho, lo_o, mask, cap, cap, a.out_hi, st);
}

}  // namespace

size_t conv_ws_bytes(int dtype, int layout, ConvSrc src, ConvDst dst, const Geo& g, const ConvArgs& a) {
    if (conv_res_fits_shape(dtype, layout, g, a)) return 0;
    if (src == SRC_PACKED && dst == DST_PACKED && igemm_fits_shape(dtype, layout, g, a))
        return igemm_ws_bytes(g, a, 3, 1);
    if (src == SRC_DENSE && dst == DST_DENSE && layer_packed_route(dtype, layout, g, a))
        return igemm_dense_fits(dtype, layout, g, a) ? igemm_dense_ws_bytes(g, a) : packed_layout(g, a).total;
    return 0;
}

hipError_t launch_conv(int dtype, int layout, ConvSrc src, ConvDst dst, const Geo& g, const uint8_t* mask,
                       const ConvArgs& a, Ws ws, hipStream_t st) {
    if (conv_res_fits(dtype, layout, g, a)) return launch_conv_res(dtype, src, dst, g, mask, a, st);
    if (src == SRC_PACKED && dst == DST_PACKED && igemm_fits(dtype, layout, g, a))
        return launch_igemm(dtype, g, mask, a, 3, 1, ws, st);
    if (src == SRC_DENSE && dst == DST_DENSE && layer_packed_route(dtype, layout, g, a) &&
        reinterpret_cast<uintptr_t>(a.in_hi) % 16 == 0 && reinterpret_cast<uintptr_t>(a.out_hi) % 16 == 0 &&
        reinterpret_cast<uintptr_t>(a.weight) % 16 == 0) {
        if (igemm_dense_fits(dtype, layout, g, a)) {
            if (ws.bytes < igemm_dense_ws_bytes(g, a)) return hipErrorInvalidValue;
            return launch_igemm_dense(dtype, g, mask, a, ws, st);
        }
        return layer_via_packed(dtype, g, mask, a, ws, st);
    }
    switch (dtype) {
    case 0: return conv_t<float>(layout, src, dst, g, mask, a, st);
    case 1: return conv_t<f16>(layout, src, dst, g, mask, a, st);
    default: return conv_t<bf16>(layout, src, dst, g, mask, a, st);
    }
}

}  // namespace sb
