// Backward pass of the block-conv layer y = combine(conv3x3(pad(split(x)))):
// the transposes of the block modules and the gradients of the block
// convolution.  BlockCombine and BlockSample transposed are the split and
// combine kernels run with their backward flag (sb_rows.hip, sb_gather.hip).
// Here:
//
//   k_pad_bwd     BlockPad transposed.  A block pixel gathers every padded
//                 pixel that read it, in the image frame: the full-resolution
//                 map Z that the high stacks' padded windows tile (with one
//                 pixel of overlap), and its half-resolution pool P that the
//                 low stacks' windows tile; Z's gradient takes P's through the
//                 2x2 average (a quarter each; all of it at the cell's
//                 top-left pixel with strided sampling), and BlockCombine's
//                 transpose hands Z's gradient to the block (copy for a high
//                 block, the sum of the cell for a low one).  No atomics: the
//                 sums run in a fixed order, so results do not depend on
//                 timing.
//   dgrad         the gradient of the valid 3x3 convolution of a padded block
//                 is a valid 3x3 convolution of the output gradient padded by
//                 two zeros, with the filters transposed (in <-> out) and
//                 rotated by 180 degrees, i.e. a zero-padded "same"
//                 convolution of the gradient padded by one: run on the
//                 implicit GEMM (channels-last fp16 / bf16, 64k output
//                 channels, blocks of 4k), else on the general block
//                 convolution kernel.
//   k_wgrad_mfma  the weight and bias gradients: sums over every output pixel
//                 of both stacks of outer products of the output gradient and
//                 the padded input around the pixel, as a GEMM whose K is the
//                 pixels (channels-last fp16 / bf16, channel counts multiples
//                 of 4).  A workgroup takes 64 output x 64 input channels over
//                 one range of pixels; its twelve waves are two sub-ranges x
//                 three tap rows x two halves of the output channels, each
//                 wave a 32 x (3 x 64) fp32 tile in v_mfma_f32_16x16x16
//                 accumulators.  Operands come straight
//                 from the stacks: a lane loads four consecutive channels of
//                 four consecutive pixels (8 bytes each) and transposes them
//                 in registers into the four K values of an MFMA operand, so
//                 lane n of an operand holds channels 4n + {0..3} of the four
//                 16-channel fragments.  The sub-ranges are added in LDS in a
//                 fixed order and the workgroup's sum goes to the workspace.
//   k_wgrad       the same sums on the vector ALU, 4 x 4 x 9 fp32 per thread
//                 over block rows (every other dtype, layout and channel
//                 count).
//   Either way the partial sums are added in a fixed order (k_wgrad_group
//   sums groups of 16 ranges, k_wgrad_reduce the groups in order), so
//   results do not depend on timing.
#include <algorithm>
#include <type_traits>

#include "sb_common.h"
#include "sb_kernels.h"
#include "sb_pixel.h"

namespace sb {

namespace {

constexpr int BPIECE = WG;

__device__ __forceinline__ void bcoords(int k, int GH, int GW, int& n, int& gy, int& gx) {
    const int per = GH * GW;
    n = k / per;
    const int rem = k - n * per;
    gy = rem / GW;
    gx = rem - gy * GW;
}

// Gradient that the padded windows of one class put on pixel (r, c) of the
// block (gy, gx) frame at extent e (block-local, 0 <= r, c < e): the windows
// of the block itself and of the neighbours whose one-pixel halo overlaps the
// pixel, counted only where that window belongs to the class `want_high`.
template <typename T, int L, int V>
__device__ __forceinline__ void window_sum(const T* __restrict__ pad, int C, int e, const Neigh& nb, int cap,
                                           bool want_high, int r, int c, int ch, float (&acc)[V]) {
    const int pe = e + 2;
#pragma unroll
    for (int dy = -1; dy <= 1; ++dy) {
        if ((dy == -1 && r != 0) || (dy == 1 && r != e - 1)) continue;
#pragma unroll
        for (int dx = -1; dx <= 1; ++dx) {
            if ((dx == -1 && c != 0) || (dx == 1 && c != e - 1)) continue;
            const int d = (dy + 1) * 3 + (dx + 1);
            if (!((nb.valid >> d) & 1) || (((nb.high >> d) & 1) != (want_high ? 1u : 0u))) continue;
            const int s = neigh_slot(nb, d);
            if (s >= cap) continue;
            const Vec<T, V> v = vload<T, V>(stack_at<T, L>(pad, s, C, pe, r - dy * e + 1, c - dx * e + 1, ch));
#pragma unroll
            for (int q = 0; q < V; ++q) acc[q] += to_f32(v.e[q]);
        }
    }
}

template <typename T, int L, int V>
__global__ __launch_bounds__(WG) void k_pad_bwd(const T* __restrict__ dhp, const T* __restrict__ dlp, int C, int H,
                                                int W, const uint8_t* __restrict__ mask, int bs, int B, int Gh, int Gl,
                                                T* __restrict__ dhi, T* __restrict__ dlo, int hi_cap, int lo_cap,
                                                int pm) {
    const int w = (int)blockIdx.x;
    bool high;
    int slot, piece;
    if (w < hi_cap * Gh) {
        high = true;
        slot = w / Gh;
        piece = w - slot * Gh;
    } else {
        high = false;
        slot = (w - hi_cap * Gh) / Gl;
        piece = (w - hi_cap * Gh) - slot * Gl;
    }
    WaveMask wm;
    wm.init(mask, B);
    const int k = wm.find_nth(slot, high);
    if (k < 0) return;
    const int GH = H / bs, GW = W / bs, lb = bs >> 1;
    int n, gy, gx;
    bcoords(k, GH, GW, n, gy, gx);
    const int e = high ? bs : lb;
    const Neigh nb = wave_neighbourhood<true>(wm, GH, GW, n, gy, gx);
    const int it = piece * BPIECE + (int)threadIdx.x;
    if (it >= e * e * C / V) return;
    int r, j, c;
    if constexpr (L == NHWC) {
        const int cv = C / V, pix = it / cv;
        c = (it - pix * cv) * V;
        r = pix / e;
        j = pix - r * e;
    } else {
        static_assert(L == NHWC || V == 1, "NCHW moves single elements");
        const int row = it / e;
        j = it - row * e;
        c = row / e;
        r = row - c * e;
    }
    float acc[V];
#pragma unroll
    for (int q = 0; q < V; ++q) acc[q] = 0.0f;
    if (pm == PM_ZERO) {  // every block was padded on its own: its interior only
        const Vec<T, V> v = vload<T, V>(stack_at<T, L>(high ? dhp : dlp, slot, C, e + 2, r + 1, j + 1, c));
#pragma unroll
        for (int q = 0; q < V; ++q) acc[q] = to_f32(v.e[q]);
    } else if (high) {
        // Z at this pixel: the high windows over it
        window_sum<T, L, V>(dhp, C, bs, nb, hi_cap, true, r, j, c, acc);
        // P at its cell: the low windows over it, through the 2x2 average (or the stride)
        if (pm == PM_AVG || ((r | j) & 1) == 0) {
            float h[V];
#pragma unroll
            for (int q = 0; q < V; ++q) h[q] = 0.0f;
            window_sum<T, L, V>(dlp, C, lb, nb, lo_cap, false, r >> 1, j >> 1, c, h);
            const float f = pm == PM_AVG ? 0.25f : 1.0f;
#pragma unroll
            for (int q = 0; q < V; ++q) acc[q] += f * h[q];
        }
    } else {
        // the four pixels of the cell in Z: the high windows over them
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
            for (int b = 0; b < 2; ++b) window_sum<T, L, V>(dhp, C, bs, nb, hi_cap, true, 2 * r + a, 2 * j + b, c, acc);
        // P at the cell, whose quarters (or whole, strided) come back through the four pixels
        window_sum<T, L, V>(dlp, C, lb, nb, lo_cap, false, r, j, c, acc);
    }
    Vec<T, V> o;
#pragma unroll
    for (int q = 0; q < V; ++q) o.e[q] = from_f32<T>(acc[q]);
    T* dst;
    if constexpr (L == NHWC) dst = (high ? dhi : dlo) + ((((size_t)slot * e + r) * e + j) * C + c);
    else                     dst = (high ? dhi : dlo) + ((((size_t)slot * C + c) * e + r) * e + j);
    vstore<T, V>(dst, o);
}

// ---------------------------------------------------------------------------
// dgrad helper
// ---------------------------------------------------------------------------

// Everything the data gradient's convolutions read, in one launch: the
// transposed-rotated weights, the all-high / all-low masks (nm bytes each)
// and both output-gradient stacks padded by `pad` zeros.
template <typename T, int L>
__global__ __launch_bounds__(WG) void k_dgrad_prep(const T* __restrict__ w, int Cout, int Cin, T* __restrict__ wt,
                                                   uint8_t* __restrict__ ones, uint8_t* __restrict__ zeros, long long nm,
                                                   const T* __restrict__ dho, int hi_cap, T* __restrict__ qh,
                                                   const T* __restrict__ dlo, int lo_cap, T* __restrict__ ql, int bs,
                                                   int pad) {
    const long long nw = (long long)Cout * Cin * 9;
    const int lb = bs >> 1, ph = bs + 2 * pad, pl = lb + 2 * pad;
    const long long nqh = (long long)hi_cap * Cout * ph * ph, nql = (long long)lo_cap * Cout * pl * pl;
    const long long total = nw + 2 * nm + nqh + nql;
    for (long long i = (long long)blockIdx.x * WG + threadIdx.x; i < total; i += (long long)gridDim.x * WG) {
        if (i < nw) {
            int ci, co, t;  // i indexes wt in its memory order
            if constexpr (L == NHWC) {  // [Cin][3][3][Cout]
                co = (int)(i % Cout);
                t = (int)((i / Cout) % 9);
                ci = (int)(i / (Cout * 9));
            } else {                    // [Cin][Cout][3][3]
                t = (int)(i % 9);
                co = (int)((i / 9) % Cout);
                ci = (int)(i / (9 * Cout));
            }
            const int ts = 8 - t;       // (2 - ky, 2 - kx)
            size_t src;
            if constexpr (L == NHWC) src = ((size_t)co * 9 + ts) * Cin + ci;
            else                     src = ((size_t)co * Cin + ci) * 9 + ts;
            wt[i] = w[src];
            continue;
        }
        long long k = i - nw;
        if (k < 2 * nm) {
            if (k < nm) ones[k] = 1;
            else zeros[k - nm] = 0;
            continue;
        }
        k -= 2 * nm;
        const bool hi = k < nqh;
        if (!hi) k -= nqh;
        const T* src = hi ? dho : dlo;
        T* dst = hi ? qh : ql;
        const int e = hi ? bs : lb, pe = hi ? ph : pl;
        int s, c, u, v;
        if constexpr (L == NHWC) {
            c = (int)(k % Cout);
            long long q = k / Cout;
            v = (int)(q % pe);
            q /= pe;
            u = (int)(q % pe);
            s = (int)(q / pe);
        } else {
            v = (int)(k % pe);
            long long q = k / pe;
            u = (int)(q % pe);
            q /= pe;
            c = (int)(q % Cout);
            s = (int)(q / Cout);
        }
        const int a = u - pad, b = v - pad;
        T val = from_f32<T>(0.0f);
        if (a >= 0 && a < e && b >= 0 && b < e) {
            if constexpr (L == NHWC) val = src[(((size_t)s * e + a) * e + b) * Cout + c];
            else                     val = src[(((size_t)s * Cout + c) * e + a) * e + b];
        }
        dst[k] = val;
    }
}

// ---------------------------------------------------------------------------
// wgrad
// ---------------------------------------------------------------------------
constexpr int WG_CO = 64, WG_CI = 64;  // output / input channels of a workgroup
constexpr int WG_PX = 32;              // output pixels of a row strip

// Number of high blocks of the mask (every thread of the workgroup gets it).
__device__ __forceinline__ int count_high(const uint8_t* __restrict__ mask, int B, int* s_red) {
    int c = 0;
    for (int i = (int)threadIdx.x; i < B; i += WG) c += mask[i] != 0;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) c += __shfl_xor(c, o, 64);
    if ((threadIdx.x & 63) == 0) s_red[threadIdx.x >> 6] = c;
    __syncthreads();
    int t = 0;
#pragma unroll
    for (int w = 0; w < WG / 64; ++w) t += s_red[w];
    __syncthreads();
    return t;
}

// Element (s, c, y, x) of a stack of extent ext as fp32 (0 outside the channel range).
template <typename T, int L>
__device__ __forceinline__ float stk(const T* __restrict__ base, int s, int C, int ext, int y, int x, int c) {
    if (c >= C) return 0.0f;
    if constexpr (L == NHWC) return to_f32(base[(((size_t)s * ext + y) * ext + x) * C + c]);
    else                     return to_f32(base[(((size_t)s * C + c) * ext + y) * ext + x]);
}

// grid: (chunk, co block, ci block).  A chunk is a range of block rows of the
// concatenation [high stack rows, low stack rows] (high_rows = nh * bs).
template <typename T, int L>
__global__ __launch_bounds__(WG) void k_wgrad(const T* __restrict__ hp, const T* __restrict__ lp,
                                              const T* __restrict__ dho, const T* __restrict__ dlo,
                                              const uint8_t* __restrict__ mask, int B, int bs, int C_in, int C_out,
                                              int hi_cap, int lo_cap, int rows_per_chunk, float* __restrict__ part,
                                              float* __restrict__ part_b) {
    __shared__ float s_o[WG_PX][WG_CO];             // output-gradient strip (pixels x co)
    __shared__ float s_p[3][WG_PX + 2][WG_CI + 1];  // three padded input rows (pixels x ci)
    __shared__ int s_red[WG / 64];
    const int tid = (int)threadIdx.x;
    const int co0 = (int)blockIdx.y * WG_CO, ci0 = (int)blockIdx.z * WG_CI;
    const int tco = (tid >> 4) * 4, tci = (tid & 15) * 4;  // this thread's 4 co x 4 ci
    const int nh_all = count_high(mask, B, s_red);
    const int nh = min(nh_all, hi_cap), nl = min(B - nh_all, lo_cap);
    const int lb = bs >> 1;
    const long long rows_h = (long long)nh * bs, rows = rows_h + (long long)nl * lb;
    float acc[4][4][9];
    float accb[4];
#pragma unroll
    for (int a = 0; a < 4; ++a) {
        accb[a] = 0.0f;
#pragma unroll
        for (int b = 0; b < 4; ++b)
#pragma unroll
            for (int t = 0; t < 9; ++t) acc[a][b][t] = 0.0f;
    }
    const long long r0 = (long long)blockIdx.x * rows_per_chunk;
    const long long r1 = min(rows, r0 + rows_per_chunk);
    for (long long rr = r0; rr < r1; ++rr) {
        const bool high = rr < rows_h;
        const int e = high ? bs : lb;
        const long long q = high ? rr : rr - rows_h;
        const int s = (int)(q / e), i = (int)(q - (long long)s * e);
        const T* P = high ? hp : lp;
        const T* O = high ? dho : dlo;
        for (int x = 0; x < e; x += WG_PX) {  // strips of up to WG_PX output pixels
            const int np = min(WG_PX, e - x);
            __syncthreads();
            for (int idx = tid; idx < np * WG_CO; idx += WG) {
                const int p = idx / WG_CO, co = idx - p * WG_CO;
                s_o[p][co] = stk<T, L>(O, s, C_out, e, i, x + p, co0 + co);
            }
            for (int idx = tid; idx < 3 * (np + 2) * WG_CI; idx += WG) {
                const int ky = idx / ((np + 2) * WG_CI);
                const int rem = idx - ky * (np + 2) * WG_CI;
                const int p = rem / WG_CI, ci = rem - p * WG_CI;
                s_p[ky][p][ci] = stk<T, L>(P, s, C_in, e + 2, i + ky, x + p, ci0 + ci);
            }
            __syncthreads();
            for (int p = 0; p < np; ++p) {
                float o[4];
#pragma unroll
                for (int a = 0; a < 4; ++a) {
                    o[a] = s_o[p][tco + a];
                    accb[a] += o[a];
                }
#pragma unroll
                for (int t = 0; t < 9; ++t) {
                    const int ky = t / 3, kx = t - ky * 3;
#pragma unroll
                    for (int b = 0; b < 4; ++b) {
                        const float pv = s_p[ky][p + kx][tci + b];
#pragma unroll
                        for (int a = 0; a < 4; ++a) acc[a][b][t] += o[a] * pv;
                    }
                }
            }
        }
    }
    // partial sums of this chunk: part[chunk][co][t][ci] over the full channel ranges
    float* pc = part + (size_t)blockIdx.x * C_out * 9 * C_in;
#pragma unroll
    for (int a = 0; a < 4; ++a) {
        const int co = co0 + tco + a;
        if (co >= C_out) continue;
#pragma unroll
        for (int t = 0; t < 9; ++t)
#pragma unroll
            for (int b = 0; b < 4; ++b) {
                const int ci = ci0 + tci + b;
                if (ci < C_in) pc[((size_t)co * 9 + t) * C_in + ci] = acc[a][b][t];
            }
        if (part_b && blockIdx.z == 0 && (tid & 15) == 0) part_b[(size_t)blockIdx.x * C_out + co] = accb[a];
    }
}

// First stage of the partial-sum reduction when there are many chunks:
// thread (i, group) adds chunks 16 group .. 16 group + 15 of element i in
// order and leaves the sum in chunk 16 group (read by no other thread).
constexpr int WR_GROUP = 16;
__global__ __launch_bounds__(WG) void k_wgrad_group(float* __restrict__ part, int chunks, int total) {
    const long long gid = (long long)blockIdx.x * WG + threadIdx.x;
    const int groups = (chunks + WR_GROUP - 1) / WR_GROUP;
    if (gid >= (long long)total * groups) return;
    const int grp = (int)(gid / total), i = (int)(gid - (long long)grp * total);
    const int q0 = grp * WR_GROUP, q1 = min(chunks, q0 + WR_GROUP);
    float v[WR_GROUP];
#pragma unroll
    for (int u = 0; u < WR_GROUP; ++u) v[u] = q0 + u < q1 ? part[(size_t)(q0 + u) * total + i] : 0.0f;
    float s = v[0];
#pragma unroll
    for (int u = 1; u < WR_GROUP; ++u)
        if (q0 + u < q1) s += v[u];
    part[(size_t)q0 * total + i] = s;
}

// dw (call's format) and db from the chunk partial sums, added in chunk order
// (gstride 1), or from the group sums of k_wgrad_group in group order
// (gstride WR_GROUP).
template <typename T, int L>
__global__ __launch_bounds__(WG) void k_wgrad_reduce(const float* __restrict__ part, const float* __restrict__ part_b,
                                                     int chunks, int gstride, int C_in, int C_out, T* __restrict__ dw,
                                                     T* __restrict__ db) {
    const int total = C_out * 9 * C_in;
    const int i = (int)(blockIdx.x * WG + threadIdx.x);
    if (i < total) {
        float s = 0.0f;
        for (int q = 0; q < chunks; q += gstride) s += part[(size_t)q * total + i];
        const int ci = i % C_in, t = (i / C_in) % 9, co = i / (9 * C_in);
        size_t o;
        if constexpr (L == NHWC) o = i;  // [Cout][3][3][Cin]
        else                     o = ((size_t)co * C_in + ci) * 9 + t;
        dw[o] = from_f32<T>(s);
    }
    if (db && i < C_out) {
        // in chunk order, sixteen loads in flight at a time
        float s = 0.0f;
        int q = 0;
        for (; q + 16 <= chunks; q += 16) {
            float v[16];
#pragma unroll
            for (int u = 0; u < 16; ++u) v[u] = part_b[(size_t)(q + u) * C_out + i];
#pragma unroll
            for (int u = 0; u < 16; ++u) s += v[u];
        }
        for (; q < chunks; ++q) s += part_b[(size_t)q * C_out + i];
        db[i] = from_f32<T>(s);
    }
}

typedef float floatx4_t __attribute__((ext_vector_type(4)));
constexpr int WM_SUB = 2;                 // pixel sub-ranges of a workgroup
constexpr int WM_WAVES = 6 * WM_SUB;      // x three tap rows x two output-channel halves
constexpr int WM_THREADS = 64 * WM_WAVES;
constexpr int WM_LDS = (64 * 9 * 64 + 64) * 4;  // the workgroup's sums: [co][tap][ci] fp32, then the bias

template <typename T> struct WMF;
template <> struct WMF<f16> {
    typedef _Float16 h4 __attribute__((ext_vector_type(4)));
    static __device__ __forceinline__ floatx4_t mma(uint2 a, uint2 b, floatx4_t c) {
        return __builtin_amdgcn_mfma_f32_16x16x16f16(__builtin_bit_cast(h4, a), __builtin_bit_cast(h4, b), c, 0, 0, 0);
    }
};
template <> struct WMF<bf16> {
    typedef short s4 __attribute__((ext_vector_type(4)));
    static __device__ __forceinline__ floatx4_t mma(uint2 a, uint2 b, floatx4_t c) {
        return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s4, a), __builtin_bit_cast(s4, b), c, 0,
                                                          0, 0);
    }
};

// 16-bit element c (0..1) of four 32-bit words (one per pixel) as an MFMA
// operand: pixel u's value in 16-bit slot u.
__device__ __forceinline__ uint2 wm_gather2(const uint32_t (&v)[4], int c) {
    // byte selector of v_perm_b32: the low (c = 0) or high (c = 1) halves of
    // its second and first source
    const uint32_t sel = c ? 0x07060302u : 0x05040100u;
    return uint2{__builtin_amdgcn_perm(v[1], v[0], sel), __builtin_amdgcn_perm(v[3], v[2], sel)};
}
// 16-bit element c (0..3) of four 64-bit words (one per pixel), the same way.
__device__ __forceinline__ uint2 wm_gather4(const uint2 (&v)[4], int c) {
    uint32_t w[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) w[u] = (c & 2) ? v[u].y : v[u].x;
    return wm_gather2(w, c & 1);
}

// grid: (pixel range, co block, ci block).  The pixels are those of the high
// stack then the low stack (counts from the mask, capped by the capacities),
// in stack order; range r is [P r / R, P (r + 1) / R).
template <typename T>
__global__ __launch_bounds__(WM_THREADS, 1) void k_wgrad_mfma(const T* __restrict__ hp, const T* __restrict__ lp,
                                                              const T* __restrict__ dho, const T* __restrict__ dlo,
                                                              const uint8_t* __restrict__ mask, int B, int bs, int C_in,
                                                              int C_out, int hi_cap, int lo_cap,
                                                              float* __restrict__ part, float* __restrict__ part_b) {
    typedef WMF<T> mf;
    extern __shared__ __align__(16) float s_sum[];
    __shared__ int s_red[WM_WAVES];
    const int tid = (int)threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int hf = wave & 1, ky = (wave >> 1) % 3, sub = wave / 6;
    const int co0 = (int)blockIdx.y * 64, ci0 = (int)blockIdx.z * 64;
    const int n = lane & 15, kq = lane >> 4;

    // class counts
    int c = 0;
    for (int i = tid; i < B; i += WM_THREADS) c += mask[i] != 0;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) c += __shfl_xor(c, o, 64);
    if (lane == 0) s_red[wave] = c;
    __syncthreads();
    int nh_all = 0;
#pragma unroll
    for (int w = 0; w < WM_WAVES; ++w) nh_all += s_red[w];
    const int nh = min(nh_all, hi_cap), nl = min(B - nh_all, lo_cap);
    const int lb = bs >> 1;
    const long long P_h = (long long)nh * bs * bs, P = P_h + (long long)nl * lb * lb;
    // range and sub-range bounds at multiples of four pixels (a lane's four
    // pixels then stay in one block row whenever rows are multiples of four)
    const long long R = gridDim.x, r = blockIdx.x;
    const long long pa = (P * r / R) & ~3LL, pb = r + 1 == R ? P : (P * (r + 1) / R) & ~3LL;
    const long long ps = sub == 0 ? pa : (pa + (pb - pa) * sub / WM_SUB) & ~3LL;
    const long long pe = sub + 1 == WM_SUB ? pb : (pa + (pb - pa) * (sub + 1) / WM_SUB) & ~3LL;

    // this lane's channels: output channels co0 + 4 n + 2 hf + {0, 1} (the
    // wave's half of fragments 0..3), input channels ci0 + 4 n + {0..3}
    const int co_l = co0 + 4 * n, ci_l = ci0 + 4 * n;
    const bool co_ok = co_l < C_out, ci_ok = ci_l < C_in;
    floatx4_t acc[3][2][4];  // [kx][co fragment 2 hf + 0, 1][ci fragment]
#pragma unroll
    for (int a = 0; a < 3; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int d = 0; d < 4; ++d) acc[a][b][d] = floatx4_t{0.f, 0.f, 0.f, 0.f};
    float bsum[2] = {0.f, 0.f};

    // one step: sixteen pixels, K values 4 kq .. 4 kq + 3 from this lane.
    // Straight-line code: a pixel past the range loads from pixel 0 and is
    // zeroed, the stack-order walk to the next pixel uses selects.
    const int pe32 = (int)pe, nh32 = nh;
    auto load_step = [&](int stp, uint32_t (&va)[4], uint2 (&vb)[3][4]) {
        int p = (int)ps + 16 * stp + 4 * kq;
        bool high = p < (int)P_h;
        int e = high ? bs : lb;
        const int q = high ? p : p - (int)P_h;
        const int ee = e * e;
        int slot = q / ee;
        const int rem = q - slot * ee;
        int i = rem / e;
        int j = rem - i * e;
        if (p >= pe32) {  // past the sub-range: nothing to load
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                va[u] = 0u;
#pragma unroll
                for (int kx = 0; kx < 3; ++kx) vb[kx][u] = uint2{0u, 0u};
            }
            return;
        }
        if (j + 3 < e && p + 3 < pe32) {
            // the four pixels are consecutive in one row: fixed strides
            const T* O = high ? dho : dlo;
            const T* X = high ? hp : lp;
            const int pe2 = e + 2;
            const T* orow = O + ((size_t)(slot * e + i) * e + j) * C_out + (co_ok ? co_l + 2 * hf : 0);
            const T* xr = X + ((size_t)(slot * pe2 + i + ky) * pe2 + j) * C_in + (ci_ok ? ci_l : 0);
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const uint32_t a0 = *reinterpret_cast<const uint32_t*>(orow + (size_t)u * C_out);
                va[u] = co_ok ? a0 : 0u;
#pragma unroll
                for (int kx = 0; kx < 3; ++kx) {
                    const uint2 b0 = *reinterpret_cast<const uint2*>(xr + (size_t)(u + kx) * C_in);
                    vb[kx][u] = ci_ok ? b0 : uint2{0u, 0u};
                }
            }
            return;
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const bool ok = p < pe32;
            // a pixel past the range reads pixel 0 of a non-empty stack
            const bool hs = ok ? high : nh32 > 0;
            const T* O = hs ? dho : dlo;
            const T* X = hs ? hp : lp;
            const int pe2 = e + 2;
            const size_t opx = ok ? ((size_t)(slot * e + i) * e + j) : 0;
            const size_t xpx = ok ? ((size_t)(slot * pe2 + i + ky) * pe2 + j) : 0;
            const uint32_t a0 = *reinterpret_cast<const uint32_t*>(O + opx * C_out + (co_ok ? co_l + 2 * hf : 0));
            va[u] = (ok && co_ok) ? a0 : 0u;
            const T* xr = X + xpx * C_in + (ci_ok ? ci_l : 0);
#pragma unroll
            for (int kx = 0; kx < 3; ++kx) {
                const uint2 b0 = *reinterpret_cast<const uint2*>(xr + (size_t)kx * C_in);
                vb[kx][u] = (ok && ci_ok) ? b0 : uint2{0u, 0u};
            }
            // next pixel in stack order
            ++p;
            const bool wj = ++j == e;
            j = wj ? 0 : j;
            i += wj;
            const bool wi = i == e;
            i = wi ? 0 : i;
            slot += wi;
            const bool sw = high && slot == nh32;
            high = high && !sw;
            slot = sw ? 0 : slot;
            e = sw ? lb : e;
        }
    };
    auto compute_step = [&](const uint32_t (&va)[4], const uint2 (&vb)[3][4]) {
        uint2 fa[2];
#pragma unroll
        for (int cb = 0; cb < 2; ++cb) fa[cb] = wm_gather2(va, cb);
        if (ky == 0) {
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                Vec<T, 2> t;
                t.raw = va[u];
#pragma unroll
                for (int cb = 0; cb < 2; ++cb) bsum[cb] += to_f32(t.e[cb]);
            }
        }
#pragma unroll
        for (int kx = 0; kx < 3; ++kx)
#pragma unroll
            for (int cib = 0; cib < 4; ++cib) {
                const uint2 fb = wm_gather4(vb[kx], cib);
#pragma unroll
                for (int cb = 0; cb < 2; ++cb) acc[kx][cb][cib] = mf::mma(fa[cb], fb, acc[kx][cb][cib]);
            }
    };
    // (a second register set for the next step's loads does not fit beside
    // the accumulators at three waves per SIMD: the three waves of a SIMD
    // overlap each other's loads instead)
    const int steps = (int)((pe - ps + 15) / 16);
    for (int stp = 0; stp < steps; ++stp) {
        uint32_t va[4];
        uint2 vb[3][4];
        load_step(stp, va, vb);
        compute_step(va, vb);
    }

    // bias: the four pixel groups of a lane column, in a fixed order
#pragma unroll
    for (int cb = 0; cb < 2; ++cb) {
        bsum[cb] += __shfl_xor(bsum[cb], 16, 64);
        bsum[cb] += __shfl_xor(bsum[cb], 32, 64);
    }
    // the sub-ranges' sums, added in LDS in sub-range order.  Lane l holds
    // rows 4 (l >> 4) + rr of each 16 x 16 fragment, column l & 15: output
    // channel 16 (l >> 4) + 4 rr + (2 hf + cb), input channel 4 (l & 15) + cib.
    float* s_b = s_sum + 64 * 9 * 64;
    for (int ph = 0; ph < WM_SUB; ++ph) {
        if (sub == ph) {
#pragma unroll
            for (int kx = 0; kx < 3; ++kx)
#pragma unroll
                for (int cb = 0; cb < 2; ++cb)
#pragma unroll
                    for (int cib = 0; cib < 4; ++cib)
#pragma unroll
                        for (int rr = 0; rr < 4; ++rr) {
                            const int co = 16 * kq + 4 * rr + 2 * hf + cb, ci = 4 * n + cib;
                            float* d = s_sum + (co * 9 + 3 * ky + kx) * 64 + ci;
                            *d = ph == 0 ? acc[kx][cb][cib][rr] : *d + acc[kx][cb][cib][rr];
                        }
            if (ky == 0 && kq == 0) {
#pragma unroll
                for (int cb = 0; cb < 2; ++cb) {
                    float* d = s_b + 4 * n + 2 * hf + cb;
                    *d = ph == 0 ? bsum[cb] : *d + bsum[cb];
                }
            }
        }
        __syncthreads();
    }
    float* pc = part + (size_t)blockIdx.x * C_out * 9 * C_in;
    for (int idx = tid; idx < 64 * 9 * 16; idx += WM_THREADS) {  // four channels per store
        const int co = idx / (9 * 16), rest = idx - co * (9 * 16);
        const int t = rest >> 4, ci = (rest & 15) * 4;
        if (co0 + co < C_out && ci0 + ci < C_in)
            *reinterpret_cast<float4*>(pc + ((size_t)(co0 + co) * 9 + t) * C_in + ci0 + ci) =
                *reinterpret_cast<const float4*>(s_sum + 4 * idx);
    }
    if (part_b && blockIdx.z == 0 && tid < 64 && co0 + tid < C_out)
        part_b[(size_t)blockIdx.x * C_out + co0 + tid] = s_b[tid];
}

inline size_t r256(size_t b) { return (b + 255) / 256 * 256; }
inline int esz(int dtype) { return dtype == 0 ? 4 : 2; }

// The data gradient of each stack as a convolution of its own (the classes
// do not mix: the padded blocks are independent).  On the implicit GEMM:
// the output gradient padded by one zero (extent e + 2) taken as a stack of
// blocks of that extent, every block high, zero-padded on its own
// (SB_FLAG_PAD_ZERO), transposed-rotated weights: a "same" convolution whose
// output is the padded block's gradient.  Otherwise the general kernel runs
// a valid convolution over the gradient padded by two.
struct DgradCall {
    Geo g;
    ConvArgs a;
};
DgradCall dgrad_call(const Geo& g, int e, int cap, int C_in, int C_out) {
    DgradCall d;
    d.g = g;
    d.g.N = 1;
    d.g.C = C_out;
    d.g.bs = e + 2;
    d.g.GH = 1;
    d.g.GW = cap;
    d.g.B = cap;
    d.g.H = e + 2;
    d.g.W = cap * (e + 2);
    d.a = ConvArgs{nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, C_out, C_in,
                   PM_ZERO << 1, cap, 0};  // zero padding of each block on its own
    return d;
}
bool dgrad_igemm_shape(int dtype, int layout, const Geo& g, int C_in, int C_out, int hi_cap, int lo_cap) {
    if (g.bs % 4) return false;  // even extents e + 2 for both classes
    const DgradCall h = dgrad_call(g, g.bs, hi_cap, C_in, C_out), l = dgrad_call(g, g.bs / 2, lo_cap, C_in, C_out);
    return (hi_cap == 0 || igemm_fits_shape(dtype, layout, h.g, h.a)) &&
           (lo_cap == 0 || igemm_fits_shape(dtype, layout, l.g, l.a));
}

struct DgradLayout {
    bool ig_shape;  // the implicit GEMM takes these shapes
    size_t qh, ql, wt, masks, ig, total;
};

DgradLayout dgrad_layout(int dtype, int layout, const Geo& g, int C_in, int C_out, int hi_cap, int lo_cap) {
    const size_t es = esz(dtype), lb = g.bs / 2;
    DgradLayout D;
    D.qh = r256((size_t)hi_cap * C_out * (g.bs + 4) * (g.bs + 4) * es);
    D.ql = r256((size_t)lo_cap * C_out * (lb + 4) * (lb + 4) * es);
    D.wt = r256((size_t)C_in * C_out * 9 * es);
    D.masks = r256((size_t)std::max<long long>({g.B, (long long)hi_cap, (long long)lo_cap}) * 2);
    D.ig = 0;
    D.ig_shape = dgrad_igemm_shape(dtype, layout, g, C_in, C_out, hi_cap, lo_cap);
    if (D.ig_shape) {
        const DgradCall h = dgrad_call(g, g.bs, hi_cap, C_in, C_out), l = dgrad_call(g, (int)lb, lo_cap, C_in, C_out);
        D.ig = r256(std::max(hi_cap ? igemm_ws_bytes(h.g, h.a, 3, 1) : 0, lo_cap ? igemm_ws_bytes(l.g, l.a, 3, 1) : 0));
    }
    D.total = D.qh + D.ql + D.wt + D.masks + D.ig;
    return D;
}

struct WgradPlan {
    bool mfma;
    int chunks, rows_per_chunk, tiles_co, tiles_ci;
    size_t part, part_b, total;
};

// The MFMA kernel takes channels-last fp16 / bf16 with channel counts that
// are multiples of 4 (8-byte operand loads) and fewer than 2^30 pixels.
bool wgrad_mfma_fits(int dtype, int layout, const Geo& g, int C_in, int C_out, int hi_cap, int lo_cap) {
    const long long px = (long long)hi_cap * g.bs * g.bs + (long long)lo_cap * (g.bs / 2) * (g.bs / 2);
    return layout == NHWC && (dtype == 1 || dtype == 2) && C_in % 4 == 0 && C_out % 4 == 0 &&
           px < (1LL << 30);  // pixel indices in 32 bits
}

// mfma: the plan of k_wgrad_mfma (else of k_wgrad)
WgradPlan wgrad_plan(const Geo& g, int C_in, int C_out, int hi_cap, int lo_cap, bool bias, bool mfma) {
    WgradPlan p;
    p.tiles_co = (C_out + WG_CO - 1) / WG_CO;
    p.tiles_ci = (C_in + WG_CI - 1) / WG_CI;
    p.mfma = mfma;
    if (mfma) {
        // pixel ranges: one workgroup per CU over the channel blocks, at least
        // 256 pixels per range (partial sums cost 147 KB per range and block)
        const long long px = (long long)hi_cap * g.bs * g.bs + (long long)lo_cap * (g.bs / 2) * (g.bs / 2);
        const long long per_block = std::max(1LL, (long long)device_cus() / (p.tiles_co * p.tiles_ci));
        p.chunks = (int)std::max(1LL, std::min(per_block, (px + 255) / 256));
        p.rows_per_chunk = 0;
        p.part = r256((size_t)p.chunks * C_out * 9 * C_in * 4);
        p.part_b = bias ? r256((size_t)p.chunks * C_out * 4) : 0;
        p.total = p.part + p.part_b;
        return p;
    }
    // rows by capacity (the counts are on the device): aim at about 2 workgroups per CU
    const long long rows = (long long)hi_cap * g.bs + (long long)lo_cap * (g.bs / 2);
    const long long want = (2LL * device_cus() + p.tiles_co * p.tiles_ci - 1) / (p.tiles_co * p.tiles_ci);
    const long long per = rows > 0 ? (rows + want - 1) / want : 1;
    p.rows_per_chunk = (int)(per > 0 ? per : 1);
    p.chunks = rows > 0 ? (int)((rows + p.rows_per_chunk - 1) / p.rows_per_chunk) : 1;
    p.part = r256((size_t)p.chunks * C_out * 9 * C_in * 4);
    p.part_b = bias ? r256((size_t)p.chunks * C_out * 4) : 0;
    p.total = p.part + p.part_b;
    return p;
}

template <typename T>
hipError_t pad_bwd_t(int layout, const Geo& g, const void* dhp, const void* dlp, const uint8_t* mask, void* dhi,
                     void* dlo, int hi_cap, int lo_cap, int pm, hipStream_t st) {
    constexpr int VM = 16 / (int)sizeof(T);
    const bool al = ((reinterpret_cast<uintptr_t>(dhp) | reinterpret_cast<uintptr_t>(dlp) |
                      reinterpret_cast<uintptr_t>(dhi) | reinterpret_cast<uintptr_t>(dlo)) & 15) == 0;
    const int lb = g.bs / 2;
    auto run = [&](auto kern, int V) -> hipError_t {
        const int Gh = (int)(((long long)g.bs * g.bs * g.C / V + BPIECE - 1) / BPIECE);
        const int Gl = (int)(((long long)lb * lb * g.C / V + BPIECE - 1) / BPIECE);
        const long long blocks = (long long)hi_cap * Gh + (long long)lo_cap * Gl;
        if (blocks == 0) return hipSuccess;
        hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(WG), 0, st, (const T*)dhp, (const T*)dlp, g.C, g.H, g.W,
                           mask, g.bs, (int)g.B, Gh, Gl, (T*)dhi, (T*)dlo, hi_cap, lo_cap, pm);
        return hipGetLastError();
    };
    if (layout == NHWC) {
        if (al && g.C % VM == 0) return run(k_pad_bwd<T, NHWC, VM>, VM);
        return run(k_pad_bwd<T, NHWC, 1>, 1);
    }
    return run(k_pad_bwd<T, NCHW, 1>, 1);
}

template <typename T, int L>
hipError_t dgrad_t(const Geo& g, const void* dho, const void* dlo, const uint8_t* mask, const void* w, int C_in,
                   int C_out, void* dhp, void* dlp, int hi_cap, int lo_cap, Ws ws, hipStream_t st) {
    (void)mask;
    constexpr int dt = sizeof(T) == 4 ? 0 : (std::is_same<T, f16>::value ? 1 : 2);
    const DgradLayout D = dgrad_layout(dt, L, g, C_in, C_out, hi_cap, lo_cap);
    if (ws.bytes < D.total || !ws.p) return hipErrorInvalidValue;
    char* base = (char*)ws.p;
    T* qh = (T*)base;
    T* ql = (T*)(base + D.qh);
    T* wt = (T*)(base + D.qh + D.ql);
    uint8_t* ones = (uint8_t*)(base + D.qh + D.ql + D.wt);
    const long long nm = std::max<long long>({g.B, (long long)hi_cap, (long long)lo_cap});
    uint8_t* zeros = ones + nm;
    void* igws = base + D.qh + D.ql + D.wt + D.masks;
    const int lb = g.bs / 2;
    const int grid = device_cus() * 4;
    hipError_t e;
    // the implicit GEMM when both calls take it (shapes and alignment)
    DgradCall h = dgrad_call(g, g.bs, hi_cap, C_in, C_out), l = dgrad_call(g, lb, lo_cap, C_in, C_out);
    h.a.in_hi = qh;
    h.a.weight = wt;
    h.a.out_hi = dhp;
    l.a.in_hi = ql;
    l.a.weight = wt;
    l.a.out_hi = dlp;
    const bool ig = D.ig_shape && (hi_cap == 0 || igemm_fits(dt, L, h.g, h.a)) &&
                    (lo_cap == 0 || igemm_fits(dt, L, l.g, l.a));
    const int pad = ig ? 1 : 2;
    hipLaunchKernelGGL((k_dgrad_prep<T, L>), dim3(grid), dim3(WG), 0, st, (const T*)w, C_out, C_in, wt, ones, zeros,
                       nm, (const T*)dho, hi_cap, qh, (const T*)dlo, lo_cap, ql, g.bs, pad);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (ig) {
        const Ws w2{igws, D.ig};
        if (hi_cap > 0 && (e = launch_igemm(dt, h.g, ones, h.a, 3, 1, w2, st)) != hipSuccess) return e;
        if (lo_cap > 0 && (e = launch_igemm(dt, l.g, ones, l.a, 3, 1, w2, st)) != hipSuccess) return e;
        return hipSuccess;
    }
    // the high stack: every block of the grid taken as high, extent bs + 2 (the padded gradient)
    if (hi_cap > 0) {
        Geo gh = g;
        gh.bs = g.bs + 2;
        gh.H = g.GH * gh.bs;
        gh.W = g.GW * gh.bs;
        const ConvArgs a{qh, nullptr, wt, nullptr, nullptr, nullptr, dhp, nullptr, C_out, C_in, 0, hi_cap, 0};
        if ((e = launch_conv(dt, L, SRC_PADDED, DST_PACKED, gh, ones, a, Ws{nullptr, 0}, st)) != hipSuccess) return e;
    }
    // the low stack: every block taken as low, low extent lb + 2
    if (lo_cap > 0) {
        Geo gl = g;
        gl.bs = g.bs + 4;
        gl.H = g.GH * gl.bs;
        gl.W = g.GW * gl.bs;
        const ConvArgs a{nullptr, ql, wt, nullptr, nullptr, nullptr, nullptr, dlp, C_out, C_in, 0, 0, lo_cap};
        if ((e = launch_conv(dt, L, SRC_PADDED, DST_PACKED, gl, zeros, a, Ws{nullptr, 0}, st)) != hipSuccess) return e;
    }
    return hipSuccess;
}

template <typename T, int L>
hipError_t wgrad_t(const Geo& g, const void* hp, const void* lp, const void* dho, const void* dlo,
                   const uint8_t* mask, int C_in, int C_out, void* dw, void* db, int hi_cap, int lo_cap, Ws ws,
                   hipStream_t st) {
    constexpr int dt = sizeof(T) == 4 ? 0 : (std::is_same<T, f16>::value ? 1 : 2);
    const bool al8 = ((reinterpret_cast<uintptr_t>(hp) | reinterpret_cast<uintptr_t>(lp) |
                       reinterpret_cast<uintptr_t>(dho) | reinterpret_cast<uintptr_t>(dlo)) & 7) == 0;
    const bool mfma = al8 && wgrad_mfma_fits(dt, L, g, C_in, C_out, hi_cap, lo_cap);
    const WgradPlan p = wgrad_plan(g, C_in, C_out, hi_cap, lo_cap, db != nullptr, mfma);
    if (ws.bytes < p.total || !ws.p) return hipErrorInvalidValue;
    float* part = (float*)ws.p;
    float* part_b = db ? (float*)((char*)ws.p + p.part) : nullptr;
    hipError_t e;
    const dim3 grid((unsigned)p.chunks, (unsigned)p.tiles_co, (unsigned)p.tiles_ci);
    if constexpr (L == NHWC && dt != 0) {
        if (mfma) {
            if ((e = ensure_dyn_lds((const void*)k_wgrad_mfma<T>, WM_LDS)) != hipSuccess) return e;
            hipLaunchKernelGGL((k_wgrad_mfma<T>), grid, dim3(WM_THREADS), WM_LDS, st, (const T*)hp, (const T*)lp,
                               (const T*)dho, (const T*)dlo, mask, (int)g.B, g.bs, C_in, C_out, hi_cap, lo_cap, part,
                               part_b);
        }
    }
    if (!mfma)
        hipLaunchKernelGGL((k_wgrad<T, L>), grid, dim3(WG), 0, st, (const T*)hp, (const T*)lp, (const T*)dho,
                           (const T*)dlo, mask, (int)g.B, g.bs, C_in, C_out, hi_cap, lo_cap, p.rows_per_chunk, part,
                           part_b);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const int total = C_out * 9 * C_in;
    int gstride = 1;
    if (p.chunks > 2 * WR_GROUP) {
        const long long threads = (long long)total * ((p.chunks + WR_GROUP - 1) / WR_GROUP);
        hipLaunchKernelGGL(k_wgrad_group, dim3((unsigned)((threads + WG - 1) / WG)), dim3(WG), 0, st, part, p.chunks,
                           total);
        gstride = WR_GROUP;
    }
    hipLaunchKernelGGL((k_wgrad_reduce<T, L>), dim3((unsigned)((total + WG - 1) / WG)), dim3(WG), 0, st,
                       (const float*)part, (const float*)part_b, p.chunks, gstride, C_in, C_out, (T*)dw, (T*)db);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_pad_bwd(int dtype, int layout, const Geo& g, const void* dhp, const void* dlp, const uint8_t* mask,
                          void* dhi, void* dlo, int hi_cap, int lo_cap, int pm, hipStream_t st) {
    switch (dtype) {
    case 0: return pad_bwd_t<float>(layout, g, dhp, dlp, mask, dhi, dlo, hi_cap, lo_cap, pm, st);
    case 1: return pad_bwd_t<f16>(layout, g, dhp, dlp, mask, dhi, dlo, hi_cap, lo_cap, pm, st);
    default: return pad_bwd_t<bf16>(layout, g, dhp, dlp, mask, dhi, dlo, hi_cap, lo_cap, pm, st);
    }
}

size_t dgrad_ws_bytes(int dtype, int layout, const Geo& g, int C_in, int C_out, int hi_cap, int lo_cap) {
    return dgrad_layout(dtype, layout, g, C_in, C_out, hi_cap, lo_cap).total;
}

hipError_t launch_dgrad(int dtype, int layout, const Geo& g, const void* dho, const void* dlo, const uint8_t* mask,
                        const void* w, int C_in, int C_out, void* dhp, void* dlp, int hi_cap, int lo_cap, Ws ws,
                        hipStream_t st) {
    if (layout == NHWC) {
        switch (dtype) {
        case 0: return dgrad_t<float, NHWC>(g, dho, dlo, mask, w, C_in, C_out, dhp, dlp, hi_cap, lo_cap, ws, st);
        case 1: return dgrad_t<f16, NHWC>(g, dho, dlo, mask, w, C_in, C_out, dhp, dlp, hi_cap, lo_cap, ws, st);
        default: return dgrad_t<bf16, NHWC>(g, dho, dlo, mask, w, C_in, C_out, dhp, dlp, hi_cap, lo_cap, ws, st);
        }
    }
    switch (dtype) {
    case 0: return dgrad_t<float, NCHW>(g, dho, dlo, mask, w, C_in, C_out, dhp, dlp, hi_cap, lo_cap, ws, st);
    case 1: return dgrad_t<f16, NCHW>(g, dho, dlo, mask, w, C_in, C_out, dhp, dlp, hi_cap, lo_cap, ws, st);
    default: return dgrad_t<bf16, NCHW>(g, dho, dlo, mask, w, C_in, C_out, dhp, dlp, hi_cap, lo_cap, ws, st);
    }
}

size_t wgrad_ws_bytes(int dtype, int layout, const Geo& g, int C_in, int C_out, int hi_cap, int lo_cap, bool bias) {
    // a misaligned call of the MFMA kernel's shapes takes the vector-ALU kernel
    const size_t v = wgrad_plan(g, C_in, C_out, hi_cap, lo_cap, bias, false).total;
    if (!wgrad_mfma_fits(dtype, layout, g, C_in, C_out, hi_cap, lo_cap)) return v;
    return std::max(v, wgrad_plan(g, C_in, C_out, hi_cap, lo_cap, bias, true).total);
}

hipError_t launch_wgrad(int dtype, int layout, const Geo& g, const void* hp, const void* lp, const void* dho,
                        const void* dlo, const uint8_t* mask, int C_in, int C_out, void* dw, void* db, int hi_cap,
                        int lo_cap, Ws ws, hipStream_t st) {
    if (layout == NHWC) {
        switch (dtype) {
        case 0: return wgrad_t<float, NHWC>(g, hp, lp, dho, dlo, mask, C_in, C_out, dw, db, hi_cap, lo_cap, ws, st);
        case 1: return wgrad_t<f16, NHWC>(g, hp, lp, dho, dlo, mask, C_in, C_out, dw, db, hi_cap, lo_cap, ws, st);
        default: return wgrad_t<bf16, NHWC>(g, hp, lp, dho, dlo, mask, C_in, C_out, dw, db, hi_cap, lo_cap, ws, st);
        }
    }
    switch (dtype) {
    case 0: return wgrad_t<float, NCHW>(g, hp, lp, dho, dlo, mask, C_in, C_out, dw, db, hi_cap, lo_cap, ws, st);
    case 1: return wgrad_t<f16, NCHW>(g, hp, lp, dho, dlo, mask, C_in, C_out, dw, db, hi_cap, lo_cap, ws, st);
    default: return wgrad_t<bf16, NCHW>(g, hp, lp, dho, dlo, mask, C_in, C_out, dw, db, hi_cap, lo_cap, ws, st);
    }
}

}  // namespace sb
