// BlockSample (split), BlockPad (pad) and BlockCombine (combine) as
// gather/scatter kernels for gfx950.
//
// Work decomposition: every workgroup writes one piece of 256 output vectors
// (4 KiB for 16-byte vectors) of one block, one vector per thread, so that a
// launch has thousands of small workgroups and the memory system always has
// both loads and stores of many workgroups in flight.  (Fewer, larger
// workgroups whose threads first load several vectors and then store them
// measured about half the bandwidth on MI355X.)
//
//   split   : grid over the output stacks: (class, slot, piece); the block
//             of a slot is found from the mask by a wavefront scan.
//   pad     : grid over the padded stacks: (class, slot, piece), plus the
//             slots of the 8 neighbours.
//   combine : grid over the dense output: (block, piece); the block's slot
//             comes from a wavefront count of the mask prefix.
//
// Every wave computes the plan it needs by itself (no LDS, no barrier).
// Items are numbered in the memory order of the output, so consecutive
// threads write consecutive vectors: along the channels for channels-last
// (NHWC) tensors, along the rows for NCHW tensors.
#include "sb_common.h"
#include "sb_kernels.h"
#include "sb_pixel.h"

namespace sb {

namespace {

constexpr int PIECE = WG;  // output vectors per workgroup

__device__ __forceinline__ void block_coords(int k, int GH, int GW, int& n, int& gy, int& gx) {
    const int per = GH * GW;
    n = k / per;
    const int rem = k - n * per;
    gy = rem / GW;
    gx = rem - gy * GW;
}

// Picks element `idx` of the concatenation of two vectors.
template <typename T, int V>
__device__ __forceinline__ T pick2(const Vec<T, V>& a, const Vec<T, V>& b, int idx) {
    return idx < V ? a.e[idx] : b.e[idx - V];
}

// Coordinates of output vector `it` of a block of extent e with C channels,
// items in memory order: NHWC (r, j, c0) with V channels, NCHW (c, r, j0)
// with V pixels along the row.
template <int L, int V>
__device__ __forceinline__ void item_coords(int it, int e, int C, int& r, int& j, int& c) {
    if constexpr (L == NHWC) {
        const int cv = C / V;
        const int pix = it / cv;
        c = (it - pix * cv) * V;
        r = pix / e;
        j = pix - r * e;
    } else {
        const int rv = e / V;
        const int row = it / rv;
        j = (it - row * rv) * V;
        c = row / e;
        r = row - c * e;
    }
}

// Decodes a workgroup of a (class, slot, piece) grid: high slots first.
__device__ __forceinline__ bool slot_piece(int w, int hi_cap, int Gh, int Gl, bool& high, int& slot, int& piece) {
    if (w < hi_cap * Gh) {
        high = true;
        slot = w / Gh;
        piece = w - slot * Gh;
        return true;
    }
    w -= hi_cap * Gh;
    high = false;
    slot = w / Gl;
    piece = w - slot * Gl;
    return true;
}

// ---------------------------------------------------------------------------
// split: x[N,C,H,W] -> hi[nh,C,bs,bs], lo[nl,C,lb,lb]
// ---------------------------------------------------------------------------
// bwd != 0: BlockCombine transposed (a low block gets the sums of its cells)
template <typename T, int L, int V>
__global__ __launch_bounds__(WG) void k_split(const T* __restrict__ x, int C, int H, int W,
                                              const uint8_t* __restrict__ mask, int bs, int B, int Gh, int Gl,
                                              T* __restrict__ hi, int hi_cap, T* __restrict__ lo, int lo_cap,
                                              int bwd) {
    bool high;
    int slot, piece;
    slot_piece((int)blockIdx.x, hi_cap, Gh, Gl, high, slot, piece);
    WaveMask wm;
    wm.init(mask, B);
    const int k = wm.find_nth(slot, high);
    if (k < 0) return;
    const int GH = H / bs, GW = W / bs, lb = bs >> 1;
    int n, gy, gx;
    block_coords(k, GH, GW, n, gy, gx);
    const int e = high ? bs : lb;
    const int items = e * e * C / V;
    const int it = piece * PIECE + (int)threadIdx.x;
    if (it >= items) return;
    int r, j, c;
    item_coords<L, V>(it, e, C, r, j, c);
    T* dst = (high ? hi : lo) + (size_t)slot * C * e * e + (size_t)it * V;
    if (high) {
        vstore<T, V>(dst, vload<T, V>(map_at<T, L>(x, n, C, H, W, gy * bs + r, gx * bs + j, c)));
        return;
    }
    const int Y = gy * bs + 2 * r, X = gx * bs + 2 * j;
    if constexpr (L == NHWC) {
        const T* p = map_at<T, L>(x, n, C, H, W, Y, X, c);
        const size_t down = (size_t)W * C;
        const Vec<T, V> a = vload<T, V>(p), b = vload<T, V>(p + C), c2 = vload<T, V>(p + down),
                        d = vload<T, V>(p + down + C);
        vstore<T, V>(dst, bwd ? vsum4<T, V>(a, b, c2, d) : vavg4<T, V>(a, b, c2, d));
    } else {
        // V low pixels along the row come from 2V input pixels of two rows
        const T* p = map_at<T, L>(x, n, C, H, W, Y, X, c);
        const Vec<T, V> t0 = vload<T, V>(p), t1 = vload<T, V>(p + V);
        const Vec<T, V> b0 = vload<T, V>(p + W), b1 = vload<T, V>(p + W + V);
        Vec<T, V> o;
#pragma unroll
        for (int q = 0; q < V; ++q) {
            const T a = pick2(t0, t1, 2 * q), b = pick2(t0, t1, 2 * q + 1), c2 = pick2(b0, b1, 2 * q),
                    d = pick2(b0, b1, 2 * q + 1);
            o.e[q] = bwd ? from_f32<T>((to_f32(a) + to_f32(b)) + (to_f32(c2) + to_f32(d))) : avg4(a, b, c2, d);
        }
        vstore<T, V>(dst, o);
    }
}

// ---------------------------------------------------------------------------
// pad: hi, lo -> hp[nh,C,bs+2,bs+2], lp[nl,C,lb+2,lb+2]
// ---------------------------------------------------------------------------
template <typename T, int L, int V>
__global__ __launch_bounds__(WG) void k_pad(const T* __restrict__ hi, const T* __restrict__ lo, int C, int H, int W,
                                            const uint8_t* __restrict__ mask, int bs, int B, int Gh, int Gl,
                                            T* __restrict__ hp, T* __restrict__ lp, int hi_cap, int lo_cap, int pm,
                                            int halo) {
    bool high;
    int slot, piece;
    slot_piece((int)blockIdx.x, hi_cap, Gh, Gl, high, slot, piece);
    WaveMask wm;
    wm.init(mask, B);
    const int k = wm.find_nth(slot, high);
    if (k < 0) return;
    const int GH = H / bs, GW = W / bs, lb = bs >> 1;
    int n, gy, gx;
    block_coords(k, GH, GW, n, gy, gx);
    const int e = high ? bs : lb, pe = e + 2 * halo;
    const int items = pe * pe * C / V;
    const int it = piece * PIECE + (int)threadIdx.x;
    const Neigh nb = wave_neighbourhood<true>(wm, GH, GW, n, gy, gx);
    if (it >= items) return;
    int u, v, c;
    item_coords<L, V>(it, pe, C, u, v, c);
    T* dst = (high ? hp : lp) + (size_t)slot * C * pe * pe + (size_t)it * V;
    if constexpr (L == NHWC || V == 1) {
        const Src<T> s = packed_src<T, L>(hi, lo, C, bs, nb, hi_cap, lo_cap, u - halo, v - halo, c, pm);
        SrcBatch<T, V, 1> b;
        b.issue(0, s);
        vstore<T, V>(dst, b.value(0));
    } else {
        static_assert(L == NHWC || V == 1, "NCHW pad moves single elements");
    }
}

// ---------------------------------------------------------------------------
// combine: hi, lo -> y[N,C,H,W]
// ---------------------------------------------------------------------------
template <typename T, int L, int V>
// bwd != 0: BlockSample transposed (a low value is spread as quarters)
__global__ __launch_bounds__(WG) void k_combine(const T* __restrict__ hi, const T* __restrict__ lo, int C, int H,
                                                int W, const uint8_t* __restrict__ mask, int bs, int B, int G,
                                                int hi_cap, int lo_cap, T* __restrict__ y, int bwd) {
    const int k = (int)blockIdx.x / G;
    const int piece = (int)blockIdx.x - k * G;
    const int GH = H / bs, GW = W / bs, lb = bs >> 1;
    int n, gy, gx;
    block_coords(k, GH, GW, n, gy, gx);
    WaveMask wm;
    wm.init(mask, B);
    const bool high = wm.high(k);
    const int slot = wm.slot(k, high);
    const bool skip = slot >= (high ? hi_cap : lo_cap);
    const int items = bs * bs * C / V;
    const int it = piece * PIECE + (int)threadIdx.x;
    if (it >= items) return;
    int r, j, c;
    item_coords<L, V>(it, bs, C, r, j, c);
    Vec<T, V> val;
    if (skip) {
        val = vzero<T, V>();
    } else if (high) {
        val = vload<T, V>(hi + (size_t)slot * C * bs * bs + (size_t)it * V);
    } else if constexpr (L == NHWC) {
        val = vload<T, V>(stack_at<T, L>(lo, slot, C, lb, r >> 1, j >> 1, c));
    } else if constexpr (V == 1) {
        val = vload<T, 1>(stack_at<T, L>(lo, slot, C, lb, r >> 1, j >> 1, c));
    } else {
        // V output pixels along the row repeat V/2 low pixels
        const Vec<T, V / 2> h = vload<T, V / 2>(stack_at<T, L>(lo, slot, C, lb, r >> 1, j >> 1, c));
#pragma unroll
        for (int q = 0; q < V; ++q) val.e[q] = h.e[q >> 1];
    }
    if (bwd && !high && !skip) val = vquarter<T, V>(val);
    T* dst;
    if constexpr (L == NHWC) dst = y + (((size_t)n * H + gy * bs + r) * W + (size_t)gx * bs + j) * C + c;
    else                     dst = y + (((size_t)n * C + c) * H + gy * bs + r) * (size_t)W + (size_t)gx * bs + j;
    vstore<T, V>(dst, val);
}

// ---------------------------------------------------------------------------
// host-side launch helpers
// ---------------------------------------------------------------------------
inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }
inline int pieces(long long vectors) { return (int)((vectors + PIECE - 1) / PIECE); }

template <typename T, int L, int V>
hipError_t run_split(const Geo& g, const void* x, const uint8_t* mask, void* hi, int hi_cap, void* lo,
                     int lo_cap, int bwd, hipStream_t st) {
    const int lb = g.bs / 2;
    const int Gh = pieces((long long)g.bs * g.bs * g.C / V), Gl = pieces((long long)lb * lb * g.C / V);
    const long long blocks = (long long)hi_cap * Gh + (long long)lo_cap * Gl;
    if (blocks == 0) return hipSuccess;
    hipLaunchKernelGGL((k_split<T, L, V>), dim3((unsigned)blocks), dim3(WG), 0, st, (const T*)x, g.C, g.H, g.W,
                       mask, g.bs, (int)g.B, Gh, Gl, (T*)hi, hi_cap, (T*)lo, lo_cap, bwd);
    return hipGetLastError();
}

template <typename T, int L, int V>
hipError_t run_pad(const Geo& g, const void* hi, const void* lo, const uint8_t* mask, void* hp, void* lp,
                   int hi_cap, int lo_cap, int pm, int halo, hipStream_t st) {
    const int ph = g.bs + 2 * halo, pl = g.bs / 2 + 2 * halo;
    const int Gh = pieces((long long)ph * ph * g.C / V), Gl = pieces((long long)pl * pl * g.C / V);
    const long long blocks = (long long)hi_cap * Gh + (long long)lo_cap * Gl;
    if (blocks == 0) return hipSuccess;
    hipLaunchKernelGGL((k_pad<T, L, V>), dim3((unsigned)blocks), dim3(WG), 0, st, (const T*)hi, (const T*)lo, g.C,
                       g.H, g.W, mask, g.bs, (int)g.B, Gh, Gl, (T*)hp, (T*)lp, hi_cap, lo_cap, pm, halo);
    return hipGetLastError();
}

template <typename T, int L, int V>
hipError_t run_combine(const Geo& g, const void* hi, const void* lo, const uint8_t* mask, int hi_cap, int lo_cap,
                       void* y, int bwd, hipStream_t st) {
    const int G = pieces((long long)g.bs * g.bs * g.C / V);
    const long long blocks = g.B * G;
    hipLaunchKernelGGL((k_combine<T, L, V>), dim3((unsigned)blocks), dim3(WG), 0, st, (const T*)hi, (const T*)lo,
                       g.C, g.H, g.W, mask, g.bs, (int)g.B, G, hi_cap, lo_cap, (T*)y, bwd);
    return hipGetLastError();
}

template <typename T>
hipError_t split_t(int layout, const Geo& g, const void* x, const uint8_t* mask, void* hi, int hi_cap, void* lo,
                   int lo_cap, int bwd, hipStream_t st) {
    constexpr int VM = 16 / (int)sizeof(T);
    const bool al = aligned16(x) && aligned16(hi) && aligned16(lo);
    if (layout == NHWC) {
        if (al && g.C % VM == 0) return run_split<T, NHWC, VM>(g, x, mask, hi, hi_cap, lo, lo_cap, bwd, st);
        return run_split<T, NHWC, 1>(g, x, mask, hi, hi_cap, lo, lo_cap, bwd, st);
    }
    if (al && (g.bs / 2) % VM == 0) return run_split<T, NCHW, VM>(g, x, mask, hi, hi_cap, lo, lo_cap, bwd, st);
    return run_split<T, NCHW, 1>(g, x, mask, hi, hi_cap, lo, lo_cap, bwd, st);
}

template <typename T>
hipError_t pad_t(int layout, const Geo& g, const void* hi, const void* lo, const uint8_t* mask, void* hp, void* lp,
                 int hi_cap, int lo_cap, int pm, int halo, hipStream_t st) {
    constexpr int VM = 16 / (int)sizeof(T);
    const bool al = aligned16(hi) && aligned16(lo) && aligned16(hp) && aligned16(lp);
    if (layout == NHWC) {
        if (al && g.C % VM == 0) return run_pad<T, NHWC, VM>(g, hi, lo, mask, hp, lp, hi_cap, lo_cap, pm, halo, st);
        return run_pad<T, NHWC, 1>(g, hi, lo, mask, hp, lp, hi_cap, lo_cap, pm, halo, st);
    }
    return run_pad<T, NCHW, 1>(g, hi, lo, mask, hp, lp, hi_cap, lo_cap, pm, halo, st);
}

template <typename T>
hipError_t combine_t(int layout, const Geo& g, const void* hi, const void* lo, const uint8_t* mask, int hi_cap,
                     int lo_cap, void* y, int bwd, hipStream_t st) {
    constexpr int VM = 16 / (int)sizeof(T);
    const bool al = aligned16(hi) && aligned16(lo) && aligned16(y);
    if (layout == NHWC) {
        if (al && g.C % VM == 0) return run_combine<T, NHWC, VM>(g, hi, lo, mask, hi_cap, lo_cap, y, bwd, st);
        return run_combine<T, NHWC, 1>(g, hi, lo, mask, hi_cap, lo_cap, y, bwd, st);
    }
    if (al && g.bs % VM == 0) return run_combine<T, NCHW, VM>(g, hi, lo, mask, hi_cap, lo_cap, y, bwd, st);
    return run_combine<T, NCHW, 1>(g, hi, lo, mask, hi_cap, lo_cap, y, bwd, st);
}

}  // namespace

hipError_t launch_split(int dtype, int layout, const Geo& g, const void* x, const uint8_t* mask, void* hi,
                        int hi_cap, void* lo, int lo_cap, hipStream_t st, bool bwd) {
    if (rows_fit(dtype, layout, g, {x, hi, lo}))
        return launch_split_rows(dtype, g, x, mask, hi, hi_cap, lo, lo_cap, st, bwd);
    switch (dtype) {
    case 0: return split_t<float>(layout, g, x, mask, hi, hi_cap, lo, lo_cap, bwd, st);
    case 1: return split_t<f16>(layout, g, x, mask, hi, hi_cap, lo, lo_cap, bwd, st);
    default: return split_t<bf16>(layout, g, x, mask, hi, hi_cap, lo, lo_cap, bwd, st);
    }
}

hipError_t launch_pad(int dtype, int layout, const Geo& g, const void* hi, const void* lo, const uint8_t* mask,
                      void* hp, void* lp, int hi_cap, int lo_cap, int pm, hipStream_t st, int halo) {
    if (halo == 1 && rows_fit(dtype, layout, g, {hi, lo, hp, lp}))
        return launch_pad_rows(dtype, g, hi, lo, mask, hp, lp, hi_cap, lo_cap, pm, st);
    switch (dtype) {
    case 0: return pad_t<float>(layout, g, hi, lo, mask, hp, lp, hi_cap, lo_cap, pm, halo, st);
    case 1: return pad_t<f16>(layout, g, hi, lo, mask, hp, lp, hi_cap, lo_cap, pm, halo, st);
    default: return pad_t<bf16>(layout, g, hi, lo, mask, hp, lp, hi_cap, lo_cap, pm, halo, st);
    }
}

hipError_t launch_combine(int dtype, int layout, const Geo& g, const void* hi, const void* lo, const uint8_t* mask,
                          int hi_cap, int lo_cap, void* y, hipStream_t st, bool bwd) {
    if (rows_fit(dtype, layout, g, {hi, lo, y}))
        return launch_combine_rows(dtype, g, hi, lo, mask, hi_cap, lo_cap, y, st, bwd);
    switch (dtype) {
    case 0: return combine_t<float>(layout, g, hi, lo, mask, hi_cap, lo_cap, y, bwd, st);
    case 1: return combine_t<f16>(layout, g, hi, lo, mask, hi_cap, lo_cap, y, bwd, st);
    default: return combine_t<bf16>(layout, g, hi, lo, mask, hi_cap, lo_cap, y, bwd, st);
    }
}

}  // namespace sb
