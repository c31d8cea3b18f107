// BlockSample (split), BlockPad (pad) and BlockCombine (combine) as
// gather/scatter kernels for gfx950.
//
// Work decomposition: one workgroup per (block k, group of rows of that
// block); block k's resolution comes from its mask byte and its slot from a
// wavefront count of the high blocks before it.  Every thread moves one
// vector of V elements per item (16 bytes in the channels-last layout, along
// the channel axis), so a wave covers 1 KiB of contiguous memory per access.
#include "sb_common.h"
#include "sb_kernels.h"
#include "sb_pixel.h"

namespace sb {

namespace {

__device__ __forceinline__ void block_coords(long long k, int GH, int GW, int& n, int& gy, int& gx) {
    const long long per = (long long)GH * GW;
    n = (int)(k / per);
    const int rem = (int)(k - (long long)n * per);
    gy = rem / GW;
    gx = rem - gy * GW;
}

// slot of block k within its class (uniform across the wave)
__device__ __forceinline__ int block_slot(const uint8_t* __restrict__ mask, long long k, bool high) {
    long long t[1] = {k};
    int c[1];
    wave_count_high<1>(mask, k + 1, t, c);
    return high ? c[0] : (int)(k - c[0]);
}

// Picks element `idx` of the concatenation of two vectors.
template <typename T, int V>
__device__ __forceinline__ T pick2(const Vec<T, V>& a, const Vec<T, V>& b, int idx) {
    return idx < V ? a.e[idx] : b.e[idx - V];
}

// ---------------------------------------------------------------------------
// split: x[N,C,H,W] -> hi[nh,C,bs,bs], lo[nl,C,lb,lb]
// R = high rows per workgroup (even); a low block's workgroup produces R/2
// low rows from the same R input rows.
// ---------------------------------------------------------------------------
template <typename T, int L, int V>
__global__ __launch_bounds__(WG) void k_split(const T* __restrict__ x, int C, int H, int W,
                                              const uint8_t* __restrict__ mask, int bs, int R, int groups,
                                              T* __restrict__ hi, int hi_cap, T* __restrict__ lo, int lo_cap) {
    const int GH = H / bs, GW = W / bs, lb = bs >> 1;
    const long long k = blockIdx.x / groups;
    const int g = (int)(blockIdx.x - k * groups);
    int n, gy, gx;
    block_coords(k, GH, GW, n, gy, gx);
    const bool high = mask[k] != 0;
    const int slot = block_slot(mask, k, high);
    if (slot >= (high ? hi_cap : lo_cap)) return;
    const int tid = threadIdx.x;
    if (high) {
        const int r0 = g * R, r1 = min(bs, r0 + R);
        if (r0 >= r1) return;
        if constexpr (L == NHWC) {
            const int rowv = bs * C / V;
            const int items = (r1 - r0) * rowv;
            for (int it = tid; it < items; it += WG) {
                const int r = r0 + it / rowv, o = (it % rowv) * V;
                const T* src = x + ((size_t)((long long)n * H + gy * bs + r) * W + (size_t)gx * bs) * C + o;
                T* dst = hi + ((size_t)slot * bs + r) * (size_t)bs * C + o;
                vstore<T, V>(dst, vload<T, V>(src));
            }
        } else {
            const int rowv = bs / V, per_c = (r1 - r0) * rowv;
            const int items = C * per_c;
            for (int it = tid; it < items; it += WG) {
                const int c = it / per_c, q = it - c * per_c;
                const int r = r0 + q / rowv, j = (q % rowv) * V;
                const T* src = x + (((size_t)n * C + c) * H + gy * bs + r) * (size_t)W + (size_t)gx * bs + j;
                T* dst = hi + (((size_t)slot * C + c) * bs + r) * (size_t)bs + j;
                vstore<T, V>(dst, vload<T, V>(src));
            }
        }
    } else {
        const int r0 = (g * R) >> 1, r1 = min(lb, (g * R + R) >> 1);
        if (r0 >= r1) return;
        if constexpr (L == NHWC) {
            const int cv = C / V, rowv = lb * cv;
            const int items = (r1 - r0) * rowv;
            for (int it = tid; it < items; it += WG) {
                const int r = r0 + it / rowv, q = it % rowv;
                const int j = q / cv, c = (q % cv) * V;
                const T* p = x + ((size_t)((long long)n * H + gy * bs + 2 * r) * W + (size_t)gx * bs + 2 * j) * C + c;
                const size_t down = (size_t)W * C;
                const Vec<T, V> a = vload<T, V>(p), b = vload<T, V>(p + C);
                const Vec<T, V> cc = vload<T, V>(p + down), d = vload<T, V>(p + down + C);
                vstore<T, V>(lo + (((size_t)slot * lb + r) * lb + j) * C + c, vavg4<T, V>(a, b, cc, d));
            }
        } else {
            const int rowv = lb / V, per_c = (r1 - r0) * rowv;
            const int items = C * per_c;
            for (int it = tid; it < items; it += WG) {
                const int c = it / per_c, q = it - c * per_c;
                const int r = r0 + q / rowv, j = (q % rowv) * V;
                const T* p = x + (((size_t)n * C + c) * H + gy * bs + 2 * r) * (size_t)W + (size_t)gx * bs + 2 * j;
                const Vec<T, V> t0 = vload<T, V>(p), t1 = vload<T, V>(p + V);
                const Vec<T, V> b0 = vload<T, V>(p + W), b1 = vload<T, V>(p + W + V);
                Vec<T, V> o;
#pragma unroll
                for (int e = 0; e < V; ++e)
                    o.e[e] = avg4(pick2(t0, t1, 2 * e), pick2(t0, t1, 2 * e + 1),
                                  pick2(b0, b1, 2 * e), pick2(b0, b1, 2 * e + 1));
                vstore<T, V>(lo + (((size_t)slot * C + c) * lb + r) * (size_t)lb + j, o);
            }
        }
    }
}

// ---------------------------------------------------------------------------
// pad: hi, lo -> hp[nh,C,bs+2,bs+2], lp[nl,C,lb+2,lb+2]
// R = padded rows per workgroup.
// ---------------------------------------------------------------------------
template <typename T, int L, int V>
__global__ __launch_bounds__(WG) void k_pad(const T* __restrict__ hi, const T* __restrict__ lo, int C, int H, int W,
                                            const uint8_t* __restrict__ mask, int bs, int R, int groups,
                                            T* __restrict__ hp, T* __restrict__ lp, int hi_cap, int lo_cap) {
    __shared__ Neigh s_nb;
    const int GH = H / bs, GW = W / bs, lb = bs >> 1;
    const long long k = blockIdx.x / groups;
    const int g = (int)(blockIdx.x - k * groups);
    int n, gy, gx;
    block_coords(k, GH, GW, n, gy, gx);
    if (threadIdx.x < 64) block_neighbourhood<true>(mask, GH, GW, n, gy, gx, &s_nb);
    __syncthreads();
    const bool high = (s_nb.high >> 4) & 1;
    const int slot = s_nb.slot[4];
    if (slot >= (high ? hi_cap : lo_cap)) return;
    const int e = high ? bs : lb, pe = e + 2;
    const int r0 = g * R, r1 = min(pe, r0 + R);
    if (r0 >= r1) return;
    T* out = high ? hp : lp;
    const int tid = threadIdx.x;
    if constexpr (L == NHWC) {
        const int cv = C / V, rowv = pe * cv;
        const int items = (r1 - r0) * rowv;
        for (int it = tid; it < items; it += WG) {
            const int u = r0 + it / rowv, q = it % rowv;
            const int v = q / cv, c = (q % cv) * V;
            const Vec<T, V> val = packed_pixel<T, L, V>(hi, lo, C, bs, s_nb, hi_cap, lo_cap, u - 1, v - 1, c);
            vstore<T, V>(out + (((size_t)slot * pe + u) * pe + v) * C + c, val);
        }
    } else {
        static_assert(L == NHWC || V == 1, "NCHW pad is scalar");
        const int per_c = (r1 - r0) * pe;
        const int items = C * per_c;
        for (int it = tid; it < items; it += WG) {
            const int c = it / per_c, q = it - c * per_c;
            const int u = r0 + q / pe, v = q % pe;
            const Vec<T, 1> val = packed_pixel<T, L, 1>(hi, lo, C, bs, s_nb, hi_cap, lo_cap, u - 1, v - 1, c);
            vstore<T, 1>(out + (((size_t)slot * C + c) * pe + u) * pe + v, val);
        }
    }
}

// ---------------------------------------------------------------------------
// combine: hi, lo -> y[N,C,H,W]
// R = output rows per workgroup.
// ---------------------------------------------------------------------------
template <typename T, int L, int V>
__global__ __launch_bounds__(WG) void k_combine(const T* __restrict__ hi, const T* __restrict__ lo, int C, int H,
                                                int W, const uint8_t* __restrict__ mask, int bs, int R, int groups,
                                                int hi_cap, int lo_cap, T* __restrict__ y) {
    const int GH = H / bs, GW = W / bs, lb = bs >> 1;
    const long long k = blockIdx.x / groups;
    const int g = (int)(blockIdx.x - k * groups);
    int n, gy, gx;
    block_coords(k, GH, GW, n, gy, gx);
    const bool high = mask[k] != 0;
    const int slot = block_slot(mask, k, high);
    const bool skip = slot >= (high ? hi_cap : lo_cap);
    const int r0 = g * R, r1 = min(bs, r0 + R);
    if (r0 >= r1) return;
    const int tid = threadIdx.x;
    if constexpr (L == NHWC) {
        const int cv = C / V, rowv = bs * cv;
        const int items = (r1 - r0) * rowv;
        for (int it = tid; it < items; it += WG) {
            const int i = r0 + it / rowv, q = it % rowv;
            const int j = q / cv, c = (q % cv) * V;
            Vec<T, V> val;
            if (skip)      val = vzero<T, V>();
            else if (high) val = vload<T, V>(hi + (((size_t)slot * bs + i) * bs + j) * C + c);
            else           val = vload<T, V>(lo + (((size_t)slot * lb + (i >> 1)) * lb + (j >> 1)) * C + c);
            vstore<T, V>(y + ((size_t)((long long)n * H + gy * bs + i) * W + (size_t)gx * bs + j) * C + c, val);
        }
    } else {
        const int rowv = bs / V, per_c = (r1 - r0) * rowv;
        const int items = C * per_c;
        for (int it = tid; it < items; it += WG) {
            const int c = it / per_c, q = it - c * per_c;
            const int i = r0 + q / rowv, j = (q % rowv) * V;
            Vec<T, V> val;
            if (skip) {
                val = vzero<T, V>();
            } else if (high) {
                val = vload<T, V>(hi + (((size_t)slot * C + c) * bs + i) * (size_t)bs + j);
            } else {
                const T* src = lo + (((size_t)slot * C + c) * lb + (i >> 1)) * (size_t)lb + (j >> 1);
                if constexpr (V == 1) {
                    val = vload<T, 1>(src);
                } else {
                    const Vec<T, V / 2> h = vload<T, V / 2>(src);
#pragma unroll
                    for (int e = 0; e < V; ++e) val.e[e] = h.e[e >> 1];
                }
            }
            vstore<T, V>(y + (((size_t)n * C + c) * H + gy * bs + i) * (size_t)W + (size_t)gx * bs + j, val);
        }
    }
}

// ---------------------------------------------------------------------------
// host-side launch helpers
// ---------------------------------------------------------------------------
constexpr int kTargetBytes = 32768;  // bytes moved per workgroup (approx.)

inline int clampi(int v, int lo, int hi) { return v < lo ? lo : (v > hi ? hi : v); }

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

template <typename T, int L, int V>
hipError_t run_split(const Geo& g, const void* x, const uint8_t* mask, void* hi, int hi_cap, void* lo,
                     int lo_cap, hipStream_t st) {
    const int row_bytes = g.bs * g.C * (int)sizeof(T);
    int R = clampi(kTargetBytes / (row_bytes > 0 ? row_bytes : 1), 2, g.bs) & ~1;
    const int groups = (g.bs + R - 1) / R;
    const long long blocks = g.B * groups;
    hipLaunchKernelGGL((k_split<T, L, V>), dim3((unsigned)blocks), dim3(WG), 0, st, (const T*)x, g.C, g.H, g.W,
                       mask, g.bs, R, groups, (T*)hi, hi_cap, (T*)lo, lo_cap);
    return hipGetLastError();
}

template <typename T, int L, int V>
hipError_t run_pad(const Geo& g, const void* hi, const void* lo, const uint8_t* mask, void* hp, void* lp,
                   int hi_cap, int lo_cap, hipStream_t st) {
    const int pe = g.bs + 2;
    const int row_bytes = pe * g.C * (int)sizeof(T);
    const int R = clampi(kTargetBytes / (row_bytes > 0 ? row_bytes : 1), 1, pe);
    const int groups = (pe + R - 1) / R;
    const long long blocks = g.B * groups;
    hipLaunchKernelGGL((k_pad<T, L, V>), dim3((unsigned)blocks), dim3(WG), 0, st, (const T*)hi, (const T*)lo, g.C,
                       g.H, g.W, mask, g.bs, R, groups, (T*)hp, (T*)lp, hi_cap, lo_cap);
    return hipGetLastError();
}

template <typename T, int L, int V>
hipError_t run_combine(const Geo& g, const void* hi, const void* lo, const uint8_t* mask, int hi_cap, int lo_cap,
                       void* y, hipStream_t st) {
    const int row_bytes = g.bs * g.C * (int)sizeof(T);
    const int R = clampi(kTargetBytes / (row_bytes > 0 ? row_bytes : 1), 1, g.bs);
    const int groups = (g.bs + R - 1) / R;
    const long long blocks = g.B * groups;
    hipLaunchKernelGGL((k_combine<T, L, V>), dim3((unsigned)blocks), dim3(WG), 0, st, (const T*)hi, (const T*)lo,
                       g.C, g.H, g.W, mask, g.bs, R, groups, hi_cap, lo_cap, (T*)y);
    return hipGetLastError();
}

template <typename T>
hipError_t split_t(int layout, const Geo& g, const void* x, const uint8_t* mask, void* hi, int hi_cap, void* lo,
                   int lo_cap, hipStream_t st) {
    constexpr int VM = 16 / (int)sizeof(T);
    const bool al = aligned16(x) && aligned16(hi) && aligned16(lo);
    if (layout == NHWC) {
        if (al && g.C % VM == 0) return run_split<T, NHWC, VM>(g, x, mask, hi, hi_cap, lo, lo_cap, st);
        return run_split<T, NHWC, 1>(g, x, mask, hi, hi_cap, lo, lo_cap, st);
    }
    if (al && (g.bs / 2) % VM == 0) return run_split<T, NCHW, VM>(g, x, mask, hi, hi_cap, lo, lo_cap, st);
    return run_split<T, NCHW, 1>(g, x, mask, hi, hi_cap, lo, lo_cap, st);
}

template <typename T>
hipError_t pad_t(int layout, const Geo& g, const void* hi, const void* lo, const uint8_t* mask, void* hp, void* lp,
                 int hi_cap, int lo_cap, hipStream_t st) {
    constexpr int VM = 16 / (int)sizeof(T);
    const bool al = aligned16(hi) && aligned16(lo) && aligned16(hp) && aligned16(lp);
    if (layout == NHWC) {
        if (al && g.C % VM == 0) return run_pad<T, NHWC, VM>(g, hi, lo, mask, hp, lp, hi_cap, lo_cap, st);
        return run_pad<T, NHWC, 1>(g, hi, lo, mask, hp, lp, hi_cap, lo_cap, st);
    }
    return run_pad<T, NCHW, 1>(g, hi, lo, mask, hp, lp, hi_cap, lo_cap, st);
}

template <typename T>
hipError_t combine_t(int layout, const Geo& g, const void* hi, const void* lo, const uint8_t* mask, int hi_cap,
                     int lo_cap, void* y, hipStream_t st) {
    constexpr int VM = 16 / (int)sizeof(T);
    const bool al = aligned16(hi) && aligned16(lo) && aligned16(y);
    if (layout == NHWC) {
        if (al && g.C % VM == 0) return run_combine<T, NHWC, VM>(g, hi, lo, mask, hi_cap, lo_cap, y, st);
        return run_combine<T, NHWC, 1>(g, hi, lo, mask, hi_cap, lo_cap, y, st);
    }
    if (al && g.bs % VM == 0) return run_combine<T, NCHW, VM>(g, hi, lo, mask, hi_cap, lo_cap, y, st);
    return run_combine<T, NCHW, 1>(g, hi, lo, mask, hi_cap, lo_cap, y, st);
}

}  // namespace

hipError_t launch_split(int dtype, int layout, const Geo& g, const void* x, const uint8_t* mask, void* hi,
                        int hi_cap, void* lo, int lo_cap, hipStream_t st) {
    switch (dtype) {
    case 0: return split_t<float>(layout, g, x, mask, hi, hi_cap, lo, lo_cap, st);
    case 1: return split_t<f16>(layout, g, x, mask, hi, hi_cap, lo, lo_cap, st);
    default: return split_t<bf16>(layout, g, x, mask, hi, hi_cap, lo, lo_cap, st);
    }
}

hipError_t launch_pad(int dtype, int layout, const Geo& g, const void* hi, const void* lo, const uint8_t* mask,
                      void* hp, void* lp, int hi_cap, int lo_cap, hipStream_t st) {
    switch (dtype) {
    case 0: return pad_t<float>(layout, g, hi, lo, mask, hp, lp, hi_cap, lo_cap, st);
    case 1: return pad_t<f16>(layout, g, hi, lo, mask, hp, lp, hi_cap, lo_cap, st);
    default: return pad_t<bf16>(layout, g, hi, lo, mask, hp, lp, hi_cap, lo_cap, st);
    }
}

hipError_t launch_combine(int dtype, int layout, const Geo& g, const void* hi, const void* lo, const uint8_t* mask,
                          int hi_cap, int lo_cap, void* y, hipStream_t st) {
    switch (dtype) {
    case 0: return combine_t<float>(layout, g, hi, lo, mask, hi_cap, lo_cap, y, st);
    case 1: return combine_t<f16>(layout, g, hi, lo, mask, hi_cap, lo_cap, y, st);
    default: return combine_t<bf16>(layout, g, hi, lo, mask, hi_cap, lo_cap, y, st);
    }
}

}  // namespace sb
