// BlockSample (split), BlockPad (pad) and BlockCombine (combine) for
// channels-last tensors whose pixels are whole 16-byte vectors (C * sizeof(T)
// a multiple of 16, 16-byte aligned buffers): row jobs on persistent waves.
//
// One wave of each workgroup copies the mask to LDS and builds the block plan
// there as a table (class and slot of every block, for up to 1024 blocks);
// every wave then looks blocks up in it (plain LDS reads, no chains of
// cross-lane reads on the CU's scalar unit) and walks jobs; a job moves whole
// rows, so every access of a wave is a run of full 128-byte lines:
//
//   split   : job (block, row pair p): dense rows 2p, 2p + 1 of the block.
//             Their addresses do not depend on the mask, so the loads are
//             issued before the plan is known; a high block stores both rows
//             to its slot, a low block stores the 2x2 averages as low row p.
//   combine : job (block, row pair p): dense rows 2p, 2p + 1 of the block,
//             from high rows 2p, 2p + 1 or low row p (each pixel twice in
//             both directions).
//   pad     : job (block, padded row u), u < e + 2; a wave takes a run of
//             consecutive jobs, so the block's neighbourhood is computed once
//             per block.  Interior and halo pixels follow BlockPad exactly as
//             the general kernels do (packed_src).
//
// A lane owns the vectors lane, lane + 64, ... of its job; with 8 vectors per
// pixel (64 channels of 16 bits) eight lanes cover one pixel, so each
// instruction moves eight whole pixels.
#include "sb_common.h"
#include "sb_kernels.h"
#include "sb_pixel.h"

namespace sb {

namespace {

constexpr int RW_WAVES = WG / 64;  // waves per workgroup

__device__ __forceinline__ void coords(int k, int GH, int GW, int& n, int& gy, int& gx) {
    const int per = GH * GW;
    n = k / per;
    const int rem = k - n * per;
    gy = rem / GW;
    gx = rem - gy * GW;
}

template <typename T>
__device__ __forceinline__ uint4 avg_raw(uint4 a, uint4 b, uint4 c, uint4 d) {
    constexpr int V = 16 / (int)sizeof(T);
    Vec<T, V> va, vb, vc, vd;
    va.raw = a;
    vb.raw = b;
    vc.raw = c;
    vd.raw = d;
    return vavg4<T, V>(va, vb, vc, vd).raw;
}

template <typename T>
__device__ __forceinline__ uint4 sum_raw(uint4 a, uint4 b, uint4 c, uint4 d) {
    constexpr int V = 16 / (int)sizeof(T);
    Vec<T, V> va, vb, vc, vd;
    va.raw = a;
    vb.raw = b;
    vc.raw = c;
    vd.raw = d;
    return vsum4<T, V>(va, vb, vc, vd).raw;
}

template <typename T>
__device__ __forceinline__ uint4 quarter_raw(uint4 a) {
    constexpr int V = 16 / (int)sizeof(T);
    Vec<T, V> va;
    va.raw = a;
    return vquarter<T, V>(va).raw;
}

__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6)); }

// The block plan of a workgroup: the LDS table for masks of up to 1024
// blocks, else the wave-level plan over the staged first 1024 bytes and the
// global mask beyond them.
template <bool ONE>
struct RPlan {
    const PlanTable* pt;
    WaveMaskT<ONE> wm;
    __device__ __forceinline__ void init(const uint8_t* mask, int B, const uint8_t* s_mask, const PlanTable* t) {
        pt = t;
        if constexpr (!ONE) wm.init_staged(mask, B, s_mask);
    }
    __device__ __forceinline__ bool high(int k) const {
        if constexpr (ONE) return table_high(pt, k);
        else return wm.high(k);
    }
    __device__ __forceinline__ int slot(int k, bool h) const {
        if constexpr (ONE) return table_slot(pt, k);
        else return wm.slot(k, h);
    }
    __device__ __forceinline__ Neigh neigh(int GH, int GW, int n, int gy, int gx) const {
        if constexpr (ONE) return table_neighbourhood(pt, GH, GW, n, gy, gx);
        else return wave_neighbourhood<true>(wm, GH, GW, n, gy, gx);
    }
};

// Every kernel starts here: wave 0 copies the mask to LDS (and builds the
// table), the workgroup synchronises.
#define ROWS_PLAN_PREAMBLE()                                               \
    __shared__ __align__(16) uint8_t s_mask[1024];                        \
    __shared__ __align__(16) PlanTable s_pt;                              \
    if (wave_id() == 0) {                                                 \
        stage_mask(mask, B, s_mask);                                      \
        if (ONE) build_plan_table(s_mask, &s_pt);                         \
    }                                                                     \
    __syncthreads()

// Cells per lane and pass for split and combine: a cell is one 16-byte vector
// position (j, c) of a low row, i.e. a 2x2 group of dense vectors; a job takes
// as many passes of 64 * MAXM cells as its row pair has.
constexpr int MAXM = 4;

// ---------------------------------------------------------------------------
// split: x -> hi, lo
// ---------------------------------------------------------------------------
// BWD: the transpose of BlockCombine instead (a low block gets its cells' sums)
template <typename T, bool ONE, bool BWD>
__global__ __launch_bounds__(WG) void k_split_rows(const T* __restrict__ x, int C, int H, int W,
                                                   const uint8_t* __restrict__ mask, int bs, int B, int GH, int GW,
                                                   T* __restrict__ hi, int hi_cap, T* __restrict__ lo, int lo_cap) {
    constexpr int V = 16 / (int)sizeof(T);
    const int lane = lane_id();
    const int CV = C / V, lb = bs >> 1, cells = lb * CV;
    const int njobs = B * lb;
    const int nw = (int)gridDim.x * RW_WAVES;
    ROWS_PLAN_PREAMBLE();
    int job = (int)blockIdx.x * RW_WAVES + wave_id();
    if (job >= njobs) return;
    RPlan<ONE> wm;
    wm.init(mask, B, s_mask, &s_pt);
    for (; job < njobs; job += nw) {
        const int k = job / lb, p = job - k * lb;
        int n, gy, gx;
        coords(k, GH, GW, n, gy, gx);
        // the block's dense rows 2p and 2p + 1: cell (j, c) is pixels 2j, 2j + 1 of both
        const T* r0 = x + ((size_t)(n * H + gy * bs + 2 * p) * W + gx * bs) * C;
        const T* r1 = r0 + (size_t)W * C;
        bool high = false;
        int s = -1;
        for (int cb = 0; cb < cells; cb += 64 * MAXM) {
            uint4 v[MAXM][4];
#pragma unroll
            for (int m = 0; m < MAXM; ++m) {
                const int cell = cb + lane + 64 * m;
                if (cell < cells) {
                    const int j = cell / CV, c = (cell - j * CV) * V;
                    const int o = 2 * j * C + c;
                    v[m][0] = ld_nt16(r0 + o);
                    v[m][1] = ld_nt16(r0 + o + C);
                    v[m][2] = ld_nt16(r1 + o);
                    v[m][3] = ld_nt16(r1 + o + C);
                }
            }
            if (s < 0) {  // the plan, after the first loads are in flight
                high = wm.high(k);
                s = wm.slot(k, high);
            }
            if (s >= (high ? hi_cap : lo_cap)) break;
            if (high) {
                T* d0 = hi + ((size_t)(s * bs + 2 * p) * bs) * C;
                T* d1 = d0 + (size_t)bs * C;
#pragma unroll
                for (int m = 0; m < MAXM; ++m) {
                    const int cell = cb + lane + 64 * m;
                    if (cell < cells) {
                        const int j = cell / CV, c = (cell - j * CV) * V;
                        const int o = 2 * j * C + c;
                        st_nt16(d0 + o, v[m][0]);
                        st_nt16(d0 + o + C, v[m][1]);
                        st_nt16(d1 + o, v[m][2]);
                        st_nt16(d1 + o + C, v[m][3]);
                    }
                }
            } else {
                T* d = lo + ((size_t)(s * lb + p) * lb) * C;
#pragma unroll
                for (int m = 0; m < MAXM; ++m) {
                    const int cell = cb + lane + 64 * m;
                    if (cell < cells) {
                        const int j = cell / CV, c = (cell - j * CV) * V;
                        st_nt16(d + j * C + c, BWD ? sum_raw<T>(v[m][0], v[m][1], v[m][2], v[m][3])
                                                   : avg_raw<T>(v[m][0], v[m][1], v[m][2], v[m][3]));
                    }
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------
// low blocks of a dense map, sampled and padded in one pass: x -> lp
// ---------------------------------------------------------------------------
// Row u of the padded tile of low block (n, gy, gx) is the 2x2 average of
// the image cells at twice its coordinates, zero outside the image: that is
// BlockSample of the block and of its neighbours, and so, with average
// sampling, BlockPad of the low stack (a high neighbour's halo cell is the
// same average).  Maps whose sides are multiples of the block size (cells
// never straddle the border).  A job is (block, padded row); the jobs of
// high blocks end at the plan, before any load.
template <typename T, bool ONE>
__global__ __launch_bounds__(WG) void k_pad_low_dense(const T* __restrict__ x, int C, int H, int W,
                                                      const uint8_t* __restrict__ mask, int bs, int B, int GH, int GW,
                                                      T* __restrict__ lp, int lo_cap) {
    constexpr int V = 16 / (int)sizeof(T);
    const int lane = lane_id();
    const int CV = C / V, lb = bs >> 1, pe = lb + 2, cells = pe * CV;
    const int njobs = B * pe;
    const int nw = (int)gridDim.x * RW_WAVES;
    ROWS_PLAN_PREAMBLE();
    int job = (int)blockIdx.x * RW_WAVES + wave_id();
    if (job >= njobs) return;
    RPlan<ONE> wm;
    wm.init(mask, B, s_mask, &s_pt);
    for (; job < njobs; job += nw) {
        const int k = job / pe, u = job - k * pe;
        if (wm.high(k)) continue;
        const int s = wm.slot(k, false);
        if (s >= lo_cap) continue;
        int n, gy, gx;
        coords(k, GH, GW, n, gy, gx);
        const int Y = gy * bs + 2 * (u - 1);
        const bool yin = Y >= 0 && Y + 1 < H;
        const T* r0 = x + ((size_t)n * H + (yin ? Y : 0)) * W * C;
        const T* r1 = r0 + (size_t)W * C;
        T* d = lp + ((size_t)(s * pe + u) * pe) * C;
        for (int cb = 0; cb < cells; cb += 64 * MAXM) {
            uint4 v[MAXM][4];
            bool in[MAXM];
#pragma unroll
            for (int m = 0; m < MAXM; ++m) {
                const int cell = cb + lane + 64 * m;
                in[m] = false;
                if (cell < cells) {
                    const int j = cell / CV, c = (cell - j * CV) * V;
                    const int X = gx * bs + 2 * (j - 1);
                    if (yin && X >= 0 && X + 1 < W) {
                        const int o = X * C + c;
                        in[m] = true;
                        v[m][0] = ld_nt16(r0 + o);
                        v[m][1] = ld_nt16(r0 + o + C);
                        v[m][2] = ld_nt16(r1 + o);
                        v[m][3] = ld_nt16(r1 + o + C);
                    }
                }
            }
#pragma unroll
            for (int m = 0; m < MAXM; ++m) {
                const int cell = cb + lane + 64 * m;
                if (cell < cells) {
                    const int j = cell / CV, c = (cell - j * CV) * V;
                    st_nt16(d + j * C + c, in[m] ? avg_raw<T>(v[m][0], v[m][1], v[m][2], v[m][3])
                                                 : uint4{0u, 0u, 0u, 0u});
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------
// combine: hi, lo -> y (blocks past a stack's capacity are written as zeros)
// ---------------------------------------------------------------------------
// BWD: the transpose of BlockSample instead (a low value is spread as quarters)
template <typename T, bool ONE, bool BWD>
__global__ __launch_bounds__(WG) void k_combine_rows(const T* __restrict__ hi, const T* __restrict__ lo, int C,
                                                     int H, int W, const uint8_t* __restrict__ mask, int bs, int B,
                                                     int GH, int GW, int hi_cap, int lo_cap, T* __restrict__ y) {
    constexpr int V = 16 / (int)sizeof(T);
    const int lane = lane_id();
    const int CV = C / V, lb = bs >> 1, cells = lb * CV;
    const int njobs = B * lb;
    const int nw = (int)gridDim.x * RW_WAVES;
    ROWS_PLAN_PREAMBLE();
    int job = (int)blockIdx.x * RW_WAVES + wave_id();
    if (job >= njobs) return;
    RPlan<ONE> wm;
    wm.init(mask, B, s_mask, &s_pt);
    for (; job < njobs; job += nw) {
        const int k = job / lb, p = job - k * lb;
        int n, gy, gx;
        coords(k, GH, GW, n, gy, gx);
        const bool high = wm.high(k);
        const int s = wm.slot(k, high);
        const bool in = s < (high ? hi_cap : lo_cap);
        const T* s0 = high ? hi + ((size_t)(s * bs + 2 * p) * bs) * C : lo + ((size_t)(s * lb + p) * lb) * C;
        const T* s1 = s0 + (size_t)bs * C;
        T* d0 = y + ((size_t)(n * H + gy * bs + 2 * p) * W + gx * bs) * C;
        T* d1 = d0 + (size_t)W * C;
        for (int cb = 0; cb < cells; cb += 64 * MAXM) {
            uint4 v[MAXM][4];
#pragma unroll
            for (int m = 0; m < MAXM; ++m) {
                const int cell = cb + lane + 64 * m;
                if (cell < cells) {
                    const int j = cell / CV, c = (cell - j * CV) * V;
                    const int o = 2 * j * C + c;
                    if (!in) {
                        v[m][0] = v[m][1] = v[m][2] = v[m][3] = uint4{0u, 0u, 0u, 0u};
                    } else if (high) {
                        v[m][0] = ld_nt16(s0 + o);
                        v[m][1] = ld_nt16(s0 + o + C);
                        v[m][2] = ld_nt16(s1 + o);
                        v[m][3] = ld_nt16(s1 + o + C);
                    } else {
                        v[m][0] = ld_nt16(s0 + j * C + c);
                        if (BWD) v[m][0] = quarter_raw<T>(v[m][0]);
                        v[m][1] = v[m][2] = v[m][3] = v[m][0];
                    }
                }
            }
#pragma unroll
            for (int m = 0; m < MAXM; ++m) {
                const int cell = cb + lane + 64 * m;
                if (cell < cells) {
                    const int j = cell / CV, c = (cell - j * CV) * V;
                    const int o = 2 * j * C + c;
                    st_nt16(d0 + o, v[m][0]);
                    st_nt16(d0 + o + C, v[m][1]);
                    st_nt16(d1 + o, v[m][2]);
                    st_nt16(d1 + o + C, v[m][3]);
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------
// pad: hi, lo -> hp, lp
//
// A job is one padded row, done in one pass of loads then stores (a second
// pass would wait for the first pass's stores: one counter covers loads and
// stores).  Jobs [0, B (lb + 2)) are rows 0 .. lb + 1 of every block (all of
// a low padded block); the rest are rows lb + 2 .. bs + 1 of the high slots,
// whose blocks come from an inverse of the plan (LDS table) or a wave-level
// search, so no job is empty.
// ---------------------------------------------------------------------------
constexpr int PADM = 5;   // vectors per lane and pass (up to four loads each)

// Where the interior (columns 1..e) of padded row u of the block comes from:
// one row of one block (uniform) -- this block's row, or the row next to it in
// the block above or below -- copied at equal resolution (kind 1),
// nearest-upsampled from a low neighbour (2), 2x2-averaged from a high
// neighbour (3), or zero outside the image or past a stack's capacity (0).
// Only the two halo columns need the per-pixel rule (packed_src).
template <typename T>
__device__ __forceinline__ const T* pad_row_source(const T* __restrict__ hi, const T* __restrict__ lo, int C, int bs,
                                                   const Neigh& nb, bool high, int hi_cap, int lo_cap, int u,
                                                   int pm, int& kind) {
    const int lb = bs >> 1, e = high ? bs : lb;
    const int r = u - 1;
    const int dy = r < 0 ? 0 : (r >= e ? 2 : 1), dn = dy * 3 + 1;
    const int nhigh = (nb.high >> dn) & 1;
    const int ns = neigh_slot(nb, dn);
    kind = 0;
    if (!((nb.valid >> dn) & 1) || ns >= (nhigh ? hi_cap : lo_cap) || (pm == PM_ZERO && dy != 1)) return nullptr;
    const int u2 = r - (dy - 1) * e;
    if (nhigh == (int)high) {
        kind = 1;
        return (nhigh ? hi : lo) + ((size_t)(ns * e + u2) * e) * C;
    }
    if (high) {
        kind = 2;
        return lo + ((size_t)(ns * lb + (u2 >> 1)) * lb) * C;
    }
    kind = pm == PM_STRIDED ? 4 : 3;  // every other pixel of the even row, averaged with the next ones or not
    return hi + ((size_t)(ns * bs + 2 * u2) * bs) * C;
}

template <typename T, bool ONE>
__global__ __launch_bounds__(WG, 4) void k_pad_rows(const T* __restrict__ hi, const T* __restrict__ lo, int C,
                                                 const uint8_t* __restrict__ mask, int bs, int B, int GH, int GW,
                                                 int per_wave, T* __restrict__ hp, T* __restrict__ lp, int hi_cap,
                                                 int lo_cap, int pm) {
    constexpr int V = 16 / (int)sizeof(T);
    const int lane = lane_id();
    const int CV = C / V, lb = bs >> 1, ph = lb + 2, ex = bs - lb;
    const int jobs_a = B * ph;
    const int njobs = jobs_a + (hp ? hi_cap * ex : 0);  // no high output: the low blocks only
    __shared__ __align__(16) uint8_t s_mask[1024];
    __shared__ __align__(16) PlanTable s_pt;
    __shared__ uint16_t s_inv[1024];  // block of each high slot (one table)
    __shared__ int s_nh;
    if (wave_id() == 0) {
        stage_mask(mask, B, s_mask);
        if (ONE) {
            build_plan_table(s_mask, &s_pt);
            const int c = __popc(nonzero_bytes16(*reinterpret_cast<const uint4*>(s_mask + 16 * lane)));
            const int tot = wave_sum5(c);
            if (lane == 0) s_nh = tot;
        }
    }
    __syncthreads();
    if (ONE) {
        for (int k = (int)threadIdx.x; k < B; k += WG)
            if ((s_pt.hi[k >> 4] >> (k & 15)) & 1) s_inv[s_pt.slot[k]] = (uint16_t)k;
        __syncthreads();
    }
    int job = ((int)blockIdx.x * RW_WAVES + wave_id()) * per_wave;
    const int end = min(njobs, job + per_wave);
    if (job >= end) return;
    RPlan<ONE> wm;
    wm.init(mask, B, s_mask, &s_pt);
    int kcur = -1;
    Neigh nb;
    bool high = false;
    int s = 0;
    for (; job < end; ++job) {
        int k, u;
        if (job < jobs_a) {
            k = job / ph;
            u = job - k * ph;
        } else {
            const int j = job - jobs_a;
            const int hs = j / ex;
            u = ph + (j - hs * ex);
            if (ONE) {
                if (hs >= s_nh) continue;
                k = s_inv[hs];
            } else {
                k = wm.wm.find_nth(hs, true);
                if (k < 0) continue;
            }
        }
        if (k != kcur) {
            int n, gy, gx;
            coords(k, GH, GW, n, gy, gx);
            nb = wm.neigh(GH, GW, n, gy, gx);
            high = (nb.high >> 4) & 1;
            s = nb.slot[4];
            kcur = k;
        }
        if (s >= (high ? hi_cap : lo_cap) || (high && !hp)) continue;
        const int e = high ? bs : lb, pe = e + 2, nv = pe * CV;
        int kind;
        const T* row = pad_row_source<T>(hi, lo, C, bs, nb, high, hi_cap, lo_cap, u, pm, kind);
        T* d = (high ? hp : lp) + ((size_t)(s * pe + u) * pe) * C;
        for (int ib = 0; ib < nv; ib += 64 * PADM) {
            uint4 v[PADM][4];
            int mode[PADM];
#pragma unroll
            for (int m = 0; m < PADM; ++m) {
                const int i = ib + lane + 64 * m;
                mode[m] = -1;
                if (i < nv) {
                    const int w = i / CV, c = (i - w * CV) * V;
                    const T* src = nullptr;
                    bool avg = false;
                    int d1c = C, d2c = bs * C;
                    if (w == 0 || w == pe - 1) {
                        const Src<T> sp =
                            packed_src<T, NHWC>(hi, lo, C, bs, nb, hi_cap, lo_cap, u - 1, w - 1, c, pm);
                        src = sp.p;
                        avg = sp.avg;
                        d1c = sp.d1;
                        d2c = sp.d2;
                    } else if (kind == 1) {
                        src = row + (w - 1) * C + c;
                    } else if (kind == 2) {
                        src = row + ((w - 1) >> 1) * C + c;
                    } else if (kind >= 3) {
                        src = row + 2 * (w - 1) * C + c;
                        avg = kind == 3;
                    }
                    if (!src) {
                        mode[m] = 0;
                    } else {
                        mode[m] = avg ? 2 : 1;
                        v[m][0] = ld_nt16(src);
                        if (avg) {
                            v[m][1] = ld_nt16(src + d1c);
                            v[m][2] = ld_nt16(src + d2c);
                            v[m][3] = ld_nt16(src + d2c + d1c);
                        }
                    }
                }
            }
#pragma unroll
            for (int m = 0; m < PADM; ++m) {
                const int i = ib + lane + 64 * m;
                if (mode[m] >= 0) {
                    uint4 o = uint4{0u, 0u, 0u, 0u};
                    if (mode[m] == 1) o = v[m][0];
                    else if (mode[m] == 2) o = avg_raw<T>(v[m][0], v[m][1], v[m][2], v[m][3]);
                    st_nt16(d + (size_t)i * V, o);
                }
            }
        }
    }
}

int rows_grid(long long waves) {
    const long long cap = (long long)device_cus() * 8;  // workgroups: up to 32 waves per CU
    const long long wgs = (waves + RW_WAVES - 1) / RW_WAVES;
    return (int)(wgs < cap ? wgs : cap);
}

template <typename T, bool ONE, bool BWD>
hipError_t split_rows(const Geo& g, const void* x, const uint8_t* mask, void* hi, int hi_cap, void* lo, int lo_cap,
                      hipStream_t st) {
    const long long jobs = g.B * (g.bs / 2);
    hipLaunchKernelGGL((k_split_rows<T, ONE, BWD>), dim3(rows_grid(jobs)), dim3(WG), 0, st, (const T*)x, g.C, g.H,
                       g.W, mask, g.bs, (int)g.B, g.GH, g.GW, (T*)hi, hi_cap, (T*)lo, lo_cap);
    return hipGetLastError();
}

template <typename T, bool ONE, bool BWD>
hipError_t combine_rows(const Geo& g, const void* hi, const void* lo, const uint8_t* mask, int hi_cap, int lo_cap,
                        void* y, hipStream_t st) {
    const long long jobs = g.B * (g.bs / 2);
    hipLaunchKernelGGL((k_combine_rows<T, ONE, BWD>), dim3(rows_grid(jobs)), dim3(WG), 0, st, (const T*)hi,
                       (const T*)lo, g.C, g.H, g.W, mask, g.bs, (int)g.B, g.GH, g.GW, hi_cap, lo_cap, (T*)y);
    return hipGetLastError();
}

template <typename T, bool ONE>
hipError_t pad_low_dense(const Geo& g, const void* x, const uint8_t* mask, void* lp, int lo_cap, hipStream_t st) {
    const long long jobs = g.B * (g.bs / 2 + 2);
    hipLaunchKernelGGL((k_pad_low_dense<T, ONE>), dim3(rows_grid(jobs)), dim3(WG), 0, st, (const T*)x, g.C, g.H, g.W,
                       mask, g.bs, (int)g.B, g.GH, g.GW, (T*)lp, lo_cap);
    return hipGetLastError();
}

template <typename T, bool ONE>
hipError_t pad_rows(const Geo& g, const void* hi, const void* lo, const uint8_t* mask, void* hp, void* lp,
                    int hi_cap, int lo_cap, int pm, hipStream_t st) {
    const long long jobs = g.B * (g.bs / 2 + 2) + (hp ? (long long)hi_cap * (g.bs - g.bs / 2) : 0LL);
    const int grid = rows_grid(jobs);
    const long long waves = (long long)grid * RW_WAVES;
    const int per_wave = (int)((jobs + waves - 1) / waves);
    hipLaunchKernelGGL((k_pad_rows<T, ONE>), dim3(grid), dim3(WG), 0, st, (const T*)hi, (const T*)lo, g.C, mask,
                       g.bs, (int)g.B, g.GH, g.GW, per_wave, (T*)hp, (T*)lp, hi_cap, lo_cap, pm);
    return hipGetLastError();
}

template <typename T>
hipError_t split_rows_t(const Geo& g, const void* x, const uint8_t* mask, void* hi, int hi_cap, void* lo, int lo_cap,
                        bool bwd, hipStream_t st) {
    if (bwd)
        return g.B <= 1024 ? split_rows<T, true, true>(g, x, mask, hi, hi_cap, lo, lo_cap, st)
                           : split_rows<T, false, true>(g, x, mask, hi, hi_cap, lo, lo_cap, st);
    return g.B <= 1024 ? split_rows<T, true, false>(g, x, mask, hi, hi_cap, lo, lo_cap, st)
                       : split_rows<T, false, false>(g, x, mask, hi, hi_cap, lo, lo_cap, st);
}
template <typename T>
hipError_t combine_rows_t(const Geo& g, const void* hi, const void* lo, const uint8_t* mask, int hi_cap, int lo_cap,
                          void* y, bool bwd, hipStream_t st) {
    if (bwd)
        return g.B <= 1024 ? combine_rows<T, true, true>(g, hi, lo, mask, hi_cap, lo_cap, y, st)
                           : combine_rows<T, false, true>(g, hi, lo, mask, hi_cap, lo_cap, y, st);
    return g.B <= 1024 ? combine_rows<T, true, false>(g, hi, lo, mask, hi_cap, lo_cap, y, st)
                       : combine_rows<T, false, false>(g, hi, lo, mask, hi_cap, lo_cap, y, st);
}
template <typename T>
hipError_t pad_rows_t(const Geo& g, const void* hi, const void* lo, const uint8_t* mask, void* hp, void* lp,
                      int hi_cap, int lo_cap, int pm, hipStream_t st) {
    return g.B <= 1024 ? pad_rows<T, true>(g, hi, lo, mask, hp, lp, hi_cap, lo_cap, pm, st)
                       : pad_rows<T, false>(g, hi, lo, mask, hp, lp, hi_cap, lo_cap, pm, st);
}

inline bool al16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

// The high stack at half resolution: one thread per (slot, cell, 8
// channels); the cell's four pixels are read as 16-byte vectors and averaged
// in the library's association (vavg4).
template <typename T>
__global__ __launch_bounds__(256) void k_sample_hs(const T* __restrict__ hi, long long items, int e, int C,
                                                   T* __restrict__ hs) {
    const long long t = (long long)blockIdx.x * 256 + threadIdx.x;
    if (t >= items) return;
    const int c8 = C >> 3, eh = e >> 1;
    const long long cell = t / c8;
    const int c = (int)(t - cell * c8) * 8;
    const long long s = cell / (eh * eh);
    const int r = (int)(cell - s * eh * eh), u = r / eh, v = r - (r / eh) * eh;
    const T* p = hi + (((size_t)s * e + 2 * u) * e + 2 * v) * C + c;
    const Vec<T, 8> a = vload<T, 8>(p), b = vload<T, 8>(p + C), cc = vload<T, 8>(p + (size_t)e * C),
                    d = vload<T, 8>(p + (size_t)e * C + C);
    *reinterpret_cast<uint4*>(hs + (size_t)cell * C + c) = vavg4<T, 8>(a, b, cc, d).raw;
}

}  // namespace

bool rows_fit(int dtype, int layout, const Geo& g, std::initializer_list<const void*> ptrs) {
    if (layout != NHWC) return false;
    const int es = dtype == 0 ? 4 : 2;
    if ((g.C * es) % 16) return false;
    for (const void* p : ptrs)
        if (!al16(p)) return false;
    return true;
}

hipError_t launch_split_rows(int dtype, const Geo& g, const void* x, const uint8_t* mask, void* hi, int hi_cap,
                             void* lo, int lo_cap, hipStream_t st, bool bwd) {
    switch (dtype) {
    case 0: return split_rows_t<float>(g, x, mask, hi, hi_cap, lo, lo_cap, bwd, st);
    case 1: return split_rows_t<f16>(g, x, mask, hi, hi_cap, lo, lo_cap, bwd, st);
    default: return split_rows_t<bf16>(g, x, mask, hi, hi_cap, lo, lo_cap, bwd, st);
    }
}

hipError_t launch_combine_rows(int dtype, const Geo& g, const void* hi, const void* lo, const uint8_t* mask,
                               int hi_cap, int lo_cap, void* y, hipStream_t st, bool bwd) {
    switch (dtype) {
    case 0: return combine_rows_t<float>(g, hi, lo, mask, hi_cap, lo_cap, y, bwd, st);
    case 1: return combine_rows_t<f16>(g, hi, lo, mask, hi_cap, lo_cap, y, bwd, st);
    default: return combine_rows_t<bf16>(g, hi, lo, mask, hi_cap, lo_cap, y, bwd, st);
    }
}

hipError_t launch_pad_low_dense(int dtype, const Geo& g, const void* x, const uint8_t* mask, void* lp, int lo_cap,
                                hipStream_t st) {
    const bool one = g.B <= 1024;
    if (dtype == 1) return one ? pad_low_dense<f16, true>(g, x, mask, lp, lo_cap, st)
                               : pad_low_dense<f16, false>(g, x, mask, lp, lo_cap, st);
    return one ? pad_low_dense<bf16, true>(g, x, mask, lp, lo_cap, st)
               : pad_low_dense<bf16, false>(g, x, mask, lp, lo_cap, st);
}

hipError_t launch_pad_rows(int dtype, const Geo& g, const void* hi, const void* lo, const uint8_t* mask, void* hp,
                           void* lp, int hi_cap, int lo_cap, int pm, hipStream_t st) {
    switch (dtype) {
    case 0: return pad_rows_t<float>(g, hi, lo, mask, hp, lp, hi_cap, lo_cap, pm, st);
    case 1: return pad_rows_t<f16>(g, hi, lo, mask, hp, lp, hi_cap, lo_cap, pm, st);
    default: return pad_rows_t<bf16>(g, hi, lo, mask, hp, lp, hi_cap, lo_cap, pm, st);
    }
}

hipError_t launch_sample_hs(int dtype, const void* hi, int hi_cap, int e, int C, void* hs, hipStream_t st) {
    if (hi_cap <= 0 || e < 2) return hipSuccess;
    if ((e & 1) || C % 8 || (dtype != 1 && dtype != 2) || (reinterpret_cast<uintptr_t>(hi) & 15) ||
        (reinterpret_cast<uintptr_t>(hs) & 15))
        return hipErrorInvalidValue;
    const long long items = (long long)hi_cap * (e / 2) * (e / 2) * (C / 8);
    const unsigned grid = (unsigned)((items + 255) / 256);
    if (dtype == 1)
        hipLaunchKernelGGL(k_sample_hs<f16>, dim3(grid), dim3(256), 0, st, (const f16*)hi, items, e, C, (f16*)hs);
    else
        hipLaunchKernelGGL(k_sample_hs<bf16>, dim3(grid), dim3(256), 0, st, (const bf16*)hi, items, e, C, (bf16*)hs);
    return hipGetLastError();
}

}  // namespace sb
