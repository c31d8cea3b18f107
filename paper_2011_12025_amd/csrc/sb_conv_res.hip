// Persistent 3x3 block convolution with LDS-resident weights, for the
// channels-last fp16/bf16 layers with up to 64 input channels (the early,
// bandwidth-bound layers of the network).
//
// One workgroup per CU (4 waves) loads its 64-output-channel slice of the
// weights into LDS once and then walks a static list of tiles.  A tile is a
// group of R image rows of one block: R rows of a high block, R/2 rows of a
// low block, so every tile covers the same image area and moves about the
// same number of bytes.  The padded input tile (all input channels, 128
// bytes per pixel) is double-buffered in LDS:
//
//   - pixels that are plain copies (interior, same-resolution halo,
//     nearest-upsampled halo) go straight from global memory to LDS with
//     global_load_lds_dwordx4 (gfx950), which needs no registers, so a whole
//     tile is in flight at once;
//   - pixels that are 2x2 averages (a low tile read from the dense map, or a
//     halo pixel across a resolution boundary) are loaded into registers,
//     averaged and written to LDS;
//   - pixels outside the image are written as zeros.
//
// The next tile is requested before the current tile's MFMAs start, so its
// loads overlap the MFMAs and the epilogue stores of the current tile.
//
// MFMA v_mfma_f32_16x16x32_{f16,bf16}: weights are the A operand (16 output
// channels), pixels the B operand (16 pixels).  Each wave owns up to four
// 16-pixel sub-tiles and the four 16-channel sub-tiles; a lane's result is
// 4 consecutive output channels of one pixel, stored directly.
//
// LDS rows (a weight row [tap][co] or a tile pixel) are 128 bytes = 8
// sub-chunks of 16 bytes; sub-chunk q of row r lives at position q ^ (r & 7)
// so that 8 consecutive rows read at one sub-chunk hit 8 distinct 16-byte
// bank groups.
#include "sb_common.h"
#include "sb_kernels.h"
#include "sb_pixel.h"

namespace sb {

namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef _Float16 halfx8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

template <typename T> struct MFR;
template <> struct MFR<f16> {
    typedef halfx8 frag;
    static __device__ __forceinline__ floatx4 mma(frag a, frag b, floatx4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
    }
};
template <> struct MFR<bf16> {
    typedef bf16x8 frag;
    static __device__ __forceinline__ floatx4 mma(frag a, frag b, floatx4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
    }
};

constexpr int RNT = 64;           // output channels per workgroup
constexpr int RROW = 128;         // LDS bytes per row: 64 channels of 16 bits
constexpr int RSUB = RROW / 16;   // 16-byte sub-chunks per row
constexpr int RW_BYTES = 9 * RNT * RROW;
constexpr int RMT = 256;          // most output pixels of one tile

typedef __attribute__((address_space(3))) void* lds_ptr;

__device__ __forceinline__ int rswz(int row, int q) { return row * RROW + ((q ^ (row & 7)) << 4); }

// One 16-byte global -> LDS copy per active lane; the wave's 64 lanes fill
// the 64 consecutive 16-byte slots starting at `window`.
__device__ __forceinline__ void dma16(const void* g, unsigned char* window) {
    __builtin_amdgcn_global_load_lds(g, (lds_ptr)window, 16, 0, 0);
}

struct RTile {
    int k, n, gy, gx, high, slot, e, pe, r0, rows, M, in_px;
    float inv_pe, inv_e;  // exact quotients p / pe, m / e for the tile's small p, m (see res_div)
};

// q = p / d for 0 <= p < 4096 and 1 <= d <= 128: (p + 0.5) / d in fp32 is at
// least 0.5 / d away from an integer and its rounding error is below 2^-11,
// so truncation gives the exact quotient.
__device__ __forceinline__ int res_div(int p, float inv_d) { return (int)(((float)p + 0.5f) * inv_d); }

template <int SRC, int DST, bool ONE>
__device__ __forceinline__ bool res_tile(const Geo& g, const ConvArgs& a, const WaveMaskT<ONE>& wm, int R, int G,
                                         int tile, RTile& t, Neigh& nb) {
    t.k = tile / G;
    const int grp = tile - t.k * G;
    const int per = g.GH * g.GW;
    t.n = t.k / per;
    const int rem = t.k - t.n * per;
    t.gy = rem / g.GW;
    t.gx = rem - t.gy * g.GW;
    constexpr bool NEED_SLOTS = !(SRC == SRC_DENSE && DST == DST_DENSE);
    nb = wave_neighbourhood<NEED_SLOTS>(wm, g.GH, g.GW, t.n, t.gy, t.gx);
    t.high = (nb.high >> 4) & 1;
    t.slot = nb.slot[4];
    if (NEED_SLOTS && t.slot >= (t.high ? a.hi_cap : a.lo_cap)) return false;
    t.e = t.high ? g.bs : (g.bs >> 1);
    const int rr = t.high ? R : (R >> 1);
    t.r0 = grp * rr;
    if (t.r0 >= t.e) return false;
    t.rows = min(rr, t.e - t.r0);
    t.M = t.rows * t.e;
    t.pe = t.e + 2;
    t.in_px = (t.rows + 2) * t.pe;
    t.inv_pe = 1.0f / (float)t.pe;
    t.inv_e = 1.0f / (float)t.e;
    return true;
}

// Where the value of tile slot (pixel p, channels c..c+7) comes from, as a
// 32-bit element offset from one of two per-call bases (0: the input map or
// the high / own stack, 1: the low stack): mode 0 = zero, 1 = copy,
// 2 = average of the 2x2 cell at off, off + C, off + row, off + row + C.
struct RLoc {
    int off, mode, which, row;
};

template <int SRC>
__device__ __forceinline__ RLoc res_loc(const Geo& g, const ConvArgs& a, const Neigh& nb, const RTile& t, int p,
                                        int c) {
    RLoc L{0, 0, 0, 0};
    const int u = res_div(p, t.inv_pe), v = p - u * t.pe;
    const int C = a.C_in;
    if constexpr (SRC == SRC_PADDED) {
        L.off = ((t.slot * t.pe + t.r0 + u) * t.pe + v) * C + c;
        L.mode = 1;
        L.which = t.high ? 0 : 1;
        return L;
    }
    const int r = t.r0 + u - 1, j = v - 1;  // block-local coordinates
    const int dy = r < 0 ? 0 : (r >= t.e ? 2 : 1);
    const int dx = j < 0 ? 0 : (j >= t.e ? 2 : 1);
    const int d = dy * 3 + dx;
    if constexpr (SRC == SRC_DENSE) {
        L.row = g.W * C;
        if (t.high) {
            const int Y = t.gy * g.bs + r, X = t.gx * g.bs + j;
            if ((unsigned)Y >= (unsigned)g.H || (unsigned)X >= (unsigned)g.W) return L;
            if ((nb.high >> d) & 1) {
                L.off = (Y * g.W + X) * C + c;
                L.mode = 1;
            } else {
                L.off = ((Y & ~1) * g.W + (X & ~1)) * C + c;
                L.mode = 2;
            }
        } else {
            const int lb = g.bs >> 1;
            const int Y = 2 * (t.gy * lb + r), X = 2 * (t.gx * lb + j);
            if ((unsigned)Y >= (unsigned)g.H || (unsigned)X >= (unsigned)g.W) return L;
            L.off = (Y * g.W + X) * C + c;
            L.mode = 2;
        }
        return L;
    } else {
        if (!((nb.valid >> d) & 1)) return L;
        const int nhigh = (nb.high >> d) & 1;
        int ns = nb.slot[0];  // nb.slot[d] with constant indices, so nb stays in registers
#pragma unroll
        for (int i = 1; i < 9; ++i)
            if (d == i) ns = nb.slot[i];
        if (ns >= (nhigh ? a.hi_cap : a.lo_cap)) return L;
        const int u2 = r - (dy - 1) * t.e, v2 = j - (dx - 1) * t.e;
        const int bs = g.bs, lb = bs >> 1;
        if (nhigh == t.high) {
            L.off = ((ns * t.e + u2) * t.e + v2) * C + c;
            L.mode = 1;
            L.which = nhigh ? 0 : 1;
        } else if (t.high) {  // low neighbour of a high block: nearest upsampling
            L.off = ((ns * lb + (u2 >> 1)) * lb + (v2 >> 1)) * C + c;
            L.mode = 1;
            L.which = 1;
        } else {              // high neighbour of a low block: 2x2 average
            L.off = ((ns * bs + 2 * u2) * bs + 2 * v2) * C + c;
            L.mode = 2;
            L.which = 0;
            L.row = bs * C;
        }
        return L;
    }
}

// The two bases of a tile's source offsets (uniform): the image of the
// tile for the dense map, else the high and the low stack.
template <typename T, int SRC>
__device__ __forceinline__ void res_bases(const Geo& g, const ConvArgs& a, const RTile& t, const T*& b0,
                                          const T*& b1) {
    if constexpr (SRC == SRC_DENSE) {
        b0 = (const T*)a.in_hi + (size_t)t.n * g.H * g.W * a.C_in;
        b1 = b0;
    } else {
        b0 = (const T*)a.in_hi;
        b1 = (const T*)a.in_lo;
    }
}

// Issues the copy part of a tile (DMA) and writes its zero slots.  Slots
// whose value is a 2x2 average are left to the average pass.
template <typename T, int SRC>
__device__ __forceinline__ void res_stage_copies(const Geo& g, const ConvArgs& a, const Neigh& nb, const RTile& t,
                                                 const T* base0, const T* base1, unsigned char* buf, int ptid) {
    const int lane = lane_id(), pwave = ptid >> 6;
    const int slots = t.in_px * RSUB;
    for (int w0 = pwave * 64; w0 < slots; w0 += WG) {
        const int s = w0 + lane;
        const int p = s >> 3, q = (s & 7) ^ (p & 7);
        const int c = q * 8;
        RLoc L{0, 0, 0, 0};
        if (s < slots && c < a.C_in) L = res_loc<SRC>(g, a, nb, t, p, c);
        if (s < slots && L.mode == 1) dma16((L.which ? base1 : base0) + L.off, buf + w0 * 16);
        if (s < slots && L.mode == 0) *reinterpret_cast<uint4*>(buf + s * 16) = uint4{0u, 0u, 0u, 0u};
    }
}

// Average pass: the slots of a tile whose value is a 2x2 average.  For a
// low tile read from the dense map that is every pixel; otherwise only halo
// pixels can be averages.  Up to AV items per thread, loaded together.
constexpr int AV = 4;

// 2x2 average of four raw 16-byte vectors of 8 elements.
template <typename T>
__device__ __forceinline__ uint4 avg4_raw(uint4 a, uint4 b, uint4 c, uint4 d) {
    Vec<T, 8> va, vb, vc, vd;
    va.raw = a;
    vb.raw = b;
    vc.raw = c;
    vd.raw = d;
    return vavg4<T, 8>(va, vb, vc, vd).raw;
}

template <typename T, int SRC>
struct ResAvg {
    uint4 v[AV][4];  // raw loaded data (kept packed until the average is taken)
    int slot[AV];    // LDS slot, -1 = none

    // item -> tile pixel: all pixels, or the halo ring
    __device__ __forceinline__ static int item_pixel(const RTile& t, bool all, int h) {
        if (all) return h;
        const int side = t.rows + 2;
        if (h < side) return h * t.pe;                      // left column
        h -= side;
        if (h < side) return h * t.pe + t.pe - 1;           // right column
        h -= side;
        if (h < t.e) return t.r0 == 0 ? 1 + h : -1;         // top row
        h -= t.e;
        return (t.r0 + t.rows == t.e) ? (t.rows + 1) * t.pe + 1 + h : -1;  // bottom row
    }
    __device__ __forceinline__ static bool all_avg(const RTile& t) {
        return SRC == SRC_DENSE && !t.high;
    }
    __device__ __forceinline__ static int n_items(const RTile& t) {
        if constexpr (SRC == SRC_PADDED) return 0;
        if constexpr (SRC == SRC_PACKED) {
            if (t.high) return 0;
        }
        const int pix = all_avg(t) ? t.in_px : 2 * (t.rows + 2) + 2 * t.e;
        return pix * RSUB;
    }
    __device__ __forceinline__ void issue(const Geo& g, const ConvArgs& a, const Neigh& nb, const RTile& t,
                                          const T* base0, const T* base1, int base, int ptid) {
        const bool all = all_avg(t);
        const int items = n_items(t);
#pragma unroll
        for (int u = 0; u < AV; ++u) {
            slot[u] = -1;
            const int it = base + u * WG + ptid;
            if (it < items) {
                const int q = it & 7;
                const int p = item_pixel(t, all, it >> 3);
                if (p >= 0 && q * 8 < a.C_in) {
                    const RLoc L = res_loc<SRC>(g, a, nb, t, p, q * 8);
                    if (L.mode == 2) {
                        const T* p0 = (L.which ? base1 : base0) + L.off;
                        slot[u] = p * RSUB + (q ^ (p & 7));
                        v[u][0] = ld_nt16(p0);
                        v[u][1] = ld_nt16(p0 + a.C_in);
                        v[u][2] = ld_nt16(p0 + L.row);
                        v[u][3] = ld_nt16(p0 + L.row + a.C_in);
                    }
                }
            }
        }
    }
    __device__ __forceinline__ void commit(unsigned char* buf) const {
#pragma unroll
        for (int u = 0; u < AV; ++u)
            if (slot[u] >= 0)
                *reinterpret_cast<uint4*>(buf + slot[u] * 16) = avg4_raw<T>(v[u][0], v[u][1], v[u][2], v[u][3]);
    }
};

// MFMA over one tile and its epilogue, for a wave owning NMS 16-pixel
// sub-tiles (pixels (wave + 4 ms) * 16 + l16) and NKS 32-channel K-steps per
// tap.  Fully unrolled; the fragments of the next K-step are read from LDS
// while the MFMAs of the current one run.
template <typename T, int DST, int NMS, int NKS>
__device__ __forceinline__ void res_compute(const Geo& g, const ConvArgs& a, const RTile& t,
                                            const unsigned char* s_w, const unsigned char* buf,
                                            const float (&bv)[4][4], int co0, int vec_out, bool relu) {
    typedef MFR<T> mf;
    typedef typename mf::frag frag;
    const int lane = lane_id(), l16 = lane & 15, kg = lane >> 4;
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    int pbase[NMS];
#pragma unroll
    for (int ms = 0; ms < NMS; ++ms) {
        const int m = min((wave + 4 * ms) * 16 + l16, t.M - 1);
        const int mi = res_div(m, t.inv_e);
        pbase[ms] = mi * t.pe + (m - mi * t.e);
    }
    // per-lane byte offsets of the weight fragments (row & 7 == l16 & 7 for every weight row used)
    int wbase[NKS];
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) wbase[ks] = l16 * RROW + (((ks * 4 + kg) ^ (l16 & 7)) << 4);

    floatx4 acc[NMS][4];
#pragma unroll
    for (int ms = 0; ms < NMS; ++ms)
#pragma unroll
        for (int ns = 0; ns < 4; ++ns) acc[ms][ns] = floatx4{0.f, 0.f, 0.f, 0.f};

    constexpr int S = 9 * NKS;
    frag wf[2][4], pf[2][NMS];
    auto load = [&](int step, int b) {
        const int tap = step / NKS, ks = step - tap * NKS;
        const int q = ks * 4 + kg;
        const int toff = (tap / 3) * t.pe + (tap % 3);
#pragma unroll
        for (int ns = 0; ns < 4; ++ns)
            wf[b][ns] = *reinterpret_cast<const frag*>(s_w + wbase[ks] + (tap * RNT + ns * 16) * RROW);
#pragma unroll
        for (int ms = 0; ms < NMS; ++ms) {
            const int r = pbase[ms] + toff;
            pf[b][ms] = *reinterpret_cast<const frag*>(buf + r * RROW + ((q ^ (r & 7)) << 4));
        }
    };
    load(0, 0);
#pragma unroll
    for (int step = 0; step < S; ++step) {
        if (step + 1 < S) load(step + 1, (step + 1) & 1);
#pragma unroll
        for (int ms = 0; ms < NMS; ++ms)
#pragma unroll
            for (int ns = 0; ns < 4; ++ns) acc[ms][ns] = mf::mma(wf[step & 1][ns], pf[step & 1][ms], acc[ms][ns]);
    }

    // -- epilogue: channels co0 + ns*16 + kg*4 + {0..3} of pixel (wave + 4*ms)*16 + l16
    const int Co = a.C_out;
    T* obase;  // the tile's block in its output stack, or the tile's image
    const T* rbase = nullptr;
    if constexpr (DST == DST_PACKED) {
        const size_t blk = (size_t)t.slot * t.e * t.e * Co;
        obase = (T*)(t.high ? a.out_hi : a.out_lo) + blk;
        const T* rb = (const T*)(t.high ? a.res_hi : a.res_lo);
        if (rb) rbase = rb + blk;
    } else {
        obase = (T*)a.out_hi + (size_t)t.n * g.H * g.W * Co;
    }
#pragma unroll
    for (int ms = 0; ms < NMS; ++ms) {
        const int m = (wave + 4 * ms) * 16 + l16;
        if (m >= t.M) continue;
        const int mi = res_div(m, t.inv_e);
        const int i = t.r0 + mi, j = m - mi * t.e;
        int off;  // element offset of channel 0 of this pixel (the first of 2x2 for a low block)
        int down = 0;
        if constexpr (DST == DST_PACKED) {
            off = (i * t.e + j) * Co;
        } else {
            const int Y = t.gy * g.bs + (t.high ? i : 2 * i), X = t.gx * g.bs + (t.high ? j : 2 * j);
            off = (Y * g.W + X) * Co;
            down = g.W * Co;
        }
#pragma unroll
        for (int ns = 0; ns < 4; ++ns) {
            const int co = co0 + ns * 16 + kg * 4;
            if (co >= Co) continue;
            const bool full = vec_out && co + 4 <= Co;
            float f[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) f[r] = acc[ms][ns][r] + bv[ns][r];
            if (rbase) {
                if (full) {
                    const Vec<T, 4> rv = vload<T, 4>(rbase + off + co);
#pragma unroll
                    for (int r = 0; r < 4; ++r) f[r] += to_f32(rv.e[r]);
                } else {
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        if (co + r < Co) f[r] += to_f32(rbase[off + co + r]);
                }
            }
            Vec<T, 4> o;
#pragma unroll
            for (int r = 0; r < 4; ++r) o.e[r] = from_f32<T>(relu ? fmaxf(f[r], 0.0f) : f[r]);
            const int reps = (DST == DST_DENSE && !t.high) ? 2 : 1;
            for (int dy = 0; dy < reps; ++dy)
                for (int dx = 0; dx < reps; ++dx) {
                    T* q = obase + off + dy * down + dx * Co + co;
                    if (full) {
                        if constexpr (sizeof(T) == 2) st_nt8(q, o.raw);
                        else vstore<T, 4>(q, o);
                    } else {
#pragma unroll
                        for (int r = 0; r < 4; ++r)
                            if (co + r < Co) q[r] = o.e[r];
                    }
                }
        }
    }
}

// Stages tile t completely into `buf`: copies by DMA, zeros, then the 2x2
// averages; returns with every write to `buf` complete.  Producer waves only
// (ptid = 0..255).
template <typename T, int SRC>
__device__ __forceinline__ void res_stage(const Geo& g, const ConvArgs& a, const Neigh& nb, const RTile& t,
                                          unsigned char* buf, int ptid) {
    const T *b0, *b1;
    res_bases<T, SRC>(g, a, t, b0, b1);
    res_stage_copies<T, SRC>(g, a, nb, t, b0, b1, buf, ptid);
    for (int base = 0; base < ResAvg<T, SRC>::n_items(t); base += WG * AV) {
        ResAvg<T, SRC> av;
        av.issue(g, a, nb, t, b0, b1, base, ptid);
        av.commit(buf);
    }
    __builtin_amdgcn_s_waitcnt(0);  // DMA (vmcnt) and LDS writes (lgkmcnt) done
}

// Workgroup barrier without the memory fences of __syncthreads: consumer
// waves must not wait for their epilogue stores here.  LDS hand-over is
// ordered by the explicit s_waitcnt of each side before it.
__device__ __forceinline__ void res_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// 8 waves: waves 0-3 compute (MFMA + epilogue) tile j from buffer j & 1 while
// waves 4-7 stage tile j + 1 into the other buffer; one barrier per tile.
template <typename T, int SRC, int DST, bool ONE>
__global__ __launch_bounds__(2 * WG, 2) void k_conv_res(Geo g, const uint8_t* __restrict__ mask, ConvArgs a, int R,
                                                        int G, int ntiles, int buf_bytes, int vec_out) {
    extern __shared__ __align__(16) unsigned char smem[];
    unsigned char* s_w = smem;
    unsigned char* s_buf0 = smem + RW_BYTES;
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const bool producer = wave >= 4;
    const int ptid = (int)threadIdx.x - WG;
    const int lane = lane_id(), kg = lane >> 4;
    const int co0 = blockIdx.y * RNT;

    WaveMaskT<ONE> wm;
    wm.init(mask, (int)g.B);

    // the tile sequence of this workgroup (every wave walks it identically)
    int tile = blockIdx.x;
    RTile t;
    Neigh nb;
    bool have = false;
    while (tile < ntiles && !(have = res_tile<SRC, DST, ONE>(g, a, wm, R, G, tile, t, nb))) tile += gridDim.x;

    if (producer) {
        // weights of this workgroup's output channels: rows [tap][co], 64 channels each
        const T* __restrict__ wgt = (const T*)a.weight;
        for (int w0 = (wave - 4) * 64; w0 < 9 * RNT * RSUB; w0 += WG) {
            const int s = w0 + lane;
            const int row = s >> 3, q = (s & 7) ^ (row & 7);
            const int tap = row / RNT, col = row - tap * RNT;
            const int co = co0 + col, ci = q * 8;
            if (co < a.C_out && ci < a.C_in) dma16(wgt + ((size_t)co * 9 + tap) * a.C_in + ci, s_w + w0 * 16);
            else *reinterpret_cast<uint4*>(s_w + s * 16) = uint4{0u, 0u, 0u, 0u};
        }
        if (have) res_stage<T, SRC>(g, a, nb, t, s_buf0, ptid);
        __builtin_amdgcn_s_waitcnt(0);
    }
    res_barrier();

    const T* __restrict__ bias = (const T*)a.bias;
    const bool relu = (a.flags & 1) != 0;
    float bv[4][4];  // bias of channels co0 + ns*16 + kg*4 + r
#pragma unroll
    for (int ns = 0; ns < 4; ++ns)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int co = co0 + ns * 16 + kg * 4 + r;
            bv[ns][r] = (bias && co < a.C_out) ? to_f32(bias[co]) : 0.0f;
        }

    int cur = 0;
    while (have) {
        unsigned char* buf = s_buf0 + cur * buf_bytes;
        unsigned char* nbuf = s_buf0 + (cur ^ 1) * buf_bytes;
        int ntile = tile + gridDim.x;
        RTile t2;
        Neigh nb2;
        bool have2 = false;
        while (ntile < ntiles && !(have2 = res_tile<SRC, DST, ONE>(g, a, wm, R, G, ntile, t2, nb2)))
            ntile += gridDim.x;
        if (producer) {
            if (have2) res_stage<T, SRC>(g, a, nb2, t2, nbuf, ptid);
        } else {
            const int nst = (t.M + 15) >> 4;
            const int nms = nst > wave ? min(4, (nst - wave + 3) >> 2) : 0;
            if (a.C_in > 32) {
                if (nms == 4) res_compute<T, DST, 4, 2>(g, a, t, s_w, buf, bv, co0, vec_out, relu);
                else if (nms == 3) res_compute<T, DST, 3, 2>(g, a, t, s_w, buf, bv, co0, vec_out, relu);
                else if (nms == 2) res_compute<T, DST, 2, 2>(g, a, t, s_w, buf, bv, co0, vec_out, relu);
                else if (nms == 1) res_compute<T, DST, 1, 2>(g, a, t, s_w, buf, bv, co0, vec_out, relu);
            } else {
                if (nms == 4) res_compute<T, DST, 4, 1>(g, a, t, s_w, buf, bv, co0, vec_out, relu);
                else if (nms == 3) res_compute<T, DST, 3, 1>(g, a, t, s_w, buf, bv, co0, vec_out, relu);
                else if (nms == 2) res_compute<T, DST, 2, 1>(g, a, t, s_w, buf, bv, co0, vec_out, relu);
                else if (nms == 1) res_compute<T, DST, 1, 1>(g, a, t, s_w, buf, bv, co0, vec_out, relu);
            }
            __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this tile's LDS reads are done
        }
        res_barrier();
        have = have2;
        t = t2;
        nb = nb2;
        tile = ntile;
        cur ^= 1;
    }
}

int cu_count() {
    static int n = 0;
    if (n == 0) {
        int dev = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
            n = 256;
    }
    return n;
}

inline bool aligned_to(const void* p, int bytes) { return (reinterpret_cast<uintptr_t>(p) & (bytes - 1)) == 0; }

template <typename T, int SRC, int DST, bool ONE>
hipError_t run_res(const Geo& g, const uint8_t* mask, const ConvArgs& a, int R, hipStream_t st) {
    const int G = (g.bs + R - 1) / R;
    const long long ntiles = g.B * G;
    const int lb = g.bs / 2;
    const int px_h = (R + 2) * (g.bs + 2), px_l = (R / 2 + 2) * (lb + 2);
    const int buf_bytes = (px_h > px_l ? px_h : px_l) * RROW;
    const int smem = RW_BYTES + 2 * buf_bytes;
    const int ob = 4 * (int)sizeof(T);
    const int vec_out = (a.C_out % 4 == 0) && aligned_to(a.out_hi, ob) && aligned_to(a.out_lo, ob) &&
                        aligned_to(a.res_hi, ob) && aligned_to(a.res_lo, ob);
    static int attr_bytes = 0;
    if (smem > attr_bytes) {
        hipError_t e = hipFuncSetAttribute((const void*)k_conv_res<T, SRC, DST, ONE>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, smem);
        if (e != hipSuccess) return e;
        attr_bytes = smem;
    }
    const int nwg = (int)(ntiles < cu_count() ? ntiles : cu_count());
    const dim3 grid((unsigned)nwg, (unsigned)((a.C_out + RNT - 1) / RNT));
    hipLaunchKernelGGL((k_conv_res<T, SRC, DST, ONE>), grid, dim3(2 * WG), smem, st, g, mask, a, R, G, (int)ntiles, buf_bytes,
                       vec_out);
    return hipGetLastError();
}

// Image rows per tile: the largest even R <= bs whose two tile buffers fit
// beside the weights (a tile covers at most RMT output pixels).
int res_rows(int bs) {
    const int budget = (160 * 1024 - RW_BYTES) / 2 / RROW;  // pixels per buffer
    int best = 0;
    for (int R = 2; R <= bs; R += 2) {
        const int lb = bs / 2;
        const int px = (R + 2) * (bs + 2) > (R / 2 + 2) * (lb + 2) ? (R + 2) * (bs + 2) : (R / 2 + 2) * (lb + 2);
        if (px <= budget && R * bs <= RMT) best = R;
    }
    return best;
}

template <typename T, bool ONE>
hipError_t res_t(ConvSrc src, ConvDst dst, const Geo& g, const uint8_t* mask, const ConvArgs& a, int R,
                 hipStream_t st) {
    if (src == SRC_PADDED) return run_res<T, SRC_PADDED, DST_PACKED, ONE>(g, mask, a, R, st);
    if (src == SRC_PACKED) return run_res<T, SRC_PACKED, DST_PACKED, ONE>(g, mask, a, R, st);
    (void)dst;
    return run_res<T, SRC_DENSE, DST_DENSE, ONE>(g, mask, a, R, st);
}

}  // namespace

bool conv_res_fits(int dtype, int layout, const Geo& g, const ConvArgs& a) {
    if (layout != NHWC || (dtype != 1 && dtype != 2)) return false;
    if (a.C_in % 8 || a.C_in > 64 || g.bs < 16 || g.bs > 64) return false;
    if (!aligned_to(a.in_hi, 16) || !aligned_to(a.in_lo, 16) || !aligned_to(a.weight, 16)) return false;
    // element offsets inside one image or one stack are 32-bit
    const long long img = (long long)g.H * g.W * (a.C_in > a.C_out ? a.C_in : a.C_out);
    const long long cap = (a.hi_cap > a.lo_cap ? a.hi_cap : a.lo_cap) + 1LL;
    const long long stk = cap * (g.bs + 2) * (g.bs + 2) * (a.C_in > a.C_out ? a.C_in : a.C_out);
    if (img >= (1LL << 31) || stk >= (1LL << 31)) return false;
    return res_rows(g.bs) > 0;
}

hipError_t launch_conv_res(int dtype, ConvSrc src, ConvDst dst, const Geo& g, const uint8_t* mask, const ConvArgs& a,
                           hipStream_t st) {
    const int R = res_rows(g.bs);
    const bool one = g.B <= 1024;
    if (dtype == 1) return one ? res_t<f16, true>(src, dst, g, mask, a, R, st) : res_t<f16, false>(src, dst, g, mask, a, R, st);
    return one ? res_t<bf16, true>(src, dst, g, mask, a, R, st) : res_t<bf16, false>(src, dst, g, mask, a, R, st);
}

}  // namespace sb
