// Persistent 3x3 block convolution with LDS-resident weights, for the
// channels-last fp16/bf16 layers with up to 64 input channels (the early,
// bandwidth-bound layers of the network).
//
// One 12-wave workgroup per CU keeps its 64-output-channel slice of the
// weights in LDS and walks a static list of tiles.  A tile is a group of R
// image rows of one block: R rows of a high block, R/2 rows of a low block,
// so every tile covers the same image area and moves about the same number of
// bytes.  The padded input tile (all input channels, 128 bytes per pixel) is
// double-buffered in LDS, and the waves are specialised:
//
//   waves 0-7  (consumers): MFMA over tile j from one buffer, then the
//              epilogue (bias, residual, ReLU, rounding) stored directly to
//              global memory;
//   waves 8-11 (producers): stage tile j+1 into the other buffer.
//
// Staging issues every load of the tile before waiting once:
//   - pixels that are plain copies (interior, same-resolution halo,
//     nearest-upsampled halo) go straight from global memory to LDS with
//     global_load_lds_dwordx4 (gfx950);
//   - pixels that are 2x2 averages (a low tile read from the dense map, or a
//     halo pixel across a resolution boundary) are loaded into registers
//     with non-temporal loads, averaged and written to LDS;
//   - pixels outside the image are written as zeros.
// One barrier per tile hands the buffer from the producers to the consumers.
// The barrier carries no memory fence, so the consumers' epilogue stores stay
// in flight while the next tile is computed.
//
// MFMA v_mfma_f32_16x16x32_{f16,bf16}: weights are the A operand (16 output
// channels), pixels the B operand (16 pixels).  Consumer wave w owns the
// 16-pixel sub-tiles w, w + 8 (of up to 16) and all four 16-channel
// sub-tiles; a lane's result is 4 consecutive output channels of one pixel.
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
constexpr int NCW = 8;            // consumer waves
constexpr int NPW = 4;            // producer waves
constexpr int RWG = 64 * (NCW + NPW);
constexpr int PT = 64 * NPW;      // producer threads

typedef __attribute__((address_space(3))) void* lds_ptr;

// One 16-byte global -> LDS copy per active lane; the wave's 64 lanes fill
// the 64 consecutive 16-byte slots starting at `window`.
__device__ __forceinline__ void dma16(const void* g, unsigned char* window) {
    __builtin_amdgcn_global_load_lds(g, (lds_ptr)window, 16, 0, 0);
}

// q = p / d for 0 <= p < 4096 and 1 <= d <= 128: (p + 0.5) / d in fp32 is at
// least 0.5 / d away from an integer and its rounding error is below 2^-11,
// so truncation gives the exact quotient.
__device__ __forceinline__ int res_div(int p, float inv_d) { return (int)(((float)p + 0.5f) * inv_d); }

struct RTile {
    int n, gy, gx, high, slot, e, pe, r0, rows, M, in_px;
    float inv_e;
};

template <int SRC, int DST, bool ONE>
__device__ __forceinline__ bool res_tile(const Geo& g, const ConvArgs& a, const WaveMaskT<ONE>& wm, int R, int G,
                                         int tile, RTile& t, Neigh& nb) {
    const int k = tile / G;
    const int grp = tile - k * G;
    const int per = g.GH * g.GW;
    t.n = k / per;
    const int rem = k - t.n * per;
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
    t.inv_e = 1.0f / (float)t.e;
    return true;
}

// Where the value of tile pixel (u, v) (row u of the padded tile, column v),
// channels c..c+7, comes from: a 32-bit element offset from one of two
// per-tile bases (0: the tile's image or the high / own stack, 1: the low
// stack); mode 0 = zero, 1 = copy, 2 = average of the 2x2 cell at off,
// off + C, off + row, off + row + C.
struct RLoc {
    int off, mode, which, row;
};

template <int SRC>
__device__ __forceinline__ RLoc res_loc(const Geo& g, const ConvArgs& a, const Neigh& nb, const RTile& t, int u,
                                        int v, int c) {
    RLoc L{0, 0, 0, 0};
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

// The two bases of a tile's source offsets (uniform): the tile's image for
// the dense map, else the high and the low stack.
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

// Average pass: the slots of a tile whose value is a 2x2 average.  For a
// low tile read from the dense map that is every pixel; otherwise only halo
// pixels can be averages.  Up to AV items per producer thread per batch.
constexpr int AV = 4;

template <typename T, int SRC>
struct ResAvg {
    uint4 v[AV][4];  // raw loaded data (kept packed until the average is taken)
    int slot[AV];    // LDS slot, -1 = none

    // item h -> tile pixel (u, v): every pixel, or the halo ring
    __device__ __forceinline__ static bool item_pixel(const RTile& t, bool all, int h, int& u, int& v) {
        if (all) {
            u = res_div(h, 1.0f / (float)t.pe);
            v = h - u * t.pe;
            return true;
        }
        const int side = t.rows + 2;
        if (h < side) { u = h; v = 0; return true; }                  // left column
        h -= side;
        if (h < side) { u = h; v = t.pe - 1; return true; }           // right column
        h -= side;
        if (h < t.e) { u = 0; v = 1 + h; return t.r0 == 0; }          // top row
        h -= t.e;
        u = t.rows + 1;                                               // bottom row
        v = 1 + h;
        return t.r0 + t.rows == t.e;
    }
    __device__ __forceinline__ static bool all_avg(const RTile& t) { return SRC == SRC_DENSE && !t.high; }
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
        for (int i = 0; i < AV; ++i) {
            slot[i] = -1;
            const int it = base + i * PT + ptid;
            int u, w;
            if (it < items && item_pixel(t, all, it >> 3, u, w)) {
                const int q = it & 7;
                if (q * 8 < a.C_in) {
                    const RLoc L = res_loc<SRC>(g, a, nb, t, u, w, q * 8);
                    if (L.mode == 2) {
                        const T* p0 = (L.which ? base1 : base0) + L.off;
                        const int p = u * t.pe + w;
                        slot[i] = p * RSUB + (q ^ (p & 7));
                        v[i][0] = ld_nt16(p0);
                        v[i][1] = ld_nt16(p0 + a.C_in);
                        v[i][2] = ld_nt16(p0 + L.row);
                        v[i][3] = ld_nt16(p0 + L.row + a.C_in);
                    }
                }
            }
        }
    }
    __device__ __forceinline__ void commit(unsigned char* buf) const {
#pragma unroll
        for (int i = 0; i < AV; ++i)
            if (slot[i] >= 0)
                *reinterpret_cast<uint4*>(buf + slot[i] * 16) = avg4_raw<T>(v[i][0], v[i][1], v[i][2], v[i][3]);
    }
};

// Stages tile t completely into `buf` (producer waves, ptid = 0..PT-1):
// every copy by DMA, every zero slot, and the first batch of averages are
// issued before a single wait; returns with every write to `buf` complete.
template <typename T, int SRC>
__device__ __forceinline__ void res_stage(const Geo& g, const ConvArgs& a, const Neigh& nb, const RTile& t,
                                          unsigned char* buf, int ptid) {
    const T *b0, *b1;
    res_bases<T, SRC>(g, a, t, b0, b1);
    const int lane = lane_id(), pwave = ptid >> 6;
    const int nwin = (t.in_px * RSUB + 63) >> 6;  // 64-slot windows = 8 pixels each
    for (int w = pwave; w < nwin; w += NPW) {
        const int pw = w * 8;                       // first pixel of the window (uniform)
        const int u0 = pw / t.pe, v0 = pw - u0 * t.pe;
        int u = u0, v = v0 + (lane >> 3);
        if (v >= t.pe) {                            // a window spans at most two rows (pe >= 10)
            v -= t.pe;
            ++u;
        }
        const int p = pw + (lane >> 3);
        const int q = (lane & 7) ^ (lane >> 3);     // p & 7 == lane >> 3 inside a window
        RLoc L{0, 0, 0, 0};
        const bool in = p < t.in_px;
        if (in && q * 8 < a.C_in) L = res_loc<SRC>(g, a, nb, t, u, v, q * 8);
        if (in && L.mode == 1) dma16((L.which ? b1 : b0) + L.off, buf + w * 1024);
        if (in && L.mode == 0) *reinterpret_cast<uint4*>(buf + w * 1024 + lane * 16) = uint4{0u, 0u, 0u, 0u};
    }
    const int navg = ResAvg<T, SRC>::n_items(t);
    for (int base = 0; base < navg; base += PT * AV) {
        ResAvg<T, SRC> av;
        av.issue(g, a, nb, t, b0, b1, base, ptid);
        av.commit(buf);
    }
    __builtin_amdgcn_s_waitcnt(0);  // DMA (vmcnt) and LDS writes (lgkmcnt) done
}

// MFMA over one tile and its epilogue, for a consumer wave cw owning NMS
// 16-pixel sub-tiles (pixels (cw + NCW * ms) * 16 + l16) and NKS 32-channel
// K-steps per tap.  Fully unrolled; the fragments of the next K-step are
// read from LDS while the MFMAs of the current one run.
template <typename T, int DST, int NMS, int NKS>
__device__ __forceinline__ void res_compute(const Geo& g, const ConvArgs& a, const RTile& t, int cw,
                                            const unsigned char* s_w, const unsigned char* buf,
                                            const float (&bv)[4][4], int co0, int vec_out, bool relu) {
    typedef MFR<T> mf;
    typedef typename mf::frag frag;
    const int lane = lane_id(), l16 = lane & 15, kg = lane >> 4;
    int pbase[NMS];
#pragma unroll
    for (int ms = 0; ms < NMS; ++ms) {
        const int m = min((cw + NCW * ms) * 16 + l16, t.M - 1);
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

    constexpr int S = 9 * NKS;  // K-steps (even: 18, or 9 with one odd step left)
    frag wf[2][4], pf[2][NMS];
    auto load = [&](int step, int b) {
        const int tap = NKS == 2 ? (step >> 1) : step, ks = NKS == 2 ? (step & 1) : 0;
        const int ky = tap >= 6 ? 2 : (tap >= 3 ? 1 : 0);
        const int toff = ky * t.pe + (tap - 3 * ky);
        const int q = ks * 4 + kg;
#pragma unroll
        for (int ns = 0; ns < 4; ++ns)
            wf[b][ns] = *reinterpret_cast<const frag*>(s_w + wbase[ks] + (tap * RNT + ns * 16) * RROW);
#pragma unroll
        for (int ms = 0; ms < NMS; ++ms) {
            const int r = pbase[ms] + toff;
            pf[b][ms] = *reinterpret_cast<const frag*>(buf + r * RROW + ((q ^ (r & 7)) << 4));
        }
    };
    auto mma = [&](int b) {
#pragma unroll
        for (int ms = 0; ms < NMS; ++ms)
#pragma unroll
            for (int ns = 0; ns < 4; ++ns) acc[ms][ns] = mf::mma(wf[b][ns], pf[b][ms], acc[ms][ns]);
    };
    load(0, 0);
#pragma unroll 1
    for (int step = 0; step + 1 < S; step += 2) {
        load(step + 1, 1);
        mma(0);
        if (step + 2 < S) load(step + 2, 0);
        mma(1);
    }
    if (S & 1) mma(0);

    // -- epilogue: channels co0 + ns*16 + kg*4 + {0..3} of pixel (cw + NCW*ms)*16 + l16
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
        const int m = (cw + NCW * ms) * 16 + l16;
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
                        st_nt8(q, o.raw);
                    } else {
#pragma unroll
                        for (int r = 0; r < 4; ++r)
                            if (co + r < Co) q[r] = o.e[r];
                    }
                }
        }
    }
}

// Workgroup barrier without the memory fences of __syncthreads: consumer
// waves must not wait for their epilogue stores here.  LDS hand-over is
// ordered by the explicit s_waitcnt of each side before it.
__device__ __forceinline__ void res_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

template <typename T, int SRC, int DST, bool ONE, int NKS>
__global__ __launch_bounds__(RWG, 1) void k_conv_res(Geo g, const uint8_t* __restrict__ mask, ConvArgs a, int R,
                                                     int G, int ntiles, int buf_bytes, int vec_out) {
    extern __shared__ __align__(16) unsigned char smem[];
    unsigned char* s_w = smem;
    unsigned char* s_buf0 = smem + RW_BYTES;
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const bool producer = wave >= NCW;
    const int ptid = (int)threadIdx.x - 64 * NCW;
    const int lane = lane_id(), kg = lane >> 4;
    const int co0 = blockIdx.y * RNT;

    if (producer) {
        // weights of this workgroup's output channels first (they do not depend on the
        // mask): rows [tap][co], 64 channels each
        const T* __restrict__ wgt = (const T*)a.weight;
        for (int w0 = (wave - NCW) * 64; w0 < 9 * RNT * RSUB; w0 += PT) {
            const int s = w0 + lane;
            const int row = s >> 3, q = (s & 7) ^ (row & 7);
            const int tap = row / RNT, col = row - tap * RNT;
            const int co = co0 + col, ci = q * 8;
            if (co < a.C_out && ci < a.C_in) dma16(wgt + ((size_t)co * 9 + tap) * a.C_in + ci, s_w + w0 * 16);
            else *reinterpret_cast<uint4*>(s_w + s * 16) = uint4{0u, 0u, 0u, 0u};
        }
    }

    WaveMaskT<ONE> wm;
    wm.init(mask, (int)g.B);

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

    // Step i: the producers stage tile i of this workgroup's sequence into buffer i & 1
    // while the consumers compute tile i - 1 from the other buffer.  Every wave walks
    // the sequence identically, so all of them leave the loop together.
    int tile = blockIdx.x;
    RTile t;            // the tile the consumers compute in this step
    bool have = false;  // ... if any
    for (int it = 0;; ++it) {
        RTile t2;
        Neigh nb2;
        bool have2 = false;
        while (tile < ntiles && !(have2 = res_tile<SRC, DST, ONE>(g, a, wm, R, G, tile, t2, nb2))) tile += gridDim.x;
        tile += gridDim.x;
        if (!have && !have2) break;
        unsigned char* sbuf = s_buf0 + (it & 1) * buf_bytes;
        unsigned char* cbuf = s_buf0 + ((it & 1) ^ 1) * buf_bytes;
        if (producer) {
            // the staging wait also covers the weight copies of the first step
            if (have2) res_stage<T, SRC>(g, a, nb2, t2, sbuf, ptid);
            __builtin_amdgcn_s_waitcnt(0);
        } else if (have) {
            const int nst = (t.M + 15) >> 4;
            const int nms = nst > wave ? min(2, (nst - wave + NCW - 1) / NCW) : 0;
            if (nms == 2) res_compute<T, DST, 2, NKS>(g, a, t, wave, s_w, cbuf, bv, co0, vec_out, relu);
            else if (nms == 1) res_compute<T, DST, 1, NKS>(g, a, t, wave, s_w, cbuf, bv, co0, vec_out, relu);
            __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this tile's LDS reads are done
        }
        res_barrier();
        t = t2;
        have = have2;
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

template <typename T, int SRC, int DST, bool ONE, int NKS>
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
        hipError_t e = hipFuncSetAttribute((const void*)k_conv_res<T, SRC, DST, ONE, NKS>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, smem);
        if (e != hipSuccess) return e;
        attr_bytes = smem;
    }
    const int nwg = (int)(ntiles < cu_count() ? ntiles : cu_count());
    const dim3 grid((unsigned)nwg, (unsigned)((a.C_out + RNT - 1) / RNT));
    hipLaunchKernelGGL((k_conv_res<T, SRC, DST, ONE, NKS>), grid, dim3(RWG), smem, st, g, mask, a, R, G, (int)ntiles,
                       buf_bytes, vec_out);
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

template <typename T, bool ONE, int NKS>
hipError_t res_k(ConvSrc src, const Geo& g, const uint8_t* mask, const ConvArgs& a, int R, hipStream_t st) {
    if (src == SRC_PADDED) return run_res<T, SRC_PADDED, DST_PACKED, ONE, NKS>(g, mask, a, R, st);
    if (src == SRC_PACKED) return run_res<T, SRC_PACKED, DST_PACKED, ONE, NKS>(g, mask, a, R, st);
    return run_res<T, SRC_DENSE, DST_DENSE, ONE, NKS>(g, mask, a, R, st);
}

template <typename T, bool ONE>
hipError_t res_t(ConvSrc src, ConvDst dst, const Geo& g, const uint8_t* mask, const ConvArgs& a, int R,
                 hipStream_t st) {
    (void)dst;
    if (a.C_in > 32) return res_k<T, ONE, 2>(src, g, mask, a, R, st);
    return res_k<T, ONE, 1>(src, g, mask, a, R, st);
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
    if (dtype == 1)
        return one ? res_t<f16, true>(src, dst, g, mask, a, R, st) : res_t<f16, false>(src, dst, g, mask, a, R, st);
    return one ? res_t<bf16, true>(src, dst, g, mask, a, R, st) : res_t<bf16, false>(src, dst, g, mask, a, R, st);
}

}  // namespace sb
