// Persistent 3x3 block convolution with register-resident weights, for the
// channels-last fp16/bf16 layers with up to 64 input channels and block sides
// 32 or 64 (the early, bandwidth-bound layers of the network).
//
// One 8-wave workgroup per CU computes a 64-output-channel slice and walks a
// static list of tiles.  A tile is a group of rows of one block: R rows of a
// high block (R = 8 for blocks of 32, 4 for blocks of 64) or, from packed or
// padded stacks, 2R rows of a low block, so every tile has the same number
// of output pixels and a low block has a quarter of a high block's tiles;
// that list holds the high blocks' tiles, then the low blocks', in slot
// order, and its length follows the class counts of the mask, so the work
// of a launch falls with the low-resolution fraction.  From the dense map a
// low tile is R/2 low rows and the list is block-major (see res_tile).  The
// padded input tile (all input channels, 128 bytes per pixel) is
// triple-buffered in LDS and the waves are specialised:
//
//   waves 0-3  (consumers): wave c owns output channels co0 + 32 * (c & 1)
//              + [0, 32) and half (c >> 1) of the tile; its 32 x 9 x C_in
//              weights are loaded into its registers at start-up and stay
//              there for the whole launch;
//   waves 4-7  (producers): finish staging tile i (wait for its copies,
//              write its 2x2 averages), then issue the copies of tile i + 1,
//              while the consumers compute tile i - 1.
//
// Staging:
//   - pixels that are plain copies (interior, same-resolution halo,
//     nearest-upsampled halo) go straight from global memory to LDS with
//     global_load_lds_dwordx4 (gfx950), issued one step before they are
//     needed;
//   - pixels that are 2x2 averages (a low tile read from the dense map, or a
//     halo pixel across a resolution boundary) are loaded into registers,
//     averaged a step later and written to LDS;
//   - pixels outside the image are written as zeros.
// One barrier per step hands the buffers over.  It carries no memory fence,
// so the consumers' epilogue stores stay in flight while the next tile is
// computed.
//
// MFMA v_mfma_f32_16x16x32_{f16,bf16}: weights are the A operand (16 output
// channels), pixels the B operand (16 consecutive pixels of one tile row).
// One B fragment of input row r serves output rows r, r - 1 and r - 2 (taps
// ky = 0, 1, 2), so a wave reads each input row once per kx and K-step.
// The 16 A rows of channel block j are channels kg * 8 + j * 4 + {0..3} of
// the wave's 32 (kg = row / 4): a lane's results are 8 consecutive channels
// of one pixel, and one store instruction writes 64 contiguous bytes of each
// of 16 pixels.
//
// A tile pixel in LDS is 128 bytes = 8 sub-chunks of 16 bytes; sub-chunk q of
// the pixel in column v lives at position q ^ ((v >> 1) & 7), so the 16
// pixels of an MFMA operand read at one sub-chunk hit all 64 banks once, and
// a pixel's position does not depend on its row.  The weights never pass
// through LDS: each consumer lane loads its A fragments (16 bytes each)
// directly.
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
constexpr int NCW = 4;            // consumer waves
constexpr int NPW = 4;            // producer waves
constexpr int RWG = 64 * (NCW + NPW);
constexpr int PT = 64 * NPW;      // producer threads
constexpr int NBUF = 3;           // tile buffers

typedef __attribute__((address_space(3))) void* lds_ptr;

// One 16-byte global -> LDS copy per active lane; the wave's 64 lanes fill
// the 64 consecutive 16-byte slots starting at `window`.
__device__ __forceinline__ void dma16(const void* g, unsigned char* window) {
    __builtin_amdgcn_global_load_lds(g, (lds_ptr)window, 16, 0, 0);
}

// 16 zero bytes to LDS.  Written in assembly so that the compiler does not
// wait for the wave's pending LDS copies first (it cannot tell that they
// fill other bytes); the LDS-counter wait before the next barrier covers it.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ void lds_zero16(unsigned char* p) {
    const uint32_t a = (uint32_t)(uintptr_t)(lds_ptr)p;
    const u32x4 z = {0u, 0u, 0u, 0u};
    asm volatile("ds_write_b128 %0, %1" ::"v"(a), "v"(z) : "memory");
}

// q = p / d for 0 <= p < 4096 and 1 <= d <= 128: (p + 0.5) / d in fp32 is at
// least 0.5 / d away from an integer and its rounding error is below 2^-11,
// so truncation gives the exact quotient.
__device__ __forceinline__ int res_div(int p, float inv_d) { return (int)(((float)p + 0.5f) * inv_d); }

struct RTile {
    int n, gy, gx, high, slot, e, pe, r0, rows, in_px;
    float inv_pe;
};

// Tile `tile` of the list.  From packed or padded stacks the list is
// class-major: first the high blocks' tiles (Gh per block, R image rows
// each), then the low blocks' (Gl per block, RL = 2R low rows each: the same
// pixels as a high tile, so a low block costs a quarter of a high one; R/2
// rows when that spreads a second round over every workgroup, see the
// kernel), in slot order; nth = high tiles in the list.  From the dense map the list is
// block-major with RL = R/2 (Gh = Gl): a low tile's pixels are 2x2 averages
// of image pixels, staged through registers, and 2R rows of them take three
// rounds of loads where R/2 rows take one; the block of a tile is then its
// index over Gh, with no search for the n-th block of a class.
template <int SRC, int DST, bool ONE>
__device__ __forceinline__ bool res_tile(const Geo& g, const ConvArgs& a, const WaveMaskT<ONE>& wm, int R, int RL,
                                         int Gh, int Gl, int nth, int tile, RTile& t, Neigh& nb) {
    bool high;
    int slot, grp, k;
    if constexpr (SRC == SRC_DENSE) {
        // block-major: Gh == Gl tiles per block of either class, and no
        // search for the n-th block of a class
        k = tile / Gh;
        grp = tile - k * Gh;
        high = wm.high(k);
        slot = 0;
    } else {
        high = tile < nth;
        const int G = high ? Gh : Gl;
        const int q = high ? tile : tile - nth;
        slot = q / G;
        grp = q - slot * G;
        k = wm.find_nth(slot, high);
        if (k < 0) return false;
    }
    const int per = g.GH * g.GW;
    t.n = k / per;
    const int rem = k - t.n * per;
    t.gy = rem / g.GW;
    t.gx = rem - t.gy * g.GW;
    constexpr bool NEED_SLOTS = !(SRC == SRC_DENSE && DST == DST_DENSE);
    nb = wave_neighbourhood<NEED_SLOTS>(wm, g.GH, g.GW, t.n, t.gy, t.gx);
    t.high = high ? 1 : 0;
    t.slot = SRC == SRC_DENSE ? (NEED_SLOTS ? nb.slot[4] : 0) : slot;
    t.e = high ? g.bs : (g.bs >> 1);
    const int rr = high ? R : RL;
    t.r0 = grp * rr;
    if (t.r0 >= t.e) return false;
    t.rows = min(rr, t.e - t.r0);
    t.pe = t.e + 2;
    t.in_px = (t.rows + 2) * t.pe;
    t.inv_pe = 1.0f / (float)t.pe;
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
        const int ns = neigh_slot(nb, d);
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

// LDS slot (16-byte unit) of sub-chunk q of tile pixel (u, v): position
// q ^ ((v >> 1) & 7) inside the pixel's 128 bytes.  The 16 consecutive pixels
// of an MFMA operand then hit 16 distinct (parity of v, position) pairs, i.e.
// all 64 banks once, whatever the row.
__device__ __forceinline__ int tile_pos(int v, int q) { return q ^ ((v >> 1) & 7); }
__device__ __forceinline__ int tile_slot(int u, int v, int pe, int q) { return (u * pe + v) * RSUB + tile_pos(v, q); }

// How the interior (columns 1..e) of padded tile row u is filled: zeros,
// a contiguous copy of e pixels, a nearest upsampling of e/2 pixels (each
// used twice), or per-pixel items (2x2 averages) of the register path.
enum RowKind { ROW_ZERO = 0, ROW_COPY = 1, ROW_NEAR = 2, ROW_ITEMS = 3 };
struct RowSrc {
    int kind, which, off;  // which: base 0 or 1; off: element offset of the row's first interior pixel
};

template <int SRC>
__device__ __forceinline__ RowSrc row_src(const Geo& g, const ConvArgs& a, const Neigh& nb, const RTile& t, int u) {
    RowSrc S{ROW_ITEMS, 0, 0};
    const int C = a.C_in;
    if constexpr (SRC == SRC_PADDED) {
        S.kind = ROW_COPY;
        S.which = t.high ? 0 : 1;
        S.off = ((t.slot * t.pe + t.r0 + u) * t.pe + 1) * C;
        return S;
    }
    const int r = t.r0 + u - 1;  // block-local row
    const int dy = r < 0 ? 0 : (r >= t.e ? 2 : 1);
    const int d = dy * 3 + 1;    // the block above, the block itself, or the block below
    if constexpr (SRC == SRC_DENSE) {
        if (!t.high) return S;   // every pixel of a low tile is a 2x2 average
        const int Y = t.gy * g.bs + r;
        if ((unsigned)Y >= (unsigned)g.H) {
            S.kind = ROW_ZERO;
            return S;
        }
        if (!((nb.high >> d) & 1)) return S;  // a low neighbour row: averages
        S.kind = ROW_COPY;
        S.off = (Y * g.W + t.gx * g.bs) * C;
        return S;
    } else {
        if (!((nb.valid >> d) & 1)) {
            S.kind = ROW_ZERO;
            return S;
        }
        const int nhigh = (nb.high >> d) & 1;
        const int ns = neigh_slot(nb, dy * 3 + 1);
        if (ns >= (nhigh ? a.hi_cap : a.lo_cap)) {
            S.kind = ROW_ZERO;
            return S;
        }
        const int u2 = r - (dy - 1) * t.e;  // row inside that block
        if (nhigh == t.high) {
            S.kind = ROW_COPY;
            S.which = nhigh ? 0 : 1;
            S.off = (ns * t.e + u2) * t.e * C;
        } else if (t.high) {                // low neighbour of a high block: nearest upsampling
            const int lb = g.bs >> 1;
            S.kind = ROW_NEAR;
            S.which = 1;
            S.off = (ns * lb + (u2 >> 1)) * lb * C;
        }                                   // else a high neighbour of a low block: averages
        return S;
    }
}

// The register path of staging: every pixel of the two halo columns, and
// every interior pixel of the rows filled by items (all rows of a low tile
// read from the dense map; otherwise at most the top and the bottom row).
// An item is one 16-byte sub-chunk: zero, one load, or four loads averaged.
// Up to AV items per producer thread per batch; a batch's loads are issued
// in one step and written to LDS in the next.
constexpr int AV = 5;

template <typename T, int SRC>
struct ResAvg {
    uint4 v[AV][4];  // raw loaded data (kept packed until the value is formed)
    int slot[AV];    // LDS slot, -1 = none
    int kind[AV];    // 0 zero, 1 copy, 2 average

    struct Plan {
        bool all;     // every pixel of the tile
        int top, bot; // 1 if row 0 / row rows+1 is filled by items
        int n;        // items
    };
    __device__ __forceinline__ static Plan plan(const Geo& g, const ConvArgs& a, const Neigh& nb, const RTile& t) {
        Plan P{false, 0, 0, 0};
        if (SRC == SRC_DENSE && !t.high) {
            P.all = true;
            P.n = t.in_px * RSUB;
            return P;
        }
        P.top = row_src<SRC>(g, a, nb, t, 0).kind == ROW_ITEMS;
        P.bot = row_src<SRC>(g, a, nb, t, t.rows + 1).kind == ROW_ITEMS;
        P.n = (2 * (t.rows + 2) + t.e * (P.top + P.bot)) * RSUB;
        return P;
    }
    // item pixel h -> tile pixel (u, v)
    __device__ __forceinline__ static void item_pixel(const RTile& t, const Plan& P, int h, int& u, int& v) {
        if (P.all) {
            u = res_div(h, t.inv_pe);
            v = h - u * t.pe;
            return;
        }
        const int ring = 2 * (t.rows + 2);
        if (h < ring) {
            u = h >> 1;
            v = (h & 1) ? t.pe - 1 : 0;
            return;
        }
        h -= ring;
        const bool top = P.top && h < t.e;
        if (!top && P.top) h -= t.e;
        u = top ? 0 : t.rows + 1;
        v = 1 + h;
    }
    __device__ __forceinline__ void clear() {
#pragma unroll
        for (int i = 0; i < AV; ++i) slot[i] = -1;
    }
    __device__ __forceinline__ void issue(const Geo& g, const ConvArgs& a, const Neigh& nb, const RTile& t,
                                          const Plan& P, const T* base0, const T* base1, int base, int ptid) {
#pragma unroll
        for (int i = 0; i < AV; ++i) {
            slot[i] = -1;
            kind[i] = 0;
            const int it = base + i * PT + ptid;
            if (it < P.n) {
                int u, w;
                item_pixel(t, P, it >> 3, u, w);
                const int q = it & 7;
                slot[i] = tile_slot(u, w, t.pe, q);
                if (q * 8 < a.C_in) {
                    const RLoc L = res_loc<SRC>(g, a, nb, t, u, w, q * 8);
                    const T* p0 = (L.which ? base1 : base0) + L.off;
                    kind[i] = L.mode;
                    if (L.mode >= 1) v[i][0] = ld_nt16(p0);
                    if (L.mode == 2) {
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
            if (slot[i] >= 0) {
                uint4 val = uint4{0u, 0u, 0u, 0u};
                if (kind[i] == 1) val = v[i][0];
                else if (kind[i] == 2) val = avg4_raw<T>(v[i][0], v[i][1], v[i][2], v[i][3]);
                *reinterpret_cast<uint4*>(buf + slot[i] * 16) = val;
            }
    }
};

// First half of staging tile t into `buf` (producer waves, ptid = 0..PT-1):
// the interiors of copied rows by DMA, 8 pixels a window (a uniform source
// address plus a per-lane constant), zero rows, and the loads of the first
// batch of register items (held in av).  Nothing is waited for.
template <typename T, int SRC>
__device__ __forceinline__ void rw_issue(const Geo& g, const ConvArgs& a, const Neigh& nb, const RTile& t,
                                         unsigned char* buf, int ptid, ResAvg<T, SRC>& av) {
    const T *b0, *b1;
    res_bases<T, SRC>(g, a, t, b0, b1);
    const int lane = lane_id(), pwave = ptid >> 6, i = lane >> 3;
    const int C = a.C_in;
    const int wpr = t.e >> 3;  // windows per row interior
    // a wave takes whole rows (their source is found once per row)
    for (int u = pwave; u < t.rows + 2; u += NPW) {
        const RowSrc S = row_src<SRC>(g, a, nb, t, u);
        if (S.kind == ROW_ITEMS) continue;
        for (int k = 0; k < wpr; ++k) {
            const int v0 = 1 + 8 * k;                           // the window's first tile column
            const int q = (lane & 7) ^ (((v0 + i) >> 1) & 7);   // the sub-chunk this lane's slot holds
            unsigned char* win = buf + (u * t.pe + v0) * RROW;
            if (S.kind != ROW_ZERO && q * 8 < C) {
                const int px = S.kind == ROW_COPY ? 8 * k + i : ((8 * k + i) >> 1);
                dma16((S.which ? b1 : b0) + S.off + px * C + q * 8, win);
            } else {
                lds_zero16(win + lane * 16);
            }
        }
    }
    const typename ResAvg<T, SRC>::Plan P = ResAvg<T, SRC>::plan(g, a, nb, t);
    av.issue(g, a, nb, t, P, b0, b1, 0, ptid);
}

// Second half: waits for the tile's copies and first-batch loads, writes the
// averages (further batches are loaded and written here).  Returns with
// every LDS write of the tile issued; the caller waits for lgkmcnt.
template <typename T, int SRC>
__device__ __forceinline__ void rw_complete(const Geo& g, const ConvArgs& a, const Neigh& nb, const RTile& t,
                                            unsigned char* buf, int ptid, ResAvg<T, SRC>& av) {
    __builtin_amdgcn_s_waitcnt(0);
    av.commit(buf);
    const typename ResAvg<T, SRC>::Plan P = ResAvg<T, SRC>::plan(g, a, nb, t);
    if (P.n > PT * AV) {
        const T *b0, *b1;
        res_bases<T, SRC>(g, a, t, b0, b1);
        for (int base = PT * AV; base < P.n; base += PT * AV) {
            av.issue(g, a, nb, t, P, b0, b1, base, ptid);
            av.commit(buf);
        }
    }
}

// MFMA over one unit of a consumer wave's part of a tile of extent E (the
// 16-pixel column strip `strip`, M output rows from row0) and NKS 32-channel
// K-steps per tap, then the epilogue: bias, optional residual, optional
// ReLU, rounding, and the stores (2x2 nearest for a low block written to the
// dense map).
template <typename T, int DST, int E, int M, int NKS>
__device__ __forceinline__ void rw_compute(const Geo& g, const ConvArgs& a, const RTile& t, int strip, int row0,
                                           const unsigned char* buf, const typename MFR<T>::frag (&Wr)[9][NKS][2],
                                           const float (&bv)[2][4], int cobase, int vec_out, bool relu) {
    typedef MFR<T> mf;
    typedef typename mf::frag frag;
    constexpr int PE = E + 2, RB = PE * RROW;  // LDS bytes per padded tile row
    const int lane = lane_id(), l16 = lane & 15, kg = lane >> 4;

    floatx4 acc[M][2];
#pragma unroll
    for (int o = 0; o < M; ++o)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[o][j] = floatx4{0.f, 0.f, 0.f, 0.f};

    // The unit's B fragments in order (ks, kx, input row ir), each read from LDS
    // PD fragments ahead of its MFMAs.
    constexpr int NIR = M + 2, F = NKS * 3 * NIR;
    int pb[3];  // per-lane byte offset of input row 0 for kx = 0, 1, 2 (without the K-step)
#pragma unroll
    for (int kx = 0; kx < 3; ++kx) {
        const int col = strip * 16 + kx + l16;
        pb[kx] = (row0 * PE + col) * RROW + (tile_pos(col, kg) << 4);
    }
    auto load = [&](int f) -> frag {
        const int ks = f / (3 * NIR), kx = (f / NIR) % 3, ir = f % NIR;
        // sub-chunk ks * 4 + kg sits at position tile_pos(col, kg) ^ (4 * ks): the K-step
        // flips bit 2 of the position, i.e. XORs 64 into the byte offset
        return *reinterpret_cast<const frag*>(buf + ((pb[kx] ^ (ks << 6)) + ir * RB));
    };
    // ring of PD + 1 fragments: fragment f + PD is read while the MFMAs of f run
    constexpr int PD = M <= 2 ? 5 : 2;
    frag P[PD + 1];
#pragma unroll
    for (int f = 0; f < PD; ++f) P[f] = load(f);
    __builtin_amdgcn_sched_group_barrier(0x100, PD, 0);  // schedule: the first PD reads
#pragma unroll
    for (int f = 0; f < F; ++f) {
        if (f + PD < F) P[(f + PD) % (PD + 1)] = load(f + PD);
        const int ks = f / (3 * NIR), kx = (f / NIR) % 3, ir = f % NIR;
        int n = 0;
#pragma unroll
        for (int ky = 0; ky < 3; ++ky) {
            const int o = ir - ky;
            if (o >= 0 && o < M) {
                n += 2;
#pragma unroll
                for (int j = 0; j < 2; ++j) acc[o][j] = mf::mma(Wr[ky * 3 + kx][ks][j], P[f % (PD + 1)], acc[o][j]);
            }
        }
        // then, per fragment: the read PD ahead, and this fragment's MFMAs
        if (f + PD < F) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        if (n == 2) __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
        else if (n == 4) __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
        else __builtin_amdgcn_sched_group_barrier(0x008, 6, 0);
    }

    // -- epilogue: channels cobase + kg*8 + {0..7} of pixel (row0 + o, strip*16 + l16)
    const int Co = a.C_out;
    const int co = cobase + kg * 8;
    if (co >= Co) return;
    const bool full = vec_out && co + 8 <= Co;
    T* obase;  // the tile's block in its output stack, or the tile's image
    const T* rbase = nullptr;
    if constexpr (DST == DST_PACKED) {
        const size_t blk = (size_t)t.slot * E * E * Co;
        obase = (T*)(t.high ? a.out_hi : a.out_lo) + blk;
        const T* rb = (const T*)(t.high ? a.res_hi : a.res_lo);
        if (rb) rbase = rb + blk;
    } else {
        obase = (T*)a.out_hi + (size_t)t.n * g.H * g.W * Co;
    }
#pragma unroll
    for (int o = 0; o < M; ++o) {
        const int i = t.r0 + row0 + o, jx = strip * 16 + l16;  // block-local output pixel
        int off, down = 0;  // element offset of channel 0 of the pixel (the first of 2x2 for a low block)
        if constexpr (DST == DST_PACKED) {
            off = (i * E + jx) * Co;
        } else {
            const int Y = t.gy * g.bs + (t.high ? i : 2 * i), X = t.gx * g.bs + (t.high ? jx : 2 * jx);
            off = (Y * g.W + X) * Co;
            down = g.W * Co;
        }
        float f[8];
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 4; ++r) f[j * 4 + r] = acc[o][j][r] + bv[j][r];
        if (rbase) {
            if (full) {
                const Vec<T, 8> rv = vload<T, 8>(rbase + off + co);
#pragma unroll
                for (int e = 0; e < 8; ++e) f[e] += to_f32(rv.e[e]);
            } else {
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    if (co + e < Co) f[e] += to_f32(rbase[off + co + e]);
            }
        }
        Vec<T, 8> ov;
#pragma unroll
        for (int e = 0; e < 8; ++e) ov.e[e] = from_f32<T>(relu ? fmaxf(f[e], 0.0f) : f[e]);
        const int reps = (DST == DST_DENSE && !t.high) ? 2 : 1;
        for (int dy = 0; dy < reps; ++dy)
            for (int dx = 0; dx < reps; ++dx) {
                T* q = obase + off + dy * down + dx * Co + co;
                if (full) {
                    st_nt16(q, ov.raw);
                } else {
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        if (co + e < Co) q[e] = ov.e[e];
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
                                                     int RL, int Gh, int Gl, int buf_bytes, int vec_out) {
    typedef typename MFR<T>::frag frag;
    extern __shared__ __align__(16) unsigned char smem[];
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const bool producer = wave >= NCW;
    const int ptid = (int)threadIdx.x - 64 * NCW;
    const int lane = lane_id(), l16 = lane & 15, kg = lane >> 4;
    const int co0 = blockIdx.y * RNT;

    // consumer c: output channels co0 + 32 * (c & 1) + [0, 32), half (c >> 1) of every tile
    const int h = wave & 1, half = wave >> 1;
    const int cobase = co0 + 32 * h;
    const int cb = cobase + kg * 8;  // the first of this lane's 8 output channels
    const T* __restrict__ bias = (const T*)a.bias;
    Vec<T, 8> braw;                  // their bias, converted once the weights are in registers
    // A consumer loads its 32 x 9 x C_in weights straight into registers while
    // the producers plan and issue tile 0 (16 bytes per lane and fragment; the
    // LDS copy engine stays free for the tile).  Row m of channel block j of a
    // fragment is channel kg' * 8 + j * 4 + (m & 3) of the wave's 32 (kg' = m >> 2).
    frag Wr[9][NKS][2];
    if (!producer) {
        const T* __restrict__ wgt = (const T*)a.weight;
        const int co = cobase + (l16 >> 2) * 8 + (l16 & 3);
#pragma unroll
        for (int tap = 0; tap < 9; ++tap)
#pragma unroll
            for (int ks = 0; ks < NKS; ++ks)
#pragma unroll
                for (int j = 0; j < 2; ++j) {
                    const int c = co + j * 4, ci = (ks * 4 + kg) * 8;
                    if (c < a.C_out && ci < a.C_in)
                        Wr[tap][ks][j] = *reinterpret_cast<const frag*>(wgt + ((size_t)c * 9 + tap) * a.C_in + ci);
                    else
                        Wr[tap][ks][j] = frag{};
                }
        if (bias) {
            if (cb + 8 <= a.C_out && (reinterpret_cast<uintptr_t>(bias) & 15) == 0) {
                braw = vload<T, 8>(bias + cb);
            } else {
#pragma unroll
                for (int e = 0; e < 8; ++e) braw.e[e] = bias[min(cb + e, a.C_out - 1)];
            }
        }
    }
    WaveMaskT<ONE> wm;
    wm.init(mask, (int)g.B);

    // This workgroup's tiles are pos, pos + nwg, ...  Workgroups are spread
    // over the XCDs round-robin; pos numbers them XCD by XCD, so the tiles of
    // one block (which share halo rows) run on one XCD and share its L2.
    // The tile list by class (the class counts come from the mask; slots past
    // a stack's capacity are skipped).
    const int nwg = (int)gridDim.x;
    int nth = 0, ntiles = (int)g.B * Gh;  // the dense map: every block, block-major
    int rl = RL, gl = Gl;                 // rows and tiles of a low block
    if constexpr (SRC != SRC_DENSE) {
        const int nh_all = wm.count_high((int)g.B);
        const int nh = min(nh_all, a.hi_cap);
        const int nl = min((int)g.B - nh_all, a.lo_cap);
        nth = nh * Gh;
        ntiles = nth + nl * gl;
        // When the high tiles fit in one round and whole-block low tiles would
        // make a second round on a few workgroups, low tiles of R/2 rows (a
        // quarter of the work each) spread that round over every workgroup.
        const int gq = (g.bs >> 1) / (R >> 1);
        if (nl > 0 && nth <= nwg && ntiles > nwg && nth + nl * gq <= 2 * nwg) {
            rl = R >> 1;
            gl = gq;
            ntiles = nth + nl * gl;
        }
    }
    const int pos = (nwg & 7) ? (int)blockIdx.x : (int)(blockIdx.x & 7) * (nwg >> 3) + (int)(blockIdx.x >> 3);
    int tile = pos;
    auto next_tile = [&](RTile& t, Neigh& nb) -> bool {
        while (tile < ntiles) {
            const bool ok = res_tile<SRC, DST, ONE>(g, a, wm, R, rl, Gh, gl, nth, tile, t, nb);
            tile += nwg;
            if (ok) return true;
        }
        return false;
    };
    auto bufn = [&](int k) { return smem + (k == 0 ? 0 : (k == 1 ? buf_bytes : 2 * buf_bytes)); };

    // Step i: the consumers compute tile i (buffer i % 3) while the producers
    // complete tile i + 1 (buffer (i + 1) % 3: wait for its copies, write its
    // register items) and issue tile i + 2 (buffer (i + 2) % 3).
    // Before the loop:
    //   producers: issue tile 0, complete tile 0 | (0) | issue tile 1
    //   consumers: weights -> registers           | (0)
    // Both roles walk the same tile sequence and take one barrier before the
    // loop and one per step, so they leave together.  The roles have separate
    // loops so that the producers' in-flight items and the consumers' weights
    // do not compete for registers.
    RTile t0, t1;  // tiles i and i + 1
    Neigh nb0, nb1;
    bool h0 = next_tile(t0, nb0);
    bool h1 = h0 ? next_tile(t1, nb1) : false;
    if (producer) {
        ResAvg<T, SRC> av;
        av.clear();
        if (h0) rw_issue<T, SRC>(g, a, nb0, t0, bufn(0), ptid, av);
        if (h0) rw_complete<T, SRC>(g, a, nb0, t0, bufn(0), ptid, av);
        __builtin_amdgcn_s_waitcnt(0xC07F);        // lgkmcnt(0): tile 0's LDS writes are done
        res_barrier();                             // (0) tile 0 is staged, the weights are in registers
        if (h1) rw_issue<T, SRC>(g, a, nb1, t1, bufn(1), ptid, av);
        int b = 0;  // i % 3
        while (h0) {
            RTile t2;
            Neigh nb2;
            const bool h2 = h1 ? next_tile(t2, nb2) : false;
            const int b1 = b == NBUF - 1 ? 0 : b + 1, b2 = b1 == NBUF - 1 ? 0 : b1 + 1;
            if (h1) rw_complete<T, SRC>(g, a, nb1, t1, bufn(b1), ptid, av);
            if (h2) rw_issue<T, SRC>(g, a, nb2, t2, bufn(b2), ptid, av);
            __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this step's LDS writes are done
            res_barrier();
            h0 = h1;
            t1 = t2;
            nb1 = nb2;
            h1 = h2;
            b = b1;
        }
        __builtin_amdgcn_s_waitcnt(0);
        return;
    }

    const bool relu = (a.flags & 1) != 0;
    float bv[2][4];
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) bv[j][r] = (bias && cb + j * 4 + r < a.C_out) ? to_f32(braw.e[j * 4 + r]) : 0.0f;
    // All counters: the weight loads, and (for the compiler's wait tracking) nothing
    // pending on this path, which keeps the waits for the MFMA operands partial.
    __builtin_amdgcn_s_waitcnt(0);
    res_barrier();  // (0)

    int b = 0;
    while (h0) {
        RTile t2;
        Neigh nb2;
        const bool h2 = h1 ? next_tile(t2, nb2) : false;
        const unsigned char* buf = bufn(b);
        if (t0.high) {
            if (t0.e == 32) {  // 8 rows x 2 strips: strip `half`, two rows at a time
#pragma unroll 1
                for (int r = 0; r < 8; r += 2)
                    rw_compute<T, DST, 32, 2, NKS>(g, a, t0, half, r, buf, Wr, bv, cobase, vec_out, relu);
            } else {           // 4 rows x 4 strips: strips 2 * half and 2 * half + 1, two rows at a time
#pragma unroll 1
                for (int u = 0; u < 4; ++u)
                    rw_compute<T, DST, 64, 2, NKS>(g, a, t0, 2 * half + (u >> 1), 2 * (u & 1), buf, Wr, bv, cobase,
                                                   vec_out, relu);
            }
        } else if (t0.rows == 2 * R) {
            if (t0.e == 16) {  // 16 rows x 1 strip: rows 8 * half .. + 8, two at a time
#pragma unroll 1
                for (int r = 0; r < 8; r += 2)
                    rw_compute<T, DST, 16, 2, NKS>(g, a, t0, 0, 8 * half + r, buf, Wr, bv, cobase, vec_out, relu);
            } else {           // 8 rows x 2 strips: strip `half`, two rows at a time
#pragma unroll 1
                for (int r = 0; r < 8; r += 2)
                    rw_compute<T, DST, 32, 2, NKS>(g, a, t0, half, r, buf, Wr, bv, cobase, vec_out, relu);
            }
        } else {               // R/2 rows
            if (t0.e == 16) rw_compute<T, DST, 16, 2, NKS>(g, a, t0, 0, 2 * half, buf, Wr, bv, cobase, vec_out, relu);
            else rw_compute<T, DST, 32, 2, NKS>(g, a, t0, half, 0, buf, Wr, bv, cobase, vec_out, relu);
        }
        __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this tile's LDS reads are done
        res_barrier();
        (void)nb2;
        t0 = t1;
        h0 = h1;
        t1 = t2;
        h1 = h2;
        b = b == NBUF - 1 ? 0 : b + 1;
    }
}

inline bool aligned_to(const void* p, int bytes) { return (reinterpret_cast<uintptr_t>(p) & (bytes - 1)) == 0; }

// Image rows per high tile (a low tile has twice as many rows of half the
// width): 8 for blocks of 32, 4 for blocks of 64, so that every tile has 256
// output pixels and each consumer half is whole 16-pixel strips of whole
// rows; 0 = not supported.
int res_rows(int bs) { return bs == 32 ? 8 : (bs == 64 ? 4 : 0); }

int res_buf_bytes(int bs, int R) {
    const int lb = bs / 2;
    const int px_h = (R + 2) * (bs + 2), px_l = (2 * R + 2) * (lb + 2);
    return (px_h > px_l ? px_h : px_l) * RROW;
}

template <typename T, int SRC, int DST, bool ONE, int NKS>
hipError_t run_res(const Geo& g, const uint8_t* mask, const ConvArgs& a, int R, hipStream_t st) {
    const int RL = SRC == SRC_DENSE ? R / 2 : 2 * R;  // rows of a low tile (see res_tile)
    const int Gh = g.bs / R;                           // tiles per high block
    const int Gl = (g.bs / 2) / RL;                    // tiles per low block
    const long long ntiles = g.B * Gh;                 // at most (every block high)
    const int buf_bytes = res_buf_bytes(g.bs, R);
    const int smem = NBUF * buf_bytes;
    const int ob = 16;
    const int vec_out = (a.C_out % 8 == 0) && aligned_to(a.out_hi, ob) && aligned_to(a.out_lo, ob) &&
                        aligned_to(a.res_hi, ob) && aligned_to(a.res_lo, ob);
    hipError_t e = ensure_dyn_lds((const void*)k_conv_res<T, SRC, DST, ONE, NKS>, smem);
    if (e != hipSuccess) return e;
    const int cus = device_cus();
    const int nwg = (int)(ntiles < cus ? ntiles : cus);
    const dim3 grid((unsigned)nwg, (unsigned)((a.C_out + RNT - 1) / RNT));
    hipLaunchKernelGGL((k_conv_res<T, SRC, DST, ONE, NKS>), grid, dim3(RWG), smem, st, g, mask, a, R, RL, Gh, Gl,
                       buf_bytes, vec_out);
    return hipGetLastError();
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
    if (!aligned_to(a.in_hi, 16) || !aligned_to(a.in_lo, 16) || !aligned_to(a.weight, 16)) return false;
    return conv_res_fits_shape(dtype, layout, g, a);
}

bool conv_res_fits_shape(int dtype, int layout, const Geo& g, const ConvArgs& a) {
    if (layout != NHWC || (dtype != 1 && dtype != 2)) return false;
    // BlockPad with average sampling only: the alternatives go to the other kernels
    if ((a.flags >> 1) & 3) return false;
    if (a.C_in % 8 || a.C_in > 64 || res_rows(g.bs) == 0) return false;
    // element offsets inside one image or one stack are 32-bit
    const long long img = (long long)g.H * g.W * (a.C_in > a.C_out ? a.C_in : a.C_out);
    const long long cap = (a.hi_cap > a.lo_cap ? a.hi_cap : a.lo_cap) + 1LL;
    const long long stk = cap * (g.bs + 2) * (g.bs + 2) * (a.C_in > a.C_out ? a.C_in : a.C_out);
    if (img >= (1LL << 31) || stk >= (1LL << 31)) return false;
    // three tile buffers
    const int bb = res_buf_bytes(g.bs, res_rows(g.bs));
    return NBUF * bb <= 160 * 1024;
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
