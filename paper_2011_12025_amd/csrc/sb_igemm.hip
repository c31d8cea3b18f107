// Block convolutions of packed channels-last stacks as one implicit GEMM over
// the pixels of many blocks (the deeper layers of the encoder, where blocks
// shrink to a few pixels and the channel counts grow).
//
// GEMM view: rows = output pixels of one class's stack, in stack order (slot,
// row, column), so a workgroup tile spans as many blocks as it takes; columns
// = output channels; K = taps x input channels, walked in steps of one tap
// and 64 channels (128 bytes of every pixel and of every weight row).
//
// BlockPad is fused into the pixel gather.  At start-up a workgroup builds
// the block plan in LDS (for every block the number of high blocks before
// it, by a workgroup-wide scan of the mask) and then, for each of its tile
// pixels and taps, a source descriptor: a pixel of the high or the low stack
// (own block, same-resolution neighbour, the low neighbour's pixel
// nearest-upsampled, the top-left pixel of a high neighbour's cell with
// strided sampling), or zero (outside the image, a neighbour past its
// stack's capacity, zero padding).  A low block's halo across a resolution
// change with average sampling (the 2x2 average of a high neighbour's cell)
// comes from the low stack padded beforehand by the pad kernel, so every
// source is a plain copy.  Stride-2 and 1x1 convolutions only change which
// padded pixel a tap reads.
//
// Pipeline (three LDS stages): weights and pixels of step s+2 go global ->
// LDS by DMA (global_load_lds, 16 bytes per lane) while the MFMAs of step s
// run, so every wave issues the same number of DMAs per step and waits for
// step s+1 with a constant count.  Rows of 128 bytes carry an XOR swizzle of
// their 16-byte chunks so that the 16 rows read by one MFMA operand hit
// distinct banks.
//
// Split K: when the tiles alone do not fill the chip, the K steps of a tile
// are divided among several workgroups that write fp32 partial tiles to the
// caller's workspace; a second kernel sums them in split order
// (deterministic) and runs the epilogue.
//
// The grid has room for every slot below the stacks' capacities; the class
// counts are only known in the kernel, so each workgroup numbers the tiles
// that hold pixels (the high class's, then the low class's) from them and
// takes its M tile in that order; with room for surplus tiles the tile
// number is the slowest grid index, so the surplus workgroups are dispatched
// last and leave after the plan.
//
// MFMA: v_mfma_f32_16x16x32_{f16,bf16}, weights as A (16 output channels),
// pixels as B (16 pixels).  Eight waves (two per SIMD, so that one wave's
// address work overlaps the other's MFMAs) in a WM x (8 / WM) grid, each
// 16 x MS pixel and 16 x NS channel fragments.  The weight rows of each 32-channel group
// are permuted in LDS so that a lane ends with 8 consecutive output channels
// of one pixel and stores them as one 16-byte write.
#include <algorithm>
#include <utility>
#include <type_traits>

#include "sb_common.h"
#include "sb_kernels.h"
#include "sb_pixel.h"

namespace sb {

namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef _Float16 halfx8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) void* lds_ptr;

template <typename T> struct GMF;
template <> struct GMF<f16> {
    typedef halfx8 frag;
    static __device__ __forceinline__ floatx4 mma(frag a, frag b, floatx4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
    }
};
template <> struct GMF<bf16> {
    typedef bf16x8 frag;
    static __device__ __forceinline__ floatx4 mma(frag a, frag b, floatx4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
    }
};

constexpr int GROWB = 128;     // LDS bytes per row: 64 channels of one pixel / one weight row
constexpr int GKC = 64;        // channels per K step
constexpr int GWAVES = 8;      // waves per workgroup
constexpr int GWG = 64 * GWAVES;
constexpr int GNST = 3;        // LDS stages
constexpr int GMAXB = 8192;    // blocks whose plan fits the LDS table
constexpr int GMAXC = 4096;    // input channels the zero row covers

// A row of zeros that pixels outside the image are copied from; device
// globals start zeroed and this one is never written.
__device__ __align__(16) uint4 g_zero_row[GMAXC * 2 / 16];

// source descriptor: kind in bits 30..31, pixel index (in its stack) below.
// A low tile that reads the input's high stack at half resolution
// (ConvArgs::in_hs) has no full-resolution high source: GK_HI then indexes
// that stack.
constexpr uint32_t GK_HI = 0u, GK_LO = 1u, GK_ZERO = 3u;
__device__ __forceinline__ uint32_t gdesc(uint32_t kind, int pix) { return (kind << 30) | (uint32_t)pix; }

// byte offset of 16-byte chunk q of LDS row r (XOR swizzle, see above)
__device__ __forceinline__ int gsw(int r, int q) { return r * GROWB + ((q ^ ((r >> 1) & 7)) << 4); }

// output channel held by LDS weight row r of a tile (within its 32-row group:
// row 16h + l, l = 4 kg + i, holds channel 8 kg + 4 h + i)
__device__ __forceinline__ int gperm(int r) {
    const int l = r & 15;
    return (r & ~31) + (l >> 2) * 8 + ((r >> 4) & 1) * 4 + (l & 3);
}

// s_waitcnt operand that waits until at most n vector-memory operations are
// outstanding (lgkm and export counts left alone)
constexpr unsigned gvm_wait(int n) { return 0x0F70u | (unsigned)(n & 0xF) | ((unsigned)(n >> 4) << 14); }

// Workgroup barrier without the memory fences of __syncthreads (which would
// wait for the DMAs of the step after next): LDS writes are waited for here,
// DMAs by the explicit count before it.
__device__ __forceinline__ void gbarrier() {
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

__device__ __forceinline__ void gdma16(const void* g, unsigned char* window) {
    __builtin_amdgcn_global_load_lds(g, (lds_ptr)window, 16, 0, 0);
}

// DMA of one step's weight rows: wrow[j] points at this lane's chunk of its
// weight row, off selects the tap and the 64 channels.
template <typename T, int AR>
__device__ __forceinline__ void gissue_a(const T* const (&wrow)[AR], unsigned char* st, int off, int wave) {
#pragma unroll
    for (int j = 0; j < AR; ++j) gdma16(wrow[j] + off, st + (wave * AR + j) * 1024);
}

// This lane's pixel-row sources of one tap, decoded once per tap: a pointer
// to chunk pq of the source row (the zero row for pixels outside the
// image).  A step then only adds its channel offset.
template <typename T, int BR>
struct GRows {
    const T* p[BR];
};

template <typename T, int BR>
__device__ __forceinline__ void gdecode(const uint32_t (&dsc)[BR], const int (&pq)[BR], const T* __restrict__ in_hi,
                                        const T* __restrict__ in_lo, const T* zrow, int C_in, GRows<T, BR>& r) {
#pragma unroll
    for (int j = 0; j < BR; ++j) {
        const uint32_t d = dsc[j];
        const uint32_t kind = d >> 30;
        const T* base = kind == GK_LO ? in_lo : (kind == GK_ZERO ? zrow : in_hi);
        const size_t pix = kind != GK_ZERO ? (size_t)(d & 0x3FFFFFFFu) : 0;
        r.p[j] = base + pix * C_in + pq[j];
    }
}

// DMA of one step's pixel rows: channel offset c of every row.
template <typename T, int BR>
__device__ __forceinline__ void gissue_b(const GRows<T, BR>& r, int c, unsigned char* st, int wave) {
#pragma unroll
    for (int j = 0; j < BR; ++j) gdma16(r.p[j] + c, st + (wave * BR + j) * 1024);
}

// This lane's pixel-row descriptors of one tap, held in registers for the
// steps of that tap.
template <int BR>
__device__ __forceinline__ void gload_desc(const uint32_t* s_desc, const int (&prow)[BR], int KT, int tap,
                                           uint32_t (&dsc)[BR]) {
#pragma unroll
    for (int j = 0; j < BR; ++j) dsc[j] = s_desc[prow[j] * KT + tap];
}

// N DMAs of zeros into a stage that no step reads (keeps the count per step constant)
template <typename T, int N>
__device__ __forceinline__ void gissue_pad(const T* zrow, unsigned char* st, int wave, int lane) {
#pragma unroll
    for (int j = 0; j < N; ++j) gdma16(zrow + (lane & 7) * 8, st + (wave * N + j) * 1024);
}

struct GParams {
    int eo_h, eo_l; // output extents
    int cpt;        // K steps per tap (C_in / 64)
    int tiles;      // M tiles of the grid (both classes)
    int tiles_n;    // output-channel tiles
    int tile_major; // grid order: 1 = M tile slowest, 0 = M tile fastest
    int splits;     // workgroups sharing the K steps of a tile
    float* part;    // fp32 partial tiles [tile][n tile][split][TM * TN] when splits > 1
    int* rows;      // per M tile, written when splits > 1: valid output rows of its class's stack and its
                    // tile number in that class (-1 - number for the low class)
    const void* lo_pad;  // the low stack with its 1-pixel halo [lo_cap][lb+2][lb+2][C_in], or nullptr
    // Dense mode (a whole layer): the high blocks' pixels come from the dense
    // map a.in_hi [N][H][W][C_in] (the low neighbours' from lo_pad, which the
    // low tiles read too), and the results go to the dense map a.out_hi
    // [N][H][W][C_out], a low pixel to its 2 x 2 cell (BlockCombine).
    int dense;
    int W;          // dense mode: width of the map
    int* dout;      // per M tile, TM dense output pixels (-1: none), written when splits > 1
    int hs_lg;      // log2 of the high output extent when the epilogue writes a.out_hs, else -1
};

// The store of 8 finished channels of one output pixel: row m of the class's
// output stack, or (dense mode, dpix >= 0) pixel dpix of the dense output
// map, a low pixel to its 2 x 2 cell (map width W).
template <typename T>
__device__ __forceinline__ void gstore8(T* out, int m, int dpix, int W, int high, int C_out, int co,
                                        const uint4& v) {
    if (dpix < 0) {
        *reinterpret_cast<uint4*>(out + (size_t)m * C_out + co) = v;
        return;
    }
    T* q = out + (size_t)dpix * C_out + co;
    *reinterpret_cast<uint4*>(q) = v;
    if (!high) {
        *reinterpret_cast<uint4*>(q + C_out) = v;
        *reinterpret_cast<uint4*>(q + (size_t)W * C_out) = v;
        *reinterpret_cast<uint4*>(q + (size_t)(W + 1) * C_out) = v;
    }
}

template <typename T>
__device__ __forceinline__ Vec<T, 8> gsel(bool c, const Vec<T, 8>& x, const Vec<T, 8>& y) {
    Vec<T, 8> r;
    r.raw.x = c ? x.raw.x : y.raw.x;
    r.raw.y = c ? x.raw.y : y.raw.y;
    r.raw.z = c ? x.raw.z : y.raw.z;
    r.raw.w = c ? x.raw.w : y.raw.w;
    return r;
}

template <typename T, int MS, int ms>
__device__ __forceinline__ void gsample_one(const Vec<T, 8> (&o)[MS], int mbase, int rows_valid, int l16, int lg,
                                            T* hs, int C_out, int co) {
    const int eo = 1 << lg, eh = eo >> 1;
    const int vstep = eo >> 4;  // fragment step of the row below (eo >= 16)
    // values selected per component, fragments by fixed index (a select
    // between array elements would put the array in scratch memory)
    const Vec<T, 8> down = gsel(eo == 16, o[ms ^ 1], o[(ms ^ 2) % MS]);
    const Vec<T, 8> right = vshfl_xor(o[ms], 1);
    const Vec<T, 8> below = gsel(eo <= 8, vshfl_xor(o[ms], eo), down);
    const Vec<T, 8> diag = vshfl_xor(gsel(eo <= 8, o[ms], down), eo <= 8 ? (eo | 1) : 1);
    const int m = mbase + ms * 16 + l16;
    const bool top = eo <= 8 ? (l16 & eo) == 0 : (ms & vstep) == 0;
    if (m < rows_valid && (l16 & 1) == 0 && top) {
        const int slot = m >> (2 * lg), rem = m & (eo * eo - 1);
        const int i = rem >> lg, j = rem & (eo - 1);
        const size_t idx = ((size_t)slot * eh + (i >> 1)) * eh + (j >> 1);
        *reinterpret_cast<uint4*>(hs + idx * C_out + co) = vavg4<T, 8>(o[ms], right, below, diag).raw;
    }
}

template <typename T, int MS, int... I>
__device__ __forceinline__ void gsample_seq(std::integer_sequence<int, I...>, const Vec<T, 8> (&o)[MS], int mbase,
                                            int rows_valid, int l16, int lg, T* hs, int C_out, int co) {
    (gsample_one<T, MS, I>(o, mbase, rows_valid, l16, lg, hs, C_out, co), ...);
}

// The 2x2 averages of a finished high tile (its blocks at half resolution,
// ConvArgs::out_hs), from the rounded results o[ms] of 8 channels (co..) of
// pixel rows mbase + 16 ms + l16.  Rows of a block of extent eo = 2^lg are
// row-major, and a 16-row group starts a block row, so the cell of a pixel
// at even (i, j) has its right partner in lane ^ 1 and the row below in
// lane ^ eo for eo <= 8, in fragment ms ^ 1 for eo = 16 and in ms ^ 2 for
// eo = 32 (MS = 4).  Every lane takes part in every shuffle (partners lie in
// the lane's own group of 16, all valid or all past rows_valid together).
template <typename T, int MS>
__device__ __forceinline__ void gsample(const Vec<T, 8> (&o)[MS], int mbase, int rows_valid, int l16, int lg, T* hs,
                                        int C_out, int co) {
    gsample_seq<T, MS>(std::make_integer_sequence<int, MS>{}, o, mbase, rows_valid, l16, lg, hs, C_out, co);
}

// Bias, residual, ReLU and the store of a finished tile: lane holds channels
// co0 + wn*NS*16 + jj*32 + kg*8 + 0..7 of pixel row m0 + wm*MS*16 + ms*16 + l16.
// dout: dense mode, the dense output pixel of each tile pixel (else nullptr).
// hs: a high tile's half-resolution output (gsample; lg = log2 of the block
// extent), or nullptr.
template <typename T, int WM, int MS, int NS>
__device__ __forceinline__ void gepilogue(const floatx4 (&acc)[MS][NS], const ConvArgs& a, int high, int m0,
                                          int rows_valid, int co0, const int* dout, int W, T* hs, int lg) {
    const int lane = (int)threadIdx.x & 63, wave = (int)threadIdx.x >> 6;
    const int wm = wave % WM, wn = wave / WM, l16 = lane & 15, kg = lane >> 4;
    const int C_out = a.C_out;
    const T* __restrict__ bias = (const T*)a.bias;
    const T* __restrict__ res = (const T*)(high ? a.res_hi : a.res_lo);
    T* __restrict__ out = (T*)(high ? a.out_hi : a.out_lo);
    const bool relu = (a.flags & 1) != 0;
#pragma unroll
    for (int jj = 0; jj < NS / 2; ++jj) {
        const int co = co0 + wn * NS * 16 + jj * 32 + kg * 8;
        if (co >= C_out) continue;
        float bv[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) bv[i] = bias ? to_f32(bias[co + i]) : 0.0f;
        if (!hs) {  // (uniform) the plain stores
#pragma unroll
            for (int ms = 0; ms < MS; ++ms) {
                const int m = m0 + wm * MS * 16 + ms * 16 + l16;
                if (m >= rows_valid) continue;
                float f[8];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    f[i] = acc[ms][2 * jj][i] + bv[i];
                    f[4 + i] = acc[ms][2 * jj + 1][i] + bv[4 + i];
                }
                const size_t off = (size_t)m * C_out + co;
                if (res) {
                    Vec<T, 8> rv;
                    rv.raw = *reinterpret_cast<const uint4*>(res + off);
#pragma unroll
                    for (int i = 0; i < 8; ++i) f[i] += to_f32(rv.e[i]);
                }
                Vec<T, 8> o;
#pragma unroll
                for (int i = 0; i < 8; ++i) o.e[i] = from_f32<T>(relu ? fmaxf(f[i], 0.0f) : f[i]);
                gstore8<T>(out, m, dout ? dout[m - m0] : -1, W, high, C_out, co, o.raw);
            }
            continue;
        }
        // with the half-resolution output: every lane computes every fragment
        // (the cell's partners are taken by shuffles), stores where valid
        Vec<T, 8> o[MS];
#pragma unroll
        for (int ms = 0; ms < MS; ++ms) {
            const int m = m0 + wm * MS * 16 + ms * 16 + l16;
            const bool valid = m < rows_valid;
            float f[8];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                f[i] = acc[ms][2 * jj][i] + bv[i];
                f[4 + i] = acc[ms][2 * jj + 1][i] + bv[4 + i];
            }
            const size_t off = (size_t)m * C_out + co;
            if (res && valid) {
                Vec<T, 8> rv;
                rv.raw = *reinterpret_cast<const uint4*>(res + off);
#pragma unroll
                for (int i = 0; i < 8; ++i) f[i] += to_f32(rv.e[i]);
            }
#pragma unroll
            for (int i = 0; i < 8; ++i) o[ms].e[i] = from_f32<T>(relu ? fmaxf(f[i], 0.0f) : f[i]);
            if (valid) gstore8<T>(out, m, dout ? dout[m - m0] : -1, W, high, C_out, co, o[ms].raw);
        }
        gsample<T, MS>(o, m0 + wm * MS * 16, rows_valid, l16, lg, hs, C_out, co);
    }
}

// fp32 partial tile of one split: fragment (ms, ns) of a wave is 64 lanes x 16 bytes, contiguous
template <int TILE, int MS, int NS>
__device__ __forceinline__ size_t gpart_off(int tile_lin, int split, int splits, int wave, int ms, int ns, int lane) {
    return ((size_t)tile_lin * splits + split) * TILE + ((size_t)((wave * MS + ms) * NS + ns) * 64 + lane) * 4;
}

template <typename T, int KS, int ST, int WM, int MS, int NS>
__global__ __launch_bounds__(GWG, 1) void k_igemm(Geo g, const uint8_t* __restrict__ mask, ConvArgs a, GParams gp) {
    typedef GMF<T> mf;
    typedef typename mf::frag frag;
    constexpr int KT = KS * KS;
    constexpr int WN = GWAVES / WM;
    constexpr int TM = WM * MS * 16, TN = WN * NS * 16;
    constexpr int A_BYTES = TN * GROWB, B_BYTES = TM * GROWB, STAGE = A_BYTES + B_BYTES;
    constexpr int BR = TM / (8 * GWAVES);   // pixel rows of 8 per wave per step (one DMA each)
    constexpr int AR = TN / (8 * GWAVES);   // weight rows of 8 per wave per step
    static_assert(BR >= 1 && AR >= 1 && NS % 2 == 0, "tile shape");
    extern __shared__ __align__(16) unsigned char smem[];
    unsigned char* s_stage = smem;
    uint32_t* s_desc = reinterpret_cast<uint32_t*>(smem + GNST * STAGE);
    int* s_pij = reinterpret_cast<int*>(smem + GNST * STAGE + TM * KT * 4);
    int* s_dout = s_pij + TM;  // dense mode: output pixel of each tile pixel
    uint16_t* s_hb = reinterpret_cast<uint16_t*>(smem + GNST * STAGE + TM * KT * 4 + 2 * TM * 4);
    // Start-up tables in the third stage, which no DMA touches before the
    // main loop: the block of each slot of this workgroup's class (uint16),
    // then for each block of the tile its nine neighbour sources (uint32).
    unsigned char* s_tmp = s_stage + 2 * STAGE;
    __shared__ int s_wsum[GWAVES];

    const int tid = (int)threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: LDS windows are scalar addresses
    const int B = (int)g.B;
    // Workgroup lin = (M tile, channel tile, split).  When the stacks have
    // room for more blocks than the mask can fill, the M tile is the slowest
    // index, so that the surplus workgroups are dispatched last; otherwise
    // the fastest, so that the channel tiles and splits of a tile, which
    // share its pixels, run on one XCD when the tile count is a multiple of 8
    // (workgroups go to the XCDs round-robin).
    const int lin = (int)blockIdx.x, per_tile = gp.tiles_n * gp.splits;
    int tx, rq;
    if (gp.tile_major) {
        tx = lin / per_tile;
        rq = lin - tx * per_tile;
    } else {
        rq = lin / gp.tiles;
        tx = lin - rq * gp.tiles;
    }
    const int ny = gp.tile_major ? rq / gp.splits : rq - (rq / gp.tiles_n) * gp.tiles_n;
    const int co0 = ny * TN;
    const int C_in = a.C_in, C_out = a.C_out;
    const int cpt = gp.cpt;
    const int nsteps = KT * cpt;
    const int z = gp.tile_major ? rq - ny * gp.splits : rq / gp.tiles_n;
    const int s_first = z * nsteps / gp.splits;
    const int n = (z + 1) * nsteps / gp.splits - s_first;  // steps of this workgroup (>= 1)
    const T* zrow = reinterpret_cast<const T*>(g_zero_row);

    // the mask byte of the thread's first block
    const int per = (B + GWG - 1) / GWG;
    const int k0 = tid * per;
    const uint8_t mv0 = mask[min(k0, B - 1)];  // the thread's first block (in bounds for every thread)

    // this lane's DMA rows and chunks: LDS slot (lane & 7) of row r holds global chunk (lane & 7) ^ ((r >> 1) & 7)
    const T* wrow[AR];
#pragma unroll
    for (int j = 0; j < AR; ++j) {
        const int r = (wave * AR + j) * 8 + (lane >> 3);
        const int co = min(co0 + gperm(r), C_out - 1);
        wrow[j] = (const T*)a.weight + (size_t)co * KT * C_in + (((lane & 7) ^ ((r >> 1) & 7)) * 8);
    }
    const int tap0 = s_first / cpt, c0 = s_first - (s_first / cpt) * cpt;
    int tap1 = tap0, c1 = c0 + 1;
    if (c1 == cpt) { c1 = 0; ++tap1; }
    const int hk0 = k0 < B && mv0 != 0;
    // The weights of steps 0 and 1 do not depend on the mask: they land while
    // the plan and the descriptors are built.  (Issued after the mask byte is
    // in: a wait for it would otherwise wait for them too.)
    gissue_a<T, AR>(wrow, s_stage, tap0 * C_in + c0 * GKC, wave);
    if (n > 1) gissue_a<T, AR>(wrow, s_stage + STAGE, tap1 * C_in + c1 * GKC, wave);
    else gissue_pad<T, AR>(zrow, s_stage + STAGE, wave, lane);

    // ---- block plan: s_hb[k] = high blocks before k (k = 0..B), and the
    // block of every slot of this workgroup's class
    uint16_t* s_inv = reinterpret_cast<uint16_t*>(s_tmp);
    int high, mt, nh_eff, nl_eff;
    bool surplus;
    {
        int c = hk0;
        for (int i = 1; i < per; ++i) c += k0 + i < B && mask[k0 + i] != 0;
        int x = c;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const int y = __shfl_up(x, d, 64);
            if (lane >= d) x += y;
        }
        if (lane == 63) s_wsum[wave] = x;
        gbarrier();
        int run = x - c, nh_all = 0;
        for (int w = 0; w < GWAVES; ++w) {
            if (w < wave) run += s_wsum[w];
            nh_all += s_wsum[w];
        }
        // This workgroup's tile, from the class counts: the filled tiles of
        // the high class come first, then those of the low class, and the
        // grid's surplus (room for blocks that the mask does not have) last.
        nh_eff = min(nh_all, a.hi_cap);
        nl_eff = min(B - nh_all, a.lo_cap);
        const int real_h = (int)(((long long)nh_eff * gp.eo_h * gp.eo_h + TM - 1) / TM);
        const int real_l = (int)(((long long)nl_eff * gp.eo_l * gp.eo_l + TM - 1) / TM);
        high = tx < real_h;
        mt = high ? tx : tx - real_h;
        surplus = !high && mt >= real_l;
        for (int i = 0; i < per; ++i) {
            const int k = k0 + i;
            if (k < B) {
                const bool hk = i == 0 ? hk0 != 0 : mask[k] != 0;
                s_hb[k] = (uint16_t)run;
                if (hk == (high != 0)) s_inv[hk ? run : k - run] = (uint16_t)k;
                run += hk;
            }
        }
        if (tid == GWG - 1) s_hb[B] = (uint16_t)run;
        gbarrier();
    }
    const int eo = high ? gp.eo_h : gp.eo_l;
    const int eo2 = eo * eo;
    const int rows_valid = surplus ? 0 : (high ? nh_eff : nl_eff) * eo2;
    const int m0 = mt * TM;
    if (gp.splits > 1 && ny == 0 && z == 0 && tid == 0) {
        gp.rows[2 * tx] = rows_valid;
        gp.rows[2 * tx + 1] = high ? mt : -1 - mt;
    }
    if (m0 >= rows_valid) {  // uniform over the workgroup; no DMA may still be writing LDS at exit
        __builtin_amdgcn_s_waitcnt(0);
        return;
    }
    const int bs = g.bs, lb = bs >> 1;
    const int e_in = high ? bs : lb;

    int prow[BR], pq[BR];
#pragma unroll
    for (int j = 0; j < BR; ++j) {
        prow[j] = (wave * BR + j) * 8 + (lane >> 3);
        pq[j] = ((lane & 7) ^ ((prow[j] >> 1) & 7)) * 8;
    }
    // a low tile reads the padded low stack when there is one (uniform); in
    // dense mode the high tiles' low neighbours come from it too
    const bool lpad = !high && gp.lo_pad != nullptr;
    const bool dense = gp.dense != 0;
    const T* __restrict__ in_lo = (lpad || dense) ? (const T*)gp.lo_pad : (const T*)a.in_lo;
    // a low tile takes a high neighbour's halo cells (average sampling) from
    // the input's high stack at half resolution when the caller gives it, and
    // then reads nothing else of the high stack: its GK_HI sources index that
    const int pm = pad_mode(a.flags);
    const bool hsrc = !high && a.in_hs != nullptr && pm == PM_AVG;
    const T* __restrict__ in_hi = (const T*)(hsrc ? a.in_hs : a.in_hi);

    // ---- source descriptors.  First, at once: the position of each tile pixel
    // (one thread each), and the nine neighbour sources of each block of the
    // tile (kind and slot: own block, neighbour block of either class, or
    // zero; one (block, direction) per thread beyond the first TM).
    const int slot0 = m0 / eo2;
    const int nblk = (min(m0 + TM, rows_valid) - 1) / eo2 - slot0 + 1;  // blocks the tile touches (<= TM + 1)
    uint32_t* s_nb = reinterpret_cast<uint32_t*>(s_tmp + ((2 * B + 15) & ~15));
    int* s_nbase = reinterpret_cast<int*>(s_nb + nblk * 9);  // dense mode: top-left pixel of each block of the tile
    if (tid < TM) {  // each tile pixel: its block among the tile's blocks, row, column
        const int m = m0 + tid;
        int pij = -1;
        if (m < rows_valid) {
            const int slot = m / eo2;
            const int rem = m - slot * eo2;
            const int i = rem / eo;
            pij = ((slot - slot0) << 22) | (i << 11) | (rem - i * eo);
        }
        s_pij[tid] = pij;
    } else if (!lpad || dense) {
        const int per_img = g.GH * g.GW;
        for (int e = tid - TM; e < nblk * 9; e += GWG - TM) {
            const int b = e / 9, d = e - (e / 9) * 9;
            const int dy = d / 3 - 1, dx = d - (d / 3) * 3 - 1;
            const int slot = slot0 + b;
            const int k = s_inv[slot];
            const int nn = k / per_img;
            const int r = k - nn * per_img;
            const int gy = r / g.GW, gx = r - (r / g.GW) * g.GW;
            const int ny = gy + dy, nx = gx + dx;
            const bool inside = ny >= 0 && ny < g.GH && nx >= 0 && nx < g.GW;
            const int k2 = inside ? (nn * g.GH + ny) * g.GW + nx : k;  // both reads in bounds, no branch
            const int before = s_hb[k2];
            const int h2 = (int)s_hb[k2 + 1] - before;
            const int s2 = h2 ? before : k2 - before;
            uint32_t ent = gdesc(GK_ZERO, 0);
            if (d == 4 && dense) s_nbase[b] = (nn * g.H + gy * bs) * g.W + gx * bs;
            if (d == 4) ent = gdesc(high ? GK_HI : GK_LO, slot);
            else if (pm != PM_ZERO && inside && s2 < (h2 ? a.hi_cap : a.lo_cap))  // zero padding: halo stays zero
                ent = gdesc(h2 ? GK_HI : GK_LO, s2);
            s_nb[e] = ent;
        }
    }
    gbarrier();
    // Then a descriptor per (tile pixel, tap), spread over the workgroup; a
    // thread reads the records of all its entries before it uses any.
    constexpr int NIT = (TM * KT + GWG - 1) / GWG;
    int pijv[NIT];
    uint32_t nbv[NIT];
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
        const int idx = tid + it * GWG;
        pijv[it] = idx < TM * KT ? s_pij[idx / KT] : -1;
    }
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
        const int idx = tid + it * GWG, t = idx - (idx / KT) * KT;
        const int pij = pijv[it];
        const int b = pij >> 22, i = (pij >> 11) & 2047, j = pij & 2047;
        const int uu = ST * i + t / KS - KS / 2, vv = ST * j + (t - (t / KS) * KS) - KS / 2;
        const int dy = uu < 0 ? -1 : (uu >= e_in ? 1 : 0);
        const int dx = vv < 0 ? -1 : (vv >= e_in ? 1 : 0);
        nbv[it] = (pij >= 0 && !lpad) ? s_nb[b * 9 + (dy + 1) * 3 + dx + 1] : gdesc(GK_ZERO, 0);
    }
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
        const int idx = tid + it * GWG;
        if (idx >= TM * KT) break;
        const int t = idx - (idx / KT) * KT;
        const int pij = pijv[it];
        uint32_t ds = gdesc(GK_ZERO, 0);
        if (pij >= 0) {
            const int b = pij >> 22, i = (pij >> 11) & 2047, j = pij & 2047;
            const int ky = t / KS, kx = t - (t / KS) * KS;
            const int uu = ST * i + ky - KS / 2, vv = ST * j + kx - KS / 2;
            if (lpad) {  // a low tile over the padded low stack: every source is a copy
                ds = gdesc(GK_LO, ((slot0 + b) * (lb + 2) + uu + 1) * (lb + 2) + vv + 1);
            } else {
                const int dy = uu < 0 ? -1 : (uu >= e_in ? 1 : 0);
                const int dx = vv < 0 ? -1 : (vv >= e_in ? 1 : 0);
                const uint32_t e = nbv[it];
                const uint32_t kind = e >> 30;
                const int s2 = (int)(e & 0x3FFFFFFFu);
                const int u2 = uu - dy * e_in, v2 = vv - dx * e_in;
                if (kind != GK_ZERO && dense) {  // a high tile: dense pixels, or a low neighbour's padded pixel
                    if (kind == GK_HI) ds = gdesc(GK_HI, s_nbase[b] + uu * g.W + vv);
                    else ds = gdesc(GK_LO, (s2 * (lb + 2) + (u2 >> 1) + 1) * (lb + 2) + (v2 >> 1) + 1);
                } else if (kind != GK_ZERO) {
                    if ((kind == GK_HI) == (high != 0)) ds = gdesc(kind, (s2 * e_in + u2) * e_in + v2);
                    else if (high) ds = gdesc(GK_LO, (s2 * lb + (u2 >> 1)) * lb + (v2 >> 1));
                    // a low block beside a high one: average sampling reads the
                    // cell's average from the half-resolution high stack (without
                    // it the low stack is padded beforehand, see igemm_plan),
                    // strided sampling the cell's top-left pixel
                    else if (hsrc) ds = gdesc(GK_HI, (s2 * lb + u2) * lb + v2);
                    else ds = gdesc(GK_HI, (s2 * bs + 2 * u2) * bs + 2 * v2);
                }
            }
        }
        s_desc[idx] = ds;
    }
    if (dense && tid < TM) {  // the dense output pixel of each tile pixel (a low one: its cell's top left)
        const int pij = s_pij[tid];
        int o = -1;
        if (pij >= 0) {
            const int b = pij >> 22, i = (pij >> 11) & 2047, j = pij & 2047;
            o = s_nbase[b] + (high ? i * g.W + j : 2 * i * g.W + 2 * j);
        }
        s_dout[tid] = o;
        if (gp.splits > 1 && ny == 0 && z == 0) gp.dout[tx * TM + tid] = o;
    }
    gbarrier();

    // ---- prologue: pixels of steps 0 and 1 (their weights went out at entry)
    uint32_t dsc[BR];
    GRows<T, BR> r0, rA, rB;  // pixel-row sources of steps 0 / s + 1 / s + 2
    gload_desc<BR>(s_desc, prow, KT, tap0, dsc);
    gdecode<T, BR>(dsc, pq, in_hi, in_lo, zrow, C_in, r0);
    gload_desc<BR>(s_desc, prow, KT, tap1 < KT ? tap1 : tap0, dsc);
    gdecode<T, BR>(dsc, pq, in_hi, in_lo, zrow, C_in, rA);
    gissue_b<T, BR>(r0, c0 * GKC, s_stage + A_BYTES, wave);
    if (n > 1) gissue_b<T, BR>(rA, c1 * GKC, s_stage + STAGE + A_BYTES, wave);
    else gissue_pad<T, BR>(zrow, s_stage + STAGE + A_BYTES, wave, lane);
    // step 0 has landed once only step 1's pixels can be outstanding
    __builtin_amdgcn_s_waitcnt(gvm_wait(BR));
    gbarrier();

    floatx4 acc[MS][NS];
#pragma unroll
    for (int ms = 0; ms < MS; ++ms)
#pragma unroll
        for (int ns = 0; ns < NS; ++ns) acc[ms][ns] = floatx4{0.f, 0.f, 0.f, 0.f};

    const int wm = wave % WM, wn = wave / WM;
    const int l16 = lane & 15, kg = lane >> 4;
    // (tap, chunk) of step s + 2
    int tb = tap1, cb = c1 + 1;
    if (cb == cpt) { cb = 0; ++tb; }
    gload_desc<BR>(s_desc, prow, KT, tb < KT ? tb : tap0, dsc);
    gdecode<T, BR>(dsc, pq, in_hi, in_lo, zrow, C_in, rB);
    int b_cur = 0;

    for (int s = 0; s < n; ++s) {
        unsigned char* cur = s_stage + b_cur * STAGE;
        const int b1 = b_cur == GNST - 1 ? 0 : b_cur + 1;
        const int b2 = b1 == GNST - 1 ? 0 : b1 + 1;
        // every fragment of the step is read first, so that the LDS latency
        // runs under the DMA issue of step s + 2 instead of between MFMAs
        frag af[2][NS], bf[2][MS];
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
            for (int ns = 0; ns < NS; ++ns)
                af[ks][ns] = *reinterpret_cast<const frag*>(cur + gsw(wn * NS * 16 + ns * 16 + l16, ks * 4 + kg));
#pragma unroll
            for (int ms = 0; ms < MS; ++ms)
                bf[ks][ms] =
                    *reinterpret_cast<const frag*>(cur + A_BYTES + gsw(wm * MS * 16 + ms * 16 + l16, ks * 4 + kg));
        }
        __builtin_amdgcn_sched_barrier(0);
        if (s + 2 < n) {
            gissue_a<T, AR>(wrow, s_stage + b2 * STAGE, tb * C_in + cb * GKC, wave);
            gissue_b<T, BR>(rB, cb * GKC, s_stage + b2 * STAGE + A_BYTES, wave);
        } else {
            gissue_pad<T, AR + BR>(zrow, s_stage + b2 * STAGE, wave, lane);
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
#pragma unroll
            for (int ms = 0; ms < MS; ++ms)
#pragma unroll
                for (int ns = 0; ns < NS; ++ns) acc[ms][ns] = mf::mma(af[ks][ns], bf[ks][ms], acc[ms][ns]);
        __builtin_amdgcn_sched_barrier(0);
        // step s + 1 has landed once only step s + 2's DMAs can be outstanding
        __builtin_amdgcn_s_waitcnt(gvm_wait(AR + BR));
        gbarrier();
        b_cur = b1;
        rA = rB;
        if (++cb == cpt) {  // a new tap: its sources (read a step before they are used)
            cb = 0;
            ++tb;
            if (tb < KT) {
                gload_desc<BR>(s_desc, prow, KT, tb, dsc);
                gdecode<T, BR>(dsc, pq, in_hi, in_lo, zrow, C_in, rB);
            }
        }
    }
    __builtin_amdgcn_s_waitcnt(0);  // the padding DMAs

    if (gp.splits == 1) {
        gepilogue<T, WM, MS, NS>(acc, a, high, m0, rows_valid, co0, dense ? s_dout : nullptr, g.W,
                                 high && gp.hs_lg >= 0 ? (T*)a.out_hs : nullptr, gp.hs_lg);
    } else {
        const int tile_lin = tx * gp.tiles_n + ny;
#pragma unroll
        for (int ms = 0; ms < MS; ++ms)
#pragma unroll
            for (int ns = 0; ns < NS; ++ns)
                *reinterpret_cast<floatx4*>(gp.part + gpart_off<TM * TN, MS, NS>(tile_lin, z, gp.splits, wave, ms, ns,
                                                                                lane)) = acc[ms][ns];
    }
}

// Sums the split partial tiles in split order and runs the epilogue.  One
// thread per (tile, wave, ms, ns pair, lane) of the multiply kernel, so the
// whole grid shares the work; a thread holds 8 consecutive output channels
// of one pixel, exactly as the multiply kernel's lane does.  Consecutive
// waves take the ns pairs of a fragment (their stores fill whole lines),
// except with the half-resolution output (a.out_hs): the MS fragments of a
// (wave, ns pair) are then consecutive waves of one workgroup, so that a
// 2x2 cell's four pixels can come from LDS: the right neighbour is thread
// ^ 1, the row below thread ^ eo for eo <= 8, the next fragment's wave
// (thread ^ 64) for eo = 16 and the one after (thread ^ 128) for eo = 32
// (MS = 4).
template <typename T, int WM, int MS, int NS>
__global__ __launch_bounds__(256) void k_igemm_reduce(ConvArgs a, GParams gp, int tiles, int tiles_n) {
    constexpr int WN = GWAVES / WM;
    constexpr int TM = WM * MS * 16, TN = WN * NS * 16;
    constexpr int PER_TILE = GWAVES * MS * (NS / 2) * 64;
    static_assert(PER_TILE % 256 == 0, "a workgroup stays in one tile");
    __shared__ uint4 s_o[256];
    const long long gid = (long long)blockIdx.x * 256 + threadIdx.x;
    if (gid >= (long long)tiles * tiles_n * PER_TILE) return;  // whole workgroups
    const int tile_lin = (int)(gid / PER_TILE);
    int r = (int)(gid - (long long)tile_lin * PER_TILE);
    const int lane = r & 63;
    r >>= 6;
    int ms, jj;
    if (gp.hs_lg >= 0) {
        ms = r % MS;
        r /= MS;
        jj = r % (NS / 2);
        r /= (NS / 2);
    } else {
        jj = r % (NS / 2);
        r /= (NS / 2);
        ms = r % MS;
        r /= MS;
    }
    const int wave = r;
    const int tx = tile_lin / tiles_n, ty = tile_lin - tx * tiles_n;
    const int rows_valid = gp.rows[2 * tx];
    const int code = gp.rows[2 * tx + 1];
    const int high = code >= 0;
    const int m0 = (high ? code : -1 - code) * TM;
    const int wm = wave % WM, wn = wave / WM, l16 = lane & 15, kg = lane >> 4;
    const int m = m0 + wm * MS * 16 + ms * 16 + l16;
    const int co = ty * TN + wn * NS * 16 + jj * 32 + kg * 8;
    Vec<T, 8> o;
    o.raw = uint4{0u, 0u, 0u, 0u};
    if (m < rows_valid && co < a.C_out) {
        floatx4 lo = *reinterpret_cast<const floatx4*>(
            gp.part + gpart_off<TM * TN, MS, NS>(tile_lin, 0, gp.splits, wave, ms, 2 * jj, lane));
        floatx4 hi = *reinterpret_cast<const floatx4*>(
            gp.part + gpart_off<TM * TN, MS, NS>(tile_lin, 0, gp.splits, wave, ms, 2 * jj + 1, lane));
        for (int z = 1; z < gp.splits; ++z) {
            lo += *reinterpret_cast<const floatx4*>(
                gp.part + gpart_off<TM * TN, MS, NS>(tile_lin, z, gp.splits, wave, ms, 2 * jj, lane));
            hi += *reinterpret_cast<const floatx4*>(
                gp.part + gpart_off<TM * TN, MS, NS>(tile_lin, z, gp.splits, wave, ms, 2 * jj + 1, lane));
        }
        const T* __restrict__ bias = (const T*)a.bias;
        const T* __restrict__ res = (const T*)(high ? a.res_hi : a.res_lo);
        T* __restrict__ out = (T*)(high ? a.out_hi : a.out_lo);
        const bool relu = (a.flags & 1) != 0;
        float f[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            f[i] = lo[i] + (bias ? to_f32(bias[co + i]) : 0.0f);
            f[4 + i] = hi[i] + (bias ? to_f32(bias[co + 4 + i]) : 0.0f);
        }
        const size_t off = (size_t)m * a.C_out + co;
        if (res) {
            Vec<T, 8> rv;
            rv.raw = *reinterpret_cast<const uint4*>(res + off);
#pragma unroll
            for (int i = 0; i < 8; ++i) f[i] += to_f32(rv.e[i]);
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) o.e[i] = from_f32<T>(relu ? fmaxf(f[i], 0.0f) : f[i]);
        gstore8<T>(out, m, gp.dense ? gp.dout[tx * TM + (m - m0)] : -1, gp.W, high, a.C_out, co, o.raw);
    }
    if (gp.hs_lg >= 0 && high) {  // uniform over the workgroup (one tile)
        const int lg = gp.hs_lg, eo = 1 << lg, eh = eo >> 1;
        const int t = (int)threadIdx.x;
        s_o[t] = o.raw;
        __syncthreads();
        const int tb = eo <= 8 ? t ^ eo : t ^ (64 * (eo >> 4));  // the row below
        const bool top = eo <= 8 ? (l16 & eo) == 0 : (ms & (eo >> 4)) == 0;
        if (m < rows_valid && co < a.C_out && (l16 & 1) == 0 && top) {
            Vec<T, 8> rt, bl, dg;
            rt.raw = s_o[t ^ 1];
            bl.raw = s_o[tb];
            dg.raw = s_o[tb ^ 1];
            const int slot = m >> (2 * lg), rem = m & (eo * eo - 1);
            const int i = rem >> lg, j = rem & (eo - 1);
            const size_t idx = ((size_t)slot * eh + (i >> 1)) * eh + (j >> 1);
            *reinterpret_cast<uint4*>((T*)a.out_hs + idx * a.C_out + co) = vavg4<T, 8>(o, rt, bl, dg).raw;
        }
    }
}

}  // namespace

namespace {

// Launch cost model, in 128 x 128 K steps (about 0.65 us each, measured):
// a workgroup's start-up (launch spread, mask plan, descriptors, first
// stages: about 6.5 us), and the partial-sum pass, which reads every split's
// partial tiles.
constexpr int GSTART_COST = 10;
constexpr int GSPLIT_COST = 12;  // plus one per split

inline bool galigned(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }
inline size_t ground256(size_t b) { return (b + 255) / 256 * 256; }

template <int TM, int TN, int KT>
constexpr int igemm_smem_fixed() {
    return GNST * (TM + TN) * GROWB + TM * KT * 4 + 2 * TM * 4;
}

inline int igemm_hb_bytes(const Geo& g) { return (((int)g.B + 1) * 2 + 15) / 16 * 16; }

// Widest workgroup tile for these shapes: 64 output channels for narrow
// layers, 256 from 256 channels on (eight 64 x 64 wave tiles: a third fewer
// LDS reads per MAC than 128) when its LDS fits, else 128.
inline int igemm_tn(const Geo& g, const ConvArgs& a) {
    if (a.C_out <= 64) return 64;
    if (a.C_out >= 256 && igemm_smem_fixed<128, 256, 9>() + igemm_hb_bytes(g) + GWAVES * 4 <= 160 * 1024) return 256;
    return 128;
}

// The 256 x 128 workgroup tile (eight 64 x 64 wave tiles over 256 pixel rows)
// when its LDS fits: three 48 KB stages and a descriptor table twice as long.
inline bool igemm_tm256_fits(const Geo& g, int ks) {
    const int fixed = ks == 3 ? igemm_smem_fixed<256, 128, 9>() : igemm_smem_fixed<256, 128, 1>();
    return fixed + igemm_hb_bytes(g) + GWAVES * 4 <= 160 * 1024;
}

// Everything about a launch that the host decides from the shapes alone:
// tile counts (from the stack capacities), the K split, the padded low stack,
// and the caller's workspace that they take.
struct IgPlan {
    int TM, TN, tiles_h, tiles_l, tiles_n, splits;
    bool pad_low;
    size_t part_bytes, pad_bytes;
};

IgPlan igemm_plan(const Geo& g, const ConvArgs& a, int ks, int stride, bool dense = false) {
    IgPlan p;
    const int eo_h = g.bs / stride, eo_l = (g.bs / 2) / stride;
    auto tiles_of = [&](int TM, long long nh, long long nl) {
        return (nh * eo_h * eo_h + TM - 1) / TM + (nl * eo_l * eo_l + TM - 1) / TM;
    };
    // The work the cost model sees: the tiles that hold pixels under the
    // worst mask.  With room for every block in both classes (the fused
    // layer's packed route) the grid has twice the tiles any mask fills; the
    // surplus workgroups leave after the plan.
    const long long nh_max = std::min<long long>(a.hi_cap, g.B);
    const long long nh_min = std::max<long long>(0, g.B - a.lo_cap);
    auto work_of = [&](int TM) {
        auto filled = [&](long long nh) { return tiles_of(TM, nh, std::min<long long>(g.B - nh, a.lo_cap)); };
        return std::min<long long>(tiles_of(TM, a.hi_cap, a.lo_cap),
                                   std::max(filled(nh_max), filled(std::min(nh_min, nh_max))));
    };
    // Workgroup tile and split K by a cost model in units of one 128 x 128 K
    // step: one workgroup per CU at a time (LDS), so a launch costs about
    // rounds x (steps per split x step cost + start-up); a 128 x 256 or
    // 256 x 128 step (eight 64 x 64 wave tiles) does twice the MACs at about
    // 1.5 times the cost; a split adds the partial-sum pass, which grows
    // with the partial tiles it reads.  Take the cheapest choice that keeps at
    // least four steps per workgroup (ties: the first of 128 x 256, 128 x 128,
    // 256 x 128).
    const int cus = device_cus();
    const int nsteps = ks * ks * (a.C_in / GKC);
    const int tn_max = igemm_tn(g, a);
    // (not in dense mode: there the wider tile measured slower at half low)
    const bool tm256 = !dense && a.C_out >= 128 && igemm_tm256_fits(g, ks);
    double best = -1.0;
    p.TM = 128;
    p.TN = tn_max;
    p.splits = 1;
    for (int cand = 0; cand < 4; ++cand) {
        int TM = 128, tn;
        if (cand < 3) {
            tn = tn_max >> cand;
            if (cand > 0 && (tn < 128 || tn_max <= 128)) continue;
        } else {
            if (!tm256) continue;
            TM = 256;
            tn = 128;
        }
        const int tiles_n = (a.C_out + tn - 1) / tn;
        const bool wide = tn == 256 || TM == 256;
        const double w = wide ? 1.5 : 1.0, wr = wide ? 2.0 : 1.0;
        const long long wgs = work_of(TM) * tiles_n;
        for (int c = 1; c <= 16 && (c == 1 || nsteps / c >= 4); ++c) {
            const long long rounds = (wgs * c + cus - 1) / cus;
            const double cost = (double)rounds * ((nsteps + c - 1) / c * w + GSTART_COST) +
                                (c > 1 ? GSPLIT_COST + c * wr : 0.0);
            if (best < 0.0 || cost < best) {
                best = cost;
                p.TM = TM;
                p.TN = tn;
                p.splits = c;
            }
        }
    }
    p.tiles_h = (int)(((long long)a.hi_cap * eo_h * eo_h + p.TM - 1) / p.TM);
    p.tiles_l = (int)(((long long)a.lo_cap * eo_l * eo_l + p.TM - 1) / p.TM);
    const int tiles = p.tiles_h + p.tiles_l;
    p.tiles_n = (a.C_out + p.TN - 1) / p.TN;
    if (tiles == 0) p.splits = 1;
    // A low block's halo across a resolution change, with average sampling, is
    // the 2x2 average of a high neighbour's cell: a 3 x 3 convolution with
    // both classes pads the low stack once beforehand (BlockPad of the low
    // blocks, one extra launch), so that every source of the K loop is a plain
    // copy.  (Averaging in the K loop instead measured 6-12 us slower at the
    // ResNet-18 stage shapes with 25 % low blocks or 128 channels, within
    // 3 us either way elsewhere.)
    // In dense mode the padded low stack comes straight from the dense map and
    // the high tiles read their low neighbours from it as well.
    p.pad_low = dense || (ks == 3 && p.tiles_l > 0 && a.hi_cap > 0 && pad_mode(a.flags) == PM_AVG && !a.in_hs);
    p.part_bytes = p.splits > 1 ? ground256((size_t)tiles * p.tiles_n * p.splits * p.TM * p.TN * 4 + (size_t)tiles * 8 +
                                            (dense ? (size_t)tiles * p.TM * 4 : 0))
                                : 0;
    p.pad_bytes = p.pad_low ? ground256((size_t)a.lo_cap * (g.bs / 2 + 2) * (g.bs / 2 + 2) * a.C_in * 2) : 0;
    return p;
}

template <typename T, int KS, int ST, int WM, int MS, int NS>
hipError_t igemm_run(const Geo& g, const uint8_t* mask, const ConvArgs& a, Ws ws, hipStream_t st, bool dense) {
    constexpr int TM = WM * MS * 16, TN = (GWAVES / WM) * NS * 16;
    const IgPlan pl = igemm_plan(g, a, KS, ST, dense);
    if (pl.TM != TM || pl.TN != TN) return hipErrorInvalidValue;
    const int tiles = pl.tiles_h + pl.tiles_l;
    if (tiles == 0) return hipSuccess;
    if (ws.bytes < pl.part_bytes + pl.pad_bytes || (pl.part_bytes + pl.pad_bytes > 0 && !ws.p))
        return hipErrorInvalidValue;  // the entry points check the workspace before anything is launched
    GParams gp;
    gp.eo_h = g.bs / ST;
    gp.eo_l = (g.bs / 2) / ST;
    gp.cpt = a.C_in / GKC;
    const int smem = igemm_smem_fixed<TM, TN, KS * KS>() + igemm_hb_bytes(g);
    hipError_t e = ensure_dyn_lds((const void*)k_igemm<T, KS, ST, WM, MS, NS>, smem);
    if (e != hipSuccess) return e;
    const int tiles_n = pl.tiles_n;
    const int S = pl.splits;
    gp.splits = S;
    gp.tiles = tiles;
    gp.tiles_n = tiles_n;
    gp.tile_major = (long long)a.hi_cap + a.lo_cap > g.B;  // room for surplus tiles
    gp.part = nullptr;
    gp.rows = nullptr;
    gp.lo_pad = nullptr;
    gp.dense = dense ? 1 : 0;
    gp.W = g.W;
    gp.dout = nullptr;
    // the half-resolution output from the epilogue when a 2x2 cell's pixels
    // lie in one wave (see gsample), else from launch_sample_hs afterwards
    const int eo_h = gp.eo_h;
    const bool hs_epi = a.out_hs != nullptr && !dense && eo_h >= 2 && (eo_h & (eo_h - 1)) == 0 &&
                        (eo_h <= 16 || (eo_h == 32 && MS == 4));
    gp.hs_lg = hs_epi ? __builtin_ctz((unsigned)eo_h) : -1;
    if (S > 1) {
        gp.part = (float*)ws.p;
        gp.rows = (int*)((char*)ws.p + (size_t)tiles * tiles_n * S * TM * TN * 4);  // 2 ints per tile
        gp.dout = gp.rows + 2 * tiles;                                              // dense mode: TM per tile
    }
    if (pl.pad_low) {
        void* lp = (char*)ws.p + pl.part_bytes;
        Geo pg = g;
        pg.C = a.C_in;
        const int dt = std::is_same<T, f16>::value ? 1 : 2;
        e = dense ? launch_pad_low_dense(dt, pg, a.in_hi, mask, lp, a.lo_cap, st)
                  : launch_pad_rows(dt, pg, a.in_hi, a.in_lo, mask, nullptr, lp, a.hi_cap, a.lo_cap, PM_AVG, st);
        if (e != hipSuccess) return e;
        gp.lo_pad = lp;
    }
    const dim3 grid((unsigned)((long long)tiles * tiles_n * S));
    hipLaunchKernelGGL((k_igemm<T, KS, ST, WM, MS, NS>), grid, dim3(GWG), smem, st, g, mask, a, gp);
    if (S > 1) {
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        const long long threads = (long long)tiles * tiles_n * GWAVES * MS * (NS / 2) * 64;
        hipLaunchKernelGGL((k_igemm_reduce<T, WM, MS, NS>), dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, st, a,
                           gp, tiles, tiles_n);
    }
    if (a.out_hs && !hs_epi && !dense) {
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        return launch_sample_hs(std::is_same<T, f16>::value ? 1 : 2, a.out_hi, a.hi_cap, eo_h, a.C_out, a.out_hs, st);
    }
    return hipGetLastError();
}

template <typename T, int KS, int ST>
hipError_t igemm_tile(const Geo& g, const uint8_t* mask, const ConvArgs& a, Ws ws, hipStream_t st,
                      bool dense = false) {
    const IgPlan pl = igemm_plan(g, a, KS, ST, dense);
    const int tn = pl.TN;
    if (pl.TM == 256) return igemm_run<T, KS, ST, 4, 4, 4>(g, mask, a, ws, st, dense);
    if (tn == 64) return igemm_run<T, KS, ST, 4, 2, 2>(g, mask, a, ws, st, dense);
    if (tn == 256) return igemm_run<T, KS, ST, 2, 4, 4>(g, mask, a, ws, st, dense);
    return igemm_run<T, KS, ST, 2, 4, 2>(g, mask, a, ws, st, dense);
}

template <typename T>
hipError_t igemm_t(const Geo& g, const uint8_t* mask, const ConvArgs& a, int ks, int stride, Ws ws,
                   hipStream_t st) {
    if (ks == 3)
        return stride == 1 ? igemm_tile<T, 3, 1>(g, mask, a, ws, st) : igemm_tile<T, 3, 2>(g, mask, a, ws, st);
    return stride == 1 ? igemm_tile<T, 1, 1>(g, mask, a, ws, st) : igemm_tile<T, 1, 2>(g, mask, a, ws, st);
}

}  // namespace

bool igemm_fits_shape(int dtype, int layout, const Geo& g, const ConvArgs& a) {
    if (layout != NHWC || (dtype != 1 && dtype != 2)) return false;
    if (a.C_in % GKC || a.C_in > GMAXC || a.C_out % 8 || g.B > GMAXB || g.bs > 2048) return false;
    // pixel indices of the stacks fit the 30 bits of a descriptor
    const long long lb = g.bs / 2;
    if ((long long)a.hi_cap * g.bs * g.bs >= (1LL << 30) || (long long)a.lo_cap * (lb + 2) * (lb + 2) >= (1LL << 30))
        return false;
    const int smem = igemm_smem_fixed<128, 128, 9>() + igemm_hb_bytes(g);
    return smem + GWAVES * 4 <= 160 * 1024;
}

bool igemm_fits(int dtype, int layout, const Geo& g, const ConvArgs& a) {
    if (!galigned(a.in_hi) || !galigned(a.in_lo) || !galigned(a.weight) || !galigned(a.out_hi) ||
        !galigned(a.out_lo) || !galigned(a.res_hi) || !galigned(a.res_lo) || !galigned(a.in_hs) ||
        !galigned(a.out_hs))
        return false;
    return igemm_fits_shape(dtype, layout, g, a);
}

size_t igemm_ws_bytes(const Geo& g, const ConvArgs& a, int ksize, int stride) {
    const IgPlan p = igemm_plan(g, a, ksize, stride);
    return p.part_bytes + p.pad_bytes;
}

hipError_t launch_igemm(int dtype, const Geo& g, const uint8_t* mask, const ConvArgs& a, int ksize, int stride, Ws ws,
                        hipStream_t st) {
    if (dtype == 1) return igemm_t<f16>(g, mask, a, ksize, stride, ws, st);
    return igemm_t<bf16>(g, mask, a, ksize, stride, ws, st);
}

bool igemm_dense_fits(int dtype, int layout, const Geo& g, const ConvArgs& a) {
    // the dense pixel indices fit a descriptor; blocks tile the map exactly;
    // average sampling (the padded low stack is then the dense map's 2x2 averages)
    if (g.H % g.bs || g.W % g.bs || (long long)g.N * g.H * g.W >= (1LL << 30) || pad_mode(a.flags) != PM_AVG)
        return false;
    ConvArgs p = a;
    p.hi_cap = p.lo_cap = (int)g.B;
    return igemm_fits_shape(dtype, layout, g, p);
}

size_t igemm_dense_ws_bytes(const Geo& g, const ConvArgs& a) {
    ConvArgs p = a;
    p.hi_cap = p.lo_cap = (int)g.B;
    const IgPlan pl = igemm_plan(g, p, 3, 1, true);
    return pl.part_bytes + pl.pad_bytes;
}

hipError_t launch_igemm_dense(int dtype, const Geo& g, const uint8_t* mask, const ConvArgs& a, Ws ws, hipStream_t st) {
    ConvArgs p = a;
    p.in_lo = nullptr;
    p.out_lo = a.out_hi;  // one dense output map for both classes
    p.res_hi = p.res_lo = nullptr;
    p.hi_cap = p.lo_cap = (int)g.B;
    if (dtype == 1) return igemm_tile<f16, 3, 1>(g, mask, p, ws, st, true);
    return igemm_tile<bf16, 3, 1>(g, mask, p, ws, st, true);
}

}  // namespace sb
