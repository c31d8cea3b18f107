// Internal device helpers of libsegblocks: storage types, fp32 conversions,
// raw vector memory access, the 2x2 average and the block-plan primitives
// (wavefront counting of high blocks).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sb {

typedef _Float16 f16;
typedef __bf16 bf16;

enum Layout { NCHW = 0, NHWC = 1 };

constexpr int WG = 256;  // threads per workgroup in every kernel

// ---------------------------------------------------------------------------
// fp32 <-> storage type.  Widening is exact; narrowing is the hardware
// round-to-nearest-even conversion (v_cvt_f16_f32 / v_cvt_pk_bf16_f32), with
// fp16 subnormals preserved (the kernels run with denormals enabled).
// ---------------------------------------------------------------------------
__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(f16 v) { return (float)v; }
__device__ __forceinline__ float to_f32(bf16 v) { return (float)v; }

template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ f16 from_f32<f16>(float v) { return (f16)v; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float v) { return (bf16)v; }

// 2x2 average in the library's fixed fp32 association: ((a + b) + (c + d)) * 0.25
// where a, b are the top and c, d the bottom pixels of the cell.
template <typename T>
__device__ __forceinline__ T avg4(T a, T b, T c, T d) {
    const float s = (to_f32(a) + to_f32(b)) + (to_f32(c) + to_f32(d));
    return from_f32<T>(s * 0.25f);
}

// ---------------------------------------------------------------------------
// Vectors of V storage elements moved as one raw load/store (V*sizeof(T) is
// 2, 4, 8 or 16 bytes; the address must be aligned to that size).
// ---------------------------------------------------------------------------
template <int BYTES> struct RawT;
template <> struct RawT<2> { typedef uint16_t type; };
template <> struct RawT<4> { typedef uint32_t type; };
template <> struct RawT<8> { typedef uint2 type; };
template <> struct RawT<16> { typedef uint4 type; };

template <typename T, int V>
struct Vec {
    static_assert(V >= 1, "vector width");
    union {
        typename RawT<(int)sizeof(T) * V>::type raw;
        T e[V];
    };
};
template <typename T>
struct Vec<T, 1> {
    T e[1];
};

template <typename T, int V>
__device__ __forceinline__ Vec<T, V> vload(const T* p) {
    Vec<T, V> v;
    if constexpr (V == 1) {
        v.e[0] = *p;
    } else {
        v.raw = *reinterpret_cast<const typename RawT<(int)sizeof(T) * V>::type*>(p);
    }
    return v;
}

template <typename T, int V>
__device__ __forceinline__ void vstore(T* p, const Vec<T, V>& v) {
    if constexpr (V == 1) {
        *p = v.e[0];
    } else {
        *reinterpret_cast<typename RawT<(int)sizeof(T) * V>::type*>(p) = v.raw;
    }
}

// Streaming (non-temporal) 16-byte loads and stores.  Data that is read or
// written once per kernel goes through these: on MI355X ordinary loads of
// streamed data reached about a third of the bandwidth of the non-temporal
// form (measured: ~1.9 vs ~5.8 TB/s into LDS).
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 ld_nt16(const void* p) {
    const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
    return uint4{v.x, v.y, v.z, v.w};
}
__device__ __forceinline__ void st_nt16(void* p, uint4 v) {
    const u32x4_t w = {v.x, v.y, v.z, v.w};
    __builtin_nontemporal_store(w, reinterpret_cast<u32x4_t*>(p));
}
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ void st_nt8(void* p, uint2 v) {
    const u32x2_t w = {v.x, v.y};
    __builtin_nontemporal_store(w, reinterpret_cast<u32x2_t*>(p));
}

template <typename T, int V>
__device__ __forceinline__ Vec<T, V> vzero() {
    Vec<T, V> v;
#pragma unroll
    for (int i = 0; i < V; ++i) v.e[i] = from_f32<T>(0.0f);
    return v;
}

// The 16-byte vector of lane (lane ^ mask) of the wave.
template <typename T>
__device__ __forceinline__ Vec<T, 8> vshfl_xor(const Vec<T, 8>& v, int mask) {
    Vec<T, 8> r;
    r.raw.x = (uint32_t)__shfl_xor((int)v.raw.x, mask, 64);
    r.raw.y = (uint32_t)__shfl_xor((int)v.raw.y, mask, 64);
    r.raw.z = (uint32_t)__shfl_xor((int)v.raw.z, mask, 64);
    r.raw.w = (uint32_t)__shfl_xor((int)v.raw.w, mask, 64);
    return r;
}

template <typename T, int V>
__device__ __forceinline__ Vec<T, V> vavg4(const Vec<T, V>& a, const Vec<T, V>& b,
                                           const Vec<T, V>& c, const Vec<T, V>& d) {
    Vec<T, V> r;
#pragma unroll
    for (int i = 0; i < V; ++i) r.e[i] = avg4(a.e[i], b.e[i], c.e[i], d.e[i]);
    return r;
}

// The transposes for the backward pass: the 2x2 cell sum ((a + b) + (c + d))
// (BlockCombine's nearest upsampling transposed) and a quarter of a value
// (BlockSample's average transposed), in fp32, rounded once.
template <typename T, int V>
__device__ __forceinline__ Vec<T, V> vsum4(const Vec<T, V>& a, const Vec<T, V>& b,
                                           const Vec<T, V>& c, const Vec<T, V>& d) {
    Vec<T, V> r;
#pragma unroll
    for (int i = 0; i < V; ++i)
        r.e[i] = from_f32<T>((to_f32(a.e[i]) + to_f32(b.e[i])) + (to_f32(c.e[i]) + to_f32(d.e[i])));
    return r;
}
template <typename T, int V>
__device__ __forceinline__ Vec<T, V> vquarter(const Vec<T, V>& a) {
    Vec<T, V> r;
#pragma unroll
    for (int i = 0; i < V; ++i) r.e[i] = from_f32<T>(to_f32(a.e[i]) * 0.25f);
    return r;
}

// ---------------------------------------------------------------------------
// Wavefront primitives and the block plan
//
// The plan (class and slot of a block, the block of a slot) is computed by
// every wave from the mask itself: each lane loads 16 mask bytes per
// 1024-block stride with one vector load, and the cross-lane sums use
// ballots (scalar bit counts of bit planes) and v_mbcnt (lanes below), so no
// LDS traffic and no barrier is involved and the results are wave-uniform.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & 63); }

// Bit b (0..15) set iff byte b of the 16-byte word is non-zero.
__device__ __forceinline__ uint32_t nonzero_bytes16(uint4 w) {
    uint32_t r = 0;
    const uint32_t q[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        // high bit of every byte set iff that byte is non-zero
        const uint32_t y = (((q[i] & 0x7F7F7F7Fu) + 0x7F7F7F7Fu) | q[i]) & 0x80808080u;
        const uint32_t nib = ((y >> 7) & 1u) | ((y >> 14) & 2u) | ((y >> 21) & 4u) | ((y >> 28) & 8u);
        r |= nib << (4 * i);
    }
    return r;
}

// Wave-wide sum of per-lane values in [0, 31]: bit plane b contributes
// popcount(ballot(bit b)) << b.
__device__ __forceinline__ int wave_sum5(int v) {
    int s = 0;
#pragma unroll
    for (int b = 0; b < 5; ++b) s += __popcll(__ballot((v >> b) & 1)) << b;
    return s;
}

// Sum of the values in [0, 31] of the lanes below this one.
__device__ __forceinline__ int wave_excl5(int v) {
    int s = 0;
#pragma unroll
    for (int b = 0; b < 5; ++b) {
        const unsigned long long m = __ballot((v >> b) & 1);
        s += (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u)) << b;
    }
    return s;
}

// The mask as seen by one wave: a mask of B bytes (block ids 0..B-1, mask
// != 0 = high), read in strides of 1024 blocks, lane l holding the non-zero
// flags of bytes [stride + 16 l, stride + 16 l + 16) as bits 0..15.  For the
// first stride every lane also keeps the number of high blocks in the lanes
// below it, so that a class, a slot or the block of a slot inside the first
// stride costs a few scalar operations (v_readlane, s_bcnt1).  Block ids
// beyond the first stride are answered by rescanning the later strides;
// ONE = true promises B <= 1024 and compiles that code out.  All 64 lanes of
// the wave must take part in every call.
template <bool ONE>
struct WaveMaskT {
    const uint8_t* __restrict__ mask;
    int B;
    bool aligned;
    uint32_t first;  // this lane's bits of the first stride
    int pre;         // high blocks in the first stride's lanes below this one
    int tot;         // high blocks in the first stride

    __device__ __forceinline__ uint32_t load(int stride) const {
        const int b0 = stride + 16 * lane_id();
        if (b0 >= B) return 0;
        if (aligned && b0 + 16 <= B) return nonzero_bytes16(*reinterpret_cast<const uint4*>(mask + b0));
        // the mask's final partial chunk: one byte at a time, all issued together
        uint8_t v[16];
#pragma unroll
        for (int b = 0; b < 16; ++b) v[b] = (b0 + b < B) ? mask[b0 + b] : (uint8_t)0;
        uint32_t r = 0;
#pragma unroll
        for (int b = 0; b < 16; ++b) r |= (uint32_t)(v[b] != 0) << b;
        return r;
    }
    __device__ __forceinline__ void init(const uint8_t* m, int nbytes) {
        mask = m;
        B = nbytes;
        aligned = (reinterpret_cast<uintptr_t>(m) & 15) == 0;
        first = load(0);
        const int c = __popc(first);
        pre = wave_excl5(c);
        tot = wave_sum5(c);
    }
    // The same as init, with the first 1024 mask bytes already copied to LDS
    // by stage_mask (bytes past B zero): many waves reading the one global
    // line of a small mask at once wait for each other, one LDS copy per
    // workgroup does not.
    __device__ __forceinline__ void init_staged(const uint8_t* m, int nbytes, const uint8_t* s_mask) {
        mask = m;
        B = nbytes;
        aligned = (reinterpret_cast<uintptr_t>(m) & 15) == 0;
        first = nonzero_bytes16(*reinterpret_cast<const uint4*>(s_mask + 16 * lane_id()));
        const int c = __popc(first);
        pre = wave_excl5(c);
        tot = wave_sum5(c);
    }
    // valid-byte bits of this lane's chunk of a stride
    __device__ __forceinline__ uint32_t inside(int stride) const {
        const int b0 = stride + 16 * lane_id();
        return b0 >= B ? 0u : (b0 + 16 <= B ? 0xFFFFu : ((1u << (B - b0)) - 1u));
    }

    // Is block t (0 <= t < B, wave-uniform) high?
    __device__ __forceinline__ bool high(int t) const {
        const int stride = ONE ? 0 : (t & ~1023);
        const uint32_t b = stride == 0 ? first : load(stride);
        const int w = __builtin_amdgcn_readlane((int)b, (t - stride) >> 4);
        return (w >> ((t - stride) & 15)) & 1;
    }
    // Number of high blocks among ids [0, t) (0 <= t <= B, wave-uniform).
    __device__ __forceinline__ int count_high(int t) const {
        if (ONE || t < 1024) {
            if (t == 0) return 0;
            const int l = (t - 1) >> 4;  // lane holding block t - 1
            const int n = t - 16 * l;    // 1..16 bits of that lane below t
            const uint32_t w = (uint32_t)__builtin_amdgcn_readlane((int)first, l);
            return __builtin_amdgcn_readlane(pre, l) + __popc(w & (n >= 16 ? 0xFFFFu : ((1u << n) - 1u)));
        }
        int cnt = tot;
        for (int stride = 1024; stride < t; stride += 1024) {
            const int n = t - (stride + 16 * lane_id());
            const uint32_t b = load(stride);
            cnt += wave_sum5(n <= 0 ? 0 : __popc(b & (n >= 16 ? 0xFFFFu : ((1u << n) - 1u))));
        }
        return cnt;
    }
    // Slot of block t: its rank among the earlier blocks of its class.
    __device__ __forceinline__ int slot(int t, bool is_high) const {
        const int c = count_high(t);
        return is_high ? c : t - c;
    }
    // Block id of the s-th block (0-based, wave-uniform) of the class
    // `want_high`, or -1 if the mask has no more than s blocks of that class.
    __device__ __forceinline__ int find_nth(int s, bool want_high) const {
        int before = 0;
        for (int stride = 0; stride < (ONE ? 1 : B); stride += 1024) {
            const uint32_t b = stride == 0 ? first : load(stride);
            const uint32_t cls = want_high ? b : (~b & inside(stride));
            const int cnt = __popc(cls);
            int excl, total;
            if (stride == 0) {
                const int below = min(16 * lane_id(), B);  // mask bytes in the lanes below
                excl = want_high ? pre : below - pre;
                total = want_high ? tot : min(B, 1024) - tot;
            } else {
                excl = wave_excl5(cnt);
                total = wave_sum5(cnt);
            }
            if (before + total > s) {
                excl += before;
                const bool mine = s >= excl && s < excl + cnt;
                const int src = __ffsll((unsigned long long)__ballot(mine)) - 1;
                uint32_t m = cls;
                for (int i = excl; mine && i < s; ++i) m &= m - 1;
                const int pos = __builtin_amdgcn_readlane(__ffs(m) - 1, src);
                return stride + 16 * src + pos;
            }
            before += total;
        }
        return -1;
    }
};
typedef WaveMaskT<false> WaveMask;

// One wave copies mask bytes [0, min(B, 1024)) to s_mask (1024 bytes, 16-byte
// aligned LDS), zero past B; the workgroup then synchronises before any wave
// calls WaveMaskT::init_staged.
__device__ __forceinline__ void stage_mask(const uint8_t* __restrict__ m, int B, uint8_t* s_mask) {
    const int b0 = 16 * lane_id();
    uint4 v = uint4{0u, 0u, 0u, 0u};
    if (b0 < B) {
        if ((reinterpret_cast<uintptr_t>(m) & 15) == 0 && b0 + 16 <= B) {
            v = *reinterpret_cast<const uint4*>(m + b0);
        } else {
            uint8_t bytes[16];
#pragma unroll
            for (int b = 0; b < 16; ++b) bytes[b] = (b0 + b < B) ? m[b0 + b] : (uint8_t)0;
            v.x = bytes[0] | (bytes[1] << 8) | (bytes[2] << 16) | ((uint32_t)bytes[3] << 24);
            v.y = bytes[4] | (bytes[5] << 8) | (bytes[6] << 16) | ((uint32_t)bytes[7] << 24);
            v.z = bytes[8] | (bytes[9] << 8) | (bytes[10] << 16) | ((uint32_t)bytes[11] << 24);
            v.w = bytes[12] | (bytes[13] << 8) | (bytes[14] << 16) | ((uint32_t)bytes[15] << 24);
        }
    }
    *reinterpret_cast<uint4*>(s_mask + b0) = v;
}

// Class and slot of a block and of its 8 neighbours.  Neighbour index
// d = (dy+1)*3 + (dx+1); d = 4 is the block itself.
struct Neigh {
    uint32_t valid;  // bit d: neighbour d lies inside the block grid
    uint32_t high;   // bit d: neighbour d is high resolution
    int slot[9];     // slot of neighbour d in its class's stack
};

// Slot of neighbour d (run-time d) as a choice between register values.  Each
// slot is read with a constant index and passed through an empty asm, so the
// optimiser cannot turn the choice back into one load at a computed offset:
// such a load keeps the Neigh in memory, and the compiler then places it in
// LDS indexed by the flat thread id, whose computation reads the work-group
// size from the dispatch packet in host memory (microseconds per wave at
// kernel start).
__device__ __forceinline__ int neigh_slot(const Neigh& nb, int d) {
    int r = 0;
#pragma unroll
    for (int i = 0; i < 9; ++i) {
        int v = nb.slot[i];
        asm("" : "+v"(v));
        r = d == i ? v : r;
    }
    return r;
}

// Neighbourhood of block (n, gy, gx): classes and, when WITH_SLOTS, slots.
// Wave-uniform; all 64 lanes of the wave must call it.
template <bool WITH_SLOTS, bool ONE>
__device__ __forceinline__ Neigh wave_neighbourhood(const WaveMaskT<ONE>& wm, int GH, int GW, int n, int gy, int gx) {
    int t[9];
    Neigh r;
    r.valid = 0;
    r.high = 0;
#pragma unroll
    for (int d = 0; d < 9; ++d) {
        const int ny = gy + d / 3 - 1, nx = gx + d % 3 - 1;
        const bool v = (ny >= 0 && ny < GH && nx >= 0 && nx < GW);
        t[d] = (n * GH + (v ? ny : gy)) * GW + (v ? nx : gx);
        r.valid |= (uint32_t)v << d;
        r.high |= (uint32_t)wm.high(t[d]) << d;
    }
#pragma unroll
    for (int d = 0; d < 9; ++d) r.slot[d] = WITH_SLOTS ? wm.slot(t[d], (r.high >> d) & 1) : 0;
    return r;
}

// Block plan of a mask of up to 1024 blocks as a table in LDS: bit (k & 15)
// of hi[k >> 4] is block k's class, slot[k] its rank among the earlier blocks
// of that class.  One wave builds it from the staged mask (stage_mask); the
// lookups are then plain LDS reads instead of chains of cross-lane reads on
// the CU's one scalar unit.
struct PlanTable {
    uint16_t hi[64];
    uint16_t slot[1024];
};

__device__ __forceinline__ void build_plan_table(const uint8_t* s_mask, PlanTable* pt) {
    const int l = lane_id();
    const uint32_t bits = nonzero_bytes16(*reinterpret_cast<const uint4*>(s_mask + 16 * l));  // zero past B
    const int pre = wave_excl5(__popc(bits));
    pt->hi[l] = (uint16_t)bits;
    uint32_t w[8];
#pragma unroll
    for (int b = 0; b < 16; b += 2) {
        uint32_t two = 0;
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int nb = pre + __popc(bits & ((1u << (b + i)) - 1u));  // high blocks before 16 l + b + i
            const uint32_t sl = ((bits >> (b + i)) & 1u) ? (uint32_t)nb : (uint32_t)(16 * l + b + i - nb);
            two |= sl << (16 * i);
        }
        w[b / 2] = two;
    }
    *reinterpret_cast<uint4*>(&pt->slot[16 * l]) = uint4{w[0], w[1], w[2], w[3]};
    *reinterpret_cast<uint4*>(&pt->slot[16 * l + 8]) = uint4{w[4], w[5], w[6], w[7]};
}

// Class and slot of block k (wave-uniform k), from the table.
__device__ __forceinline__ bool table_high(const PlanTable* pt, int k) {
    return __builtin_amdgcn_readfirstlane((int)((pt->hi[k >> 4] >> (k & 15)) & 1u)) != 0;
}
__device__ __forceinline__ int table_slot(const PlanTable* pt, int k) {
    return __builtin_amdgcn_readfirstlane((int)pt->slot[k]);
}

// Neighbourhood of block (n, gy, gx) from the table: lane d < 9 looks up
// neighbour d, then the results are made wave-uniform.
__device__ __forceinline__ Neigh table_neighbourhood(const PlanTable* pt, int GH, int GW, int n, int gy, int gx) {
    const int l = lane_id();
    int vd = 0, hb = 0, sl = 0;
    if (l < 9) {
        const int ny = gy + l / 3 - 1, nx = gx + l % 3 - 1;
        vd = (ny >= 0 && ny < GH && nx >= 0 && nx < GW);
        const int t = (n * GH + (vd ? ny : gy)) * GW + (vd ? nx : gx);
        hb = (pt->hi[t >> 4] >> (t & 15)) & 1;
        sl = pt->slot[t];
    }
    Neigh r;
    r.valid = (uint32_t)__ballot(vd) & 0x1FFu;
    r.high = (uint32_t)__ballot(hb) & 0x1FFu;
#pragma unroll
    for (int d = 0; d < 9; ++d) r.slot[d] = __builtin_amdgcn_readlane(sl, d);
    return r;
}

}  // namespace sb
