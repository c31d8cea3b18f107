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

template <typename T, int V>
__device__ __forceinline__ Vec<T, V> vzero() {
    Vec<T, V> v;
#pragma unroll
    for (int i = 0; i < V; ++i) v.e[i] = from_f32<T>(0.0f);
    return v;
}

template <typename T, int V>
__device__ __forceinline__ Vec<T, V> vavg4(const Vec<T, V>& a, const Vec<T, V>& b,
                                           const Vec<T, V>& c, const Vec<T, V>& d) {
    Vec<T, V> r;
#pragma unroll
    for (int i = 0; i < V; ++i) r.e[i] = avg4(a.e[i], b.e[i], c.e[i], d.e[i]);
    return r;
}

// ---------------------------------------------------------------------------
// Wavefront primitives
// ---------------------------------------------------------------------------
__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & 63); }

__device__ __forceinline__ int wave_sum(int v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

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

// Block plan by wavefront counting.  For each of NT target block ids t[i]
// (0 <= t[i] <= B) returns, uniformly across the wave, the number of high
// blocks (mask != 0) among ids [0, t[i]).  Every lane covers 16 mask bytes per
// 1024-block stride with one vector load; partial counts are summed across
// the wave.  All 64 lanes of the wave must call it.
template <int NT>
__device__ __forceinline__ void wave_count_high(const uint8_t* __restrict__ mask, long long B,
                                                const long long (&t)[NT], int (&out)[NT]) {
    long long tmax = 0;
#pragma unroll
    for (int i = 0; i < NT; ++i) tmax = t[i] > tmax ? t[i] : tmax;
    const bool aligned = (reinterpret_cast<uintptr_t>(mask) & 15) == 0;
    int cnt[NT];
#pragma unroll
    for (int i = 0; i < NT; ++i) cnt[i] = 0;
    for (long long base = (long long)lane_id() * 16; base < tmax; base += 1024) {
        uint32_t bits = 0;
        if (aligned && base + 16 <= B) {
            bits = nonzero_bytes16(*reinterpret_cast<const uint4*>(mask + base));
        } else {
            for (int b = 0; b < 16; ++b)
                if (base + b < B && mask[base + b]) bits |= 1u << b;
        }
#pragma unroll
        for (int i = 0; i < NT; ++i) {
            const long long n = t[i] - base;
            if (n > 0) cnt[i] += __popc(bits & (n >= 16 ? 0xFFFFu : ((1u << n) - 1u)));
        }
    }
#pragma unroll
    for (int i = 0; i < NT; ++i) out[i] = wave_sum(cnt[i]);
}

// Class and slot of a block and of its 8 neighbours.  Neighbour index
// d = (dy+1)*3 + (dx+1); d = 4 is the block itself.  Lives in LDS so that
// every thread of the workgroup can index it with a run-time d.
struct Neigh {
    uint32_t valid;  // bit d: neighbour d lies inside the block grid
    uint32_t high;   // bit d: neighbour d is high resolution
    int slot[9];     // slot of neighbour d in its class's stack
};

// Fills *out (in LDS) with the neighbourhood of block (n, gy, gx): classes and,
// when WITH_SLOTS, slots from one wavefront count over the image's mask
// prefix.  Must be called by one whole wave; lane 0 writes.  The caller
// synchronises the workgroup before other waves read *out.
template <bool WITH_SLOTS>
__device__ __forceinline__ void block_neighbourhood(const uint8_t* __restrict__ mask, int GH, int GW,
                                                    int n, int gy, int gx, Neigh* out) {
    long long t[9];
    uint32_t valid = 0, high = 0;
#pragma unroll
    for (int d = 0; d < 9; ++d) {
        const int ny = gy + d / 3 - 1, nx = gx + d % 3 - 1;
        const bool v = (ny >= 0 && ny < GH && nx >= 0 && nx < GW);
        const long long k = ((long long)n * GH + (v ? ny : gy)) * GW + (v ? nx : gx);
        t[d] = k;
        valid |= (uint32_t)v << d;
        high |= (uint32_t)(mask[k] != 0) << d;
    }
    int c[9] = {0, 0, 0, 0, 0, 0, 0, 0, 0};
    if constexpr (WITH_SLOTS) {
        wave_count_high<9>(mask, ((long long)n + 1) * GH * GW, t, c);
    }
    if (lane_id() == 0) {
        out->valid = valid;
        out->high = high;
#pragma unroll
        for (int d = 0; d < 9; ++d)
            out->slot[d] = WITH_SLOTS ? (((high >> d) & 1) ? c[d] : (int)(t[d] - c[d])) : 0;
    }
}

}  // namespace sb
