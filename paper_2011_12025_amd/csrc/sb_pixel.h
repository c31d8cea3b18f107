// Where one padded-tile pixel comes from, for BlockPad and for the
// convolutions that fuse BlockPad (and BlockSample) into their tile load.
//
// A source is either nothing (the pixel is zero), one location (a copy), or
// the 2x2 cell p, p + d1, p + d2, p + d2 + d1 whose average is the value.
// Kernels first compute the sources of a batch of pixels, then issue every
// load of the batch, then combine: the loads of a batch are in flight
// together instead of one dependent round trip per pixel.
#pragma once

#include "sb_common.h"

namespace sb {

template <typename T>
struct Src {
    const T* p;  // nullptr -> zero
    int avg;     // 1 -> average of the 2x2 cell at p
    int d1, d2;  // element offsets of the right and of the lower pixel of the cell
};

template <typename T>
__device__ __forceinline__ Src<T> src_zero() {
    return Src<T>{nullptr, 0, 0, 0};
}
template <typename T>
__device__ __forceinline__ Src<T> src_copy(const T* p) {
    return Src<T>{p, 0, 0, 0};
}
template <typename T>
__device__ __forceinline__ Src<T> src_avg(const T* p, int d1, int d2) {
    return Src<T>{p, 1, d1, d2};
}

// How BlockPad fills a halo (the `pm` argument below): PM_AVG is BlockPad
// with average sampling (a high neighbour's 2x2 cell averaged into a low
// block's halo), PM_STRIDED takes that cell's top-left pixel instead
// (strided subsampling), PM_ZERO pads every block with zeros.  A call's
// flags carry it in bits 1-2 (SB_FLAG_PAD_STRIDED, SB_FLAG_PAD_ZERO).
constexpr int PM_AVG = 0, PM_STRIDED = 1, PM_ZERO = 2;
__host__ __device__ __forceinline__ int pad_mode(int flags) { return (flags >> 1) & 3; }

// Element (s, c, y, x) of a block stack of extent `ext` with C channels.
template <typename T, int L>
__device__ __forceinline__ const T* stack_at(const T* base, int s, int C, int ext, int y, int x, int c) {
    if constexpr (L == NHWC) return base + (((size_t)s * ext + y) * ext + x) * C + c;
    else                     return base + (((size_t)s * C + c) * ext + y) * ext + x;
}

// Element (n, c, Y, X) of a dense [N, C, H, W] map.
template <typename T, int L>
__device__ __forceinline__ const T* map_at(const T* base, int n, int C, int H, int W, int Y, int X, int c) {
    if constexpr (L == NHWC) return base + (((size_t)n * H + Y) * W + X) * C + c;
    else                     return base + (((size_t)n * C + c) * H + Y) * W + X;
}

// BlockPad from packed stacks.  (uu, vv) in [-1, e] are coordinates in the
// block's own grid (e = bs for a high block, bs/2 for a low one); the value
// is the block's own pixel inside, else the neighbour's pixel in that
// direction (the diagonal neighbour for a corner): copied at equal
// resolution, nearest-upsampled from a low neighbour into a high block,
// 2x2-averaged from a high neighbour into a low block, zero outside the
// image or for a neighbour beyond its stack's capacity.
template <typename T, int L>
__device__ __forceinline__ Src<T> packed_src(const T* __restrict__ hi, const T* __restrict__ lo, int C, int bs,
                                             const Neigh& nb, int hi_cap, int lo_cap, int uu, int vv, int c,
                                             int pm = PM_AVG) {
    const int own_high = (nb.high >> 4) & 1;
    const int lb = bs >> 1, e = own_high ? bs : lb;
    const int dy = uu < 0 ? -1 : (uu >= e ? 1 : 0);
    const int dx = vv < 0 ? -1 : (vv >= e ? 1 : 0);
    const int d = (dy + 1) * 3 + (dx + 1);
    if (!((nb.valid >> d) & 1) || (pm == PM_ZERO && d != 4)) return src_zero<T>();
    const int nhigh = (nb.high >> d) & 1;
    const int ns = neigh_slot(nb, d);
    if (ns >= (nhigh ? hi_cap : lo_cap)) return src_zero<T>();
    const int u2 = uu - dy * e, v2 = vv - dx * e;
    if (nhigh == own_high) return src_copy<T>(stack_at<T, L>(nhigh ? hi : lo, ns, C, e, u2, v2, c));
    if (own_high) return src_copy<T>(stack_at<T, L>(lo, ns, C, lb, u2 >> 1, v2 >> 1, c));
    const int px = (L == NHWC) ? C : 1;
    if (pm == PM_STRIDED) return src_copy<T>(stack_at<T, L>(hi, ns, C, bs, 2 * u2, 2 * v2, c));
    return src_avg<T>(stack_at<T, L>(hi, ns, C, bs, 2 * u2, 2 * v2, c), px, px * bs);
}

// BlockSample + BlockPad straight from the dense map x (block (n, gy, gx)).
// High block: the image pixel when the block it lies in is high, else the
// 2x2 average of the image cell containing it (= the low neighbour's value,
// nearest-upsampled).  Low block: the 2x2 average of the image cell at twice
// the low-resolution coordinate, whatever the neighbour's resolution (a high
// neighbour's 2x2 average and a low neighbour's own value are both that
// cell's average).  Zero outside the image.
//
// With strided sampling a low block's halo pixel whose cell lies in a high
// neighbour is that cell's top-left image pixel; with zero padding every
// halo pixel is zero.
template <typename T, int L>
__device__ __forceinline__ Src<T> dense_src(const T* __restrict__ x, int n, int C, int H, int W, int bs, int gy,
                                            int gx, const Neigh& nb, int uu, int vv, int c, int pm = PM_AVG) {
    const int own_high = (nb.high >> 4) & 1;
    const int px = (L == NHWC) ? C : 1;
    const int row = px * W;
    const int e = own_high ? bs : (bs >> 1);
    const int dy = uu < 0 ? -1 : (uu >= e ? 1 : 0);
    const int dx = vv < 0 ? -1 : (vv >= e ? 1 : 0);
    const int d = (dy + 1) * 3 + (dx + 1);
    if (pm == PM_ZERO && d != 4) return src_zero<T>();
    if (own_high) {
        const int Y = gy * bs + uu, X = gx * bs + vv;
        if (Y < 0 || Y >= H || X < 0 || X >= W) return src_zero<T>();
        if ((nb.high >> d) & 1) return src_copy<T>(map_at<T, L>(x, n, C, H, W, Y, X, c));
        return src_avg<T>(map_at<T, L>(x, n, C, H, W, Y & ~1, X & ~1, c), px, row);
    }
    const int lb = bs >> 1;
    const int Yl = gy * lb + uu, Xl = gx * lb + vv;
    if (Yl < 0 || 2 * Yl >= H || Xl < 0 || 2 * Xl >= W) return src_zero<T>();
    if (pm == PM_STRIDED && d != 4 && ((nb.high >> d) & 1))
        return src_copy<T>(map_at<T, L>(x, n, C, H, W, 2 * Yl, 2 * Xl, c));
    return src_avg<T>(map_at<T, L>(x, n, C, H, W, 2 * Yl, 2 * Xl, c), px, row);
}

// A batch of U vectors of V elements: sources first, then every load, then
// the combination.  Lanes whose item is past the end use a zero source.
template <typename T, int V, int U>
struct SrcBatch {
    Vec<T, V> v[U][4];
    int mode[U];  // 0 zero, 1 copy, 2 average

    __device__ __forceinline__ void issue(int u, const Src<T>& s) {
        if (!s.p) {
            mode[u] = 0;
        } else if (!s.avg) {
            mode[u] = 1;
            v[u][0] = vload<T, V>(s.p);
        } else {
            mode[u] = 2;
            v[u][0] = vload<T, V>(s.p);
            v[u][1] = vload<T, V>(s.p + s.d1);
            v[u][2] = vload<T, V>(s.p + s.d2);
            v[u][3] = vload<T, V>(s.p + s.d2 + s.d1);
        }
    }
    __device__ __forceinline__ Vec<T, V> value(int u) const {
        if (mode[u] == 0) return vzero<T, V>();
        if (mode[u] == 1) return v[u][0];
        return vavg4<T, V>(v[u][0], v[u][1], v[u][2], v[u][3]);
    }
};

}  // namespace sb
