// Source of one padded-tile pixel (a vector of V channels starting at c) for
// BlockPad and for the convolutions that fuse BlockPad / BlockSample into
// their tile load.
#pragma once

#include "sb_common.h"

namespace sb {

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
// direction: copied at equal resolution, nearest-upsampled from a low
// neighbour into a high block, 2x2-averaged from a high neighbour into a low
// block, zero outside the image or for a neighbour beyond the stack capacity.
// For NCHW, V must be 1.
template <typename T, int L, int V>
__device__ __forceinline__ Vec<T, V> packed_pixel(const T* __restrict__ hi, const T* __restrict__ lo, int C, int bs,
                                                  const Neigh& nb, int hi_cap, int lo_cap, int uu, int vv, int c) {
    const int own_high = (nb.high >> 4) & 1;
    const int lb = bs >> 1, e = own_high ? bs : lb;
    const int dy = uu < 0 ? -1 : (uu >= e ? 1 : 0);
    const int dx = vv < 0 ? -1 : (vv >= e ? 1 : 0);
    const int d = (dy + 1) * 3 + (dx + 1);
    if (!((nb.valid >> d) & 1)) return vzero<T, V>();
    const int nhigh = (nb.high >> d) & 1;
    const int ns = nb.slot[d];
    if (ns >= (nhigh ? hi_cap : lo_cap)) return vzero<T, V>();
    const int u2 = uu - dy * e, v2 = vv - dx * e;
    if (nhigh == own_high)
        return vload<T, V>(stack_at<T, L>(nhigh ? hi : lo, ns, C, e, u2, v2, c));
    if (own_high)  // low neighbour: nearest upsampling
        return vload<T, V>(stack_at<T, L>(lo, ns, C, lb, u2 >> 1, v2 >> 1, c));
    // high neighbour of a low block: average sampling over the 2x2 cell
    const int r = 2 * u2, s = 2 * v2;
    const Vec<T, V> a = vload<T, V>(stack_at<T, L>(hi, ns, C, bs, r, s, c));
    const Vec<T, V> b = vload<T, V>(stack_at<T, L>(hi, ns, C, bs, r, s + 1, c));
    const Vec<T, V> cc = vload<T, V>(stack_at<T, L>(hi, ns, C, bs, r + 1, s, c));
    const Vec<T, V> dd = vload<T, V>(stack_at<T, L>(hi, ns, C, bs, r + 1, s + 1, c));
    return vavg4<T, V>(a, b, cc, dd);
}

// BlockSample + BlockPad straight from the dense map x (block (n, gy, gx)).
// High block: the image pixel if its block is high, else the 2x2 average of
// the image cell containing it (= the low neighbour's value, nearest-
// upsampled).  Low block: the 2x2 average of the image cell at twice the
// low-resolution coordinate, whatever the neighbour's resolution (a high
// neighbour's 2x2 average and a low neighbour's own value are both that
// cell's average).  Zero outside the image.  For NCHW, V must be 1.
template <typename T, int L, int V>
__device__ __forceinline__ Vec<T, V> dense_pixel(const T* __restrict__ x, int n, int C, int H, int W, int bs,
                                                 int gy, int gx, const Neigh& nb, int uu, int vv, int c) {
    const int own_high = (nb.high >> 4) & 1;
    if (own_high) {
        const int Y = gy * bs + uu, X = gx * bs + vv;
        if (Y < 0 || Y >= H || X < 0 || X >= W) return vzero<T, V>();
        const int dy = uu < 0 ? -1 : (uu >= bs ? 1 : 0);
        const int dx = vv < 0 ? -1 : (vv >= bs ? 1 : 0);
        const int d = (dy + 1) * 3 + (dx + 1);
        if ((nb.high >> d) & 1) return vload<T, V>(map_at<T, L>(x, n, C, H, W, Y, X, c));
        const int Y0 = Y & ~1, X0 = X & ~1;
        const Vec<T, V> a = vload<T, V>(map_at<T, L>(x, n, C, H, W, Y0, X0, c));
        const Vec<T, V> b = vload<T, V>(map_at<T, L>(x, n, C, H, W, Y0, X0 + 1, c));
        const Vec<T, V> cc = vload<T, V>(map_at<T, L>(x, n, C, H, W, Y0 + 1, X0, c));
        const Vec<T, V> dd = vload<T, V>(map_at<T, L>(x, n, C, H, W, Y0 + 1, X0 + 1, c));
        return vavg4<T, V>(a, b, cc, dd);
    }
    const int lb = bs >> 1;
    const int Yl = gy * lb + uu, Xl = gx * lb + vv;
    if (Yl < 0 || 2 * Yl >= H || Xl < 0 || 2 * Xl >= W) return vzero<T, V>();
    const int Y0 = 2 * Yl, X0 = 2 * Xl;
    const Vec<T, V> a = vload<T, V>(map_at<T, L>(x, n, C, H, W, Y0, X0, c));
    const Vec<T, V> b = vload<T, V>(map_at<T, L>(x, n, C, H, W, Y0, X0 + 1, c));
    const Vec<T, V> cc = vload<T, V>(map_at<T, L>(x, n, C, H, W, Y0 + 1, X0, c));
    const Vec<T, V> dd = vload<T, V>(map_at<T, L>(x, n, C, H, W, Y0 + 1, X0 + 1, c));
    return vavg4<T, V>(a, b, cc, dd);
}

}  // namespace sb
