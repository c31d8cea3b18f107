// Heuristic downsampling policy: the per-block detail score and the per-image
// selection of the blocks to process at high resolution (the policy of the
// short paper SegBlocks grew out of, which its ablation on execution
// policies compares with; the paper's reinforcement-learned policy network
// needs trained weights and is out of scope).
//
// Score of block k: for every pixel of the block the Euclidean distance over
// the channels between the pixel and the block's low-resolution version at
// that pixel (the 2x2 average of its cell, computed and rounded as
// BlockSample does, nearest-upsampled), averaged over the bs x bs pixels.
// One workgroup per block; a thread takes 2x2 cells and all their channels
// (the four pixel norms need every channel of the cell), sums in fp32, and
// the workgroup reduces in a fixed tree.
//
// Selection: per image, the k = round(tau * GH * GW) blocks with the highest
// scores are high resolution; equal scores are ranked by block id (lower
// first).  One workgroup per image ranks every block against all others in
// LDS: exact and independent of timing.
#include "sb_common.h"
#include "sb_kernels.h"

namespace sb {

namespace {

// Element (n, c, Y, X) of a dense map.
template <typename T, int L>
__device__ __forceinline__ T px(const T* __restrict__ x, int n, int C, int H, int W, int Y, int X, int c) {
    if constexpr (L == NHWC) return x[(((size_t)n * H + Y) * W + X) * C + c];
    else                     return x[(((size_t)n * C + c) * H + Y) * W + X];
}

template <typename T, int L>
__global__ __launch_bounds__(WG) void k_policy_score(const T* __restrict__ x, int C, int H, int W, int bs, int GH,
                                                     int GW, float* __restrict__ score) {
    const int k = (int)blockIdx.x;
    const int per = GH * GW;
    const int n = k / per, r = k - n * per, gy = r / GW, gx = r - gy * GW;
    const int lb = bs >> 1, cells = lb * lb;
    float acc = 0.0f;
    for (int cell = (int)threadIdx.x; cell < cells; cell += WG) {
        const int ci = cell / lb, cj = cell - ci * lb;
        const int Y = gy * bs + 2 * ci, X = gx * bs + 2 * cj;
        float d2[4] = {0.f, 0.f, 0.f, 0.f};
        for (int c = 0; c < C; ++c) {
            const T a = px<T, L>(x, n, C, H, W, Y, X, c);
            const T b = px<T, L>(x, n, C, H, W, Y, X + 1, c);
            const T cc = px<T, L>(x, n, C, H, W, Y + 1, X, c);
            const T d = px<T, L>(x, n, C, H, W, Y + 1, X + 1, c);
            const float m = to_f32(avg4(a, b, cc, d));
            const float e0 = to_f32(a) - m, e1 = to_f32(b) - m, e2 = to_f32(cc) - m, e3 = to_f32(d) - m;
            d2[0] += e0 * e0;
            d2[1] += e1 * e1;
            d2[2] += e2 * e2;
            d2[3] += e3 * e3;
        }
        acc += (__builtin_sqrtf(d2[0]) + __builtin_sqrtf(d2[1])) + (__builtin_sqrtf(d2[2]) + __builtin_sqrtf(d2[3]));
    }
    // fixed-order reduction: lanes of a wave, then the waves in order
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o, 64);
    __shared__ float s_part[WG / 64];
    if ((threadIdx.x & 63) == 0) s_part[threadIdx.x >> 6] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
        float t = 0.0f;
#pragma unroll
        for (int w = 0; w < WG / 64; ++w) t += s_part[w];
        score[k] = t / (float)(bs * bs);
    }
}

constexpr int POL_MAXB = 8192;  // blocks per image the LDS score table holds

__global__ __launch_bounds__(WG) void k_policy_select(const float* __restrict__ score, int per, int khigh,
                                                      uint8_t* __restrict__ mask) {
    __shared__ float s[POL_MAXB];
    const int n = (int)blockIdx.x;
    const float* sc = score + (size_t)n * per;
    for (int i = (int)threadIdx.x; i < per; i += WG) s[i] = sc[i];
    __syncthreads();
    for (int b = (int)threadIdx.x; b < per; b += WG) {
        const float v = s[b];
        int rank = 0;
        for (int j = 0; j < per; ++j) {
            const float t = s[j];
            rank += (t > v || (t == v && j < b)) ? 1 : 0;
        }
        mask[(size_t)n * per + b] = rank < khigh ? 1 : 0;
    }
}

template <typename T>
hipError_t policy_t(int layout, const void* x, int N, int C, int H, int W, int bs, float* score, int khigh,
                    uint8_t* mask, hipStream_t st) {
    const int GH = H / bs, GW = W / bs;
    const long long B = (long long)N * GH * GW;
    if (layout == NHWC)
        hipLaunchKernelGGL((k_policy_score<T, NHWC>), dim3((unsigned)B), dim3(WG), 0, st, (const T*)x, C, H, W, bs,
                           GH, GW, score);
    else
        hipLaunchKernelGGL((k_policy_score<T, NCHW>), dim3((unsigned)B), dim3(WG), 0, st, (const T*)x, C, H, W, bs,
                           GH, GW, score);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_policy_select, dim3((unsigned)N), dim3(WG), 0, st, (const float*)score, GH * GW, khigh, mask);
    return hipGetLastError();
}

}  // namespace

int policy_max_blocks() { return POL_MAXB; }

hipError_t launch_policy(int dtype, int layout, const void* x, int N, int C, int H, int W, int bs, float* score,
                         int khigh, uint8_t* mask, hipStream_t st) {
    switch (dtype) {
    case 0: return policy_t<float>(layout, x, N, C, H, W, bs, score, khigh, mask, st);
    case 1: return policy_t<f16>(layout, x, N, C, H, W, bs, score, khigh, mask, st);
    default: return policy_t<bf16>(layout, x, N, C, H, W, bs, score, khigh, mask, st);
    }
}

}  // namespace sb
