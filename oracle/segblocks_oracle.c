/*
 * SegBlocks CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, obviously-correct C implementation of the block modules of
 * SegBlocks (Verelst & Tuytelaars, "SegBlocks: Block-Based Dynamic Resolution
 * Networks for Real-Time Segmentation", arXiv 2011.12025), written from the
 * paper's Method section ("Block modules": BlockSample, BlockPad,
 * BlockCombine) and its description of the block convolution (the same
 * filters applied to the high- and the low-resolution block stacks).
 *
 * Only the test suite, the smoke check and the CPU-baseline leg of the
 * benchmark may load this file's library.  The GPU product path never links,
 * imports or calls it, and the two share no code, headers or tables.
 *
 * Conventions
 *   - Every tensor is a float array in logical N,C,H,W order (row-major).
 *     For fp16/bf16 runs the arrays hold values that are exactly
 *     representable in that type (the wrapper converts bit-exactly).
 *   - dtype: 0 = fp32, 1 = fp16, 2 = bf16.
 *   - mask[n][gy][gx] != 0 means the block is processed at HIGH resolution
 *     (the paper's action a_b = 1).
 *   - Blocks are packed into each stack in row-major (n, gy, gx) order
 *     (stable compaction); the paper leaves the order open.
 *
 * Build: gcc -O2 -ffp-contract=off (no fast-math) so that the fp32
 * arithmetic below is performed exactly as written; -fopenmp lets the
 * convolutions hand whole output planes (one block or image and one output
 * channel each) to separate host threads.  Each output value is still
 * accumulated by one thread in the fixed order stated at each function, so
 * the result does not depend on the thread count.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_F32 0
#define ORC_F16 1
#define ORC_BF16 2

/* Host threads used by the convolutions (n <= 0: OpenMP's default). */
void orc_set_threads(int n)
{
    if (n > 0) omp_set_num_threads(n);
}

int orc_get_threads(void)
{
    return omp_get_max_threads();
}

/* ------------------------------------------------------------------------ */
/* Rounding to the storage type, from the IEEE-754 definition.               */
/* ------------------------------------------------------------------------ */

/* Round v to the nearest value of a binary format with p significand bits
 * (implicit bit included), minimum normal exponent emin and maximum exponent
 * emax; ties go to the even significand; overflow goes to +-inf.  The
 * quantum inside a binade is 2^(E-(p-1)); below the normal range it is fixed
 * at 2^(emin-(p-1)) (gradual underflow). */
static double round_binary(double v, int p, int emin, int emax)
{
    if (v != v || v == 0.0 || isinf(v)) return v;
    double a = fabs(v);
    int e2;
    frexp(a, &e2);          /* a = m * 2^e2, 0.5 <= m < 1 */
    int E = e2 - 1;         /* a = 1.f * 2^E              */
    if (E < emin) E = emin;
    double q = ldexp(1.0, E - (p - 1));
    double r = nearbyint(a / q) * q;     /* a/q is exact: scaling by 2^k */
    double maxf = ldexp(2.0 - ldexp(1.0, 1 - p), emax);
    if (r > maxf) r = INFINITY;
    return copysign(r, v);
}

double orc_round(double v, int dtype)
{
    switch (dtype) {
    case ORC_F16:  return round_binary(v, 11, -14, 15);
    case ORC_BF16: return round_binary(v, 8, -126, 127);
    default:       return round_binary(v, 24, -126, 127);
    }
}

void orc_round_array(const double* in, float* out, long n, int dtype)
{
    for (long i = 0; i < n; ++i) out[i] = (float)orc_round(in[i], dtype);
}

/* 2x2 average used by BlockSample's downsampling and by BlockPad's average
 * sampling.  The paper specifies average pooling but not its arithmetic;
 * this implementation fixes it as fp32 ((a+b)+(c+d)) * 0.25, rounded once
 * to the storage type.  a,b are the top-left/top-right and c,d the
 * bottom-left/bottom-right pixels of the 2x2 cell. */
float orc_avg4(float a, float b, float c, float d, int dtype)
{
    float s = (a + b) + (c + d);
    float m = s * 0.25f;
    return (float)orc_round((double)m, dtype);
}

/* ------------------------------------------------------------------------ */
/* Block plan: class and slot of every block.                                */
/* ------------------------------------------------------------------------ */

/* For each block k (row-major over n, gy, gx): slot[k] = number of earlier
 * blocks of the same class.  inv_hi[s] / inv_lo[s] give the block id of the
 * s-th high / low block.  counts[0] = #high, counts[1] = #low. */
void orc_plan(const uint8_t* mask, long B, int32_t* slot, int32_t* inv_hi,
              int32_t* inv_lo, int32_t* counts)
{
    int32_t nh = 0, nl = 0;
    for (long k = 0; k < B; ++k) {
        if (mask[k]) { slot[k] = nh; if (inv_hi) inv_hi[nh] = (int32_t)k; ++nh; }
        else         { slot[k] = nl; if (inv_lo) inv_lo[nl] = (int32_t)k; ++nl; }
    }
    counts[0] = nh;
    counts[1] = nl;
}

/* ------------------------------------------------------------------------ */
/* BlockSample: split into blocks, 2x average-pool the low-resolution ones.  */
/* ------------------------------------------------------------------------ */

/* x[N][C][H][W] -> hi[nh][C][bs][bs], lo[nl][C][bs/2][bs/2]. */
void orc_split(const float* x, int N, int C, int H, int W, const uint8_t* mask,
               int bs, int dtype, float* hi, float* lo)
{
    const int GH = H / bs, GW = W / bs, lb = bs / 2;
    long nh = 0, nl = 0;
    for (int n = 0; n < N; ++n)
    for (int gy = 0; gy < GH; ++gy)
    for (int gx = 0; gx < GW; ++gx) {
        const long k = ((long)n * GH + gy) * GW + gx;
        for (int c = 0; c < C; ++c) {
            const float* img = x + ((long)n * C + c) * H * W;
            if (mask[k]) {
                float* dst = hi + (nh * C + c) * (long)bs * bs;
                for (int i = 0; i < bs; ++i)
                    for (int j = 0; j < bs; ++j)
                        dst[i * bs + j] = img[(long)(gy * bs + i) * W + gx * bs + j];
            } else {
                float* dst = lo + (nl * C + c) * (long)lb * lb;
                for (int i = 0; i < lb; ++i)
                    for (int j = 0; j < lb; ++j) {
                        const long r0 = (long)(gy * bs + 2 * i) * W + gx * bs + 2 * j;
                        dst[i * lb + j] = orc_avg4(img[r0], img[r0 + 1],
                                                   img[r0 + W], img[r0 + W + 1], dtype);
                    }
            }
        }
        if (mask[k]) ++nh; else ++nl;
    }
}

/* ------------------------------------------------------------------------ */
/* BlockPad: one-pixel halo filled from the neighbouring blocks.             */
/* ------------------------------------------------------------------------ */

/* hi[nh][C][bs][bs], lo[nl][C][lb][lb] -> hp[nh][C][bs+2][bs+2],
 * lp[nl][C][lb+2][lb+2].  For a halo pixel the neighbour is the block in
 * the direction of the pixel (diagonal blocks for the corners):
 *   outside the image                 -> 0
 *   neighbour at the same resolution  -> copy
 *   high block, low neighbour         -> nearest-upsampled neighbour value
 *   low block, high neighbour         -> depends on `sampling` (the two
 *       options the BlockPad section weighs, and the zero padding its
 *       ablation compares them with):
 *       ORC_PAD_AVG     2x2 average of the neighbour's cell (average sampling)
 *       ORC_PAD_STRIDED the cell's top-left pixel (strided subsampling)
 *   ORC_PAD_ZERO: every halo pixel is 0 (each block zero-padded on its own,
 *       the padding BlockPad replaces).                                     */
#define ORC_PAD_AVG 0
#define ORC_PAD_STRIDED 1
#define ORC_PAD_ZERO 2

/* The same with a halo of p pixels (1 <= p <= bs/2, so that every halo pixel
 * lies in the adjacent block): padded extent e + 2p, halo coordinates
 * u, v in [-p, e + p), the neighbour in the direction of the pixel as above.
 * Wider halos serve kernels larger than 3x3 (a 7x7 stem needs 3 pixels) and
 * dilated kernels; p = 1 is BlockPad itself. */
void orc_pad_halo(const float* hi, const float* lo, int N, int C, int H, int W,
                  const uint8_t* mask, int bs, int dtype, int sampling, int p, float* hp, float* lp)
{
    const int GH = H / bs, GW = W / bs, lb = bs / 2;
    const long B = (long)N * GH * GW;
    int32_t* slot = (int32_t*)malloc(sizeof(int32_t) * (size_t)(B > 0 ? B : 1));
    int32_t counts[2];
    orc_plan(mask, B, slot, NULL, NULL, counts);

    for (int n = 0; n < N; ++n)
    for (int gy = 0; gy < GH; ++gy)
    for (int gx = 0; gx < GW; ++gx) {
        const long k = ((long)n * GH + gy) * GW + gx;
        const int high = mask[k] != 0;
        const int e = high ? bs : lb;          /* own extent */
        const int pe = e + 2 * p;              /* padded extent */
        const float* own = high ? hi + (long)slot[k] * C * bs * bs
                                : lo + (long)slot[k] * C * lb * lb;
        float* out = high ? hp + (long)slot[k] * C * pe * pe
                          : lp + (long)slot[k] * C * pe * pe;
        for (int c = 0; c < C; ++c)
        for (int u = -p; u < e + p; ++u)
        for (int v = -p; v < e + p; ++v) {
            const int dy = u < 0 ? -1 : (u >= e ? 1 : 0);
            const int dx = v < 0 ? -1 : (v >= e ? 1 : 0);
            float val;
            if (dy == 0 && dx == 0) {
                val = own[((long)c * e + u) * e + v];
            } else if (sampling == ORC_PAD_ZERO) {
                val = 0.0f;
            } else {
                const int ny = gy + dy, nx = gx + dx;
                if (ny < 0 || ny >= GH || nx < 0 || nx >= GW) {
                    val = 0.0f;
                } else {
                    const long nk = ((long)n * GH + ny) * GW + nx;
                    const int nhigh = mask[nk] != 0;
                    const int u2 = u - dy * e, v2 = v - dx * e; /* coords in neighbour */
                    if (nhigh && high) {
                        val = hi[(((long)slot[nk] * C + c) * bs + u2) * bs + v2];
                    } else if (!nhigh && !high) {
                        val = lo[(((long)slot[nk] * C + c) * lb + u2) * lb + v2];
                    } else if (high) { /* low neighbour: nearest upsampling */
                        val = lo[(((long)slot[nk] * C + c) * lb + (u2 >> 1)) * lb + (v2 >> 1)];
                    } else {           /* high neighbour: average or strided sampling */
                        const float* q = hi + ((long)slot[nk] * C + c) * bs * bs;
                        const int r = 2 * u2, s = 2 * v2;
                        if (sampling == ORC_PAD_STRIDED)
                            val = q[r * bs + s];
                        else
                            val = orc_avg4(q[r * bs + s], q[r * bs + s + 1],
                                           q[(r + 1) * bs + s], q[(r + 1) * bs + s + 1], dtype);
                    }
                }
            }
            out[((long)c * pe + (u + p)) * pe + (v + p)] = val;
        }
    }
    free(slot);
}

void orc_pad_ex(const float* hi, const float* lo, int N, int C, int H, int W,
                const uint8_t* mask, int bs, int dtype, int sampling, float* hp, float* lp)
{
    orc_pad_halo(hi, lo, N, C, H, W, mask, bs, dtype, sampling, 1, hp, lp);
}

/* BlockPad with average sampling, the module as the paper uses it. */
void orc_pad(const float* hi, const float* lo, int N, int C, int H, int W,
             const uint8_t* mask, int bs, int dtype, float* hp, float* lp)
{
    orc_pad_ex(hi, lo, N, C, H, W, mask, bs, dtype, ORC_PAD_AVG, hp, lp);
}

/* ------------------------------------------------------------------------ */
/* Block convolution: 3x3 "valid" convolution of every padded block.        */
/* ------------------------------------------------------------------------ */

/* P[S][Cin][E+2][E+2], w[Cout][Cin][3][3], bias[Cout] (or NULL)
 * -> out[S][Cout][E][E] in fp64:
 *    out = bias[co] + sum_ci sum_ky sum_kx w[co][ci][ky][kx] * P[ci][i+ky][j+kx]
 * (cross-correlation, as in every CNN framework), accumulated in fp64 in
 * the fixed order ci, ky, kx.  The products of fp16/bf16/fp32 operands are
 * exact in fp64. */
void orc_conv3x3_valid(const float* P, long S, int Cin, int E, const float* w,
                       const float* bias, int Cout, double* out)
{
    const int pe = E + 2;
    #pragma omp parallel for collapse(2) schedule(dynamic)
    for (long s = 0; s < S; ++s)
    for (int co = 0; co < Cout; ++co)
    for (int i = 0; i < E; ++i)
    for (int j = 0; j < E; ++j) {
        double acc = 0.0;
        for (int ci = 0; ci < Cin; ++ci) {
            const float* p = P + ((s * Cin + ci) * pe) * (long)pe;
            const float* wk = w + ((long)co * Cin + ci) * 9;
            for (int ky = 0; ky < 3; ++ky)
                for (int kx = 0; kx < 3; ++kx)
                    acc += (double)wk[ky * 3 + kx] * (double)p[(i + ky) * pe + (j + kx)];
        }
        if (bias) acc += (double)bias[co];
        out[((s * Cout + co) * E + i) * (long)E + j] = acc;
    }
}

/* ------------------------------------------------------------------------ */
/* Strided block convolution (the encoder's convolutions on block stacks).  */
/* ------------------------------------------------------------------------ */

/* P[S][Cin][E+2][E+2] (padded blocks), w[Cout][Cin][K][K] with K = 1 or 3,
 * stride st = 1 or 2 dividing E, bias[Cout] (or NULL)
 * -> out[S][Cout][E/st][E/st] in fp64:
 *    out[i][j] = bias[co] + sum_ci sum_ky sum_kx
 *                w[co][ci][ky][kx] * P[ci][st*i + ky + o][st*j + kx + o],
 *    o = 1 - K/2.
 * A 3x3 kernel is centred on block pixel (st*i, st*j) with one pixel of
 * padding (row 0 of a padded block is block row -1, so a stride-2 output
 * only ever reads the top and left halo); a 1x1 kernel reads block pixel
 * (st*i, st*j).  This is an ordinary strided convolution of the block with
 * the halo BlockPad gives it.  Accumulated in fp64 in the order ci, ky, kx. */
void orc_conv_block(const float* P, long S, int Cin, int E, const float* w, int K, int st,
                    const float* bias, int Cout, double* out)
{
    const int pe = E + 2, Eo = E / st, o = 1 - K / 2;
    #pragma omp parallel for collapse(2) schedule(dynamic)
    for (long s = 0; s < S; ++s)
    for (int co = 0; co < Cout; ++co)
    for (int i = 0; i < Eo; ++i)
    for (int j = 0; j < Eo; ++j) {
        double acc = 0.0;
        for (int ci = 0; ci < Cin; ++ci) {
            const float* p = P + ((s * Cin + ci) * pe) * (long)pe;
            const float* wk = w + ((long)co * Cin + ci) * K * K;
            for (int ky = 0; ky < K; ++ky)
                for (int kx = 0; kx < K; ++kx)
                    acc += (double)wk[ky * K + kx] * (double)p[(st * i + ky + o) * pe + (st * j + kx + o)];
        }
        if (bias) acc += (double)bias[co];
        out[((s * Cout + co) * Eo + i) * (long)Eo + j] = acc;
    }
}

/* ------------------------------------------------------------------------ */
/* Dense layers of the encoder around the block stages.                     */
/* ------------------------------------------------------------------------ */

/* x[N][Cin][H][W], w[Cout][Cin][K][K], zero padding `pad`, stride st,
 * bias[Cout] (or NULL) -> out[N][Cout][Ho][Wo] in fp64 with
 * Ho = (H + 2 pad - K) / st + 1 (likewise Wo); order ci, ky, kx. */
void orc_conv_dense(const float* x, int N, int Cin, int H, int W, const float* w, int K, int st, int pad,
                    const float* bias, int Cout, double* out)
{
    const int Ho = (H + 2 * pad - K) / st + 1, Wo = (W + 2 * pad - K) / st + 1;
    #pragma omp parallel for collapse(2) schedule(dynamic)
    for (int n = 0; n < N; ++n)
    for (int co = 0; co < Cout; ++co)
    for (int i = 0; i < Ho; ++i)
    for (int j = 0; j < Wo; ++j) {
        double acc = 0.0;
        for (int ci = 0; ci < Cin; ++ci) {
            const float* img = x + ((long)n * Cin + ci) * H * (long)W;
            const float* wk = w + ((long)co * Cin + ci) * K * K;
            for (int ky = 0; ky < K; ++ky) {
                const int y = st * i + ky - pad;
                if (y < 0 || y >= H) continue;
                for (int kx = 0; kx < K; ++kx) {
                    const int xx = st * j + kx - pad;
                    if (xx < 0 || xx >= W) continue;
                    acc += (double)wk[ky * K + kx] * (double)img[(long)y * W + xx];
                }
            }
        }
        if (bias) acc += (double)bias[co];
        out[(((long)n * Cout + co) * Ho + i) * (long)Wo + j] = acc;
    }
}

/* x[N][C][H][W] -> y[N][C][Ho][Wo]: maximum over the K x K window at stride
 * st with `pad` pixels of padding that never win (they are not candidates). */
void orc_maxpool(const float* x, int N, int C, int H, int W, int K, int st, int pad, float* y)
{
    const int Ho = (H + 2 * pad - K) / st + 1, Wo = (W + 2 * pad - K) / st + 1;
    for (int n = 0; n < N; ++n)
    for (int c = 0; c < C; ++c) {
        const float* img = x + ((long)n * C + c) * H * (long)W;
        for (int i = 0; i < Ho; ++i)
        for (int j = 0; j < Wo; ++j) {
            float m = -INFINITY;
            for (int ky = 0; ky < K; ++ky) {
                const int yy = st * i + ky - pad;
                if (yy < 0 || yy >= H) continue;
                for (int kx = 0; kx < K; ++kx) {
                    const int xx = st * j + kx - pad;
                    if (xx < 0 || xx >= W) continue;
                    if (img[(long)yy * W + xx] > m) m = img[(long)yy * W + xx];
                }
            }
            y[(((long)n * C + c) * Ho + i) * (long)Wo + j] = m;
        }
    }
}

/* ------------------------------------------------------------------------ */
/* BlockCombine: nearest-upsample the low blocks and reassemble the map.     */
/* ------------------------------------------------------------------------ */

/* hi[nh][C][bs][bs], lo[nl][C][lb][lb] -> y[N][C][H][W]. */
void orc_combine(const float* hi, const float* lo, int N, int C, int H, int W,
                 const uint8_t* mask, int bs, float* y)
{
    const int GH = H / bs, GW = W / bs, lb = bs / 2;
    long nh = 0, nl = 0;
    for (int n = 0; n < N; ++n)
    for (int gy = 0; gy < GH; ++gy)
    for (int gx = 0; gx < GW; ++gx) {
        const long k = ((long)n * GH + gy) * GW + gx;
        for (int c = 0; c < C; ++c) {
            float* img = y + ((long)n * C + c) * H * W;
            for (int i = 0; i < bs; ++i)
                for (int j = 0; j < bs; ++j) {
                    float v;
                    if (mask[k]) v = hi[((nh * C + c) * bs + i) * (long)bs + j];
                    else         v = lo[((nl * C + c) * lb + (i >> 1)) * (long)lb + (j >> 1)];
                    img[(long)(gy * bs + i) * W + gx * bs + j] = v;
                }
        }
        if (mask[k]) ++nh; else ++nl;
    }
}

/* ------------------------------------------------------------------------ */
/* Heuristic downsampling policy (the earlier short paper's policy, which    */
/* the ablation on execution policies compares with): a block's score is     */
/* how much detail its low-resolution version loses.                         */
/* ------------------------------------------------------------------------ */

/* x[N][C][H][W] -> score[N][GH][GW] (fp64): for every pixel of the block the
 * Euclidean distance over the channels between the pixel and the block's
 * low-resolution version at that pixel (the 2x2 average of its cell, as
 * BlockSample computes and rounds it, nearest-upsampled), averaged over the
 * block's bs*bs pixels. */
void orc_policy_scores(const float* x, int N, int C, int H, int W, int bs, int dtype, double* score)
{
    const int GH = H / bs, GW = W / bs;
    for (int n = 0; n < N; ++n)
    for (int gy = 0; gy < GH; ++gy)
    for (int gx = 0; gx < GW; ++gx) {
        double total = 0.0;
        for (int i = 0; i < bs; ++i)
        for (int j = 0; j < bs; ++j) {
            const int Y = gy * bs + i, X = gx * bs + j;
            const int Y0 = Y & ~1, X0 = X & ~1;     /* the 2x2 cell containing the pixel */
            double d2 = 0.0;
            for (int c = 0; c < C; ++c) {
                const float* img = x + ((long)n * C + c) * H * (long)W;
                const float m = orc_avg4(img[(long)Y0 * W + X0], img[(long)Y0 * W + X0 + 1],
                                         img[(long)(Y0 + 1) * W + X0], img[(long)(Y0 + 1) * W + X0 + 1], dtype);
                const double d = (double)img[(long)Y * W + X] - (double)m;
                d2 += d * d;
            }
            total += sqrt(d2);
        }
        score[((long)n * GH + gy) * GW + gx] = total / ((double)bs * bs);
    }
}

/* score[N][B] -> mask[N][B]: per image, the k blocks with the highest scores
 * are high resolution (1), the others low (0); equal scores are ranked by
 * block id, lower first. */
void orc_policy_select(const double* score, int N, int B, int k, uint8_t* mask)
{
    for (int n = 0; n < N; ++n)
        for (int b = 0; b < B; ++b) {
            const double s = score[(long)n * B + b];
            int rank = 0;  /* blocks ahead of b in the order */
            for (int j = 0; j < B; ++j) {
                const double t = score[(long)n * B + j];
                if (t > s || (t == s && j < b)) ++rank;
            }
            mask[(long)n * B + b] = rank < k ? 1 : 0;
        }
}

/* ------------------------------------------------------------------------ */
/* Backward pass of the block modules and of the block convolution: the     */
/* transposes of the linear maps above (the paper notes the modules serve    */
/* training as well as inference).  Gradients are stored in the storage      */
/* type like the forward values.                                             */
/* ------------------------------------------------------------------------ */

/* BlockCombine transposed: dy[N][C][H][W] -> dhi[nh][C][bs][bs] (copy of the
 * block's gradient) and dlo[nl][C][lb][lb] (the sum of the 2x2 cell of
 * gradients that the low pixel was copied to), summed in fp32 as
 * ((a + b) + (c + d)) with a, b the top pixels, rounded once. */
void orc_combine_bwd(const float* dy, int N, int C, int H, int W, const uint8_t* mask, int bs, int dtype,
                     float* dhi, float* dlo)
{
    const int GH = H / bs, GW = W / bs, lb = bs / 2;
    long nh = 0, nl = 0;
    for (int n = 0; n < N; ++n)
    for (int gy = 0; gy < GH; ++gy)
    for (int gx = 0; gx < GW; ++gx) {
        const long k = ((long)n * GH + gy) * GW + gx;
        for (int c = 0; c < C; ++c) {
            const float* img = dy + ((long)n * C + c) * H * W;
            if (mask[k]) {
                for (int i = 0; i < bs; ++i)
                    for (int j = 0; j < bs; ++j)
                        dhi[((nh * C + c) * bs + i) * (long)bs + j] = img[(long)(gy * bs + i) * W + gx * bs + j];
            } else {
                for (int i = 0; i < lb; ++i)
                    for (int j = 0; j < lb; ++j) {
                        const long r0 = (long)(gy * bs + 2 * i) * W + gx * bs + 2 * j;
                        const float sum = (img[r0] + img[r0 + 1]) + (img[r0 + W] + img[r0 + W + 1]);
                        dlo[((nl * C + c) * lb + i) * (long)lb + j] = (float)orc_round((double)sum, dtype);
                    }
            }
        }
        if (mask[k]) ++nh; else ++nl;
    }
}

/* BlockSample transposed: dhi, dlo -> dx[N][C][H][W]: a high block's
 * gradient copied back; a low pixel's gradient times 0.25 (its share of the
 * average) on each pixel of its cell, rounded. */
void orc_split_bwd(const float* dhi, const float* dlo, int N, int C, int H, int W, const uint8_t* mask, int bs,
                   int dtype, float* dx)
{
    const int GH = H / bs, GW = W / bs, lb = bs / 2;
    long nh = 0, nl = 0;
    for (int n = 0; n < N; ++n)
    for (int gy = 0; gy < GH; ++gy)
    for (int gx = 0; gx < GW; ++gx) {
        const long k = ((long)n * GH + gy) * GW + gx;
        for (int c = 0; c < C; ++c) {
            float* img = dx + ((long)n * C + c) * H * W;
            for (int i = 0; i < bs; ++i)
                for (int j = 0; j < bs; ++j) {
                    float v;
                    if (mask[k]) v = dhi[((nh * C + c) * bs + i) * (long)bs + j];
                    else v = (float)orc_round(0.25 * (double)dlo[((nl * C + c) * lb + (i >> 1)) * (long)lb + (j >> 1)],
                                              dtype);
                    img[(long)(gy * bs + i) * W + gx * bs + j] = v;
                }
        }
        if (mask[k]) ++nh; else ++nl;
    }
}

/* BlockPad transposed: dhp[nh][C][bs+2][bs+2], dlp[nl][C][lb+2][lb+2]
 * -> dhi, dlo.  Every padded pixel hands its gradient back to the pixels
 * orc_pad_ex read it from: the block's own pixel (interior), the neighbour's
 * pixel at equal resolution, the low neighbour's pixel a high block's halo
 * nearest-upsampled, the 2x2 cell of a high neighbour a low block's halo
 * averaged (a quarter to each; all of it to the top-left pixel with strided
 * sampling); zero-padding and the image border read nothing.  Accumulated in
 * fp64 in block order, then rounded. */
void orc_pad_bwd(const float* dhp, const float* dlp, int N, int C, int H, int W, const uint8_t* mask, int bs,
                 int dtype, int sampling, float* dhi, float* dlo)
{
    const int GH = H / bs, GW = W / bs, lb = bs / 2;
    const long B = (long)N * GH * GW;
    int32_t* slot = (int32_t*)malloc(sizeof(int32_t) * (size_t)(B > 0 ? B : 1));
    int32_t counts[2];
    orc_plan(mask, B, slot, NULL, NULL, counts);
    const long nhi = (long)counts[0] * C * bs * bs, nlo = (long)counts[1] * C * lb * lb;
    double* ah = (double*)calloc((size_t)(nhi > 0 ? nhi : 1), sizeof(double));
    double* al = (double*)calloc((size_t)(nlo > 0 ? nlo : 1), sizeof(double));
    for (int n = 0; n < N; ++n)
    for (int gy = 0; gy < GH; ++gy)
    for (int gx = 0; gx < GW; ++gx) {
        const long k = ((long)n * GH + gy) * GW + gx;
        const int high = mask[k] != 0;
        const int e = high ? bs : lb, pe = e + 2;
        const float* g = high ? dhp + (long)slot[k] * C * pe * pe : dlp + (long)slot[k] * C * pe * pe;
        for (int c = 0; c < C; ++c)
        for (int u = -1; u <= e; ++u)
        for (int v = -1; v <= e; ++v) {
            const double gv = (double)g[((long)c * pe + (u + 1)) * pe + (v + 1)];
            const int dy = u < 0 ? -1 : (u >= e ? 1 : 0);
            const int dx = v < 0 ? -1 : (v >= e ? 1 : 0);
            if (dy == 0 && dx == 0) {
                double* own = high ? ah + (long)slot[k] * C * bs * bs : al + (long)slot[k] * C * lb * lb;
                own[((long)c * e + u) * e + v] += gv;
                continue;
            }
            if (sampling == ORC_PAD_ZERO) continue;
            const int ny = gy + dy, nx = gx + dx;
            if (ny < 0 || ny >= GH || nx < 0 || nx >= GW) continue;
            const long nk = ((long)n * GH + ny) * GW + nx;
            const int nhigh = mask[nk] != 0;
            const int u2 = u - dy * e, v2 = v - dx * e;
            if (nhigh && high) {
                ah[(((long)slot[nk] * C + c) * bs + u2) * bs + v2] += gv;
            } else if (!nhigh && !high) {
                al[(((long)slot[nk] * C + c) * lb + u2) * lb + v2] += gv;
            } else if (high) {
                al[(((long)slot[nk] * C + c) * lb + (u2 >> 1)) * lb + (v2 >> 1)] += gv;
            } else {
                double* q = ah + ((long)slot[nk] * C + c) * bs * bs;
                const int r = 2 * u2, s = 2 * v2;
                if (sampling == ORC_PAD_STRIDED) {
                    q[r * bs + s] += gv;
                } else {
                    q[r * bs + s] += 0.25 * gv;
                    q[r * bs + s + 1] += 0.25 * gv;
                    q[(r + 1) * bs + s] += 0.25 * gv;
                    q[(r + 1) * bs + s + 1] += 0.25 * gv;
                }
            }
        }
    }
    orc_round_array(ah, dhi, nhi, dtype);
    orc_round_array(al, dlo, nlo, dtype);
    free(ah);
    free(al);
    free(slot);
}

/* Gradient of the 3x3 valid block convolution with respect to its padded
 * input: dO[S][Cout][E][E], w[Cout][Cin][3][3] -> dP[S][Cin][E+2][E+2] (fp64):
 *   dP[s][ci][u][v] = sum_co sum_ky sum_kx w[co][ci][ky][kx] * dO[s][co][u-ky][v-kx]
 * over the (u-ky, v-kx) inside the block, in the order co, ky, kx. */
void orc_conv3x3_bwd_data(const float* dO, long S, int Cout, int E, const float* w, int Cin, double* dP)
{
    const int pe = E + 2;
    #pragma omp parallel for collapse(2) schedule(dynamic)
    for (long s = 0; s < S; ++s)
    for (int ci = 0; ci < Cin; ++ci)
    for (int u = 0; u < pe; ++u)
    for (int v = 0; v < pe; ++v) {
        double acc = 0.0;
        for (int co = 0; co < Cout; ++co) {
            const float* g = dO + ((s * Cout + co) * E) * (long)E;
            const float* wk = w + ((long)co * Cin + ci) * 9;
            for (int ky = 0; ky < 3; ++ky) {
                const int i = u - ky;
                if (i < 0 || i >= E) continue;
                for (int kx = 0; kx < 3; ++kx) {
                    const int j = v - kx;
                    if (j < 0 || j >= E) continue;
                    acc += (double)wk[ky * 3 + kx] * (double)g[i * E + j];
                }
            }
        }
        dP[((s * Cin + ci) * pe + u) * (long)pe + v] = acc;
    }
}

/* Gradient with respect to the weights and the bias, accumulated over one
 * stack (call once per stack and add): P[S][Cin][E+2][E+2], dO[S][Cout][E][E]
 *   dw[co][ci][ky][kx] += sum_s sum_i sum_j dO[s][co][i][j] * P[s][ci][i+ky][j+kx]
 *   db[co]             += sum_s sum_i sum_j dO[s][co][i][j]        (db may be NULL)
 * in fp64, in the order s, i, j. */
void orc_conv3x3_bwd_weight(const float* P, const float* dO, long S, int Cin, int Cout, int E, double* dw, double* db)
{
    const int pe = E + 2;
    #pragma omp parallel for collapse(2) schedule(dynamic)
    for (int co = 0; co < Cout; ++co)
    for (int ci = 0; ci < Cin; ++ci)
    for (int t = 0; t < 9; ++t) {
        const int ky = t / 3, kx = t % 3;
        double acc = 0.0;
        for (long s = 0; s < S; ++s) {
            const float* g = dO + ((s * Cout + co) * E) * (long)E;
            const float* p = P + ((s * Cin + ci) * pe) * (long)pe;
            for (int i = 0; i < E; ++i)
                for (int j = 0; j < E; ++j) acc += (double)g[i * E + j] * (double)p[(i + ky) * pe + (j + kx)];
        }
        dw[((long)co * Cin + ci) * 9 + t] += acc;
    }
    if (db)
        for (int co = 0; co < Cout; ++co) {
            double acc = 0.0;
            for (long s = 0; s < S; ++s) {
                const float* g = dO + ((s * Cout + co) * E) * (long)E;
                for (int i = 0; i < E * E; ++i) acc += (double)g[i];
            }
            db[co] += acc;
        }
}

/* ------------------------------------------------------------------------ */
/* Layers beyond 3x3 on block stacks: every padded layer of the network can  */
/* run blockwise once BlockPad supplies a halo as wide as the kernel reaches */
/* (the blocks then persist from the image to the last stage).              */
/* ------------------------------------------------------------------------ */

/* P[S][Cin][E+2p][E+2p] (halo p), w[Cout][Cin][K][K] (K odd), stride st
 * dividing E, dilation dl with dl*(K-1)/2 <= p, bias or NULL
 * -> out[S][Cout][E/st][E/st] (fp64):
 *    out[i][j] = bias + sum_ci sum_ky sum_kx w * P[st*i + dl*ky + o][st*j + dl*kx + o],
 *    o = p - dl*(K-1)/2,
 * i.e. the kernel centred on block pixel (st*i, st*j); order ci, ky, kx. */
void orc_conv_block_general(const float* P, long S, int Cin, int E, int p, const float* w, int K, int st, int dl,
                            const float* bias, int Cout, double* out)
{
    const int pe = E + 2 * p, Eo = E / st, o = p - dl * (K - 1) / 2;
    #pragma omp parallel for collapse(2) schedule(dynamic)
    for (long s = 0; s < S; ++s)
    for (int co = 0; co < Cout; ++co)
    for (int i = 0; i < Eo; ++i)
    for (int j = 0; j < Eo; ++j) {
        double acc = 0.0;
        for (int ci = 0; ci < Cin; ++ci) {
            const float* q = P + ((s * Cin + ci) * pe) * (long)pe;
            const float* wk = w + ((long)co * Cin + ci) * K * K;
            for (int ky = 0; ky < K; ++ky)
                for (int kx = 0; kx < K; ++kx)
                    acc += (double)wk[ky * K + kx] * (double)q[(st * i + dl * ky + o) * pe + (st * j + dl * kx + o)];
        }
        if (bias) acc += (double)bias[co];
        out[((s * Cout + co) * Eo + i) * (long)Eo + j] = acc;
    }
}

/* P[S][C][E+2p][E+2p] -> out[S][C][E/st][E/st]: maximum over the K x K window
 * centred on block pixel (st*i, st*j) (o = p - (K-1)/2), halo values included
 * (zeros at the image border, which never exceed a ReLU output). */
void orc_maxpool_block(const float* P, long S, int C, int E, int p, int K, int st, float* out)
{
    const int pe = E + 2 * p, Eo = E / st, o = p - (K - 1) / 2;
    for (long s = 0; s < S; ++s)
    for (int c = 0; c < C; ++c)
    for (int i = 0; i < Eo; ++i)
    for (int j = 0; j < Eo; ++j) {
        const float* q = P + ((s * C + c) * pe) * (long)pe;
        float m = -INFINITY;
        for (int ky = 0; ky < K; ++ky)
            for (int kx = 0; kx < K; ++kx) {
                const float v = q[(st * i + ky + o) * pe + (st * j + kx + o)];
                if (v > m) m = v;
            }
        out[((s * C + c) * Eo + i) * (long)Eo + j] = m;
    }
}
