/*
 * segblocks.h -- C ABI of libsegblocks.so, block-based dynamic-resolution
 * convolution for AMD Instinct MI355X (gfx950).
 *
 * Method: SegBlocks (Verelst & Tuytelaars, arXiv 2011.12025), Method section,
 * "Block modules".  A feature map is cut into a grid of bs x bs blocks; a
 * per-block mask selects high or low resolution for every block; low blocks
 * are 2x average-pooled (BlockSample), every block gets a one-pixel halo
 * taken from its neighbours (BlockPad), the same 3x3 filters run on both
 * block stacks, and the results are reassembled into a full-resolution map
 * with the low blocks nearest-upsampled (BlockCombine).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Pointers are DEVICE pointers unless stated otherwise.  The caller owns
 *    every buffer; the library allocates no device memory.  Four calls may
 *    need scratch memory beyond their inputs and outputs (fp32 partial tiles
 *    of a reduction split over several workgroups, a padded copy of the low
 *    stack, the packed stacks of a fused layer with many channels):
 *    segblocks_block_conv3x3, segblocks_block_conv_ex,
 *    segblocks_block_conv_chain and segblocks_layer take it as a `workspace` pointer with its size `ws_bytes`.  The size a
 *    call needs depends only on its shapes, capacities and device, and is
 *    given by segblocks_block_conv3x3_workspace_size,
 *    segblocks_block_conv_ex_workspace_size,
 *    segblocks_block_conv_chain_workspace_size and
 *    segblocks_layer_workspace_size (0 = none needed; NULL is then fine).  A
 *    workspace must be 256-byte aligned and must not overlap any argument;
 *    a smaller one (or NULL when one is needed) fails with SB_ENOMEM before
 *    anything is launched.  The workspace holds no state between calls, but
 *    it is in use until the call's kernels finish on `stream`: calls that
 *    may overlap need workspaces of their own.
 *  - Logical dimensions are always N, C, H, W.  `layout` selects the memory
 *    format of every 4-d tensor of the call (input, stacks, output and the
 *    convolution weight):
 *      SB_NCHW  contiguous [N][C][H][W]          (PyTorch default)
 *      SB_NHWC  contiguous [N][H][W][C]          (PyTorch channels_last)
 *    A block stack with S blocks of extent e is a tensor of logical shape
 *    [S, C, e, e] in the same memory format.
 *  - dtype is the storage type of every feature tensor, weight and bias of
 *    the call: SB_F32, SB_F16 or SB_BF16.  Arithmetic is fp32.
 *  - mask is uint8 [N][H/bs][W/bs] (row-major).  mask != 0 selects HIGH
 *    resolution for that block (the paper's action a_b = 1).  Block id
 *    k = (n*GH + gy)*GW + gx with GH = H/bs, GW = W/bs.
 *  - Blocks are packed into the high stack and into the low stack in
 *    increasing block id (stable compaction): the slot of block k is the
 *    number of blocks before k with the same resolution.  nh = number of
 *    high blocks, nl = number of low blocks.
 *  - Stack capacities hi_cap / lo_cap are the number of blocks each stack
 *    buffer can hold.  The kernels read the true nh / nl from the mask on
 *    the device; a block whose slot is >= the capacity of its stack is
 *    skipped (not read, not written; BlockPad reads it as zeros; BlockCombine
 *    writes zeros for it).  Allocate nh / nl blocks after segblocks_count, or
 *    N*GH*GW blocks for each stack to avoid the synchronisation.
 *  - bs must be even and >= 2, and divide H and W.  Low blocks have extent
 *    lb = bs/2.
 *  - Every call except segblocks_count is asynchronous on `stream` and
 *    performs no host synchronisation.  Calls may come from several host
 *    threads at once (the library's launch-setup state is per device and
 *    guarded).  Arguments are validated on the host
 *    before anything is launched; on failure nothing is launched, the call
 *    returns a negative sb_status and segblocks_last_error() describes it.
 *    Device faults surface at the caller's next synchronisation.
 *  - Output buffers must not overlap input buffers.
 *
 * Arithmetic
 *  - The 2x2 average (BlockSample's pooling and BlockPad's average sampling)
 *    is computed in fp32 as ((a + b) + (c + d)) * 0.25 with a, b the top
 *    and c, d the bottom pixels of the cell, then rounded to nearest-even.
 *    Split, pad and combine are therefore bit-exact and deterministic.
 *  - Convolutions accumulate in fp32 (MFMA), add the bias in fp32 and round
 *    once to the storage type (nearest-even).
 */
#ifndef SEGBLOCKS_H
#define SEGBLOCKS_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { SB_F32 = 0, SB_F16 = 1, SB_BF16 = 2 } sb_dtype;
typedef enum { SB_NCHW = 0, SB_NHWC = 1 } sb_layout;
typedef enum {
    SB_OK = 0,
    SB_EINVAL = -1, /* null pointer, bad enum, non-positive size, aliasing   */
    SB_ESHAPE = -2, /* bs odd or < 2, bs does not divide H or W, too large   */
    SB_EHIP = -3,   /* a HIP runtime call failed (message from the runtime)  */
    SB_ENOMEM = -4  /* the workspace argument is NULL or smaller than needed */
} sb_status;

/* Flags of the convolutions (segblocks_block_conv3x3, segblocks_block_conv_ex,
 * segblocks_layer). */
#define SB_FLAG_RELU 1 /* max(0, .) after bias (and residual) */
/* BlockPad alternatives (paper: Method > Block modules > BlockPad weighs
 * strided subsampling against average sampling for a low block's halo taken
 * from a high neighbour; Experiments > Ablation studies, sampling pattern,
 * also compares plain zero padding).  At most one of the two: */
#define SB_FLAG_PAD_STRIDED 2 /* the high neighbour's cell gives its top-left pixel */
#define SB_FLAG_PAD_ZERO 4    /* every block is zero-padded on its own (no BlockPad) */

/* Sampling of segblocks_pad_ex (the same three choices). */
#define SB_PAD_AVG 0
#define SB_PAD_STRIDED 1
#define SB_PAD_ZERO 2

/* Number of high (mask != 0) and low blocks of a mask.  BLOCKING: copies the
 * mask to the host on `stream` and waits for it.  n_high / n_low are HOST
 * pointers.  Not needed on the hot path (see the capacity convention). */
int segblocks_count(const uint8_t* mask, int N, int GH, int GW,
                    int* n_high, int* n_low, hipStream_t stream);

/* BlockSample (paper: Method > Block modules > BlockSample).
 * x [N,C,H,W] -> hi [nh,C,bs,bs] (block copied) and lo [nl,C,bs/2,bs/2]
 * (2x2 average of the block). */
int segblocks_split(const void* x, int dtype, int layout, int N, int C, int H, int W,
                    const uint8_t* mask, int bs,
                    void* hi, int hi_cap, void* lo, int lo_cap, hipStream_t stream);

/* BlockPad with average sampling (paper: Method > Block modules > BlockPad).
 * hi [nh,C,bs,bs], lo [nl,C,lb,lb] -> hi_pad [nh,C,bs+2,bs+2],
 * lo_pad [nl,C,lb+2,lb+2].  Interior: the block itself.  A halo pixel is
 * taken from the neighbouring block in its direction (the diagonal block for
 * corners): same resolution -> copied; low neighbour of a high block ->
 * nearest-upsampled; high neighbour of a low block -> 2x2 average; outside
 * the image -> 0.  hi/hi_pad hold hi_cap blocks, lo/lo_pad lo_cap blocks. */
int segblocks_pad(const void* hi, const void* lo, int dtype, int layout,
                  int N, int C, int H, int W, const uint8_t* mask, int bs,
                  void* hi_pad, void* lo_pad, int hi_cap, int lo_cap, hipStream_t stream);

/* segblocks_pad with a choice of how a low block's halo samples a high
 * neighbour (paper: Method > Block modules > BlockPad, the two options it
 * weighs; Experiments > Ablation studies, sampling pattern):
 *   SB_PAD_AVG      the 2x2 average of the neighbour's cell (= segblocks_pad)
 *   SB_PAD_STRIDED  the cell's top-left pixel (strided subsampling)
 *   SB_PAD_ZERO     no BlockPad: every halo pixel of every block is 0
 * Any other value is SB_EINVAL.  Bit-exact like segblocks_pad. */
int segblocks_pad_ex(const void* hi, const void* lo, int dtype, int layout,
                     int N, int C, int H, int W, const uint8_t* mask, int bs,
                     void* hi_pad, void* lo_pad, int hi_cap, int lo_cap, int sampling,
                     hipStream_t stream);

/* Block convolution on padded stacks (paper: Method -- the same filters are
 * applied to the high- and the low-resolution blocks).  3x3, stride 1,
 * "valid" on every padded block:
 *   out[s,co,i,j] = bias[co] + sum_{ci,ky,kx} w[co,ci,ky,kx] * pad[s,ci,i+ky,j+kx]
 * hi_pad [nh,C_in,bs+2,bs+2], lo_pad [nl,C_in,lb+2,lb+2]
 *   -> hi_out [nh,C_out,bs,bs], lo_out [nl,C_out,lb,lb].
 * weight: logical [C_out][C_in][3][3] in the call's memory format: OIHW
 * memory for SB_NCHW, OHWI memory ([C_out][3][3][C_in], a channels_last
 * weight tensor) for SB_NHWC.  bias [C_out] or NULL.  Both in `dtype`. */
int segblocks_conv3x3(const void* hi_pad, const void* lo_pad, int dtype, int layout,
                      int N, int C_in, int H, int W, const uint8_t* mask, int bs,
                      const void* weight, const void* bias, int C_out,
                      void* hi_out, void* lo_out, int hi_cap, int lo_cap, hipStream_t stream);

/* BlockCombine (paper: Method > Block modules > BlockCombine).
 * hi [nh,C,bs,bs], lo [nl,C,lb,lb] -> y [N,C,H,W]; a low block is written
 * nearest-upsampled (each value covers 2x2 output pixels). */
int segblocks_combine(const void* hi, const void* lo, int dtype, int layout,
                      int N, int C, int H, int W, const uint8_t* mask, int bs,
                      int hi_cap, int lo_cap, void* y, hipStream_t stream);

/* Block convolution with BlockPad fused into the tile load: packed stacks in,
 * packed stacks out, no padded stacks in memory.  Equal to
 * segblocks_conv3x3(segblocks_pad(hi, lo)) followed by the optional epilogue
 *   out = act(conv + bias + residual)
 * with residual_hi / residual_lo stacks shaped like the outputs (or both
 * NULL) and act = ReLU when flags & SB_FLAG_RELU.  SB_FLAG_PAD_STRIDED or
 * SB_FLAG_PAD_ZERO replace the fused BlockPad by its alternatives (as
 * segblocks_pad_ex with SB_PAD_STRIDED / SB_PAD_ZERO).  hi/hi_out/residual_hi hold
 * hi_cap blocks, lo/lo_out/residual_lo lo_cap blocks. */
int segblocks_block_conv3x3(const void* hi, const void* lo, int dtype, int layout,
                            int N, int C_in, int H, int W, const uint8_t* mask, int bs,
                            const void* weight, const void* bias, int C_out, int flags,
                            const void* residual_hi, const void* residual_lo,
                            void* hi_out, void* lo_out, int hi_cap, int lo_cap,
                            void* workspace, size_t ws_bytes, hipStream_t stream);

/* One complete block-conv layer:
 *   y = combine(conv3x3(pad(split(x))))
 * x [N,C_in,H,W] -> y [N,C_out,H,W]; weight/bias as in segblocks_conv3x3.
 * Channels-last fp16/bf16 with C_in <= 64 and blocks of 32 or 64 run as one
 * kernel (the packed stacks never reach memory); channels-last fp16/bf16
 * with C_in % 64 == 0 and C_in > 64 run on the implicit GEMM of
 * segblocks_block_conv3x3: with average sampling as two kernels (the padded
 * low stack straight from x into the workspace, then the GEMM reading the
 * high blocks from x and writing y), with the other samplings as split, the
 * block convolution and combine over packed stacks in the workspace (for
 * 128 < C_in <= 256 only above 8192 pixels, N * H * W); everything else runs
 * as one general kernel.  Intermediate values are rounded to `dtype` exactly where the
 * four-call chain stores them, so the result equals that chain's up to the
 * order of the fp32 accumulation.  flags: SB_FLAG_RELU (after the bias) and
 * the BlockPad alternatives, as for segblocks_block_conv3x3. */
int segblocks_layer(const void* x, int dtype, int layout, int N, int C_in, int H, int W,
                    const uint8_t* mask, int bs, const void* weight, const void* bias,
                    int C_out, int flags, void* y, void* workspace, size_t ws_bytes,
                    hipStream_t stream);

/* The encoder's block convolutions (paper: Method -- the network keeps its
 * blocks through the downsampling stages, so blocks shrink with the map):
 * K x K convolution, K in {1, 3}, at stride S in {1, 2}, of every block of
 * the packed stacks, BlockPad fused for K = 3 (one pixel of halo; a stride-2
 * output only reads the top and left halo), with the epilogue of
 * segblocks_block_conv3x3 (bias, residual, SB_FLAG_RELU, one rounding):
 *   out[s,co,i,j] = bias[co] + sum_{ci,ky,kx} w[co,ci,ky,kx]
 *                   * padded[s,ci, S*i + ky + 1 - K/2, S*j + kx + 1 - K/2]
 * hi [nh,C_in,bs,bs], lo [nl,C_in,bs/2,bs/2]
 *   -> hi_out [nh,C_out,bs/S,bs/S], lo_out [nl,C_out,bs/(2S),bs/(2S)];
 * residual_hi / residual_lo (or NULL) have the outputs' shapes.  H, W, bs
 * describe the INPUT map.  weight: OHWI memory [C_out][K][K][C_in].
 * Channels-last (SB_NHWC) fp16 / bf16 with C_in % 8 == 0 only (else
 * SB_EINVAL); bs / 2 must be divisible by S. */
int segblocks_block_conv_ex(const void* hi, const void* lo, int dtype, int layout,
                            int N, int C_in, int H, int W, const uint8_t* mask, int bs,
                            const void* weight, const void* bias, int C_out,
                            int ksize, int stride, int flags,
                            const void* residual_hi, const void* residual_lo,
                            void* hi_out, void* lo_out, int hi_cap, int lo_cap,
                            void* workspace, size_t ws_bytes, hipStream_t stream);

/* segblocks_block_conv_ex for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): the same arguments, results and kernels, without the
 * workspace.  Scratch space comes from a fixed buffer of
 * SB_NOALLOC_SCRATCH_BYTES that the library holds on every device it runs on
 * until the process ends; a call that would need more (see
 * segblocks_block_conv_ex_workspace_size) fails with SB_ENOMEM before
 * anything is launched.  The call allocates nothing.  Every call on one
 * device shares that device's buffer: calls that may overlap on one device
 * (different streams, or host threads) race and must be ordered by the
 * caller.  The buffer keeps the last call's contents; each call writes every
 * scratch byte it reads, so nothing has to be cleared. */
#define SB_NOALLOC_SCRATCH_BYTES (16u << 20)
int segblocks_block_conv_ex_noalloc(const void* hi, const void* lo, int dtype, int layout,
                                    int N, int C_in, int H, int W, const uint8_t* mask, int bs,
                                    const void* weight, const void* bias, int C_out,
                                    int ksize, int stride, int flags,
                                    const void* residual_hi, const void* residual_lo,
                                    void* hi_out, void* lo_out, int hi_cap, int lo_cap,
                                    hipStream_t stream);

/* A block convolution for chains of them (paper: Method > Block modules >
 * BlockPad -- with average sampling a low block's halo cell facing a high
 * neighbour is the 2x2 average of that neighbour's cell, i.e. a pixel of the
 * high block at half resolution).  The arguments and results of
 * segblocks_block_conv_ex (3x3 at stride 1 takes the routes of
 * segblocks_block_conv3x3), plus:
 *   hi_half [nh, C_in, bs/2, bs/2] (input, or NULL): the high input blocks at
 *     half resolution, hi_half[s,c,u,v] = the 2x2 average of
 *     hi[s,c,2u..2u+1,2v..2v+1] rounded to dtype, as hi_out_half of the call
 *     that wrote `hi` gives it.  With average sampling the implicit GEMM then
 *     takes those halo cells from it instead of padding the low stack in a
 *     launch of its own; the other routes ignore it.  The result is the same
 *     bit for bit either way; a hi_half that is not those averages gives
 *     wrong results.
 *   hi_out_half [nh, C_out, bo/2, bo/2] (output, or NULL; bo = bs/stride must
 *     be even and C_out % 8 == 0): receives hi_out at half resolution, from
 *     the GEMM's epilogue where its tile layout allows, else from one extra
 *     launch after the convolution.
 * hi_half and hi_out_half are 16-byte aligned (with hi_out_half, hi_out as
 * well); they hold hi_cap blocks (slots past the mask's high count are
 * written with don't-care values).  Workspace:
 * segblocks_block_conv_chain_workspace_size (enough with or without
 * hi_half). */
int segblocks_block_conv_chain(const void* hi, const void* lo, const void* hi_half, int dtype,
                               int layout, int N, int C_in, int H, int W, const uint8_t* mask,
                               int bs, const void* weight, const void* bias, int C_out,
                               int ksize, int stride, int flags,
                               const void* residual_hi, const void* residual_lo,
                               void* hi_out, void* lo_out, void* hi_out_half, int hi_cap,
                               int lo_cap, void* workspace, size_t ws_bytes, hipStream_t stream);

/* Whether segblocks_block_conv_chain with these shapes, flags and
 * capacities (16-byte aligned buffers) reads hi_half, so that the call
 * producing its input knows whether to ask for hi_out_half: *reads (HOST
 * pointer) = 1 or 0.  Pure host function; arguments are validated as in
 * the workspace queries. */
int segblocks_block_conv_chain_reads_half(int dtype, int layout, int N, int C_in, int H, int W,
                                          int bs, int C_out, int ksize, int stride, int flags,
                                          int hi_cap, int lo_cap, int* reads);

/* Workspace sizes (bytes, HOST out-parameter) of segblocks_block_conv3x3,
 * segblocks_block_conv_ex, segblocks_block_conv_chain and segblocks_layer for the given shapes and
 * stack capacities on the current device; the arguments mean what they mean
 * in those calls and are validated the same way.  The size covers every
 * flag combination (a call checks only what its own route needs) and assumes
 * 16-byte aligned buffers (a call with less aligned buffers takes a route
 * that needs no more).  Pure host functions: nothing is launched. */
int segblocks_block_conv3x3_workspace_size(int dtype, int layout, int N, int C_in, int H, int W,
                                           int bs, int C_out, int hi_cap, int lo_cap, size_t* bytes);
int segblocks_block_conv_ex_workspace_size(int dtype, int layout, int N, int C_in, int H, int W,
                                           int bs, int C_out, int ksize, int stride,
                                           int hi_cap, int lo_cap, size_t* bytes);
int segblocks_block_conv_chain_workspace_size(int dtype, int layout, int N, int C_in, int H, int W,
                                              int bs, int C_out, int ksize, int stride,
                                              int hi_cap, int lo_cap, size_t* bytes);
int segblocks_layer_workspace_size(int dtype, int layout, int N, int C_in, int H, int W, int bs,
                                   int C_out, size_t* bytes);

/* ------------------------------------------------------------------------
 * Wider halos (paper: Method > Block modules -- BlockPad replaces the zero
 * padding of every padded layer and the blocks shrink with the map, so a
 * network can keep its blocks from the image on).  A K x K layer needs a
 * halo of (K-1)/2 pixels, a dilated one dilation*(K-1)/2.
 * ------------------------------------------------------------------------ */

/* BlockPad with a halo of `halo` pixels, 1 <= halo <= bs/2 (every halo pixel
 * then lies in the adjacent block, taken by the rules of segblocks_pad_ex):
 * hi [nh,C,bs,bs], lo [nl,C,lb,lb] -> hi_pad [nh,C,bs+2h,bs+2h],
 * lo_pad [nl,C,lb+2h,lb+2h].  halo = 1 is segblocks_pad_ex. */
int segblocks_pad_halo(const void* hi, const void* lo, int dtype, int layout, int N, int C, int H,
                       int W, const uint8_t* mask, int bs, int halo, int sampling, void* hi_pad,
                       void* lo_pad, int hi_cap, int lo_cap, hipStream_t stream);

/* K x K convolution (K odd) at stride 1 or 2 with dilation on stacks padded
 * by `halo` >= dilation*(K-1)/2 (e.g. the 7x7/2 stem on image blocks with a
 * 3-pixel halo):
 *   out[s,co,i,j] = bias[co] + sum w[co,ci,ky,kx] *
 *                   pad[s,ci, st*i + dil*ky + o, st*j + dil*kx + o],  o = halo - dil*(K-1)/2
 * -> hi_out [nh,C_out,bs/st,bs/st], lo_out [nl,C_out,lb/st,lb/st];
 * weight [C_out][C_in][K][K] in the call's memory format (OHWI for
 * SB_NHWC), bias [C_out] or NULL, flags: SB_FLAG_RELU.  H, W, bs describe
 * the unpadded map.  fp32 sums, one rounding. */
int segblocks_conv_halo(const void* hi_pad, const void* lo_pad, int dtype, int layout, int N, int C_in,
                        int H, int W, const uint8_t* mask, int bs, int halo, const void* weight,
                        const void* bias, int C_out, int ksize, int stride, int dilation, int flags,
                        void* hi_out, void* lo_out, int hi_cap, int lo_cap, hipStream_t stream);

/* K x K max-pooling (K odd) at stride 1 or 2 of stacks padded by
 * halo >= (K-1)/2; the halo values take part (zeros at the image border,
 * which never exceed a ReLU output).  Same shapes as segblocks_conv_halo. */
int segblocks_maxpool_halo(const void* hi_pad, const void* lo_pad, int dtype, int layout, int N, int C,
                           int H, int W, const uint8_t* mask, int bs, int halo, int ksize, int stride,
                           void* hi_out, void* lo_out, int hi_cap, int lo_cap, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Backward pass (the block modules and the block convolution are linear maps;
 * these are their transposes, for training through the block-conv path).
 * For y = combine(conv3x3(pad(split(x)))) and an output gradient dy:
 *   (dho, dlo_o) = segblocks_combine_backward(dy)
 *   dw, db       = segblocks_conv3x3_backward_weight(hp, lp, dho, dlo_o)
 *   (dhp, dlp)   = segblocks_conv3x3_backward_data(dho, dlo_o, w)
 *   (dhi, dlo)   = segblocks_pad_backward(dhp, dlp)
 *   dx           = segblocks_split_backward(dhi, dlo)
 * Shapes, layouts, masks and capacities follow the forward calls; every
 * gradient is stored in `dtype` with fp32 arithmetic.  Blocks past a stack's
 * capacity are skipped as in the forward calls.
 * ------------------------------------------------------------------------ */

/* BlockCombine transposed: dy [N,C,H,W] -> dhi [nh,C,bs,bs] (the block's
 * gradient copied), dlo [nl,C,lb,lb] (the fp32 sum ((a + b) + (c + d)) of the
 * 2x2 cell of gradients each low pixel was copied to, rounded once). */
int segblocks_combine_backward(const void* dy, int dtype, int layout, int N, int C, int H, int W,
                               const uint8_t* mask, int bs, void* dhi, int hi_cap, void* dlo,
                               int lo_cap, hipStream_t stream);

/* BlockSample transposed: dhi, dlo -> dx [N,C,H,W]: a high block's gradient
 * copied back, a low pixel's gradient times 0.25 on each pixel of its cell. */
int segblocks_split_backward(const void* dhi, const void* dlo, int dtype, int layout, int N, int C,
                             int H, int W, const uint8_t* mask, int bs, int hi_cap, int lo_cap,
                             void* dx, hipStream_t stream);

/* BlockPad transposed (sampling as in segblocks_pad_ex): dhp [nh,C,bs+2,bs+2],
 * dlp [nl,C,lb+2,lb+2] -> dhi, dlo.  Each block pixel receives the gradient
 * of every padded pixel that was read from it: its own interior pixel, the
 * halo pixels of neighbours at the same resolution, the halo pixels of a high
 * neighbour it was nearest-upsampled into, and a quarter of each low
 * neighbour's halo pixel averaged from its 2x2 cell (all of it at the cell's
 * top-left pixel with SB_PAD_STRIDED; nothing with SB_PAD_ZERO).  Summed in
 * fp32 in a fixed order (no atomics), rounded once. */
int segblocks_pad_backward(const void* dhp, const void* dlp, int dtype, int layout, int N, int C,
                           int H, int W, const uint8_t* mask, int bs, int sampling, void* dhi,
                           void* dlo, int hi_cap, int lo_cap, hipStream_t stream);

/* Gradient of segblocks_conv3x3 with respect to its padded input:
 *   dP[s,ci,u,v] = sum_{co,ky,kx} w[co,ci,ky,kx] * dO[s,co,u-ky,v-kx]
 * dho [nh,C_out,bs,bs], dlo [nl,C_out,lb,lb] -> dhp [nh,C_in,bs+2,bs+2],
 * dlp [nl,C_in,lb+2,lb+2]; weight as in segblocks_conv3x3.  Needs a
 * workspace (the gradients padded by two zeros, the transposed filters):
 * segblocks_conv3x3_backward_data_workspace_size. */
int segblocks_conv3x3_backward_data(const void* dho, const void* dlo, int dtype, int layout, int N,
                                    int C_in, int H, int W, const uint8_t* mask, int bs,
                                    const void* weight, int C_out, void* dhp, void* dlp, int hi_cap,
                                    int lo_cap, void* workspace, size_t ws_bytes, hipStream_t stream);
int segblocks_conv3x3_backward_data_workspace_size(int dtype, int layout, int N, int C_in, int H, int W,
                                                   int bs, int C_out, int hi_cap, int lo_cap,
                                                   size_t* bytes);

/* Gradient of segblocks_conv3x3 with respect to its weight and bias over both
 * stacks:
 *   dw[co,ci,ky,kx] = sum_{s,i,j} dO[s,co,i,j] * P[s,ci,i+ky,j+kx],  db[co] = sum dO[s,co,i,j]
 * hp, lp: the padded inputs of the forward call; dho, dlo: the output
 * gradients; dweight in the call's weight format, dbias [C_out] or NULL.
 * fp32 partial sums per range of block rows in the workspace, added in a
 * fixed order: segblocks_conv3x3_backward_weight_workspace_size (with_bias
 * != 0 when dbias is given). */
int segblocks_conv3x3_backward_weight(const void* hp, const void* lp, const void* dho, const void* dlo,
                                      int dtype, int layout, int N, int C_in, int H, int W,
                                      const uint8_t* mask, int bs, int C_out, void* dweight,
                                      void* dbias, int hi_cap, int lo_cap, void* workspace,
                                      size_t ws_bytes, hipStream_t stream);
int segblocks_conv3x3_backward_weight_workspace_size(int dtype, int layout, int N, int C_in, int H,
                                                     int W, int bs, int C_out, int hi_cap, int lo_cap,
                                                     int with_bias, size_t* bytes);

/* Heuristic downsampling policy (the policy of the short paper SegBlocks
 * extends, compared with in Experiments > Ablation studies, execution
 * policies): it selects the blocks where half resolution loses the most
 * detail.  x [N,C,H,W] (the image or a feature map) ->
 *   score [N][H/bs][W/bs] (fp32, device): for every pixel of the block the
 *     Euclidean distance over the channels between the pixel and the
 *     block's low-resolution version there (the BlockSample 2x2 average of
 *     its cell), averaged over the block's pixels;
 *   mask [N][H/bs][W/bs] (uint8, device): per image the
 *     k = floor(tau_high * GH * GW + 0.5) blocks with the highest scores are
 *     high resolution (1), the rest low (0); equal scores rank by block id,
 *     lower first.
 * tau_high in [0, 1] is the high-resolution fraction (the paper's target
 * tau).  At most 8192 blocks per image.  Any dtype and layout. */
int segblocks_policy_heuristic(const void* x, int dtype, int layout, int N, int C, int H, int W,
                               int bs, double tau_high, float* score, uint8_t* mask,
                               hipStream_t stream);

/* Dense convolution around the block stages (the encoder's 7x7/2 stem):
 * x [N,C_in,H,W] -> y [N,C_out,Ho,Wo], Ho = (H + 2 pad - K) / stride + 1,
 *   y = bias + sum w * x (zero padding), then max(0, .) if SB_FLAG_RELU.
 * weight OHWI memory [C_out][K][K][C_in], bias [C_out] or NULL.
 * Channels-last fp16 / bf16; the workgroup's LDS (weights padded to a
 * multiple of 32 K values plus one input patch) must fit in 160 KiB. */
int segblocks_conv2d(const void* x, int dtype, int layout, int N, int C_in, int H, int W,
                     const void* weight, const void* bias, int C_out, int ksize, int stride,
                     int pad, int flags, void* y, hipStream_t stream);

/* Max-pooling (the encoder's 3x3/2 pool after the stem): y = max over the
 * K x K window at `stride`, padding positions never win.  Channels-last,
 * any dtype; pad < ksize. */
int segblocks_maxpool(const void* x, int dtype, int layout, int N, int C, int H, int W,
                      int ksize, int stride, int pad, void* y, hipStream_t stream);

/* Description of the last failure on the calling thread ("" if none).  The
 * string stays valid until the next call on the same thread. */
const char* segblocks_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* SEGBLOCKS_H */
