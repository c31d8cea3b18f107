// Internal launcher interface between the C ABI (sb_api.hip) and the kernels.
#pragma once

#include <initializer_list>

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sb {

// Launch-setup state kept per device (sb_host.hip): the number of compute
// units, and the dynamic-LDS limit of a kernel raised to at least `bytes`.
int device_cus();
hipError_t ensure_dyn_lds(const void* kernel, int bytes);

// Geometry of one call: logical N, C, H, W; block size; block grid.
struct Geo {
    int N, C, H, W, bs, GH, GW;
    long long B;  // N * GH * GW
};

enum ConvSrc { SRC_PADDED = 0, SRC_PACKED = 1, SRC_DENSE = 2 };
enum ConvDst { DST_PACKED = 0, DST_DENSE = 1 };

struct ConvArgs {
    const void* in_hi;   // padded or packed high stack, or the dense map
    const void* in_lo;   // padded or packed low stack (unused for dense input)
    const void* weight;  // OIHW [C_out][C_in][3][3]
    const void* bias;    // [C_out] or nullptr
    const void* res_hi;  // residual stacks (packed output only) or nullptr
    const void* res_lo;
    void* out_hi;        // packed output stacks, or the dense output map
    void* out_lo;
    int C_in, C_out, flags, hi_cap, lo_cap;
    // The high stacks at half resolution (each block's 2x2 averages, the
    // values BlockPad with average sampling gives a low neighbour's halo):
    // in_hs [hi_cap][bs/2][bs/2][C_in] of the input, read by the implicit
    // GEMM instead of padding the low stack beforehand; out_hs
    // [hi_cap][bo/2][bo/2][C_out] of the output (bo = bs / stride), written
    // from the results.  nullptr = not given / not wanted.
    const void* in_hs = nullptr;
    void* out_hs = nullptr;
};

// bwd: the transposes for the backward pass instead: split of a gradient map
// is BlockCombine transposed (low blocks get 2x2 sums), combine of gradient
// stacks is BlockSample transposed (low values spread as quarters).
hipError_t launch_split(int dtype, int layout, const Geo& g, const void* x, const uint8_t* mask,
                        void* hi, int hi_cap, void* lo, int lo_cap, hipStream_t st, bool bwd = false);
// pm: how the halo is filled (PM_AVG, PM_STRIDED, PM_ZERO of sb_pixel.h);
// halo: its width in pixels (1 <= halo <= bs/2)
hipError_t launch_pad(int dtype, int layout, const Geo& g, const void* hi, const void* lo,
                      const uint8_t* mask, void* hp, void* lp, int hi_cap, int lo_cap, int pm, hipStream_t st,
                      int halo = 1);
hipError_t launch_combine(int dtype, int layout, const Geo& g, const void* hi, const void* lo,
                          const uint8_t* mask, int hi_cap, int lo_cap, void* y, hipStream_t st, bool bwd = false);
// Device memory that a launch needs beyond its inputs and outputs, supplied
// by the caller (at least the bytes that the matching *_ws_bytes function
// returns for the same shapes, 256-byte aligned).
struct Ws {
    void* p;
    size_t bytes;
};

// g.C is ignored by the convolution launcher (C_in / C_out are in ConvArgs).
hipError_t launch_conv(int dtype, int layout, ConvSrc src, ConvDst dst, const Geo& g,
                       const uint8_t* mask, const ConvArgs& a, Ws ws, hipStream_t st);
// Workspace of launch_conv for these shapes and capacities, assuming every
// buffer is 16-byte aligned (a call with less aligned buffers needs no more).
size_t conv_ws_bytes(int dtype, int layout, ConvSrc src, ConvDst dst, const Geo& g, const ConvArgs& a);

// Row-job split / pad / combine for channels-last tensors of whole 16-byte
// pixels with 16-byte aligned buffers; rows_fit tells whether they apply.
// launch_pad_rows with hp == nullptr pads the low blocks only (into lp).
bool rows_fit(int dtype, int layout, const Geo& g, std::initializer_list<const void*> ptrs);
hipError_t launch_split_rows(int dtype, const Geo& g, const void* x, const uint8_t* mask, void* hi, int hi_cap,
                             void* lo, int lo_cap, hipStream_t st, bool bwd = false);
hipError_t launch_pad_rows(int dtype, const Geo& g, const void* hi, const void* lo, const uint8_t* mask, void* hp,
                           void* lp, int hi_cap, int lo_cap, int pm, hipStream_t st);
hipError_t launch_combine_rows(int dtype, const Geo& g, const void* hi, const void* lo, const uint8_t* mask,
                               int hi_cap, int lo_cap, void* y, hipStream_t st, bool bwd = false);
// The padded low stack (1-pixel halo, average sampling) straight from the
// dense map, for fp16 / bf16 maps whose sides are multiples of the block size.
hipError_t launch_pad_low_dense(int dtype, const Geo& g, const void* x, const uint8_t* mask, void* lp, int lo_cap,
                                hipStream_t st);
// The high stack at half resolution: hs[s][u][v] = the 2x2 average of cell
// (2u, 2v) of block s of hi [hi_cap][e][e][C] (e even), for every slot below
// hi_cap (fp16 / bf16, channels-last, 16-byte aligned, C % 8 == 0).
hipError_t launch_sample_hs(int dtype, const void* hi, int hi_cap, int e, int C, void* hs, hipStream_t st);

// Encoder kernels (channels-last fp16/bf16): block convolution K x K
// (K = 1, 3) at stride 1 or 2 on packed stacks, dense convolution, and
// max-pooling (any dtype).  conv2d_lds_bytes: LDS of one dense-conv workgroup.
// multi-block implicit GEMM on packed channels-last stacks (fp16 / bf16,
// C_in % 64 == 0, C_out % 8 == 0, at most 8192 blocks), BlockPad fused;
// igemm_fits_shape leaves out the pointer alignment that igemm_fits checks.
bool igemm_fits_shape(int dtype, int layout, const Geo& g, const ConvArgs& a);
bool igemm_fits(int dtype, int layout, const Geo& g, const ConvArgs& a);
size_t igemm_ws_bytes(const Geo& g, const ConvArgs& a, int ksize, int stride);
// launch_igemm writes a.out_hs (when given) from its epilogue where the tile
// layout keeps every 2x2 cell within a wave, else with launch_sample_hs after.
hipError_t launch_igemm(int dtype, const Geo& g, const uint8_t* mask, const ConvArgs& a, int ksize, int stride,
                        Ws ws, hipStream_t st);
hipError_t launch_bconv(int dtype, const Geo& g, const uint8_t* mask, const ConvArgs& a, int ksize, int stride,
                        hipStream_t st);
// A whole 3x3 layer on the implicit GEMM (dense map a.in_hi in, dense map
// a.out_hi out, average sampling): the padded low stack straight from the
// map, then the GEMM with the high blocks' pixels read from the map and the
// results written to the map (BlockCombine fused).
bool igemm_dense_fits(int dtype, int layout, const Geo& g, const ConvArgs& a);
size_t igemm_dense_ws_bytes(const Geo& g, const ConvArgs& a);
hipError_t launch_igemm_dense(int dtype, const Geo& g, const uint8_t* mask, const ConvArgs& a, Ws ws, hipStream_t st);
int conv2d_lds_bytes(int dtype, int C_in, int K, int S);
int stem_lds_bytes(int K, int S);
hipError_t launch_conv2d(int dtype, const void* x, int N, int C_in, int H, int W, const void* w, const void* bias,
                         int C_out, int K, int S, int P, int flags, void* y, hipStream_t st);
hipError_t launch_maxpool(int dtype, const void* x, int N, int C, int H, int W, int K, int S, int P, void* y,
                          hipStream_t st);

// Backward pass (sb_backward.hip): BlockPad transposed, the block
// convolution's gradient with respect to its padded input (dgrad, on the
// general kernel; workspace: dgrad_ws_bytes) and to its weights and bias
// (wgrad; workspace: wgrad_ws_bytes).  BlockCombine / BlockSample transposed
// are launch_split / launch_combine with bwd.
hipError_t launch_pad_bwd(int dtype, int layout, const Geo& g, const void* dhp, const void* dlp, const uint8_t* mask,
                          void* dhi, void* dlo, int hi_cap, int lo_cap, int pm, hipStream_t st);
size_t dgrad_ws_bytes(int dtype, int layout, const Geo& g, int C_in, int C_out, int hi_cap, int lo_cap);
hipError_t launch_dgrad(int dtype, int layout, const Geo& g, const void* dho, const void* dlo, const uint8_t* mask,
                        const void* w, int C_in, int C_out, void* dhp, void* dlp, int hi_cap, int lo_cap, Ws ws,
                        hipStream_t st);
size_t wgrad_ws_bytes(int dtype, int layout, const Geo& g, int C_in, int C_out, int hi_cap, int lo_cap, bool bias);
hipError_t launch_wgrad(int dtype, int layout, const Geo& g, const void* hp, const void* lp, const void* dho,
                        const void* dlo, const uint8_t* mask, int C_in, int C_out, void* dw, void* db, int hi_cap,
                        int lo_cap, Ws ws, hipStream_t st);

// Layers beyond 3x3 on stacks padded with a halo of `halo` pixels
// (sb_halo.hip): K x K convolution (K odd) at stride st with dilation dl, and
// K x K max-pooling; g.C is the channel count of the max-pooling.
hipError_t launch_conv_halo(int dtype, int layout, const Geo& g, const void* hp, const void* lp, const uint8_t* mask,
                            int halo, const void* w, const void* bias, int C_in, int C_out, int K, int st, int dl,
                            int flags, void* ho, void* lo, int hi_cap, int lo_cap, hipStream_t s);
hipError_t launch_maxpool_halo(int dtype, int layout, const Geo& g, const void* hp, const void* lp,
                               const uint8_t* mask, int halo, int K, int st, void* ho, void* lo, int hi_cap,
                               int lo_cap, hipStream_t s);

// Heuristic downsampling policy: per-block scores [N*GH*GW] (fp32), then the
// mask with khigh high blocks per image (at most policy_max_blocks() per image).
int policy_max_blocks();
hipError_t launch_policy(int dtype, int layout, const void* x, int N, int C, int H, int W, int bs, float* score,
                         int khigh, uint8_t* mask, hipStream_t st);

// Persistent convolution with LDS-resident weights (channels-last fp16/bf16,
// C_in <= 64, blocks of 32 or 64); conv_res_fits tells whether it applies,
// conv_res_fits_shape the same without the pointer alignment.
bool conv_res_fits_shape(int dtype, int layout, const Geo& g, const ConvArgs& a);
bool conv_res_fits(int dtype, int layout, const Geo& g, const ConvArgs& a);
hipError_t launch_conv_res(int dtype, ConvSrc src, ConvDst dst, const Geo& g, const uint8_t* mask,
                           const ConvArgs& a, hipStream_t st);

}  // namespace sb
