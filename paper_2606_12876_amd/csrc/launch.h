// Kernel launchers (defined in the .hip files). Arguments are already validated.
#pragma once
#include <hip/hip_runtime.h>

#include "layer.h"

namespace aqmb {

// Re-tile n_planes plane-major code planes [n_planes][d_out][G] into out (n_planes tiled planes);
// for 4-bit codes a value above 15 sets *bad (device int).
hipError_t launch_retile(const Layer& L, const void* codes_plane_major, int n_planes, unsigned char* out, int* bad,
                         hipStream_t st);
hipError_t launch_dequant(const Layer& L, int k, void* W, aqmb_dtype w_dtype, hipStream_t st);
// Direct-gather GEMV of a layer with 8-bit codes; it serves the call when gemv_cw_fits.
bool gemv_cw_fits(const Layer& L, int k, int batch, aqmb_dtype x_dtype);
hipError_t launch_gemv_cw(const Layer& L, int k, const void* x, aqmb_dtype x_dtype, int batch, void* y,
                          aqmb_dtype y_dtype, hipStream_t st);
// Decode GEMV of a layer with 16-bit codes (codewords gathered through L2), any k, batch and row.
hipError_t launch_gemv_b16(const Layer& L, int k, const void* x, aqmb_dtype x_dtype, int batch, void* y,
                           aqmb_dtype y_dtype, hipStream_t st);
// Lookup-table GEMV (8-bit codes): split-K partial sums in `scratch` (gemv_lut_scratch_bytes bytes,
// owned by the caller for the duration of the launch on st).
size_t gemv_lut_scratch_bytes(const Layer& L, int batch);
hipError_t launch_gemv_lut(const Layer& L, int k, const void* x, aqmb_dtype x_dtype, int batch, void* y,
                           aqmb_dtype y_dtype, float* scratch, hipStream_t st);
// Decode GEMV of a layer with 8- or 4-bit codes on the matrix cores (batch 1..16).
hipError_t launch_gemv_mma(const Layer& L, int k, const void* x, aqmb_dtype x_dtype, int batch, void* y,
                           aqmb_dtype y_dtype, hipStream_t st);
// The same for n layers with the same d_in, code width and device, in one launch (results equal to
// launch_gemv_mma's for each layer); n <= AQMB_MAX_MULTI.
hipError_t launch_gemv_mma_multi(const Layer* const* Ls, int n, int k, const void* x, aqmb_dtype x_dtype, int batch,
                                 void* const* ys, aqmb_dtype y_dtype, hipStream_t st);
// Decode GEMV of a layer with 4-bit codes (16-codeword codebooks).
hipError_t launch_gemv_b4(const Layer& L, int k, const void* x, aqmb_dtype x_dtype, int batch, void* y,
                          aqmb_dtype y_dtype, hipStream_t st);
// Several layers with the same d_in and device, already validated; n <= AQMB_MAX_MULTI.
hipError_t launch_gemv_multi(const Layer* const* Ls, int n, int k, const void* x, aqmb_dtype x_dtype, int batch,
                             void* const* ys, aqmb_dtype y_dtype, hipStream_t st);
// All prefix distortions D[0..M-1] of the layer against fp16 W [d_out][d_in] and fp16 inputs
// X [n][d_in]; the per-workgroup sums go to `scratch` (distortion_scratch_bytes bytes).
hipError_t launch_distortion(const Layer& L, const void* W, const void* X, int n, double* D, double* scratch,
                             hipStream_t st);
size_t distortion_scratch_bytes();
// The device address of the distortion's file-scope scratch array on `device` (which must be
// current), looked up on the first call per device; *bytes is its size.
hipError_t distortion_static_scratch(int device, double** out, size_t* bytes);
// Beam search of codes for every group of W [d_out][d_in] fp16 over codebooks 0..k-1 (8-bit).
hipError_t launch_beam_search(const aqmb_desc& d, int k, int beam_width, const void* W, const uint16_t* codebooks,
                              const uint16_t* scales, unsigned char* codes, float* errors, hipStream_t st);
// The same search for the data-aware objective d^T H_jj d (H: [G][8][8] fp32 symmetric blocks).
hipError_t launch_beam_search_weighted(const aqmb_desc& d, int k, int beam_width, const void* W,
                                       const uint16_t* codebooks, const uint16_t* scales, const float* H,
                                       unsigned char* codes, float* errors, hipStream_t st);
// Prefill GEMM tiled for small token counts (same arithmetic as launch_gemm).
hipError_t launch_gemm_small(const Layer& L, int k, const void* X, int n_tokens, void* Y, aqmb_dtype y_dtype,
                             hipStream_t st);
// Large-tile prefill GEMM; tile: -1 = chosen by the number of workgroup rounds, 0 = 256 x 128,
// 1 = 128 x 128, 2 = 128 x 64 (tokens x weight rows).
hipError_t launch_gemm(const Layer& L, int k, const void* X, int n_tokens, void* Y, aqmb_dtype y_dtype, int tile,
                       hipStream_t st);
// Two-pass prefill GEMM (bit-identical to the 256 x 128 tiling): workspace bytes (0 where it does
// not apply) and the launch (workspace of at least that many bytes, 256-byte aligned).
size_t gemm_two_pass_bytes(const Layer& L, int k, int n_tokens);
hipError_t launch_gemm_two_pass(const Layer& L, int k, const void* X, int n_tokens, void* Y, aqmb_dtype y_dtype,
                                void* workspace, hipStream_t st);

}  // namespace aqmb
