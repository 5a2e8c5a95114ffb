/*
 * aqmb - multi-bitwidth additive-codebook linear layers on AMD Instinct MI355X (gfx950).
 *
 * A quantized linear layer stores a weight matrix W (d_out rows, d_in columns) as
 *   - M code planes: plane m holds, for every output row i and input group j
 *     (g consecutive weights of row i), the index b_{ijm} of a codeword of codebook m;
 *   - M codebooks C_0..C_{M-1}, each 2^B codewords of g fp16 values;
 *   - one fp16 scale s_i per output row.
 * At precision level k (1 <= k <= M) the layer uses only the first k codebooks:
 *   W_k[i, j*g + t] = s_i * sum_{m<k} C_m[b_{ijm}][t]
 * (Drop-by-Drop, section 5: partial reconstruction from the first k codebooks;
 * section 3.2: groups are consecutive along d_in and concatenated; the per-row
 * scale is the "Scales: d_out*16" term of the size estimate in appendix C).
 * One stored set of codes serves every k; planes m >= k are never read.
 *
 * Conventions for every entry point:
 *   - Data pointers passed to aqmb_create/gemv/gemm/dequant are DEVICE pointers on
 *     the current HIP device. Row-major, densely packed, 16-byte aligned
 *     (x, y, X, Y, W, codes, codebooks and scales).
 *   - `stream` is a hipStream_t (0 = the null stream). gemv/gemm/dequant only
 *     enqueue work on it and return; results are valid once the stream is synced.
 *   - Arguments are validated on the host before anything is enqueued. On any
 *     error nothing is launched and no output byte is written; the status says
 *     why and aqmb_last_error() gives a message for the calling thread.
 *   - No exception or abort crosses this interface.
 *   - A layer is read-only after creation (it is the stored format (C, b, s) that
 *     Alg. 1 returns): every compute call reads the layer and writes only the
 *     caller's outputs, so calls on one layer may run concurrently on different
 *     streams. Only aqmb_load_planes, aqmb_drop_planes and aqmb_destroy change a
 *     layer, and they must not overlap other calls on it.
 *   - Device scratch memory that a kernel needs for partial results (the lookup-
 *     table GEMV, the prefix distortion) is taken per call from the device's
 *     stream-ordered pool (hipMallocAsync / hipFreeAsync on `stream`), so two
 *     calls never share it. Every other call needs no scratch. Kernel choice does
 *     not depend on environment variables: aqmb_gemv_select and aqmb_gemm_select
 *     choose a kernel explicitly.
 */
#ifndef AQMB_H
#define AQMB_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct aqmb_layer_s* aqmb_layer_t;
typedef void* aqmb_stream_t; /* a hipStream_t */

typedef enum {
  AQMB_OK = 0,
  AQMB_EINVAL = 1,        /* bad argument: null pointer, k outside [1, M], sizes that do not fit */
  AQMB_EUNSUPPORTED = 2,  /* valid in the method but not implemented: g != 8, B not 8 or 16, batch > 16, dtype */
  AQMB_ENOMEM = 3,        /* device allocation failed */
  AQMB_EHIP = 4           /* a HIP runtime call or kernel launch failed; see aqmb_last_error() */
} aqmb_status;

typedef enum { AQMB_F16 = 0, AQMB_BF16 = 1, AQMB_F32 = 2 } aqmb_dtype;

typedef struct {
  int32_t d_out;          /* output rows of W, >= 1 */
  int32_t d_in;           /* input columns of W, >= g, a multiple of g */
  int32_t group_size;     /* g: weights per group; 8 is supported */
  int32_t num_codebooks;  /* M: 1..8 */
  int32_t code_bits;      /* B: 4 (16 codewords), 8 (uint8 codes, 256 codewords) or 16 (uint16 codes, 65536 codewords) */
} aqmb_desc;

/* Largest batch accepted by aqmb_gemv. */
#define AQMB_MAX_BATCH 16

/*
 * Create a layer from device buffers (Alg. 1 stores a layer as AQLMFormat(C, b, s)).
 *   codes     [M][d_out][d_in/g] uint8 (B = 8), uint16 (B = 16), or uint8 holding values 0..15
 *             (B = 4; stored two per byte): plane-major.
 *   codebooks [M][2^B][g] fp16 bit patterns; codeword c of codebook m is g contiguous values.
 *   scales    [d_out] fp16 bit patterns.
 * The library copies everything into device memory it owns, re-tiling the codes
 * inside each plane for coalesced reads while keeping planes outermost, so that
 * level k reads only the first k planes. Synchronous: returns after the copy on
 * `stream` has finished; the caller may free its buffers afterwards.
 * Code values >= 2^B cannot occur for B = 8 or 16 (they fill their type); for B = 4 they are
 * refused (EINVAL).
 * Errors: EINVAL (null pointer, bad sizes, 4-bit codes above 15), EUNSUPPORTED (g, B or M not supported),
 * ENOMEM, EHIP. On error *out is set to NULL.
 */
aqmb_status aqmb_create(aqmb_layer_t* out, const aqmb_desc* desc, const void* codes,
                        const uint16_t* codebooks, const uint16_t* scales, aqmb_stream_t stream);

/*
 * Run-time loading of code planes (the dynamic loading the paper's discussion of future work
 * names as an application of droppable codebooks: a device keeps only the planes its precision
 * level needs). Planes are stored outermost, so level k needs exactly planes 0..k-1.
 *   aqmb_create_prefix  like aqmb_create with only the first `resident` planes in device memory
 *                       (1 <= resident <= M); codes is [resident][d_out][d_in/g], codebooks and
 *                       scales are complete ([M][2^B][g], [d_out]).
 *   aqmb_load_planes    append the next n_planes planes (codes [n_planes][d_out][d_in/g], plane
 *                       `resident` first); the layer's code memory is reallocated.
 *   aqmb_drop_planes    keep planes 0..keep-1 (1 <= keep <= resident) and free the others.
 *   aqmb_resident_planes  the number of resident planes.
 * Every compute call with k above the resident count returns EINVAL; aqmb_prefix_distortion
 * covers the resident levels. load and drop are synchronous, wait for the device before the old
 * code memory is freed, and must not run concurrently with other calls on the same layer.
 * Errors: EINVAL (bad handle, null pointer, plane counts out of range, 4-bit codes above 15),
 * ENOMEM, EHIP. On error the layer is unchanged.
 */
aqmb_status aqmb_create_prefix(aqmb_layer_t* out, const aqmb_desc* desc, int resident, const void* codes,
                               const uint16_t* codebooks, const uint16_t* scales, aqmb_stream_t stream);
aqmb_status aqmb_load_planes(aqmb_layer_t layer, int n_planes, const void* codes, aqmb_stream_t stream);
aqmb_status aqmb_drop_planes(aqmb_layer_t layer, int keep);
aqmb_status aqmb_resident_planes(aqmb_layer_t layer, int* resident);

/* Free a layer and its device memory (waits for the device first). NULL is a no-op.
 * (The counterpart of aqmb_create: the stored format (C, b, s) of Alg. 1 is released.)
 * EINVAL for a handle that is not a live layer. */
aqmb_status aqmb_destroy(aqmb_layer_t layer);

/* Copy the layer's descriptor into *out. EINVAL for a bad handle or a null out. */
aqmb_status aqmb_get_desc(aqmb_layer_t layer, aqmb_desc* out);

/*
 * Decode GEMV: y[b][i] = sum_t x[b][t] * W_k[i][t] for b < batch (section 5 reconstruction,
 * applied as a product without forming W_k).
 *   x  [batch][d_in],  dtype x_dtype in {F16, BF16}
 *   y  [batch][d_out], dtype y_dtype in {F16, BF16, F32}
 * Products and sums are carried in fp32; the result is rounded once to y_dtype
 * (round to nearest even). 1 <= batch <= AQMB_MAX_BATCH.
 * Errors: EINVAL (bad handle, null pointer, k outside [1, M], batch < 1),
 * EUNSUPPORTED (batch > AQMB_MAX_BATCH, dtype), EHIP.
 */
aqmb_status aqmb_gemv(aqmb_layer_t layer, int k, const void* x, aqmb_dtype x_dtype, int batch,
                      void* y, aqmb_dtype y_dtype, aqmb_stream_t stream);

/*
 * The GEMV kernels. Each computes the quantity aqmb_gemv defines, to the same contract (fp32
 * products and sums, one rounding to y_dtype); they differ in speed only.
 *   AQMB_GEMV_AUTO    the library's choice for the layer, k, batch and x dtype (what aqmb_gemv runs)
 *   AQMB_GEMV_DIRECT  the direct-gather kernel of the layer's code width: codewords gathered per
 *                     code and dotted with x on the vector ALUs, 16 rows per workgroup. 8-bit
 *                     codes: k <= 4 and rows of at most 2048 groups (16384 inputs); 4- and 16-bit
 *                     codes: every k and row
 *   AQMB_GEMV_MMA     the matrix-core kernel (8- and 4-bit codes; every k, batch and row length)
 *   AQMB_GEMV_LUT     per-group lookup tables LUT_m[j][c] = <x_j, C_m[c]> in LDS, one read per
 *                     code (8-bit codes); its split-K partial sums take per-call scratch from the
 *                     stream-ordered pool (ENOMEM if that fails)
 * DIRECT with 8-bit codes also refuses when its codebook replicas and x tile do not fit in LDS
 * for the row length and batch (batch above 2 on rows of several thousand inputs).
 */
typedef enum {
  AQMB_GEMV_AUTO = 0,
  AQMB_GEMV_DIRECT = 1,
  AQMB_GEMV_MMA = 2,
  AQMB_GEMV_LUT = 3
} aqmb_gemv_kernel;

/*
 * aqmb_gemv with the kernel named by `kernel` (section 5 reconstruction, as aqmb_gemv). For
 * tests and tuning: every kernel can be checked against the same reference whatever the default
 * choice is. Arguments as aqmb_gemv.
 * Errors: those of aqmb_gemv; EUNSUPPORTED when the kernel cannot serve this layer, k, batch
 * or row length (see aqmb_gemv_kernel); EINVAL for an unknown kernel; ENOMEM (LUT scratch).
 */
aqmb_status aqmb_gemv_select(aqmb_layer_t layer, int k, const void* x, aqmb_dtype x_dtype, int batch,
                             void* y, aqmb_dtype y_dtype, aqmb_gemv_kernel kernel, aqmb_stream_t stream);

/* Most layers accepted by one aqmb_gemv_multi call. */
#define AQMB_MAX_MULTI 16

/*
 * Decode GEMV of several layers that read the same input (fused projections such as q/k/v or
 * gate/up): for each l < n_layers, ys[l][b][i] = sum_t x[b][t] * W_k^(l)[i][t], exactly what
 * aqmb_gemv(layers[l], k, x, x_dtype, batch, ys[l], y_dtype, stream) computes (same arithmetic,
 * same rounding), in one launch when either
 *   - every layer has 8-bit codes, k <= 4, aqmb_gemv would use the direct-gather kernel (batch 1;
 *     on rows of more than 512 groups only bf16 x at k < 3) and, for rows of more than 512
 *     groups, k = 1 (one workgroup per row block walks through the layers, loading the next
 *     layer's codes while it works on the current one), or
 *   - n_layers >= 2, every layer would take the matrix-core kernel (batch >= 2, and batch 1 on
 *     rows of more than 512 groups: see aqmb_gemv's kernel choice in the library source), all
 *     have the same code width and none has more 16-row blocks than the device has compute units
 *     (one grid over all the layers' row blocks);
 * otherwise the layers are launched one after another.
 *   layers  n_layers live handles, all with the same d_in and on the same device
 *   x       [batch][d_in], dtype x_dtype in {F16, BF16}
 *   ys      n_layers device pointers, ys[l] is [batch][d_out of layer l], dtype y_dtype
 * 1 <= n_layers <= AQMB_MAX_MULTI; k must be valid for every layer. Nothing is launched when
 * validation fails.
 * Errors: EINVAL (null pointer, bad handle, n_layers < 1, d_in or device differ, k outside
 * [1, M] of some layer, batch < 1), EUNSUPPORTED (n_layers > AQMB_MAX_MULTI, batch >
 * AQMB_MAX_BATCH, dtype), EHIP.
 */
aqmb_status aqmb_gemv_multi(const aqmb_layer_t* layers, int n_layers, int k, const void* x, aqmb_dtype x_dtype,
                            int batch, void* const* ys, aqmb_dtype y_dtype, aqmb_stream_t stream);

/*
 * Prefill GEMM (the section 5 partial reconstruction applied to n_tokens inputs at once, the
 * product Y = W X of section 2.2 in row-major form): Y[n][i] = s_i * sum_t X[n][t] * Wb_k[i][t]
 * for n < n_tokens, where Wb_k is the
 * unscaled reconstruction sum_{m<k} C_m[b_{ijm}] formed as a binary32 left fold over m and
 * rounded to nearest-even bf16 (the operand fed to bf16 matrix cores); accumulation is fp32.
 *   X  [n_tokens][d_in]  bf16 (no other activation dtype: convert before the call)
 *   Y  [n_tokens][d_out] dtype y_dtype in {BF16, F32}
 * Requires B = 8 or B = 4. Errors: EINVAL (bad handle, null pointer, k outside [1, M],
 * n_tokens < 1), EUNSUPPORTED (B = 16, dtype), EHIP.
 */
aqmb_status aqmb_gemm(aqmb_layer_t layer, int k, const void* X, int n_tokens, void* Y,
                      aqmb_dtype y_dtype, aqmb_stream_t stream);

/*
 * The prefill GEMM's tilings (the same arithmetic and rounding; they differ in speed only).
 *   AQMB_GEMM_AUTO     the library's choice (what aqmb_gemm runs): 16-row tiles up to 144 tokens,
 *                      else the large tile that needs the fewest rounds of workgroups
 *   AQMB_GEMM_ROWS16   16 weight rows per workgroup, all tokens in tiles of 16 (made for few tokens)
 *   AQMB_GEMM_256x128, AQMB_GEMM_128x128, AQMB_GEMM_128x64
 *                      tokens x weight rows per workgroup of the large-tile kernel
 */
typedef enum {
  AQMB_GEMM_AUTO = 0,
  AQMB_GEMM_ROWS16 = 1,
  AQMB_GEMM_256x128 = 2,
  AQMB_GEMM_128x128 = 3,
  AQMB_GEMM_128x64 = 4
} aqmb_gemm_tiling;

/* aqmb_gemm with the tiling named by `tiling` (tests and tuning). Errors: those of aqmb_gemm;
 * EINVAL for an unknown tiling. */
aqmb_status aqmb_gemm_select(aqmb_layer_t layer, int k, const void* X, int n_tokens, void* Y,
                             aqmb_dtype y_dtype, aqmb_gemm_tiling tiling, aqmb_stream_t stream);

/*
 * The prefill GEMM of aqmb_gemm (section 5 partial reconstruction, same definition, arguments and
 * errors) with a caller-owned device workspace. Where aqmb_gemm_workspace_bytes reports a
 * non-zero size and `workspace_bytes` is at least that size, the call runs in two passes: the
 * unscaled bf16 weights Wb_k (the same binary32 fold and rounding) are written once into the
 * workspace, tiled in matrix-core operand order, and a dense kernel multiplies X by them. The
 * output is bit-identical to aqmb_gemm's for the same arguments. Otherwise (workspace null or too
 * small, or the size is 0) the call is exactly aqmb_gemm.
 *   workspace        device memory, 256-byte aligned, owned by the caller; the call writes it
 *                    (stream-ordered on `stream`), so calls that share a workspace must be ordered
 *   workspace_bytes  its size in bytes
 * Errors: those of aqmb_gemm; EINVAL for a workspace that is not 256-byte aligned.
 */
aqmb_status aqmb_gemm_ws(aqmb_layer_t layer, int k, const void* X, int n_tokens, void* Y,
                         aqmb_dtype y_dtype, void* workspace, size_t workspace_bytes,
                         aqmb_stream_t stream);

/*
 * *bytes = the workspace aqmb_gemm_ws needs to run the two-pass GEMM for (k, n_tokens) on this
 * layer (2 bytes per weight, rows rounded up to 32 and d_in to 64), or 0 where that path does not
 * apply: it is taken for k >= 3 with 4- or 8-bit codes when the one-pass choice is the 256 x 128
 * tiling and that tiling fills every compute unit. Errors: EINVAL (bad handle, null bytes, k
 * outside [1, M], n_tokens < 1).
 */
aqmb_status aqmb_gemm_workspace_bytes(aqmb_layer_t layer, int k, int n_tokens, size_t* bytes);

/*
 * Dequantize (the section 5 partial reconstruction W_k written out as a dense matrix):
 * W[i][t] = W_k[i][t] in w_dtype in {F16, BF16, F32}, bit-exact to this evaluation
 * order: each fp16 codebook entry is taken exactly to binary32; the entries of planes
 * 0..k-1 are summed as a binary32 left fold (C_0 + C_1, then + C_2, ...), each sum rounded
 * to nearest even; the fold is multiplied by s_i in binary32 (one rounding, no fused
 * multiply-add); the product is rounded to nearest even into w_dtype. Subnormals are kept.
 *   W  [d_out][d_in]
 * Errors: EINVAL (bad handle, null pointer, k outside [1, M]), EUNSUPPORTED (dtype), EHIP.
 */
aqmb_status aqmb_dequant(aqmb_layer_t layer, int k, void* W, aqmb_dtype w_dtype, aqmb_stream_t stream);

/*
 * Distortion of every precision level in one pass (section 5: the error of each partial
 * reconstruction, which the training loop of Alg. 1 drives down level by level; the weighted
 * MSE of section 2.2, Eq. wmse-task): for k = 1..M,
 *   D[k-1] = ||(W - W_k) X||_F^2 / (d_out * n)
 * with the calibration inputs given as the rows of Xt = X^T.
 *   W   [d_out][d_in] fp16: the weights being quantized (w_dtype must be F16)
 *   Xt  [n][d_in]     fp16: one calibration input per row (x_dtype must be F16)
 *   D   one double per resident level (M unless planes were dropped or never loaded), device memory
 * The products W X and C_m[b_m] X run on fp16 matrix cores (each product of two fp16 values
 * exact, sums in fp32), the per-output differences W X - s_i sum_{m<k} (C_m[b_m] X) in fp32, the
 * sums of their squares in fp64, added in a fixed order: the result is reproducible.
 * The Hessian form of the same quantity, tr[(W - W_k) H (W - W_k)^T] / d_out with H = X X^T / n,
 * is obtained by passing any factor F with F F^T = H (e.g. a Cholesky factor) as Xt = F^T,
 * n = d_in, and multiplying D by d_in.
 * Requires B = 8 or B = 4. The per-workgroup sums (at most 256 x 8 doubles) take per-call scratch
 * from the stream-ordered pool, freed on `stream` after the final sum.
 * Errors: EINVAL (bad handle, null pointer, n < 1, misaligned pointer), EUNSUPPORTED (B = 16,
 * dtype other than F16, n > 2^30), ENOMEM (scratch), EHIP.
 */
aqmb_status aqmb_prefix_distortion(aqmb_layer_t layer, const void* W, aqmb_dtype w_dtype, const void* Xt,
                                   aqmb_dtype x_dtype, int n, double* D, aqmb_stream_t stream);

/*
 * aqmb_prefix_distortion without any device allocation, for callers that cannot allocate (code
 * under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc). Same arguments,
 * kernels, arithmetic and result as aqmb_prefix_distortion. Its per-workgroup sums live in a
 * fixed array of the library, 16 KiB per device (256 workgroups x 8 levels of doubles; the need is
 * the same for every layer and n), held until the process ends; the call allocates and frees
 * nothing. Every call on one device shares that device's array, so calls that overlap on one
 * device (different streams, or other threads) race and give wrong results: order them.
 * Errors: those of aqmb_prefix_distortion except ENOMEM; EUNSUPPORTED if the kernels ever need
 * more scratch than the array holds.
 */
aqmb_status aqmb_prefix_distortion_noalloc(aqmb_layer_t layer, const void* W, aqmb_dtype w_dtype, const void* Xt,
                                           aqmb_dtype x_dtype, int n, double* D, aqmb_stream_t stream);

/* Widest beam accepted by aqmb_beam_search. */
#define AQMB_MAX_BEAM 16

/*
 * Code search (Appendix C, code optimisation: a beam search over combinations of codewords that
 * minimise the quantization error; Algorithm 1 updates the assignments b this way): for every
 * group (row i, group j) of a dense weight matrix, beam search over codebooks 0..k-1 for the
 * codes c_0..c_{k-1} that minimise the group's squared error ||w_ij - s_i sum_m C_m[c_m]||^2.
 * Stage m extends each kept partial tuple by every codeword of codebook m and keeps the `beam`
 * best; the last stage keeps the best one (beam 1 is greedy residual coding). Groups are
 * independent (the plain squared error of the weights, X = I in the weighted MSE of §2.2).
 * Every comparison is decided in binary32 in this order: S_m[c][t] = s_i * C_m[c][t] (exact for
 * fp16 operands); the residual of a kept tuple is w - S_0[c_0] - ... with each subtraction
 * rounded; a candidate's d_t = fl(r_t - S_m[c][t]) and e = d_0 d_0 + d_1 d_1 + ... + d_7 d_7
 * with every product and every sum rounded, left to right, no fused multiply-add; candidates are
 * ordered by e, equal e by the code tuple (lexicographically).
 *   desc       the layer shape: d_out, d_in, g = 8, M codebooks, B = 8 or 4
 *   W          [d_out][d_in] fp16 (device, 16-byte aligned): the weights to encode
 *   codebooks  [M][2^B][8] fp16 (device, 16-byte aligned); codebooks 0..k-1 are used
 *   scales     [d_out] fp16 (device)
 *   codes      [k][d_out][d_in/8] uint8 (device, output; values < 2^B): plane-major, the layout
 *              aqmb_create takes
 *   errors     [d_out][d_in/8] float (device, output; may be NULL): e of the chosen tuple
 * 1 <= k <= M, 1 <= beam <= AQMB_MAX_BEAM. Work: 2^B (1 + (k - 1) beam) candidates per group.
 * Errors: EINVAL (null pointer, misaligned W or codebooks, k outside [1, M], beam < 1),
 * EUNSUPPORTED (B = 16, beam > AQMB_MAX_BEAM), EHIP.
 */
aqmb_status aqmb_beam_search(const aqmb_desc* desc, int k, int beam, const void* W, const uint16_t* codebooks,
                             const uint16_t* scales, uint8_t* codes, float* errors, aqmb_stream_t stream);

/*
 * The same code search with the data-aware objective of §2.2 (Eq. wmse-task: the weighted MSE
 * (1/n) ||(W - W_hat) X||_F^2 over calibration inputs X, which App. C's code optimisation
 * minimises): the error of group (i, j) is d^T H_j d with d = w_ij - s_i sum_m C_m[c_m] and H_j
 * the 8 x 8 diagonal block of H = X X^T / n for inputs 8 j .. 8 j + 7 (terms coupling different
 * groups are left out, so groups stay independent; with every H_j = I this is aqmb_beam_search's
 * objective). Every comparison is decided in binary32 in this order, with r the kept tuple's
 * residual (as in aqmb_beam_search) and C the unscaled candidate codeword:
 *   b_t = sum_u H_tu r_u and A = sum_t r_t b_t per kept tuple; Q = sum_t C_t (sum_u H_tu C_u) per
 *   codeword; T = sum_t C_t b_t and e = (A - (2 s_i) T) + (s_i s_i) Q per candidate,
 * every product and sum rounded, sums left to right over t, u = 0..7, no fused multiply-add;
 * candidates ordered by e, equal e by the code tuple.
 *   H       [d_in/8][8][8] fp32 (device, 4-byte aligned): the symmetric blocks H_j, row-major
 *   others  as for aqmb_beam_search; errors receive e of the chosen tuple
 * Work: 2^B (1 + (k - 1) beam) candidates per group, one workgroup per group j and 256 rows.
 * Errors: those of aqmb_beam_search; EINVAL also for a NULL or misaligned H.
 */
aqmb_status aqmb_beam_search_weighted(const aqmb_desc* desc, int k, int beam, const void* W,
                                      const uint16_t* codebooks, const uint16_t* scales, const float* H,
                                      uint8_t* codes, float* errors, aqmb_stream_t stream);

/*
 * Average storage bits per weight at level k (appendix C, Eq. avg_bits): codebooks
 * 16*g*k*2^B bits, codes d_out*(d_in/g)*B bits per used plane, scales 16*d_out bits,
 * over d_out*d_in weights. The printed codes term lacks the per-plane factor; the
 * worked example there (about 2.002 bits for d_in=8192, d_out=28672, g=8, M=2, B=8)
 * needs it. Returns a negative value for a null or invalid descriptor or k outside [1, M].
 */
double aqmb_bits_per_weight(const aqmb_desc* desc, int k);

/* Static description of a status code. Never NULL. */
const char* aqmb_strerror(aqmb_status status);

/* Message describing the last error on the calling thread ("" if none). Never NULL. */
const char* aqmb_last_error(void);

/* Validate arguments exactly as the entry points do, without touching the GPU.
 * op: 0 = gemv, 1 = gemm, 2 = dequant, 3 = prefix distortion, 4 = beam search. For gemv `n` is
 * the batch, for gemm the token count, for the distortion the number of inputs, for the beam
 * search the beam width (in = W, out = codes, dtypes ignored), ignored for dequant;
 * `in_dtype` is x's dtype (gemv) or Xt's (distortion), `out_dtype` the output dtype or, for
 * the distortion, W's dtype; `in`/`out` are x/y, X/Y, -/W, or Xt/D. `k` is not checked for
 * the distortion. Returns the status the entry point would return before launching anything
 * (the distortion's W pointer is checked by the entry point itself). */
aqmb_status aqmb_validate(const aqmb_desc* desc, int op, int k, int n, aqmb_dtype in_dtype,
                          aqmb_dtype out_dtype, const void* in, const void* out);

#ifdef __cplusplus
}
#endif

#endif /* AQMB_H */
