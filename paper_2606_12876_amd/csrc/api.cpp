// The C-ABI entry points: layer registry, creation (copy + re-tile), dispatch.
#include <hip/hip_runtime.h>

#include <mutex>
#include <new>
#include <unordered_set>

#include "launch.h"
#include "layer.h"

namespace aqmb {
aqmb_status fail(aqmb_status s, const char* fmt, ...);
void clear_error();
aqmb_status validate_desc(const aqmb_desc* d);
aqmb_status validate_call(const aqmb_desc* d, int op, int k, int n, aqmb_dtype in_dt, aqmb_dtype out_dt,
                          const void* in, const void* out);

static std::mutex g_mu;
static std::unordered_set<Layer*> g_live;

static bool is_live(Layer* L) {
  std::lock_guard<std::mutex> lk(g_mu);
  return L && g_live.count(L) && L->magic == kMagic;
}

static aqmb_status hip_fail(hipError_t e, const char* what) {
  return fail(AQMB_EHIP, "%s: %s", what, hipGetErrorString(e));
}

static void free_layer(Layer* L) {
  if (L->codes) (void)hipFree(L->codes);
  if (L->codebooks) (void)hipFree(L->codebooks);
  if (L->scales) (void)hipFree(L->scales);
  if (L->aux) (void)hipFree(L->aux);
  L->magic = 0;
  delete L;
}

// The layer's memory lives on one device; launching on another would address foreign memory.
static aqmb_status check_device(const Layer* L) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev != L->device) return fail(AQMB_EINVAL, "layer lives on device %d but device %d is current", L->device, dev);
  return AQMB_OK;
}

}  // namespace aqmb

using namespace aqmb;

extern "C" {

}  // extern "C"

namespace aqmb {

// Re-tile n plane-major code planes into dst (n tiled planes) and, for 4-bit codes, refuse values
// above 15 (the re-tiling flags them in the workspace). Synchronous.
static aqmb_status upload_planes(Layer* L, const void* codes, int n, unsigned char* dst, hipStream_t st,
                                 const char* where) {
  int* flag = L->upload_flag();
  hipError_t e;
  if ((e = hipMemsetAsync(flag, 0, sizeof(int), st)) != hipSuccess ||
      (e = launch_retile(*L, codes, n, dst, flag, st)) != hipSuccess || (e = hipStreamSynchronize(st)) != hipSuccess)
    return fail(AQMB_EHIP, "%s: upload: %s", where, hipGetErrorString(e));
  if (L->d.code_bits == 4) {
    int bad = 0;
    if ((e = hipMemcpy(&bad, flag, sizeof(int), hipMemcpyDeviceToHost)) != hipSuccess)
      return fail(AQMB_EHIP, "%s: code check: %s", where, hipGetErrorString(e));
    if (bad) return fail(AQMB_EINVAL, "%s: a 4-bit code is above 15", where);
  }
  return AQMB_OK;
}

static aqmb_status create_impl(aqmb_layer_t* out, const aqmb_desc* desc, int resident, const void* codes,
                               const uint16_t* codebooks, const uint16_t* scales, aqmb_stream_t stream) {
  if (!out) return fail(AQMB_EINVAL, "create: out is NULL");
  *out = nullptr;
  aqmb_status s = validate_desc(desc);
  if (s != AQMB_OK) return s;
  if (resident < 1 || resident > desc->num_codebooks)
    return fail(AQMB_EINVAL, "create: resident planes = %d outside [1, M = %d]", resident, desc->num_codebooks);
  if (!codes || !codebooks || !scales) return fail(AQMB_EINVAL, "create: codes, codebooks or scales is NULL");
  hipStream_t st = (hipStream_t)stream;

  Layer* L = new (std::nothrow) Layer();
  if (!L) return fail(AQMB_ENOMEM, "create: host allocation failed");
  L->magic = kMagic;
  L->d = *desc;
  hipError_t e = hipGetDevice(&L->device);
  if (e != hipSuccess) { free_layer(L); return hip_fail(e, "create: hipGetDevice"); }
  e = hipDeviceGetAttribute(&L->n_cu, hipDeviceAttributeMultiprocessorCount, L->device);
  if (e != hipSuccess) { free_layer(L); return hip_fail(e, "create: hipDeviceGetAttribute"); }
  L->G = desc->d_in / desc->group_size;
  L->J = kSliceBytes * 8 / desc->code_bits;     // groups per 16-byte slice: 32, 16 or 8
  L->S = (L->G + L->J - 1) / L->J;
  L->plane_bytes = (size_t)L->S * desc->d_out * kSliceBytes;
  L->resident = resident;
  const size_t n_codewords = (size_t)1 << desc->code_bits;
  const size_t cb_bytes = (size_t)desc->num_codebooks * n_codewords * desc->group_size * 2;

  struct { void** p; size_t n; const char* what; } allocs[] = {
      {(void**)&L->codes, (size_t)resident * L->plane_bytes, "codes"},
      {(void**)&L->codebooks, cb_bytes, "codebooks"},
      {(void**)&L->scales, (size_t)desc->d_out * 2, "scales"},
      {(void**)&L->aux, kAuxBytes, "zero page"},
  };
  for (auto& a : allocs) {
    e = hipMalloc(a.p, a.n);
    if (e != hipSuccess) {
      *a.p = nullptr;
      (void)hipGetLastError();
      free_layer(L);
      return fail(AQMB_ENOMEM, "create: hipMalloc(%zu) for %s failed: %s", a.n, a.what, hipGetErrorString(e));
    }
  }
  // The zero page that kernels read in place of out-of-range inputs (never written afterwards).
  if ((e = hipMemsetAsync(L->aux, 0, kAuxBytes, st)) != hipSuccess ||
      (e = hipMemcpyAsync(L->codebooks, codebooks, cb_bytes, hipMemcpyDeviceToDevice, st)) != hipSuccess ||
      (e = hipMemcpyAsync(L->scales, scales, (size_t)desc->d_out * 2, hipMemcpyDeviceToDevice, st)) != hipSuccess) {
    free_layer(L);
    return hip_fail(e, "create: upload");
  }
  if ((s = upload_planes(L, codes, resident, L->codes, st, "create")) != AQMB_OK) {
    free_layer(L);
    return s;
  }
  {
    std::lock_guard<std::mutex> lk(g_mu);
    g_live.insert(L);
  }
  *out = (aqmb_layer_t)L;
  return AQMB_OK;
}

// GEMV kernel choice (AQMB_GEMV_AUTO), measured faster in each case: 4-bit codes -> the
// matrix-core kernel at batch >= 2 and, for fp16 x at k >= 2, at batch 1 on rows of more than 512
// groups; their direct-gather kernel otherwise. 8-bit codes -> the matrix-core kernel at batch >= 2
// and at batch 1 on rows of more than 512 groups for fp16 x, and for bf16 x from k = 3 (4096 x
// 11008, mean of three runs, direct gathers against the matrix cores: 5.77 / 7.44 / 8.92 / 10.74
// against 5.60 / 7.55 / 8.69 / 9.92 us at k = 1..4; in a bench run 7.4 against 8.2 us at k = 2
// and even at k = 1); otherwise the direct-gather kernel when it fits (k <= 4, rows of at most
// 16384 inputs), else the matrix-core kernel. 16-bit codes -> their direct-gather kernel.
// (At batch 1 on rows of at most 512 groups the matrix cores are 3-5 % faster with fp16 x from
// k = 2 on a 4096 x 4096 layer, but the direct-gather kernel stays: aqmb_gemv_multi runs such
// layers in one direct-gather launch and must return what aqmb_gemv returns.)
static aqmb_gemv_kernel gemv_auto(const Layer& L, int k, int batch, aqmb_dtype x_dtype) {
  if (L.d.code_bits == 16) return AQMB_GEMV_DIRECT;
  const bool wide = L.S * L.J > 512;
  if (L.d.code_bits == 4)
    return batch >= 2 || (x_dtype == AQMB_F16 && wide && k >= 2) ? AQMB_GEMV_MMA : AQMB_GEMV_DIRECT;
  if (batch >= 2 || (wide && (x_dtype == AQMB_F16 || k >= 3))) return AQMB_GEMV_MMA;
  return gemv_cw_fits(L, k, batch, x_dtype) ? AQMB_GEMV_DIRECT : AQMB_GEMV_MMA;
}

// Whether `kernel` can serve this call (AUTO always can).
static bool gemv_kernel_serves(const Layer& L, int k, int batch, aqmb_dtype x_dtype, aqmb_gemv_kernel kernel) {
  switch (kernel) {
    case AQMB_GEMV_AUTO: return true;
    case AQMB_GEMV_DIRECT: return L.d.code_bits != 8 || gemv_cw_fits(L, k, batch, x_dtype);
    case AQMB_GEMV_MMA: return L.d.code_bits != 16;
    case AQMB_GEMV_LUT: return L.d.code_bits == 8;
  }
  return false;
}

// Stream-ordered scratch for one call: allocated from the device's default pool on st and freed on
// st after the kernels that use it, so calls on different streams never share it.
struct CallScratch {
  void* p = nullptr;
  hipStream_t st = nullptr;
  hipError_t alloc(size_t bytes, hipStream_t s) {
    st = s;
    return hipMallocAsync(&p, bytes, s);
  }
  hipError_t release() {
    if (!p) return hipSuccess;
    hipError_t e = hipFreeAsync(p, st);
    p = nullptr;
    return e;
  }
};

static aqmb_status launch_gemv_kernel(const Layer& L, int k, const void* x, aqmb_dtype x_dtype, int batch, void* y,
                                      aqmb_dtype y_dtype, aqmb_gemv_kernel kernel, hipStream_t st,
                                      const char* where) {
  if (kernel == AQMB_GEMV_AUTO) kernel = gemv_auto(L, k, batch, x_dtype);
  hipError_t e = hipSuccess;
  switch (kernel) {
    case AQMB_GEMV_MMA: e = launch_gemv_mma(L, k, x, x_dtype, batch, y, y_dtype, st); break;
    case AQMB_GEMV_DIRECT:
      e = L.d.code_bits == 4    ? launch_gemv_b4(L, k, x, x_dtype, batch, y, y_dtype, st)
          : L.d.code_bits == 16 ? launch_gemv_b16(L, k, x, x_dtype, batch, y, y_dtype, st)
                                : launch_gemv_cw(L, k, x, x_dtype, batch, y, y_dtype, st);
      break;
    default: {  // AQMB_GEMV_LUT
      CallScratch sc;
      if ((e = sc.alloc(gemv_lut_scratch_bytes(L, batch), st)) != hipSuccess) {
        (void)hipGetLastError();
        return fail(AQMB_ENOMEM, "%s: scratch for the lookup-table kernel: %s", where, hipGetErrorString(e));
      }
      e = launch_gemv_lut(L, k, x, x_dtype, batch, y, y_dtype, (float*)sc.p, st);
      const hipError_t e2 = sc.release();
      if (e == hipSuccess) e = e2;
    }
  }
  return e == hipSuccess ? AQMB_OK : hip_fail(e, where);
}

// GEMM tiling: small token counts take the 16-row tiling (every CU busy), larger ones the
// large-tile kernel with the tile shape that needs the fewest rounds of workgroups.
constexpr int kGemmSmallMax = 144;   // tokens: the 16-row tiling re-gathers per 64 tokens; measured break-even with 128 x 64 tiles near 150

// k must name resident planes.
static aqmb_status check_resident(const Layer* L, int k, const char* where) {
  if (k > L->resident)
    return fail(AQMB_EINVAL, "%s: k = %d needs planes that are not resident (%d of %d loaded)", where, k, L->resident,
                L->d.num_codebooks);
  return AQMB_OK;
}

// Replace the layer's planes by the first `keep` of them followed by n new planes from `codes`.
static aqmb_status resize_planes(Layer* L, int keep, const void* codes, int n, hipStream_t st, const char* where) {
  unsigned char* fresh = nullptr;
  hipError_t e = hipMalloc(&fresh, (size_t)(keep + n) * L->plane_bytes);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(AQMB_ENOMEM, "%s: hipMalloc(%zu) failed: %s", where, (size_t)(keep + n) * L->plane_bytes,
                hipGetErrorString(e));
  }
  // no kernel may still read the old planes when they are freed: wait for the device
  if ((e = hipDeviceSynchronize()) != hipSuccess ||
      (e = hipMemcpyAsync(fresh, L->codes, (size_t)keep * L->plane_bytes, hipMemcpyDeviceToDevice, st)) != hipSuccess) {
    (void)hipFree(fresh);
    return hip_fail(e, where);
  }
  if (n > 0) {
    aqmb_status s = upload_planes(L, codes, n, fresh + (size_t)keep * L->plane_bytes, st, where);
    if (s != AQMB_OK) {
      (void)hipStreamSynchronize(st);
      (void)hipFree(fresh);
      return s;
    }
  } else if ((e = hipStreamSynchronize(st)) != hipSuccess) {
    (void)hipFree(fresh);
    return hip_fail(e, where);
  }
  (void)hipFree(L->codes);
  L->codes = fresh;
  L->resident = keep + n;
  return AQMB_OK;
}

}  // namespace aqmb

extern "C" {

aqmb_status aqmb_create(aqmb_layer_t* out, const aqmb_desc* desc, const void* codes, const uint16_t* codebooks,
                        const uint16_t* scales, aqmb_stream_t stream) {
  clear_error();
  return create_impl(out, desc, desc ? desc->num_codebooks : 1, codes, codebooks, scales, stream);
}

aqmb_status aqmb_create_prefix(aqmb_layer_t* out, const aqmb_desc* desc, int resident, const void* codes,
                               const uint16_t* codebooks, const uint16_t* scales, aqmb_stream_t stream) {
  clear_error();
  return create_impl(out, desc, resident, codes, codebooks, scales, stream);
}

aqmb_status aqmb_load_planes(aqmb_layer_t layer, int n_planes, const void* codes, aqmb_stream_t stream) {
  clear_error();
  Layer* L = (Layer*)layer;
  if (!is_live(L)) return fail(AQMB_EINVAL, "load_planes: not a live layer");
  if (!codes) return fail(AQMB_EINVAL, "load_planes: codes is NULL");
  if (n_planes < 1 || L->resident + n_planes > L->d.num_codebooks)
    return fail(AQMB_EINVAL, "load_planes: %d more planes do not fit (%d of %d resident)", n_planes, L->resident,
                L->d.num_codebooks);
  aqmb_status s = check_device(L);
  if (s != AQMB_OK) return s;
  return resize_planes(L, L->resident, codes, n_planes, (hipStream_t)stream, "load_planes");
}

aqmb_status aqmb_drop_planes(aqmb_layer_t layer, int keep) {
  clear_error();
  Layer* L = (Layer*)layer;
  if (!is_live(L)) return fail(AQMB_EINVAL, "drop_planes: not a live layer");
  if (keep < 1 || keep > L->resident)
    return fail(AQMB_EINVAL, "drop_planes: keep = %d outside [1, %d resident]", keep, L->resident);
  if (keep == L->resident) return AQMB_OK;
  aqmb_status s = check_device(L);
  if (s != AQMB_OK) return s;
  return resize_planes(L, keep, nullptr, 0, nullptr, "drop_planes");
}

aqmb_status aqmb_resident_planes(aqmb_layer_t layer, int* resident) {
  clear_error();
  Layer* L = (Layer*)layer;
  if (!is_live(L)) return fail(AQMB_EINVAL, "resident_planes: not a live layer");
  if (!resident) return fail(AQMB_EINVAL, "resident_planes: resident is NULL");
  *resident = L->resident;
  return AQMB_OK;
}

aqmb_status aqmb_destroy(aqmb_layer_t layer) {
  clear_error();
  if (!layer) return AQMB_OK;
  Layer* L = (Layer*)layer;
  {
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_live.count(L) || L->magic != kMagic) return fail(AQMB_EINVAL, "destroy: not a live layer");
    g_live.erase(L);
  }
  int prev = -1;
  (void)hipGetDevice(&prev);
  (void)hipSetDevice(L->device);
  hipError_t e = hipDeviceSynchronize();
  free_layer(L);
  if (prev >= 0) (void)hipSetDevice(prev);
  if (e != hipSuccess) return hip_fail(e, "destroy: hipDeviceSynchronize");
  return AQMB_OK;
}

aqmb_status aqmb_get_desc(aqmb_layer_t layer, aqmb_desc* out) {
  clear_error();
  if (!is_live((Layer*)layer)) return fail(AQMB_EINVAL, "get_desc: not a live layer");
  if (!out) return fail(AQMB_EINVAL, "get_desc: out is NULL");
  *out = ((Layer*)layer)->d;
  return AQMB_OK;
}

static aqmb_status gemv_impl(aqmb_layer_t layer, int k, const void* x, aqmb_dtype x_dtype, int batch, void* y,
                             aqmb_dtype y_dtype, aqmb_gemv_kernel kernel, aqmb_stream_t stream, const char* where) {
  Layer* L = (Layer*)layer;
  if (!is_live(L)) return fail(AQMB_EINVAL, "%s: not a live layer", where);
  aqmb_status s = validate_call(&L->d, 0, k, batch, x_dtype, y_dtype, x, y);
  if (s != AQMB_OK) return s;
  if ((int)kernel < AQMB_GEMV_AUTO || (int)kernel > AQMB_GEMV_LUT)
    return fail(AQMB_EINVAL, "%s: unknown kernel %d", where, (int)kernel);
  if (!gemv_kernel_serves(*L, k, batch, x_dtype, kernel))
    return fail(AQMB_EUNSUPPORTED, "%s: kernel %d cannot serve B = %d, k = %d, batch = %d, d_in = %d", where,
                (int)kernel, L->d.code_bits, k, batch, L->d.d_in);
  if ((s = check_resident(L, k, where)) != AQMB_OK) return s;
  if ((s = check_device(L)) != AQMB_OK) return s;
  return launch_gemv_kernel(*L, k, x, x_dtype, batch, y, y_dtype, kernel, (hipStream_t)stream, where);
}

aqmb_status aqmb_gemv(aqmb_layer_t layer, int k, const void* x, aqmb_dtype x_dtype, int batch, void* y,
                      aqmb_dtype y_dtype, aqmb_stream_t stream) {
  clear_error();
  return gemv_impl(layer, k, x, x_dtype, batch, y, y_dtype, AQMB_GEMV_AUTO, stream, "gemv");
}

aqmb_status aqmb_gemv_select(aqmb_layer_t layer, int k, const void* x, aqmb_dtype x_dtype, int batch, void* y,
                             aqmb_dtype y_dtype, aqmb_gemv_kernel kernel, aqmb_stream_t stream) {
  clear_error();
  return gemv_impl(layer, k, x, x_dtype, batch, y, y_dtype, kernel, stream, "gemv_select");
}

aqmb_status aqmb_gemv_multi(const aqmb_layer_t* layers, int n_layers, int k, const void* x, aqmb_dtype x_dtype,
                            int batch, void* const* ys, aqmb_dtype y_dtype, aqmb_stream_t stream) {
  clear_error();
  if (!layers || !ys) return fail(AQMB_EINVAL, "gemv_multi: null layers or outputs");
  if (n_layers < 1) return fail(AQMB_EINVAL, "gemv_multi: n_layers < 1");
  if (n_layers > AQMB_MAX_MULTI) return fail(AQMB_EUNSUPPORTED, "gemv_multi: more than AQMB_MAX_MULTI layers");
  const Layer* Ls[AQMB_MAX_MULTI];
  for (int i = 0; i < n_layers; ++i) {
    const Layer* L = (const Layer*)layers[i];
    if (!is_live((Layer*)L)) return fail(AQMB_EINVAL, "gemv_multi: not a live layer");
    if (i > 0 && (L->d.d_in != Ls[0]->d.d_in || L->device != Ls[0]->device))
      return fail(AQMB_EINVAL, "gemv_multi: layers differ in d_in or device");
    aqmb_status s = validate_call(&L->d, 0, k, batch, x_dtype, y_dtype, x, ys[i]);
    if (s != AQMB_OK) return s;
    if ((s = check_resident(L, k, "gemv_multi")) != AQMB_OK) return s;
    Ls[i] = L;
  }
  aqmb_status s = check_device((Layer*)Ls[0]);
  if (s != AQMB_OK) return s;
  // The one-launch kernels share the single-layer kernels' arithmetic, so the results are always
  // those of aqmb_gemv: the direct-gather multi-layer kernel when every layer would take the
  // direct-gather kernel; the matrix-core grid over all layers' row blocks when every layer would
  // take the one-block matrix-core kernel (same code width, at most one block per compute unit:
  // taller layers run their persistent kernel, one launch each); otherwise one launch per layer.
  bool per_layer = false, all_mma = true;
  for (int i = 0; i < n_layers; ++i) {
    const aqmb_gemv_kernel kern = gemv_auto(*Ls[i], k, batch, x_dtype);
    const bool mma = kern == AQMB_GEMV_MMA;
    per_layer = per_layer || Ls[i]->d.code_bits != 8 || kern != AQMB_GEMV_DIRECT;
    all_mma = all_mma && mma && Ls[i]->d.code_bits == Ls[0]->d.code_bits &&
              (Ls[i]->d.d_out + 15) / 16 <= Ls[i]->n_cu;
  }
  if (all_mma && n_layers >= 2) {
    hipError_t e = launch_gemv_mma_multi(Ls, n_layers, k, x, x_dtype, batch, ys, y_dtype, (hipStream_t)stream);
    return e == hipSuccess ? AQMB_OK : hip_fail(e, "gemv_multi: launch");
  }
  if (per_layer) {
    for (int i = 0; i < n_layers; ++i) {
      s = launch_gemv_kernel(*Ls[i], k, x, x_dtype, batch, ys[i], y_dtype, AQMB_GEMV_AUTO, (hipStream_t)stream,
                             "gemv_multi: launch");
      if (s != AQMB_OK) return s;
    }
    return AQMB_OK;
  }
  hipError_t e = launch_gemv_multi(Ls, n_layers, k, x, x_dtype, batch, ys, y_dtype, (hipStream_t)stream);
  return e == hipSuccess ? AQMB_OK : hip_fail(e, "gemv_multi: launch");
}

static aqmb_status gemm_impl(aqmb_layer_t layer, int k, const void* X, int n_tokens, void* Y, aqmb_dtype y_dtype,
                             aqmb_gemm_tiling tiling, aqmb_stream_t stream, const char* where) {
  Layer* L = (Layer*)layer;
  if (!is_live(L)) return fail(AQMB_EINVAL, "%s: not a live layer", where);
  aqmb_status s = validate_call(&L->d, 1, k, n_tokens, AQMB_BF16, y_dtype, X, Y);
  if (s != AQMB_OK) return s;
  if ((int)tiling < AQMB_GEMM_AUTO || (int)tiling > AQMB_GEMM_128x64)
    return fail(AQMB_EINVAL, "%s: unknown tiling %d", where, (int)tiling);
  if ((s = check_resident(L, k, where)) != AQMB_OK) return s;
  if ((s = check_device(L)) != AQMB_OK) return s;
  const bool small = tiling == AQMB_GEMM_ROWS16 || (tiling == AQMB_GEMM_AUTO && n_tokens <= kGemmSmallMax);
  const int tile = tiling == AQMB_GEMM_256x128 ? 0 : tiling == AQMB_GEMM_128x128 ? 1 : tiling == AQMB_GEMM_128x64 ? 2 : -1;
  hipError_t e = small ? launch_gemm_small(*L, k, X, n_tokens, Y, y_dtype, (hipStream_t)stream)
                       : launch_gemm(*L, k, X, n_tokens, Y, y_dtype, tile, (hipStream_t)stream);
  return e == hipSuccess ? AQMB_OK : hip_fail(e, where);
}

aqmb_status aqmb_gemm(aqmb_layer_t layer, int k, const void* X, int n_tokens, void* Y, aqmb_dtype y_dtype,
                      aqmb_stream_t stream) {
  clear_error();
  return gemm_impl(layer, k, X, n_tokens, Y, y_dtype, AQMB_GEMM_AUTO, stream, "gemm");
}

aqmb_status aqmb_gemm_select(aqmb_layer_t layer, int k, const void* X, int n_tokens, void* Y, aqmb_dtype y_dtype,
                             aqmb_gemm_tiling tiling, aqmb_stream_t stream) {
  clear_error();
  return gemm_impl(layer, k, X, n_tokens, Y, y_dtype, tiling, stream, "gemm_select");
}

aqmb_status aqmb_gemm_workspace_bytes(aqmb_layer_t layer, int k, int n_tokens, size_t* bytes) {
  clear_error();
  Layer* L = (Layer*)layer;
  if (!is_live(L)) return fail(AQMB_EINVAL, "gemm_workspace_bytes: not a live layer");
  if (!bytes) return fail(AQMB_EINVAL, "gemm_workspace_bytes: null bytes");
  if (k < 1 || k > L->d.num_codebooks)
    return fail(AQMB_EINVAL, "gemm_workspace_bytes: k = %d outside [1, %d]", k, L->d.num_codebooks);
  if (n_tokens < 1) return fail(AQMB_EINVAL, "gemm_workspace_bytes: n_tokens = %d", n_tokens);
  *bytes = gemm_two_pass_bytes(*L, k, n_tokens);
  return AQMB_OK;
}

aqmb_status aqmb_gemm_ws(aqmb_layer_t layer, int k, const void* X, int n_tokens, void* Y, aqmb_dtype y_dtype,
                         void* workspace, size_t workspace_bytes, aqmb_stream_t stream) {
  clear_error();
  Layer* L = (Layer*)layer;
  if (!is_live(L)) return fail(AQMB_EINVAL, "gemm_ws: not a live layer");
  if ((uintptr_t)workspace % 256 != 0) return fail(AQMB_EINVAL, "gemm_ws: workspace is not 256-byte aligned");
  aqmb_status s = validate_call(&L->d, 1, k, n_tokens, AQMB_BF16, y_dtype, X, Y);
  if (s != AQMB_OK) return s;
  const size_t need = gemm_two_pass_bytes(*L, k, n_tokens);
  if (need == 0 || !workspace || workspace_bytes < need)
    return gemm_impl(layer, k, X, n_tokens, Y, y_dtype, AQMB_GEMM_AUTO, stream, "gemm_ws");
  if ((s = check_resident(L, k, "gemm_ws")) != AQMB_OK) return s;
  if ((s = check_device(L)) != AQMB_OK) return s;
  const hipError_t e = launch_gemm_two_pass(*L, k, X, n_tokens, Y, y_dtype, workspace, (hipStream_t)stream);
  return e == hipSuccess ? AQMB_OK : hip_fail(e, "gemm_ws");
}

aqmb_status aqmb_prefix_distortion(aqmb_layer_t layer, const void* W, aqmb_dtype w_dtype, const void* X,
                                   aqmb_dtype x_dtype, int n, double* D, aqmb_stream_t stream) {
  clear_error();
  Layer* L = (Layer*)layer;
  if (!is_live(L)) return fail(AQMB_EINVAL, "prefix_distortion: not a live layer");
  if (!W) return fail(AQMB_EINVAL, "prefix_distortion: W is NULL");
  if ((uintptr_t)W % 16) return fail(AQMB_EINVAL, "prefix_distortion: W must be 16-byte aligned");
  aqmb_status s = validate_call(&L->d, 3, 0, n, x_dtype, w_dtype, X, D);
  if (s != AQMB_OK) return s;
  if ((s = check_device(L)) != AQMB_OK) return s;
  const hipStream_t st = (hipStream_t)stream;
  CallScratch sc;
  hipError_t e = sc.alloc(distortion_scratch_bytes(), st);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(AQMB_ENOMEM, "prefix_distortion: scratch: %s", hipGetErrorString(e));
  }
  e = launch_distortion(*L, W, X, n, D, (double*)sc.p, st);
  const hipError_t e2 = sc.release();
  if (e == hipSuccess) e = e2;
  return e == hipSuccess ? AQMB_OK : hip_fail(e, "prefix_distortion: launch");
}

aqmb_status aqmb_prefix_distortion_noalloc(aqmb_layer_t layer, const void* W, aqmb_dtype w_dtype, const void* X,
                                           aqmb_dtype x_dtype, int n, double* D, aqmb_stream_t stream) {
  clear_error();
  Layer* L = (Layer*)layer;
  if (!is_live(L)) return fail(AQMB_EINVAL, "prefix_distortion_noalloc: not a live layer");
  if (!W) return fail(AQMB_EINVAL, "prefix_distortion_noalloc: W is NULL");
  if ((uintptr_t)W % 16) return fail(AQMB_EINVAL, "prefix_distortion_noalloc: W must be 16-byte aligned");
  aqmb_status s = validate_call(&L->d, 3, 0, n, x_dtype, w_dtype, X, D);
  if (s != AQMB_OK) return s;
  if ((s = check_device(L)) != AQMB_OK) return s;
  double* sc = nullptr;
  size_t have = 0;
  hipError_t e = distortion_static_scratch(L->device, &sc, &have);
  if (e != hipSuccess) return hip_fail(e, "prefix_distortion_noalloc: scratch address");
  if (distortion_scratch_bytes() > have)
    return fail(AQMB_EUNSUPPORTED, "prefix_distortion_noalloc: needs %zu bytes of scratch, the library holds %zu",
                distortion_scratch_bytes(), have);
  e = launch_distortion(*L, W, X, n, D, sc, (hipStream_t)stream);
  return e == hipSuccess ? AQMB_OK : hip_fail(e, "prefix_distortion_noalloc: launch");
}

aqmb_status aqmb_beam_search(const aqmb_desc* desc, int k, int beam, const void* W, const uint16_t* codebooks,
                             const uint16_t* scales, uint8_t* codes, float* errors, aqmb_stream_t stream) {
  clear_error();
  aqmb_status s = validate_call(desc, 4, k, beam, AQMB_F16, AQMB_F16, W, codes);
  if (s != AQMB_OK) return s;
  if (!codebooks || !scales) return fail(AQMB_EINVAL, "beam_search: codebooks or scales is NULL");
  if ((uintptr_t)codebooks % 16) return fail(AQMB_EINVAL, "beam_search: codebooks must be 16-byte aligned");
  if ((uintptr_t)scales % 2 || (uintptr_t)errors % 4) return fail(AQMB_EINVAL, "beam_search: misaligned scales or errors");
  hipError_t e = launch_beam_search(*desc, k, beam, W, codebooks, scales, codes, errors, (hipStream_t)stream);
  return e == hipSuccess ? AQMB_OK : hip_fail(e, "beam_search: launch");
}

aqmb_status aqmb_beam_search_weighted(const aqmb_desc* desc, int k, int beam, const void* W,
                                      const uint16_t* codebooks, const uint16_t* scales, const float* H,
                                      uint8_t* codes, float* errors, aqmb_stream_t stream) {
  clear_error();
  aqmb_status s = validate_call(desc, 4, k, beam, AQMB_F16, AQMB_F16, W, codes);
  if (s != AQMB_OK) return s;
  if (!codebooks || !scales || !H) return fail(AQMB_EINVAL, "beam_search_weighted: codebooks, scales or H is NULL");
  if ((uintptr_t)codebooks % 16) return fail(AQMB_EINVAL, "beam_search_weighted: codebooks must be 16-byte aligned");
  if ((uintptr_t)scales % 2 || (uintptr_t)errors % 4 || (uintptr_t)H % 4)
    return fail(AQMB_EINVAL, "beam_search_weighted: misaligned scales, H or errors");
  hipError_t e = launch_beam_search_weighted(*desc, k, beam, W, codebooks, scales, H, codes, errors,
                                             (hipStream_t)stream);
  return e == hipSuccess ? AQMB_OK : hip_fail(e, "beam_search_weighted: launch");
}

aqmb_status aqmb_dequant(aqmb_layer_t layer, int k, void* W, aqmb_dtype w_dtype, aqmb_stream_t stream) {
  clear_error();
  Layer* L = (Layer*)layer;
  if (!is_live(L)) return fail(AQMB_EINVAL, "dequant: not a live layer");
  aqmb_status s = validate_call(&L->d, 2, k, 0, AQMB_F16, w_dtype, nullptr, W);
  if (s != AQMB_OK) return s;
  if ((s = check_resident(L, k, "dequant")) != AQMB_OK) return s;
  if ((s = check_device(L)) != AQMB_OK) return s;
  hipError_t e = launch_dequant(*L, k, W, w_dtype, (hipStream_t)stream);
  return e == hipSuccess ? AQMB_OK : hip_fail(e, "dequant: launch");
}

}  // extern "C"
