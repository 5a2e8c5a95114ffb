// Host-side argument validation, status strings and the bits-per-weight formula.
// Nothing here touches the GPU, so it is exercised by CPU-only tests.
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>

#include "layer.h"

namespace aqmb {

static thread_local std::string g_last_error;

aqmb_status fail(aqmb_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
aqmb_status fail(aqmb_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

void clear_error() { g_last_error.clear(); }

aqmb_status validate_desc(const aqmb_desc* d) {
  if (!d) return fail(AQMB_EINVAL, "descriptor is NULL");
  if (d->d_out < 1) return fail(AQMB_EINVAL, "d_out = %d must be >= 1", d->d_out);
  if (d->group_size != 8) return fail(AQMB_EUNSUPPORTED, "group_size = %d: only g = 8 is supported", d->group_size);
  if (d->d_in < d->group_size || d->d_in % d->group_size)
    return fail(AQMB_EINVAL, "d_in = %d must be a positive multiple of g = %d", d->d_in, d->group_size);
  if (d->code_bits != 4 && d->code_bits != 8 && d->code_bits != 16)
    return fail(AQMB_EUNSUPPORTED, "code_bits = %d: only B = 4, 8 and 16 are supported", d->code_bits);
  if (d->num_codebooks < 1) return fail(AQMB_EINVAL, "num_codebooks = %d must be >= 1", d->num_codebooks);
  if (d->num_codebooks > 8) return fail(AQMB_EUNSUPPORTED, "num_codebooks = %d: at most 8", d->num_codebooks);
  if ((uint64_t)d->d_out * (uint64_t)d->d_in >= (1ull << 32))
    return fail(AQMB_EINVAL, "d_out * d_in = %llu must be below 2^32",
                (unsigned long long)d->d_out * (unsigned long long)d->d_in);
  return AQMB_OK;
}

static bool valid_dtype(int t) { return t == AQMB_F16 || t == AQMB_BF16 || t == AQMB_F32; }

aqmb_status validate_call(const aqmb_desc* d, int op, int k, int n, aqmb_dtype in_dt, aqmb_dtype out_dt,
                          const void* in, const void* out) {
  aqmb_status s = validate_desc(d);
  if (s != AQMB_OK) return s;
  if (op != 3 && (k < 1 || k > d->num_codebooks))   // the distortion covers every k at once
    return fail(AQMB_EINVAL, "k = %d outside [1, M = %d]", k, d->num_codebooks);
  if (op == 4) {  // beam search: n = beam width, in = W, out = codes
    if (!in || !out) return fail(AQMB_EINVAL, "beam_search: W or codes is NULL");
    if (n < 1) return fail(AQMB_EINVAL, "beam_search: beam = %d must be >= 1", n);
    if (n > AQMB_MAX_BEAM) return fail(AQMB_EUNSUPPORTED, "beam_search: beam = %d above %d", n, AQMB_MAX_BEAM);
    if (d->code_bits == 16) return fail(AQMB_EUNSUPPORTED, "beam_search: only B = 4 and B = 8 codebooks are supported");
    if ((uintptr_t)in % 16) return fail(AQMB_EINVAL, "beam_search: W must be 16-byte aligned");
    const uint64_t chunks = ((uint64_t)(d->d_in / d->group_size) + 255) / 256;
    if (chunks * (uint64_t)d->d_out >= (1ull << 31)) return fail(AQMB_EINVAL, "beam_search: matrix too large");
    return AQMB_OK;
  }
  if (!valid_dtype(out_dt)) return fail(AQMB_EUNSUPPORTED, "output dtype %d is not F16, BF16 or F32", (int)out_dt);
  switch (op) {
    case 0:  // gemv
      if (!in || !out) return fail(AQMB_EINVAL, "gemv: x or y is NULL");
      if (n < 1) return fail(AQMB_EINVAL, "gemv: batch = %d must be >= 1", n);
      if (n > AQMB_MAX_BATCH) return fail(AQMB_EUNSUPPORTED, "gemv: batch = %d above %d", n, AQMB_MAX_BATCH);
      if (in_dt != AQMB_F16 && in_dt != AQMB_BF16)
        return fail(AQMB_EUNSUPPORTED, "gemv: x dtype must be F16 or BF16");
      if ((uintptr_t)in % 16 || (uintptr_t)out % 16) return fail(AQMB_EINVAL, "gemv: x and y must be 16-byte aligned");
      return AQMB_OK;
    case 1:  // gemm
      if (!in || !out) return fail(AQMB_EINVAL, "gemm: X or Y is NULL");
      if (n < 1) return fail(AQMB_EINVAL, "gemm: n_tokens = %d must be >= 1", n);
      if (d->code_bits == 16) return fail(AQMB_EUNSUPPORTED, "gemm: only B = 4 and B = 8 layers are supported");
      if (out_dt != AQMB_BF16 && out_dt != AQMB_F32)
        return fail(AQMB_EUNSUPPORTED, "gemm: Y dtype must be BF16 or F32");
      if ((uint64_t)n * (uint64_t)(d->d_in > d->d_out ? d->d_in : d->d_out) >= (1ull << 32))
        return fail(AQMB_EINVAL, "gemm: n_tokens * max(d_in, d_out) must be below 2^32");
      if ((uintptr_t)in % 16 || (uintptr_t)out % 16) return fail(AQMB_EINVAL, "gemm: X and Y must be 16-byte aligned");
      return AQMB_OK;
    case 2:  // dequant
      if (!out) return fail(AQMB_EINVAL, "dequant: W is NULL");
      if ((uintptr_t)out % 16) return fail(AQMB_EINVAL, "dequant: W must be 16-byte aligned");
      return AQMB_OK;
    case 3:  // prefix distortion: in = X (dtype in_dt), out = D, out_dt = W's dtype
      if (!in || !out) return fail(AQMB_EINVAL, "prefix_distortion: X or D is NULL");
      if (n < 1) return fail(AQMB_EINVAL, "prefix_distortion: n = %d must be >= 1", n);
      if (n > (1 << 30)) return fail(AQMB_EUNSUPPORTED, "prefix_distortion: n = %d above 2^30", n);
      if (d->code_bits == 16) return fail(AQMB_EUNSUPPORTED, "prefix_distortion: only B = 4 and B = 8 layers are supported");
      if (in_dt != AQMB_F16 || out_dt != AQMB_F16)
        return fail(AQMB_EUNSUPPORTED, "prefix_distortion: W and X must be F16");
      if ((uintptr_t)in % 16) return fail(AQMB_EINVAL, "prefix_distortion: X must be 16-byte aligned");
      if ((uintptr_t)out % 8) return fail(AQMB_EINVAL, "prefix_distortion: D must be 8-byte aligned");
      return AQMB_OK;
    default:
      return fail(AQMB_EINVAL, "unknown op %d", op);
  }
}

}  // namespace aqmb

extern "C" {

const char* aqmb_strerror(aqmb_status s) {
  switch (s) {
    case AQMB_OK: return "success";
    case AQMB_EINVAL: return "invalid argument";
    case AQMB_EUNSUPPORTED: return "unsupported configuration";
    case AQMB_ENOMEM: return "out of device memory";
    case AQMB_EHIP: return "HIP runtime error";
  }
  return "unknown status";
}

const char* aqmb_last_error(void) { return aqmb::g_last_error.c_str(); }

double aqmb_bits_per_weight(const aqmb_desc* d, int k) {
  if (aqmb::validate_desc(d) != AQMB_OK) return -1.0;
  if (k < 1 || k > d->num_codebooks) return -1.0;
  const double g = d->group_size, B = d->code_bits, dout = d->d_out, din = d->d_in;
  const double codebook_bits = 16.0 * g * k * (double)(1ull << d->code_bits);
  const double code_bits = dout * (din / g) * B * k;
  const double scale_bits = 16.0 * dout;
  return (codebook_bits + code_bits + scale_bits) / (dout * din);
}

aqmb_status aqmb_validate(const aqmb_desc* desc, int op, int k, int n, aqmb_dtype in_dtype, aqmb_dtype out_dtype,
                          const void* in, const void* out) {
  aqmb::clear_error();
  return aqmb::validate_call(desc, op, k, n, in_dtype, out_dtype, in, out);
}

}  // extern "C"
