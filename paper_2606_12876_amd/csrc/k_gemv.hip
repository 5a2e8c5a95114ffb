// Decode GEMV: y[b][i] = s_i * sum_j sum_{m<k} <x[b, group j], C_m[code(m,i,j)]>.
//
// Work split: a workgroup owns a chunk of rows and one slice (16 consecutive groups for
// 8-bit codes, 8 for 16-bit codes); every row's sum over slices is a split-K reduction.
// Each workgroup writes fp32 partial sums for its rows to the layer's workspace; a second,
// small kernel adds the partials of all slices in slice order, applies the row scale and
// rounds once to the output dtype. The kernel boundary orders the two phases (no
// device-wide fences inside the main kernel), and the result does not depend on scheduling.
//
// 8-bit codes (256 codewords): lookup tables in LDS. For the slice's groups and every used
// plane m, LUT_m[j][c] = <x[b, group j], C_m[c]> is built once per workgroup (one codeword per
// thread, fp32 dot products of exact fp16 products), then every code byte costs one LDS read
// and one fp32 add. Rows map to threads, so each thread's accumulators need no cross-lane
// reduction. Code planes m >= k are never read.
//
// 16-bit codes (65536 codewords, 1 MiB per codebook): codewords are gathered from global
// memory (resident in L2), summed over planes, and dotted with x staged in LDS.
#include "device.h"
#include "launch.h"

namespace aqmb {

constexpr int kThreads = 512;       // 8 waves: two per SIMD
constexpr int kRowsPerThread = 1;
constexpr int kRowsPerWG = kThreads * kRowsPerThread;
constexpr int kReduceThreads = 256;

struct GemvArgs {
  const unsigned char* codes;
  const uint16_t* codebooks;
  const uint16_t* scales;
  const void* x;
  void* y;
  float* partials;     // [S][batch][d_out]
  size_t plane_bytes;
  int d_out, d_in, G, S, k, batch;
  int y_dtype;
};

size_t gemv_workspace_floats(const aqmb_desc& d, int G, int S) {
  (void)G;
  return (size_t)S * AQMB_MAX_BATCH * d.d_out + 64;
}

// Partial sums of one batch tile of this workgroup's rows.
template <int NB>
__device__ __forceinline__ void store_partials(const GemvArgs& a, int b0, const float (&acc)[kRowsPerThread][NB]) {
  const int tid = threadIdx.x, slice = blockIdx.y;
  const int row0 = blockIdx.x * kRowsPerWG;
#pragma unroll
  for (int r = 0; r < kRowsPerThread; ++r) {
    const int row = row0 + tid + r * kThreads;
    if (row < a.d_out) {
#pragma unroll
      for (int b = 0; b < NB; ++b)
        if (b0 + b < a.batch)
          a.partials[((size_t)slice * a.batch + b0 + b) * a.d_out + row] = acc[r][b];
    }
  }
}

// y[b][i] = s_i * sum over slices of the partials. A block takes 64 row quads (16-byte
// loads of four consecutive rows); its four waves take interleaved quarters of the slices with
// all their loads in flight, and the four quarter sums are added in a fixed order, so the
// result does not depend on scheduling.
__global__ __launch_bounds__(kReduceThreads) void gemv_reduce_kernel(GemvArgs a) {
  constexpr int kQuads = 64, kParts = kReduceThreads / kQuads, kInflight = 8;
  __shared__ float4 part_sum[kParts][kQuads];
  const int quads = (a.d_out + 3) / 4;
  const int lane = threadIdx.x % kQuads, part = threadIdx.x / kQuads;
  const int item = blockIdx.x * kQuads + lane;     // (batch row, row quad)
  const bool active = item < a.batch * quads;
  const int b = active ? item / quads : 0, r0 = active ? (item % quads) * 4 : 0;
  const bool vec = (a.d_out % 4) == 0;  // 16-byte aligned row quads
  float4 sum = make_float4(0.f, 0.f, 0.f, 0.f);
  if (active) {
    for (int s0 = part; s0 < a.S; s0 += kParts * kInflight) {
      float4 v[kInflight];
#pragma unroll
      for (int u = 0; u < kInflight; ++u) {
        const int sl = s0 + u * kParts;
        v[u] = make_float4(0.f, 0.f, 0.f, 0.f);
        if (sl < a.S) {
          const float* p = a.partials + ((size_t)sl * a.batch + b) * a.d_out + r0;
          if (vec) {
            v[u] = *(const float4*)p;
          } else {
            v[u].x = p[0];
            if (r0 + 1 < a.d_out) v[u].y = p[1];
            if (r0 + 2 < a.d_out) v[u].z = p[2];
            if (r0 + 3 < a.d_out) v[u].w = p[3];
          }
        }
      }
#pragma unroll
      for (int u = 0; u < kInflight; ++u) {
        sum.x += v[u].x; sum.y += v[u].y; sum.z += v[u].z; sum.w += v[u].w;
      }
    }
  }
  part_sum[part][lane] = sum;
  __syncthreads();
  if (part != 0 || !active) return;
#pragma unroll
  for (int p2 = 1; p2 < kParts; ++p2) {
    const float4 o = part_sum[p2][lane];
    sum.x += o.x; sum.y += o.y; sum.z += o.z; sum.w += o.w;
  }
  const float v[4] = {sum.x, sum.y, sum.z, sum.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int row = r0 + e;
    if (row >= a.d_out) break;
    const float val = v[e] * f16_to_f32(a.scales[row]);
    const size_t o = (size_t)b * a.d_out + row;
    if (a.y_dtype == AQMB_F16) OutT<AQMB_F16>::store(a.y, o, val);
    else if (a.y_dtype == AQMB_BF16) OutT<AQMB_BF16>::store(a.y, o, val);
    else OutT<AQMB_F32>::store(a.y, o, val);
  }
}

// x element pair -> fp32 values (XDT = F16 or BF16).
template <int XDT>
__device__ __forceinline__ void x_pair(uint32_t w, float& lo, float& hi) {
  if constexpr (XDT == AQMB_F16) { lo = f16lo(w); hi = f16hi(w); }
  else { lo = bf16lo(w); hi = bf16hi(w); }
}

// <x group (8 values in 4 words), codeword (8 fp16 in 4 words)> in fp32.
template <int XDT>
__device__ __forceinline__ float group_dot(uint4 xw, uint4 cw) {
  if constexpr (XDT == AQMB_F16) {
    float s = dot2_f16(xw.x, cw.x, 0.f);
    s = dot2_f16(xw.y, cw.y, s);
    s = dot2_f16(xw.z, cw.z, s);
    return dot2_f16(xw.w, cw.w, s);
  } else {
    float x0, x1, x2, x3, x4, x5, x6, x7;
    x_pair<XDT>(xw.x, x0, x1); x_pair<XDT>(xw.y, x2, x3); x_pair<XDT>(xw.z, x4, x5); x_pair<XDT>(xw.w, x6, x7);
    float s = x0 * f16lo(cw.x);
    s = __builtin_fmaf(x1, f16hi(cw.x), s);
    s = __builtin_fmaf(x2, f16lo(cw.y), s);
    s = __builtin_fmaf(x3, f16hi(cw.y), s);
    s = __builtin_fmaf(x4, f16lo(cw.z), s);
    s = __builtin_fmaf(x5, f16hi(cw.z), s);
    s = __builtin_fmaf(x6, f16lo(cw.w), s);
    return __builtin_fmaf(x7, f16hi(cw.w), s);
  }
}

// LUT kernel for 8-bit codes, K = k planes (a template parameter: the plane loop is
// straight-line code). BT batch rows share one LUT entry (BT floats); batch tiles of BT rows
// are processed one after another with the codes kept in registers. The LUT covers JH = 16/BT
// groups of the slice at a time, so it needs K * 16 KiB of LDS for every BT.
template <int K, int BT, int XDT>
__global__ __launch_bounds__(kThreads) void gemv_lut_kernel(GemvArgs a) {
  constexpr int JH = 16 / BT;
  extern __shared__ float lut[];                          // [K][JH][256][BT]
  __shared__ uint4 xs[AQMB_MAX_BATCH * 16];               // x of the slice: [batch][16 groups] x 8 values
  const int tid = threadIdx.x;
  const int slice = blockIdx.y;
  const int row0 = blockIdx.x * kRowsPerWG;

  // 1. Loads, oldest first: x of the slice, then the code planes 0..K-1 of this thread's rows,
  //    then this thread's codeword of each codebook. The code loads stay in flight while the
  //    x staging and the LUT construction proceed.
  static_assert(kThreads == 512, "the LUT build assigns two threads per codeword");
  uint4 xw = make_uint4(0, 0, 0, 0);
  const int xb = tid >> 4, xj = slice * 16 + (tid & 15);
  if (xb < a.batch && xj < a.G) xw = *(const uint4*)((const uint16_t*)a.x + (size_t)xb * a.d_in + (size_t)xj * 8);
  uint4 v[kRowsPerThread][K];
#pragma unroll
  for (int r = 0; r < kRowsPerThread; ++r) {
    const int row = row0 + tid + r * kThreads;
#pragma unroll
    for (int m = 0; m < K; ++m) {
      v[r][m] = make_uint4(0, 0, 0, 0);
      if (row < a.d_out)
        v[r][m] = load_stream16(a.codes + m * a.plane_bytes + ((size_t)slice * a.d_out + row) * 16);
    }
  }
  const int c = tid & 255, jhalf = tid >> 8;  // LUT column and half of the groups this thread builds
  uint4 cw[K];
#pragma unroll
  for (int m = 0; m < K; ++m) cw[m] = ((const uint4*)a.codebooks)[m * 256 + c];
  if (tid < AQMB_MAX_BATCH * 16) xs[tid] = xw;  // groups past G and batch rows past `batch` are zero
  __syncthreads();

  for (int b0 = 0; b0 < a.batch; b0 += BT) {
    float acc[kRowsPerThread][BT][2];
#pragma unroll
    for (int r = 0; r < kRowsPerThread; ++r)
#pragma unroll
      for (int bt = 0; bt < BT; ++bt) acc[r][bt][0] = acc[r][bt][1] = 0.f;
#pragma unroll
    for (int h = 0; h < BT; ++h) {  // parts of JH groups
      if (b0 + h > 0) __syncthreads();  // the previous part's lookups are done
      // 2. LUT entries of codeword c for every plane, batch row and this thread's half of
      //    the part's groups (two threads per codeword).
#pragma unroll
      for (int j2 = 0; j2 < JH / 2; ++j2) {
        const int jj = jhalf * (JH / 2) + j2;
        uint4 xv[BT];
#pragma unroll
        for (int bt = 0; bt < BT; ++bt) xv[bt] = xs[(b0 + bt) * 16 + h * JH + jj];
#pragma unroll
        for (int m = 0; m < K; ++m) {
          float e[BT];
#pragma unroll
          for (int bt = 0; bt < BT; ++bt) e[bt] = group_dot<XDT>(xv[bt], cw[m]);
          float* dst = lut + ((m * JH + jj) * 256 + c) * BT;
          if constexpr (BT == 1) dst[0] = e[0];
          else if constexpr (BT == 2) *(float2*)dst = make_float2(e[0], e[1]);
          else *(float4*)dst = make_float4(e[0], e[1], e[2], e[3]);
        }
      }
      __syncthreads();
      // 3. Gather: one LDS lookup (BT floats) per code byte; two accumulators per output
      //    shorten the dependency chains.
#pragma unroll
      for (int r = 0; r < kRowsPerThread; ++r) {
#pragma unroll
        for (int m = 0; m < K; ++m) {
#pragma unroll
          for (int jj = 0; jj < JH; ++jj) {
            const int q = h * JH + jj;  // byte index in the 16-byte chunk
            const uint32_t word = (&v[r][m].x)[q >> 2];
            const uint32_t c = (word >> (8 * (q & 3))) & 0xFFu;
            const float* src = lut + ((m * JH + jj) * 256 + c) * BT;
            const int p = jj & 1;
            if constexpr (BT == 1) {
              acc[r][0][p] += src[0];
            } else if constexpr (BT == 2) {
              const float2 e2 = *(const float2*)src;
              acc[r][0][p] += e2.x;
              acc[r][1][p] += e2.y;
            } else {
              const float4 e4 = *(const float4*)src;
              acc[r][0][p] += e4.x;
              acc[r][1][p] += e4.y;
              acc[r][2][p] += e4.z;
              acc[r][3][p] += e4.w;
            }
          }
        }
      }
    }
    float out[kRowsPerThread][BT];
#pragma unroll
    for (int r = 0; r < kRowsPerThread; ++r)
#pragma unroll
      for (int bt = 0; bt < BT; ++bt) out[r][bt] = acc[r][bt][0] + acc[r][bt][1];
    store_partials<BT>(a, b0, out);
  }
}

// 16-bit codes: codewords from global memory. One slice = 8 groups per row.
template <int XDT, int NB>
__global__ __launch_bounds__(kThreads) void gemv_b16_kernel(GemvArgs a) {
  __shared__ float xs[AQMB_MAX_BATCH][64];  // x of the slice's 8 groups, fp32
  const int tid = threadIdx.x;
  const int slice = blockIdx.y;
  const int row0 = blockIdx.x * kRowsPerWG;
  const int k = a.k;
  for (int q = tid; q < a.batch * 64; q += kThreads) {
    const int b = q / 64, e = q % 64;
    const int col = slice * 64 + e;
    float v = 0.f;
    if (col < a.d_in) {
      const uint16_t bits = ((const uint16_t*)a.x)[(size_t)b * a.d_in + col];
      v = XDT == AQMB_F16 ? f16_to_f32(bits) : __builtin_bit_cast(float, (uint32_t)bits << 16);
    }
    xs[b][e] = v;
  }
  uint4 v[kRowsPerThread][8];
#pragma unroll
  for (int r = 0; r < kRowsPerThread; ++r) {
    const int row = row0 + tid + r * kThreads;
#pragma unroll
    for (int m = 0; m < 8; ++m) {
      v[r][m] = make_uint4(0, 0, 0, 0);
      if (m < k && row < a.d_out)
        v[r][m] = load_stream16(
            (a.codes + m * a.plane_bytes + ((size_t)slice * a.d_out + row) * 16));
    }
  }
  __syncthreads();
  float acc[kRowsPerThread][NB];
#pragma unroll
  for (int r = 0; r < kRowsPerThread; ++r)
#pragma unroll
    for (int b = 0; b < NB; ++b) acc[r][b] = 0.f;
  const uint4* cb = (const uint4*)a.codebooks;
#pragma unroll
  for (int r = 0; r < kRowsPerThread; ++r) {
    if (row0 + tid + r * kThreads >= a.d_out) continue;
#pragma unroll
    for (int jj = 0; jj < 8; ++jj) {
      const int j = slice * 8 + jj;
      if (j >= a.G) continue;
      float w[8];
#pragma unroll
      for (int m = 0; m < 8; ++m) {
        if (m < k) {
          const uint32_t word = (&v[r][m].x)[jj >> 1];
          const uint32_t c = (word >> (16 * (jj & 1))) & 0xFFFFu;
          const uint4 cwv = cb[((size_t)m << 16) + c];
          const float f[8] = {f16lo(cwv.x), f16hi(cwv.x), f16lo(cwv.y), f16hi(cwv.y),
                              f16lo(cwv.z), f16hi(cwv.z), f16lo(cwv.w), f16hi(cwv.w)};
#pragma unroll
          for (int e = 0; e < 8; ++e) w[e] = m == 0 ? f[e] : w[e] + f[e];
        }
      }
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        if (b < a.batch) {
          float s = acc[r][b];
#pragma unroll
          for (int e = 0; e < 8; ++e) s = __builtin_fmaf(xs[b][jj * 8 + e], w[e], s);
          acc[r][b] = s;
        }
      }
    }
  }
  store_partials<NB>(a, 0, acc);
}

template <int K, int XDT>
static void launch_lut(const GemvArgs& a, dim3 grid, hipStream_t st) {
  const size_t lds = (size_t)K * 16 * 256 * sizeof(float);  // K * JH * 256 * BT floats, JH * BT = 16
  if (a.batch == 1) gemv_lut_kernel<K, 1, XDT><<<grid, kThreads, lds, st>>>(a);
  else if (a.batch == 2) gemv_lut_kernel<K, 2, XDT><<<grid, kThreads, lds, st>>>(a);
  else gemv_lut_kernel<K, 4, XDT><<<grid, kThreads, lds, st>>>(a);
}

template <int XDT>
static void launch_x(const GemvArgs& a, bool b16, dim3 grid, hipStream_t st) {
  if (b16) {
    if (a.batch <= 4) gemv_b16_kernel<XDT, 4><<<grid, kThreads, 0, st>>>(a);
    else gemv_b16_kernel<XDT, AQMB_MAX_BATCH><<<grid, kThreads, 0, st>>>(a);
    return;
  }
  switch (a.k) {
    case 1: launch_lut<1, XDT>(a, grid, st); break;
    case 2: launch_lut<2, XDT>(a, grid, st); break;
    case 3: launch_lut<3, XDT>(a, grid, st); break;
    case 4: launch_lut<4, XDT>(a, grid, st); break;
    case 5: launch_lut<5, XDT>(a, grid, st); break;
    case 6: launch_lut<6, XDT>(a, grid, st); break;
    case 7: launch_lut<7, XDT>(a, grid, st); break;
    default: launch_lut<8, XDT>(a, grid, st); break;
  }
}

hipError_t launch_gemv(const Layer& L, int k, const void* x, aqmb_dtype x_dtype, int batch, void* y,
                       aqmb_dtype y_dtype, hipStream_t st) {
  GemvArgs a;
  a.codes = L.codes;
  a.codebooks = L.codebooks;
  a.scales = L.scales;
  a.x = x;
  a.y = y;
  a.partials = L.ws;
  a.plane_bytes = L.plane_bytes;
  a.d_out = L.d.d_out;
  a.d_in = L.d.d_in;
  a.G = L.G;
  a.S = L.S;
  a.k = k;
  a.batch = batch;
  a.y_dtype = (int)y_dtype;
  const dim3 grid((L.d.d_out + kRowsPerWG - 1) / kRowsPerWG, L.S);
  const bool b16 = L.d.code_bits == 16;
  if (x_dtype == AQMB_F16) launch_x<AQMB_F16>(a, b16, grid, st);
  else launch_x<AQMB_BF16>(a, b16, grid, st);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int items = batch * ((L.d.d_out + 3) / 4);
  gemv_reduce_kernel<<<(items + 63) / 64, kReduceThreads, 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace aqmb
