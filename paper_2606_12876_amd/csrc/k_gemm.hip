// Prefill GEMM: Y[n][i] = s_i * sum_t X[n][t] * Wb[i][t], where Wb is the unscaled
// reconstruction from the first k codebooks (binary32 left fold over planes), rounded to bf16,
// and the products run on the bf16 matrix cores (v_mfma_f32_32x32x16_bf16, fp32 accumulate).
//
// A workgroup computes a BM x BN tile of Y (BM tokens, BN output rows). For each BK-wide step
// along d_in it stages the X tile in LDS and dequantizes the BN x BK weight tile into LDS:
// every thread gathers the k codewords of its groups from the codebooks held in LDS, folds
// them in binary32 and rounds to bf16. Four waves then run the MFMA K-loop on the two tiles.
// The row scales are applied to the fp32 accumulators in the epilogue.
#include "device.h"
#include "launch.h"

namespace aqmb {

namespace gemm {
constexpr int BM = 128, BN = 128, BK = 64;
constexpr int kThreads = 256;
constexpr int LDA = BK + 8;  // row pitch in bf16 elements: 144 bytes keeps 16-byte fragment reads conflict-free
}  // namespace gemm

template <int YDT>
__global__ __launch_bounds__(gemm::kThreads) void gemm_kernel(const unsigned char* __restrict__ codes,
                                                              const uint16_t* __restrict__ codebooks,
                                                              const uint16_t* __restrict__ scales,
                                                              const uint16_t* __restrict__ X, void* __restrict__ Y,
                                                              int n_tokens, int d_out, int d_in, int G, int k,
                                                              size_t plane_bytes) {
  using namespace gemm;
  extern __shared__ uint4 smem[];
  uint16_t* As = (uint16_t*)smem;              // [BM][LDA] bf16
  uint16_t* Bs = As + BM * LDA;                // [BN][LDA] bf16
  uint4* cbs = (uint4*)(Bs + BN * LDA);        // [k][256] codewords (fp16 x 8)

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n0 = blockIdx.y * BM, i0 = blockIdx.x * BN;
  const int wm = wave >> 1, wn = wave & 1;     // 2 x 2 waves, 64 x 64 each

  for (int q = tid; q < k * 256; q += kThreads) cbs[q] = ((const uint4*)codebooks)[q];

  f32x16_t acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[a][b][e] = 0.f;

  const int n_ksteps = (d_in + BK - 1) / BK;
  for (int ks = 0; ks < n_ksteps; ++ks) {
    const int k0 = ks * BK;
    __syncthreads();  // previous step's fragment reads are done (and the codebooks are staged)
    // X tile: BM rows x BK columns = BM * 8 chunks of 16 bytes.
#pragma unroll
    for (int p = 0; p < BM * 8 / kThreads; ++p) {
      const int q = tid + p * kThreads;
      const int row = q >> 3, c8 = (q & 7) * 8;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (n0 + row < n_tokens && k0 + c8 < d_in) v = *(const uint4*)(X + (size_t)(n0 + row) * d_in + k0 + c8);
      *(uint4*)(As + row * LDA + c8) = v;
    }
    // Weight tile: BN rows x 8 groups; each thread dequantizes 4 groups of one row.
    {
      const int row = tid >> 1, g4 = (tid & 1) * 4;
      const int j0 = k0 / 8 + g4;          // first group; the 4 groups share one code slice
      const int s = j0 >> 4, jj0 = j0 & 15;
      const bool row_ok = i0 + row < d_out;
      uint32_t cw[8];
#pragma unroll
      for (int m = 0; m < 8; ++m) {
        cw[m] = 0;
        if (m < k && row_ok && j0 < G)
          cw[m] = *(const uint32_t*)(codes + m * plane_bytes + ((size_t)s * d_out + i0 + row) * 16 + jj0);
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float w[8];
#pragma unroll
        for (int m = 0; m < 8; ++m) {
          if (m < k) {
            const uint4 c = cbs[m * 256 + ((cw[m] >> (8 * q)) & 0xFF)];
            const float f[8] = {f16lo(c.x), f16hi(c.x), f16lo(c.y), f16hi(c.y),
                                f16lo(c.z), f16hi(c.z), f16lo(c.w), f16hi(c.w)};
#pragma unroll
            for (int t = 0; t < 8; ++t) w[t] = m == 0 ? f[t] : w[t] + f[t];
          }
        }
        uint4 packed = make_uint4(pack_bf16x2(w[0], w[1]), pack_bf16x2(w[2], w[3]), pack_bf16x2(w[4], w[5]),
                                  pack_bf16x2(w[6], w[7]));
        if (!row_ok || j0 + q >= G) packed = make_uint4(0, 0, 0, 0);
        *(uint4*)(Bs + row * LDA + (g4 + q) * 8) = packed;
      }
    }
    __syncthreads();
    // MFMA: 4 sub-steps of K = 16.
#pragma unroll
    for (int kk = 0; kk < BK; kk += 16) {
      bf16x8_t af[2], bfr[2];
#pragma unroll
      for (int a = 0; a < 2; ++a) {
        const int row = wm * 64 + a * 32 + (lane & 31);
        af[a] = *(const bf16x8_t*)(As + row * LDA + kk + (lane >> 5) * 8);
      }
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const int col = wn * 64 + b * 32 + (lane & 31);
        bfr[b] = *(const bf16x8_t*)(Bs + col * LDA + kk + (lane >> 5) * 8);
      }
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b) acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[a], bfr[b], acc[a][b], 0, 0, 0);
    }
  }
  // Epilogue. Accumulator element e of lane l in a 32 x 32 block holds
  // row 8 * (e / 4) + 4 * (l / 32) + e % 4, column l % 32.
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    const int col = i0 + wn * 64 + b * 32 + (lane & 31);
    if (col >= d_out) continue;
    const float scale = f16_to_f32(scales[col]);
#pragma unroll
    for (int a = 0; a < 2; ++a) {
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int row = n0 + wm * 64 + a * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
        if (row < n_tokens) OutT<YDT>::store(Y, (size_t)row * d_out + col, acc[a][b][e] * scale);
      }
    }
  }
}

hipError_t launch_gemm(const Layer& L, int k, const void* X, int n_tokens, void* Y, aqmb_dtype y_dtype,
                       hipStream_t st) {
  using namespace gemm;
  const dim3 grid((L.d.d_out + BN - 1) / BN, (n_tokens + BM - 1) / BM);
  const size_t lds = (size_t)(BM + BN) * LDA * 2 + (size_t)k * 256 * 16;
  if (y_dtype == AQMB_BF16)
    gemm_kernel<AQMB_BF16><<<grid, kThreads, lds, st>>>(L.codes, L.codebooks, L.scales, (const uint16_t*)X, Y,
                                                         n_tokens, L.d.d_out, L.d.d_in, L.G, k, L.plane_bytes);
  else
    gemm_kernel<AQMB_F32><<<grid, kThreads, lds, st>>>(L.codes, L.codebooks, L.scales, (const uint16_t*)X, Y,
                                                        n_tokens, L.d.d_out, L.d.d_in, L.G, k, L.plane_bytes);
  return hipGetLastError();
}

}  // namespace aqmb
