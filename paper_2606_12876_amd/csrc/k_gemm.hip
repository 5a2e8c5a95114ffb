// Prefill GEMM: Y[n][i] = s_i * sum_t X[n][t] * Wb[i][t], where Wb is the unscaled
// reconstruction from the first k codebooks (binary32 left fold over planes), rounded to bf16,
// and the products run on the bf16 matrix cores (v_mfma_f32_32x32x16_bf16, fp32 accumulate).
//
// A workgroup computes a BM x BN tile of Y (BM = 256 tokens, BN = 128 output rows) with eight
// waves in two roles that share each SIMD:
//   - four consumer waves, each owning a 128 x 64 block of the tile (4 x 2 MFMA blocks of
//     32 x 32), load their X fragments straight from global memory into registers one K step
//     ahead and run the MFMAs;
//   - four producer waves dequantize the next BK = 32 slab of the weight tile into a
//     double-buffered LDS tile: per group, gather the k codewords from the codebooks held in
//     LDS, fold them in binary32, round to bf16.
// One barrier per K step hands a finished weight slab to the consumers and a consumed one back
// to the producers. Within a step the MFMA K dimension is mapped so that each lane's X
// fragments are one contiguous 32-byte piece of a row (K offsets 16h + 8i for half h and
// sub-step i); the weight fragments follow the same mapping, which leaves the product unchanged.
// (BK = 32 keeps the consumers' accumulators plus two steps of X fragments within the 256
// registers a wave has at two waves per SIMD.)
// Row scales are applied to the fp32 accumulators in the epilogue.
#include "device.h"
#include "launch.h"

namespace aqmb {

namespace gemm {
constexpr int BM = 256, BN = 128, BK = 32;
constexpr int kThreads = 512;          // waves 0-3 consume, waves 4-7 produce
constexpr int LDB = BK + 8;            // weight tile pitch in bf16: 80 bytes, conflict-free fragment reads
constexpr int kTileElems = BN * LDB;   // one weight slab buffer
}  // namespace gemm

// Binary32 left fold of one group's k codewords (fp16) and rounding to bf16 pairs.
template <int K>
__device__ __forceinline__ uint4 dequant_group_bf16(const uint4* __restrict__ cbs, const uint32_t (&word)[K], int sh) {
  float w[8];
#pragma unroll
  for (int m = 0; m < K; ++m) {
    const uint4 c = cbs[m * 256 + ((word[m] >> sh) & 0xFFu)];
    const float f[8] = {f16lo(c.x), f16hi(c.x), f16lo(c.y), f16hi(c.y), f16lo(c.z), f16hi(c.z), f16lo(c.w), f16hi(c.w)};
#pragma unroll
    for (int t = 0; t < 8; ++t) w[t] = m == 0 ? f[t] : w[t] + f[t];
  }
  return make_uint4(pack_bf16x2(w[0], w[1]), pack_bf16x2(w[2], w[3]), pack_bf16x2(w[4], w[5]), pack_bf16x2(w[6], w[7]));
}

template <int K, int YDT>
__global__ __launch_bounds__(gemm::kThreads) void gemm_kernel(const unsigned char* __restrict__ codes,
                                                              const uint16_t* __restrict__ codebooks,
                                                              const uint16_t* __restrict__ scales,
                                                              const uint16_t* __restrict__ X, void* __restrict__ Y,
                                                              int n_tokens, int d_out, int d_in, int G,
                                                              size_t plane_bytes, int n_tb) {
  using namespace gemm;
  extern __shared__ uint4 smem[];
  uint16_t* Bs = (uint16_t*)smem;                 // [2][BN][LDB] bf16
  uint4* cbs = (uint4*)(Bs + 2 * kTileElems);     // [K][256] codewords (fp16 x 8)

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // Token blocks fastest: consecutive workgroup ids (which the dispatcher spreads over the
  // XCDs) share a column block, and the workgroups of one token block land on one XCD when
  // there are 8 token blocks, so that XCD's L2 keeps those X rows.
  const int tb = blockIdx.x % n_tb, cb = blockIdx.x / n_tb;
  const int n0 = tb * BM, i0 = cb * BN;
  const int nsteps = (d_in + BK - 1) / BK;

  for (int q = tid; q < K * 256; q += kThreads) cbs[q] = ((const uint4*)codebooks)[q];

  if (wave >= 4) {
    // ------------------------------------------------------------------ producers
    const int p = tid - 256;                       // 0..255
    const int col = p >> 1, g2 = (p & 1) * 2;     // two groups of one weight row per step
    const bool col_ok = i0 + col < d_out;
    uint32_t cur[K], nxt[K];
    auto load_codes = [&](int step, uint32_t (&w)[K]) {
      const int j0 = step * (BK / 8) + g2;         // first of the two groups (same slice, even)
#pragma unroll
      for (int m = 0; m < K; ++m) {
        w[m] = 0;
        if (col_ok && j0 < G)
          w[m] = *(const uint32_t*)(codes + m * plane_bytes + ((size_t)(j0 >> 4) * d_out + i0 + col) * 16 + (j0 & 12));
      }
    };
    auto produce = [&](int step, const uint32_t (&w)[K]) {
      uint16_t* dst = Bs + (step & 1) * kTileElems + col * LDB + g2 * 8;
      const int j0 = step * (BK / 8) + g2;
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        uint4 v = dequant_group_bf16<K>(cbs, w, 8 * ((j0 & 3) + q));
        if (!col_ok || j0 + q >= G) v = make_uint4(0, 0, 0, 0);
        *(uint4*)(dst + q * 8) = v;
      }
    };
    load_codes(0, cur);
    if (nsteps > 1) load_codes(1, nxt);
    __syncthreads();                                // codebooks staged
    produce(0, cur);
    __syncthreads();                                // slab 0 ready
    for (int s = 0; s < nsteps; ++s) {
      if (s + 1 < nsteps) {
#pragma unroll
        for (int m = 0; m < K; ++m) cur[m] = nxt[m];
        if (s + 2 < nsteps) load_codes(s + 2, nxt);
        produce(s + 1, cur);
      }
      __syncthreads();
    }
    return;
  }

  // -------------------------------------------------------------------- consumers
  const int wm = wave >> 1, wn = wave & 1;          // 128 x 64 block of the tile
  const int half = lane >> 5, r32 = lane & 31;
  f32x16_t acc[4][2];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[a][b][e] = 0.f;

  // X fragments of one step: for each of the 4 row blocks, 16 bf16 (32 bytes) of one row.
  uint4 xa[4][2], xn[4][2];
  auto load_x = [&](int step, uint4 (&dst)[4][2]) {
    const int kc = step * BK + half * 16;
#pragma unroll
    for (int a = 0; a < 4; ++a) {
      const int row = n0 + wm * 128 + a * 32 + r32;
      const uint16_t* src = X + (size_t)row * d_in + kc;
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        dst[a][c] = make_uint4(0, 0, 0, 0);
        if (row < n_tokens && kc + c * 8 < d_in) dst[a][c] = *(const uint4*)(src + c * 8);
      }
    }
  };
  load_x(0, xa);
  __syncthreads();                                  // codebooks staged
  __syncthreads();                                  // slab 0 ready
  for (int s = 0; s < nsteps; ++s) {
    if (s + 1 < nsteps) load_x(s + 1, xn);
    const uint16_t* Bt = Bs + (s & 1) * kTileElems;
#pragma unroll
    for (int i = 0; i < 2; ++i) {                   // sub-step: K offsets 16 * half + 8 * i
      bf16x8_t bf[2];
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const int col = wn * 64 + b * 32 + r32;
        bf[b] = *(const bf16x8_t*)(Bt + col * LDB + half * 16 + i * 8);
      }
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        const bf16x8_t af = __builtin_bit_cast(bf16x8_t, xa[a][i]);
#pragma unroll
        for (int b = 0; b < 2; ++b) acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af, bf[b], acc[a][b], 0, 0, 0);
      }
    }
    if (s + 1 < nsteps) {
#pragma unroll
      for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int c = 0; c < 2; ++c) xa[a][c] = xn[a][c];
    }
    __syncthreads();
  }
  // Epilogue. Accumulator element e of lane l in a 32 x 32 block holds
  // row 8 * (e / 4) + 4 * (l / 32) + e % 4, column l % 32.
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    const int col = i0 + wn * 64 + b * 32 + r32;
    if (col >= d_out) continue;
    const float scale = f16_to_f32(scales[col]);
#pragma unroll
    for (int a = 0; a < 4; ++a) {
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int row = n0 + wm * 128 + a * 32 + 8 * (e >> 2) + 4 * half + (e & 3);
        if (row < n_tokens) OutT<YDT>::store(Y, (size_t)row * d_out + col, acc[a][b][e] * scale);
      }
    }
  }
}

template <int K>
static void launch_k(const Layer& L, const void* X, int n_tokens, void* Y, aqmb_dtype y_dtype, hipStream_t st) {
  using namespace gemm;
  const int n_tb = (n_tokens + BM - 1) / BM, n_cb = (L.d.d_out + BN - 1) / BN;
  const size_t lds = (size_t)2 * kTileElems * 2 + (size_t)K * 256 * 16;
  const dim3 grid(n_tb * n_cb);
  if (y_dtype == AQMB_BF16)
    gemm_kernel<K, AQMB_BF16><<<grid, kThreads, lds, st>>>(L.codes, L.codebooks, L.scales, (const uint16_t*)X, Y,
                                                            n_tokens, L.d.d_out, L.d.d_in, L.G, L.plane_bytes, n_tb);
  else
    gemm_kernel<K, AQMB_F32><<<grid, kThreads, lds, st>>>(L.codes, L.codebooks, L.scales, (const uint16_t*)X, Y,
                                                           n_tokens, L.d.d_out, L.d.d_in, L.G, L.plane_bytes, n_tb);
}

hipError_t launch_gemm(const Layer& L, int k, const void* X, int n_tokens, void* Y, aqmb_dtype y_dtype,
                       hipStream_t st) {
  switch (k) {
    case 1: launch_k<1>(L, X, n_tokens, Y, y_dtype, st); break;
    case 2: launch_k<2>(L, X, n_tokens, Y, y_dtype, st); break;
    case 3: launch_k<3>(L, X, n_tokens, Y, y_dtype, st); break;
    case 4: launch_k<4>(L, X, n_tokens, Y, y_dtype, st); break;
    case 5: launch_k<5>(L, X, n_tokens, Y, y_dtype, st); break;
    case 6: launch_k<6>(L, X, n_tokens, Y, y_dtype, st); break;
    case 7: launch_k<7>(L, X, n_tokens, Y, y_dtype, st); break;
    default: launch_k<8>(L, X, n_tokens, Y, y_dtype, st); break;
  }
  return hipGetLastError();
}

}  // namespace aqmb
