// Decode GEMV for 4-bit codes (codebooks of 16 codewords; the 4 x 4-bit configuration of the
// paper's ablation on codebook precision against codebook count): y[b][i] = s_i sum_j sum_{m<k}
// <x[b, group j], C_m[b_{ijm}]>.
//
// A 16-codeword codebook is 256 bytes: its codewords occupy the 64 LDS banks exactly once, so a
// wave's random 16-byte codeword reads never collide (equal codewords are broadcast) and no
// replicas are needed. A workgroup of 1024 threads owns 16 rows; the 64 threads of a row each
// take 8 groups of every 512-group block (one 4-byte code word per plane: 8 codes packed two to
// a byte), gather the codewords and accumulate <x_group, codeword> in fp32. x is staged in LDS by
// direct global->LDS loads, 2048 groups at a time (zeros past d_in from the zero page, so the
// padding groups of the last slice, which hold code 0, contribute nothing). Batches above one
// run in tiles of 4 rows over the same code words. A row's 64 partial sums are added in a fixed
// order (two shuffles, then the 16 waves through LDS), scaled once and rounded once.
#include "device.h"
#include "launch.h"

namespace aqmb {

namespace b4 {
constexpr int kThreads = 1024, kRows = 16, kWaves = 16;
}  // namespace b4

struct Gemv4Args {
  const unsigned char* codes;
  const uint16_t* codebooks;
  const uint16_t* scales;
  const void* x;
  void* y;
  const void* zero_page;
  size_t plane_bytes;
  int d_out, d_in, S, batch, y_dtype;
};

// <x group (8 values), codeword (8 fp16)> in fp32: fp16 products are exact (dot2), bf16 values are
// widened exactly and multiplied in fp32.
template <int XDT>
__device__ __forceinline__ float dot8(uint4 xw, uint4 cw) {
  if constexpr (XDT == AQMB_F16) {
    float s = dot2_f16(xw.x, cw.x, 0.f);
    s = dot2_f16(xw.y, cw.y, s);
    s = dot2_f16(xw.z, cw.z, s);
    return dot2_f16(xw.w, cw.w, s);
  } else {
    float s = bf16lo(xw.x) * f16lo(cw.x);
    s = __builtin_fmaf(bf16hi(xw.x), f16hi(cw.x), s);
    s = __builtin_fmaf(bf16lo(xw.y), f16lo(cw.y), s);
    s = __builtin_fmaf(bf16hi(xw.y), f16hi(cw.y), s);
    s = __builtin_fmaf(bf16lo(xw.z), f16lo(cw.z), s);
    s = __builtin_fmaf(bf16hi(xw.z), f16hi(cw.z), s);
    s = __builtin_fmaf(bf16lo(xw.w), f16lo(cw.w), s);
    return __builtin_fmaf(bf16hi(xw.w), f16hi(cw.w), s);
  }
}

// <x group, codeword> of fp16 values added to s.
__device__ __forceinline__ float dot8_acc_f16(uint4 xw, uint4 cw, float s) {
  s = dot2_f16(xw.x, cw.x, s);
  s = dot2_f16(xw.y, cw.y, s);
  s = dot2_f16(xw.z, cw.z, s);
  return dot2_f16(xw.w, cw.w, s);
}

// UB = 512-group blocks per x stage: 1 when a row has at most 512 groups (no load is issued for
// blocks past the row), else 4.
// bf16 x at batch 1: every staged 16-byte group is converted in place to fp16 by the thread that
// loaded it, with a power-of-two scale per group (largest magnitude put in [2^14, 2^15), where
// bf16's 8 significant bits are exact in fp16; values below 2^-29 of the group maximum are
// rounded to a multiple of 2^-39 of it), so the fp16 dot products apply; a group's sums over the
// planes are multiplied by its scale.
template <int K, int NB, int XDT, int UB>
__global__ __launch_bounds__(b4::kThreads) void gemv_b4_kernel(Gemv4Args a) {
  constexpr int kTiles = NB == 1 ? 1 : 4;    // batch <= 16
  constexpr int kChunk = UB * 512;
  constexpr bool kXS = XDT == AQMB_BF16 && NB == 1;
  extern __shared__ uint4 smem_b4[];
  uint4* cb = smem_b4;                                       // [K][16] codewords
  char* xs = (char*)(smem_b4 + K * 16);                      // [NB][kChunk][16 bytes]
  float* scl = (float*)(xs + (size_t)NB * kChunk * 16);      // kXS: [kChunk] group scales
  __shared__ float red[b4::kWaves][b4::kRows][NB];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int rw = lane & 15, part = tid >> 4;                 // row in the block, part 0..63
  const int row = blockIdx.x * b4::kRows + rw;
  const bool row_ok = row < a.d_out;
  const int rowc = row_ok ? row : a.d_out - 1;
  const int Gp = a.S * 32;                                   // padded groups per row
  const int n_tiles = (a.batch + NB - 1) / NB;
  const uint32_t xs_base = lds_addr(xs);

  if (tid < K * 16) cb[tid] = ((const uint4*)a.codebooks)[tid];
  const float scale = f16_to_f32(a.scales[rowc]);
  float acc[kTiles][NB];
#pragma unroll
  for (int t = 0; t < kTiles; ++t)
#pragma unroll
    for (int b = 0; b < NB; ++b) acc[t][b] = 0.f;

  for (int g0 = 0; g0 < Gp; g0 += kChunk) {
    // code words of this chunk: block u, plane m -> 8 groups g0 + 512 u + 8 part .. + 7. At batch 1
    // they are requested after x (the small, cache-resident loads go first: a CU's requests leave in
    // order) and awaited where each is used; with tiles of 4 batch rows, before the tiles.
    uint32_t code[UB][K];
    auto load_codes = [&]() {
#pragma unroll
      for (int u = 0; u < UB; ++u) {
        int j0 = g0 + u * 512 + part * 8;
        j0 = j0 < Gp ? j0 : Gp - 8;                          // unused blocks reload a valid word
#pragma unroll
        for (int m = 0; m < K; ++m)
          code[u][m] = __builtin_nontemporal_load(
              (const uint32_t*)(a.codes + m * a.plane_bytes + ((size_t)(j0 >> 5) * a.d_out + rowc) * 16 + ((j0 & 31) >> 1)));
      }
    };
    const int n_ch = ((Gp - g0 < kChunk ? Gp - g0 : kChunk) + 63) / 64;   // 1 KiB pieces per x row
    if constexpr (NB > 1) load_codes();
#pragma unroll
    for (int t = 0; t < kTiles; ++t) {
      if (t < n_tiles) {
        __syncthreads();                                     // codebooks in; xs free
        for (int q = wave; q < NB * n_ch; q += b4::kWaves) {
          const int b = q / n_ch, ch = q % n_ch;
          const int xb = t * NB + b;
          const int e = (g0 + ch * 64 + lane) * 8;           // element offset in the row
          const void* src = (xb < a.batch && e < a.d_in) ? (const void*)((const uint16_t*)a.x + (size_t)xb * a.d_in + e)
                                                         : a.zero_page;
          load_lds16(src, xs_base + (uint32_t)(b * kChunk * 16 + ch * 1024));
        }
        if constexpr (NB == 1) {
          asm volatile("" ::: "memory");
          __builtin_amdgcn_s_barrier();                      // every wave's x requests before any code words
          asm volatile("" ::: "memory");
          load_codes();
          wait_vmcnt<UB * K>();                              // this thread's x pieces are in
        } else {
          wait_vmcnt<0>();
        }
        if constexpr (kXS) {                                 // the groups this thread loaded
          for (int q = wave; q < n_ch; q += b4::kWaves) {
            const int gq = q * 64 + lane;
            char* p = xs + (size_t)gq * 16;
            const uint4 v = *(const uint4*)p;
            uint32_t w[4] = {v.x, v.y, v.z, v.w};
            uint32_t e = 0;
#pragma unroll
            for (int h = 0; h < 4; ++h) e = max(e, max((w[h] >> 7) & 0xFFu, (w[h] >> 23) & 0xFFu));
            const int sh = (int)e - 141;                     // (e - 127) - 14
#pragma unroll
            for (int h = 0; h < 4; ++h) {
              const _Float16 lo = (_Float16)ldexpf(bf16lo(w[h]), -sh);
              const _Float16 hi = (_Float16)ldexpf(bf16hi(w[h]), -sh);
              w[h] = (uint32_t)__builtin_bit_cast(uint16_t, lo) | ((uint32_t)__builtin_bit_cast(uint16_t, hi) << 16);
            }
            *(uint4*)p = make_uint4(w[0], w[1], w[2], w[3]);
            scl[gq] = ldexpf(1.0f, sh);
          }
        }
        __syncthreads();
#pragma unroll
        for (int u = 0; u < UB; ++u) {
          const int j0 = u * 512 + part * 8;                 // group within the chunk
          if (g0 + j0 < Gp) {
            auto group = [&](int jj) {
              uint4 xg[NB];
#pragma unroll
              for (int b = 0; b < NB; ++b) xg[b] = *(const uint4*)(xs + (size_t)b * kChunk * 16 + (size_t)(j0 + jj) * 16);
              // batch 1 with fp16 values (fp16 x, or bf16 x converted): the group's products are
              // chained over the planes into one sum (one v_dot2 per code word pair)
              constexpr bool kChain = NB == 1 && (kXS || XDT == AQMB_F16);
              float gs = 0.f;
#pragma unroll
              for (int m = 0; m < K; ++m) {
                const uint4 cwv = cb[m * 16 + ((code[u][m] >> (4 * jj)) & 15u)];
                if constexpr (kChain) {
                  gs = dot8_acc_f16(xg[0], cwv, gs);
                } else {
#pragma unroll
                  for (int b = 0; b < NB; ++b) acc[t][b] += dot8<XDT>(xg[b], cwv);
                }
              }
              if constexpr (kXS) acc[t][0] = __builtin_fmaf(gs, scl[j0 + jj], acc[t][0]);
              else if constexpr (kChain) acc[t][0] += gs;
            };
            if constexpr (NB == 1) {
#pragma unroll
              for (int jj = 0; jj < 8; ++jj) group(jj);
            } else {                                         // fewer reads in flight: no spills
#pragma unroll 2
              for (int jj = 0; jj < 8; ++jj) group(jj);
            }
          }
        }
      }
    }
  }
  // row sums per tile: lanes rw, rw + 16, rw + 32, rw + 48 of a wave, then the 16 waves in order
#pragma unroll
  for (int t = 0; t < kTiles; ++t) {
    if (t < n_tiles) {
      float v[NB];
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        v[b] = acc[t][b];
        v[b] += __shfl_xor(v[b], 16);
        v[b] += __shfl_xor(v[b], 32);
      }
      __syncthreads();                                       // red free
      if (lane < 16) {
#pragma unroll
        for (int b = 0; b < NB; ++b) red[wave][rw][b] = v[b];
      }
      __syncthreads();
      if (wave == 0 && lane < 16 && row_ok) {
#pragma unroll
        for (int b = 0; b < NB; ++b) {
          const int xb = t * NB + b;
          if (xb < a.batch) {
            float sum = 0.f;
#pragma unroll
            for (int w = 0; w < b4::kWaves; ++w) sum += red[w][rw][b];
            const size_t o = (size_t)xb * a.d_out + row;
            const float yv = sum * scale;
            if (a.y_dtype == AQMB_F16) OutT<AQMB_F16>::store(a.y, o, yv);
            else if (a.y_dtype == AQMB_BF16) OutT<AQMB_BF16>::store(a.y, o, yv);
            else OutT<AQMB_F32>::store(a.y, o, yv);
          }
        }
      }
    }
  }
}

template <int K, int XDT, int UB>
static hipError_t launch_b4_ub(const Gemv4Args& a, hipStream_t st) {
  const unsigned grid = (unsigned)((a.d_out + b4::kRows - 1) / b4::kRows);
  const size_t row_bytes = (size_t)UB * 512 * 16;
  const size_t scl_bytes = XDT == AQMB_BF16 ? (size_t)UB * 512 * 4 : 0;   // bf16 x: group scales
  if (a.batch == 1) gemv_b4_kernel<K, 1, XDT, UB><<<grid, b4::kThreads, (size_t)K * 256 + row_bytes + scl_bytes, st>>>(a);
  else gemv_b4_kernel<K, 4, XDT, UB><<<grid, b4::kThreads, (size_t)K * 256 + 4 * row_bytes, st>>>(a);
  return hipGetLastError();
}

template <int K, int XDT>
static hipError_t launch_b4_k(const Gemv4Args& a, hipStream_t st) {
  return a.S * 32 <= 512 ? launch_b4_ub<K, XDT, 1>(a, st) : launch_b4_ub<K, XDT, 4>(a, st);
}

template <int XDT>
static hipError_t launch_b4_x(const Gemv4Args& a, int k, hipStream_t st) {
  switch (k) {
    case 1: return launch_b4_k<1, XDT>(a, st);
    case 2: return launch_b4_k<2, XDT>(a, st);
    case 3: return launch_b4_k<3, XDT>(a, st);
    case 4: return launch_b4_k<4, XDT>(a, st);
    case 5: return launch_b4_k<5, XDT>(a, st);
    case 6: return launch_b4_k<6, XDT>(a, st);
    case 7: return launch_b4_k<7, XDT>(a, st);
    default: return launch_b4_k<8, XDT>(a, st);
  }
}

hipError_t launch_gemv_b4(const Layer& L, int k, const void* x, aqmb_dtype x_dtype, int batch, void* y,
                          aqmb_dtype y_dtype, hipStream_t st) {
  Gemv4Args a{};
  a.codes = L.codes;
  a.codebooks = L.codebooks;
  a.scales = L.scales;
  a.x = x;
  a.y = y;
  a.zero_page = L.zero_page();
  a.plane_bytes = L.plane_bytes;
  a.d_out = L.d.d_out;
  a.d_in = L.d.d_in;
  a.S = L.S;
  a.batch = batch;
  a.y_dtype = (int)y_dtype;
  return x_dtype == AQMB_F16 ? launch_b4_x<AQMB_F16>(a, k, st) : launch_b4_x<AQMB_BF16>(a, k, st);
}

}  // namespace aqmb
