// Measured ceilings of the MI355X for the roofline report of the benchmark (not part of the
// quantized layer: libaqmb_ceilings.so is loaded by the benchmark only). Each kernel isolates one
// resource the layer's kernels are bound by:
//   - hbm_read:   streaming 16-byte loads over a buffer, a persistent grid of 1024-thread
//                 workgroups (the decode GEMV's grid): attainable HBM read rate for a launch of
//                 that many bytes;
//   - hbm_write:  streaming 16-byte stores (the dequantization's output stream);
//   - lds_gather: random 16-byte LDS reads from 256-codeword codebooks stored nrep times,
//                 interleaved as the direct-gather GEMV stores them (codeword c of replica r at
//                 (c nrep + r) 16 bytes, lane l reads replica l % nrep), with (dot = 1) or without
//                 the four fp16 dot products the batch-1 GEMV spends on each codeword;
//   - lds_gather_paired: the same reads from the matrix-core GEMV's conflict-free paired layout;
//   - l2_gather:  random 16-byte global loads from a table that stays in the L2 caches (the
//                 16-bit-code GEMV's codebooks);
//   - mfma_bf16:  back-to-back v_mfma_f32_32x32x16_bf16 on operands taken from a buffer (random
//                 data draws more power than zeros, so the rate depends on the operands).
// Every kernel folds what it reads into a value that is stored only if it equals an impossible
// constant, so nothing is optimised away and nothing is written in the normal case.
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

constexpr int kThreads = 1024;
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef _Float16 half2_t __attribute__((ext_vector_type(2)));

__global__ __launch_bounds__(kThreads) void hbm_read_kernel(const u32x4_t* __restrict__ buf, size_t n16,
                                                            unsigned* sink) {
  const size_t stride = (size_t)gridDim.x * kThreads;
  size_t i = (size_t)blockIdx.x * kThreads + threadIdx.x;
  u32x4_t acc = {0, 0, 0, 0};
  for (; i + 3 * stride < n16; i += 4 * stride) {          // four loads in flight per lane
    const u32x4_t a = __builtin_nontemporal_load(buf + i);
    const u32x4_t b = __builtin_nontemporal_load(buf + i + stride);
    const u32x4_t c = __builtin_nontemporal_load(buf + i + 2 * stride);
    const u32x4_t d = __builtin_nontemporal_load(buf + i + 3 * stride);
    acc ^= a ^ b ^ c ^ d;
  }
  for (; i < n16; i += stride) acc ^= __builtin_nontemporal_load(buf + i);
  const unsigned v = acc.x ^ acc.y ^ acc.z ^ acc.w;
  if (v == 0x9E3779B9u) sink[0] = v;
}

__global__ __launch_bounds__(kThreads) void hbm_write_kernel(u32x4_t* __restrict__ buf, size_t n16) {
  const size_t stride = (size_t)gridDim.x * kThreads;
  const u32x4_t v = {threadIdx.x, blockIdx.x, 1u, 2u};
  for (size_t i = (size_t)blockIdx.x * kThreads + threadIdx.x; i < n16; i += stride)
    __builtin_nontemporal_store(v, buf + i);
}

// codes: 16 code bytes per thread of the first workgroup-sized block (kThreads x 4 words), reused
// by every workgroup; each round XORs them with a different byte pattern (still uniform).
template <int NREP, bool DOT>
__global__ __launch_bounds__(kThreads) void lds_gather_kernel(const uint32_t* __restrict__ codes, int rounds,
                                                              unsigned* sink) {
  constexpr int kBooks = 4, kShift = NREP == 8 ? 7 : NREP == 16 ? 8 : NREP == 4 ? 6 : 4;
  extern __shared__ u32x4_t cb[];                          // [kBooks][256][NREP]
  const int tid = threadIdx.x, lane = tid & 63;
  for (int q = tid; q < kBooks * 256 * NREP; q += kThreads) {
    const u32x4_t v = {(uint32_t)q * 0x3C003C00u, (uint32_t)q, 0x3C00u, 0x3C003C00u};
    cb[q] = v;
  }
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) w[i] = codes[tid * 4 + i];
  const uint32_t rep = (uint32_t)(lane % NREP) * 16;
  const u32x4_t xg = {0x3C003C00u, 0x3C003C00u, 0x3C003C00u, 0x3C003C00u};
  __syncthreads();
  float facc[4] = {0.f, 0.f, 0.f, 0.f};
  u32x4_t acc = {0, 0, 0, 0};
  for (int r = 0; r < rounds; ++r) {
    const uint32_t pat = 0x01010101u * (uint32_t)(r * 37 + 11);
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const uint32_t c = ((w[j >> 2] ^ pat) >> (8 * (j & 3))) & 0xFFu;
      const uint32_t addr = ((uint32_t)(j & 3) * 256 * NREP * 16) + (c << kShift) + rep;
      const u32x4_t v = *(const u32x4_t*)((const char*)cb + addr);
      if constexpr (DOT) {
        float s = facc[j & 3];
        s = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, xg.x), __builtin_bit_cast(half2_t, v.x), s, false);
        s = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, xg.y), __builtin_bit_cast(half2_t, v.y), s, false);
        s = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, xg.z), __builtin_bit_cast(half2_t, v.z), s, false);
        s = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, xg.w), __builtin_bit_cast(half2_t, v.w), s, false);
        facc[j & 3] = s;
      } else {
        acc ^= v;
      }
    }
  }
  const unsigned v = acc.x ^ acc.y ^ acc.z ^ acc.w ^ __builtin_bit_cast(unsigned, facc[0] + facc[1] + facc[2] + facc[3]);
  if (v == 0x9E3779B9u) sink[0] = v;
}

// The matrix-core GEMV's paired layout: two 64 KiB regions of 256 rows of 256 bytes, row c holding
// 8 copies of codeword c of two codebooks (bytes 0..127 and 128..255); in gather j, lanes with
// (lane % 16) < 8 read the first codebook's copy lane % 8 when j is even, the second when j is
// odd, and the other lanes the reverse, so every 16 lanes hit the 64 banks once.
__global__ __launch_bounds__(kThreads) void lds_gather_paired_kernel(const uint32_t* __restrict__ codes, int rounds,
                                                                    unsigned* sink) {
  extern __shared__ u32x4_t cb[];                          // [2][256][16]
  const int tid = threadIdx.x, lane = tid & 63;
  for (int q = tid; q < 2 * 256 * 16; q += kThreads) {
    const u32x4_t v = {(uint32_t)q * 0x3C003C00u, (uint32_t)q, 0x3C00u, 0x3C003C00u};
    cb[q] = v;
  }
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) w[i] = codes[tid * 4 + i];
  const uint32_t rep = (uint32_t)(lane & 7) * 16, upper = (uint32_t)((lane >> 3) & 1);
  __syncthreads();
  u32x4_t acc = {0, 0, 0, 0};
  for (int r = 0; r < rounds; ++r) {
    const uint32_t pat = 0x01010101u * (uint32_t)(r * 37 + 11);
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const uint32_t c = ((w[j >> 2] ^ pat) >> (8 * (j & 3))) & 0xFFu;
      const uint32_t half = (uint32_t)(j & 1) ^ upper;
      const uint32_t addr = (uint32_t)((j >> 1) & 1) * 65536 + (c << 8) + (half << 7) + rep;
      acc ^= *(const u32x4_t*)((const char*)cb + addr);
    }
  }
  const unsigned v = acc.x ^ acc.y ^ acc.z ^ acc.w;
  if (v == 0x9E3779B9u) sink[0] = v;
}

// table: 2^log2n entries of 16 bytes. Each lane walks its own linear congruential sequence and
// keeps 8 loads in flight.
__global__ __launch_bounds__(kThreads) void l2_gather_kernel(const u32x4_t* __restrict__ table, int log2n, int rounds,
                                                             unsigned* sink) {
  uint32_t s = (blockIdx.x * kThreads + threadIdx.x) * 2654435761u + 12345u;
  const int sh = 32 - log2n;
  u32x4_t acc = {0, 0, 0, 0};
  for (int r = 0; r < rounds; ++r) {
    u32x4_t v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      s = s * 1664525u + 1013904223u;
      v[j] = table[s >> sh];
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) acc ^= v[j];
  }
  const unsigned x = acc.x ^ acc.y ^ acc.z ^ acc.w;
  if (x == 0x9E3779B9u) sink[0] = x;
}

// Eight independent 32x32 accumulators per wave, operands loaded once per wave from `ops`
// (random bf16 data: 4 A and 4 B fragments of 8 values per lane), rotated between the MFMAs.
__global__ __launch_bounds__(256) void mfma_bf16_kernel(const bf16x8_t* __restrict__ ops, int rounds, float* sink) {
  const int lane = threadIdx.x & 63;
  bf16x8_t a[4], b[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    a[i] = ops[i * 64 + lane];
    b[i] = ops[(4 + i) * 64 + lane];
  }
  f32x16_t acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = f32x16_t{};
  for (int r = 0; r < rounds; r += 4) {                   // operand indices known at compile time
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int i = 0; i < 8; ++i)
        acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[(i + q) & 3], b[(i + 2 * q) & 3], acc[i], 0, 0, 0);
  }
  float t = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i) t += acc[i][0] + acc[i][15];
  if (t == 1.2345e30f) sink[0] = t;
}

}  // namespace

// C entry points (device pointers; launches on `stream`; return hipError_t as int).
extern "C" {

int aqmbc_hbm_read(const void* buf, size_t bytes, int n_wg, unsigned* sink, void* stream) {
  hbm_read_kernel<<<n_wg, kThreads, 0, (hipStream_t)stream>>>((const u32x4_t*)buf, bytes / 16, sink);
  return (int)hipGetLastError();
}

int aqmbc_hbm_write(void* buf, size_t bytes, int n_wg, void* stream) {
  hbm_write_kernel<<<n_wg, kThreads, 0, (hipStream_t)stream>>>((u32x4_t*)buf, bytes / 16);
  return (int)hipGetLastError();
}

// codes: at least 4096 words (16 code bytes for each of the 1024 threads).
int aqmbc_lds_gather(const uint32_t* codes, int n_wg, int rounds, int nrep, int dot, unsigned* sink, void* stream) {
  const hipStream_t st = (hipStream_t)stream;
  const size_t lds = (size_t)4 * 256 * nrep * 16;
  if (nrep == 8) {
    if (dot) lds_gather_kernel<8, true><<<n_wg, kThreads, lds, st>>>(codes, rounds, sink);
    else lds_gather_kernel<8, false><<<n_wg, kThreads, lds, st>>>(codes, rounds, sink);
  } else if (nrep == 4) {
    if (dot) lds_gather_kernel<4, true><<<n_wg, kThreads, lds, st>>>(codes, rounds, sink);
    else lds_gather_kernel<4, false><<<n_wg, kThreads, lds, st>>>(codes, rounds, sink);
  } else if (nrep == 1) {
    if (dot) lds_gather_kernel<1, true><<<n_wg, kThreads, lds, st>>>(codes, rounds, sink);
    else lds_gather_kernel<1, false><<<n_wg, kThreads, lds, st>>>(codes, rounds, sink);
  } else {
    return (int)hipErrorInvalidValue;
  }
  return (int)hipGetLastError();
}

// codes: at least 4096 words; 128 KiB of LDS per workgroup.
int aqmbc_lds_gather_paired(const uint32_t* codes, int n_wg, int rounds, unsigned* sink, void* stream) {
  lds_gather_paired_kernel<<<n_wg, kThreads, 2 * 65536, (hipStream_t)stream>>>(codes, rounds, sink);
  return (int)hipGetLastError();
}

int aqmbc_l2_gather(const void* table, int log2n, int n_wg, int rounds, unsigned* sink, void* stream) {
  if (log2n < 1 || log2n > 28) return (int)hipErrorInvalidValue;
  l2_gather_kernel<<<n_wg, kThreads, 0, (hipStream_t)stream>>>((const u32x4_t*)table, log2n, rounds, sink);
  return (int)hipGetLastError();
}

// ops: 512 entries of 8 bf16 values (8 KiB); rounds is rounded up to a multiple of 4.
int aqmbc_mfma_bf16(const void* ops, int n_wg, int rounds, float* sink, void* stream) {
  mfma_bf16_kernel<<<n_wg, 256, 0, (hipStream_t)stream>>>((const bf16x8_t*)ops, rounds, sink);
  return (int)hipGetLastError();
}

}  // extern "C"
