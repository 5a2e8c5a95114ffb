// Code re-tiling (layer creation) and the bit-exact dequantization kernel.
#include <algorithm>

#include "device.h"
#include "launch.h"

namespace aqmb {

// [M][d_out][G] plane-major codes -> [M][S][d_out][16 bytes]. CB = code bits: 16-bit codes are
// 2 bytes each, 8-bit and 4-bit codes 1 byte each in the input; a slice holds J = 128 / CB
// consecutive groups of one row, 4-bit codes packed two to a byte (group 2b in the low nibble of
// byte b, group 2b + 1 in the high nibble). A 4-bit code above 15 sets *bad (the layer is refused).
template <int CB>
__global__ __launch_bounds__(256) void retile_kernel(const unsigned char* __restrict__ in, unsigned char* __restrict__ out,
                                                     int M, int d_out, int G, int S, int* bad) {
  constexpr int J = 128 / CB, CS = CB == 16 ? 2 : 1;
  const size_t total = (size_t)M * S * d_out;
  for (size_t q = (size_t)blockIdx.x * blockDim.x + threadIdx.x; q < total; q += (size_t)gridDim.x * blockDim.x) {
    const int i = (int)(q % d_out);
    const size_t ms = q / d_out;
    const int s = (int)(ms % S), m = (int)(ms / S);
    unsigned char chunk[16];
    if constexpr (CB == 4) {
      unsigned high = 0;
#pragma unroll
      for (int b = 0; b < 16; ++b) {
        const int j0 = s * J + 2 * b, j1 = j0 + 1;
        const unsigned c0 = j0 < G ? in[((size_t)m * d_out + i) * G + j0] : 0u;
        const unsigned c1 = j1 < G ? in[((size_t)m * d_out + i) * G + j1] : 0u;
        high |= (c0 | c1) >> 4;
        chunk[b] = (unsigned char)((c0 & 15u) | ((c1 & 15u) << 4));
      }
      if (high) *bad = 1;
    } else {
#pragma unroll
      for (int jj = 0; jj < J; ++jj) {
        const int j = s * J + jj;
#pragma unroll
        for (int b = 0; b < CS; ++b)
          chunk[jj * CS + b] = j < G ? in[(((size_t)m * d_out + i) * G + j) * CS + b] : (unsigned char)0;
      }
    }
    uint4 v;
    __builtin_memcpy(&v, chunk, 16);
    *(uint4*)(out + q * 16) = v;
  }
}

hipError_t launch_retile(const Layer& L, const void* codes, int n_planes, unsigned char* out, int* bad,
                         hipStream_t st) {
  const size_t total = (size_t)n_planes * L.S * L.d.d_out;
  const unsigned grid = (unsigned)((total + 255) / 256 < 65536 ? (total + 255) / 256 : 65536);
  const auto* in = (const unsigned char*)codes;
  if (L.d.code_bits == 8)
    retile_kernel<8><<<grid, 256, 0, st>>>(in, out, n_planes, L.d.d_out, L.G, L.S, bad);
  else if (L.d.code_bits == 4)
    retile_kernel<4><<<grid, 256, 0, st>>>(in, out, n_planes, L.d.d_out, L.G, L.S, bad);
  else
    retile_kernel<16><<<grid, 256, 0, st>>>(in, out, n_planes, L.d.d_out, L.G, L.S, bad);
  return hipGetLastError();
}

// The stated evaluation order for W_k: binary32 left fold over planes, one binary32
// multiply by the row scale, one rounding to the output format. Contraction into a
// fused multiply-add is off so every step rounds on its own.
#pragma clang fp contract(off)

// The output is written once and not read back by this kernel: streaming (nontemporal) stores.
__device__ __forceinline__ void store_stream16(void* p, uint32_t a, uint32_t b, uint32_t c, uint32_t d) {
  const u32x4_t v = {a, b, c, d};
  __builtin_nontemporal_store(v, (u32x4_t*)p);
}

template <int OUT>
__device__ __forceinline__ void store_group(void* W, size_t elem, const float (&w)[8]) {
  if constexpr (OUT == AQMB_F32) {
    float* p = (float*)W + elem;
    store_stream16(p, __float_as_uint(w[0]), __float_as_uint(w[1]), __float_as_uint(w[2]), __float_as_uint(w[3]));
    store_stream16(p + 4, __float_as_uint(w[4]), __float_as_uint(w[5]), __float_as_uint(w[6]), __float_as_uint(w[7]));
  } else if constexpr (OUT == AQMB_F16) {
    store_stream16((uint16_t*)W + elem, pack_f16x2(w[0], w[1]), pack_f16x2(w[2], w[3]),
                   pack_f16x2(w[4], w[5]), pack_f16x2(w[6], w[7]));
  } else {
    store_stream16((uint16_t*)W + elem, pack_bf16x2(w[0], w[1]), pack_bf16x2(w[2], w[3]),
                   pack_bf16x2(w[4], w[5]), pack_bf16x2(w[6], w[7]));
  }
}

// acc = the first codeword (exact in binary32), or acc + the codeword, one rounding per element
__device__ __forceinline__ void fold_codeword(float (&acc)[8], uint4 cw, bool first) {
  if (first) {
    acc[0] = f16lo(cw.x); acc[1] = f16hi(cw.x); acc[2] = f16lo(cw.y); acc[3] = f16hi(cw.y);
    acc[4] = f16lo(cw.z); acc[5] = f16hi(cw.z); acc[6] = f16lo(cw.w); acc[7] = f16hi(cw.w);
  } else {
    acc[0] = add_f16_lo(cw.x, acc[0]); acc[1] = add_f16_hi(cw.x, acc[1]);
    acc[2] = add_f16_lo(cw.y, acc[2]); acc[3] = add_f16_hi(cw.y, acc[3]);
    acc[4] = add_f16_lo(cw.z, acc[4]); acc[5] = add_f16_hi(cw.z, acc[5]);
    acc[6] = add_f16_lo(cw.w, acc[6]); acc[7] = add_f16_hi(cw.w, acc[7]);
  }
}

// c0 + c1 for the fp16 values in the low (or high) halves of a and b, rounded once to binary32:
// the first two steps of the fold in one instruction (an fma with 1.0 and both sources fp16).
__device__ __forceinline__ float add2_f16_lo(uint32_t a, uint32_t b) {
  float d;
  asm("v_fma_mix_f32 %0, %1, 1.0, %2 op_sel_hi:[1,0,1]" : "=v"(d) : "v"(b), "v"(a));
  return d;
}
__device__ __forceinline__ float add2_f16_hi(uint32_t a, uint32_t b) {
  float d;
  asm("v_fma_mix_f32 %0, %1, 1.0, %2 op_sel:[1,0,1] op_sel_hi:[1,0,1]" : "=v"(d) : "v"(b), "v"(a));
  return d;
}

// acc = (binary32) c0 + c1, elementwise
__device__ __forceinline__ void fold_first_two(float (&acc)[8], uint4 c0, uint4 c1) {
  acc[0] = add2_f16_lo(c0.x, c1.x); acc[1] = add2_f16_hi(c0.x, c1.x);
  acc[2] = add2_f16_lo(c0.y, c1.y); acc[3] = add2_f16_hi(c0.y, c1.y);
  acc[4] = add2_f16_lo(c0.z, c1.z); acc[5] = add2_f16_hi(c0.z, c1.z);
  acc[6] = add2_f16_lo(c0.w, c1.w); acc[7] = add2_f16_hi(c0.w, c1.w);
}

// 16 times byte j of w (the LDS byte offset of that code's codeword), one instruction; j must be
// a constant after unrolling.
__device__ __forceinline__ uint32_t code_x16(uint32_t w, int j) {
  uint32_t d;
  switch (j) {
    case 0: asm("v_lshlrev_b32_sdwa %0, 4, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_0" : "=v"(d) : "v"(w)); break;
    case 1: asm("v_lshlrev_b32_sdwa %0, 4, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_1" : "=v"(d) : "v"(w)); break;
    case 2: asm("v_lshlrev_b32_sdwa %0, 4, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_2" : "=v"(d) : "v"(w)); break;
    default: asm("v_lshlrev_b32_sdwa %0, 4, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_3" : "=v"(d) : "v"(w)); break;
  }
  return d;
}

// Used for 16-bit and 4-bit codes (and as the general fallback). CB = code bits. One thread per
// group: the J = 128 / CB lanes of a (row, slice) pair take its J groups, so a wave writes whole
// row segments (J groups x 8 values) and the lanes of one row share one 16-byte code chunk per
// plane (a single cache line). 16- and 256-entry codebooks are staged in LDS; 65536-entry
// codebooks are read through the caches.
template <int OUT, int CB>
__global__ __launch_bounds__(256) void dequant_kernel(const unsigned char* __restrict__ codes,
                                                      const uint16_t* __restrict__ codebooks,
                                                      const uint16_t* __restrict__ scales, void* __restrict__ W,
                                                      int d_out, int d_in, int G, int S, int k, size_t plane_bytes) {
  constexpr int J = 128 / CB, PER_WORD = 32 / CB;
  extern __shared__ uint4 cb_lds[];  // [k][2^CB] codewords (CB <= 8)
  if constexpr (CB <= 8) {
    for (int q = threadIdx.x; q < (k << CB); q += blockDim.x) cb_lds[q] = ((const uint4*)codebooks)[q];
    __syncthreads();
  }
  // Each thread takes U groups per pass and issues all their code loads before using any.
  constexpr int U = 4;
  const size_t n = (size_t)S * d_out * J;
  const size_t stride = (size_t)gridDim.x * blockDim.x * U;
  for (size_t base = (size_t)blockIdx.x * blockDim.x * U + threadIdx.x; base < n; base += stride) {
    uint32_t words[U][8];
    int row[U], grp[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const size_t t = base + (size_t)u * blockDim.x;
      const int jj = (int)(t % J);
      const size_t pair = t / J;  // (slice, row) pair, rows fastest
      row[u] = (int)(pair % d_out);
      const int s = (int)(pair / d_out);
      grp[u] = (t < n) ? s * J + jj : G;
      const size_t chunk = pair * 16 + (size_t)(jj / PER_WORD) * 4;  // the code word holding this group
#pragma unroll
      for (int m = 0; m < 8; ++m) {
        words[u][m] = 0;
        if (m < k && grp[u] < G) words[u][m] = *(const uint32_t*)(codes + m * plane_bytes + chunk);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (grp[u] >= G) continue;
      const int jj = grp[u] % J;
      float acc[8];
#pragma unroll
      for (int m = 0; m < 8; ++m) {
        if (m < k) {
          uint4 cw;
          const uint32_t code = (words[u][m] >> (CB * (jj % PER_WORD))) & ((1u << CB) - 1u);
          if constexpr (CB <= 8) {
            cw = cb_lds[(m << CB) + code];
          } else {
            cw = ((const uint4*)codebooks)[((size_t)m << 16) + code];
          }
          fold_codeword(acc, cw, m == 0);
        }
      }
      const float scale = f16_to_f32(scales[row[u]]);
      float w[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        w[e] = acc[e] * scale;
        // Keep the binary32 product: without this the backend may fuse the multiply and the
        // fp16 conversion into one mixed-precision instruction that rounds only once.
        asm volatile("" : "+v"(w[e]));
      }
      store_group<OUT>(W, (size_t)row[u] * d_in + (size_t)grp[u] * 8, w);
    }
  }
}

// 8-bit codes, K = k planes, thread per group: the 16 lanes of a (slice, row) pair take its 16
// groups, so every store instruction of a wave writes four whole 256-byte row segments. Each
// thread takes U groups per pass (slots t, t + 256, ...; U = 1 measured best) and passes are
// grid-strided; the code
// words and row scales of the next pass are requested before the current pass is folded, with
// two register sets used in turn so that no copy waits for them. The codebooks go straight to
// LDS and the first pass's code words are requested right behind them; loads complete in order,
// so the wait for the codebooks does not wait for the code words. Code words are read once,
// with a streaming hint. The pointers are deliberately not restrict-qualified: that would let
// the compiler treat the loads as invariant and move them next to their uses.
template <int OUT, int K>
__global__ __launch_bounds__(256) void dequant8_kernel(const unsigned char* codes, const uint16_t* codebooks,
                                                       const uint16_t* scales, void* W,
                                                       int d_out, int d_in, int G, int S, size_t plane_bytes) {
  constexpr int U = 1;
  extern __shared__ uint4 cb8[];  // [K][256] codewords
  // group slots fit in 32 bits (the launcher checks 16 S d_out < 2^30)
  const uint32_t nslot = (uint32_t)S * (uint32_t)d_out * 16u;
  const uint32_t stride = gridDim.x * blockDim.x * U;
  uint32_t t = blockIdx.x * blockDim.x * U + threadIdx.x;
  // code words (the 4-byte word holding each group's code, per plane) and row scales of the U
  // slots of pass tt; slots past the end re-read the last slot and are not used
  auto load = [&](uint32_t tt, uint32_t (&w)[U][K], uint32_t (&sc)[U]) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      uint32_t slot = tt + u * blockDim.x;
      slot = slot < nslot ? slot : nslot - 1;
      const uint32_t pair = slot >> 4;
      sc[u] = scales[pair % (uint32_t)d_out];
#pragma unroll
      for (int m = 0; m < K; ++m)
        w[u][m] = __builtin_nontemporal_load(
            (const uint32_t*)(codes + m * plane_bytes + (size_t)pair * 16 + (slot & 12)));
    }
  };
  const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
#pragma unroll
  for (int i = 0; i < K; ++i)
    load_lds16((const uint4*)codebooks + i * 256 + threadIdx.x, lds_addr(cb8 + i * 256 + wave * 64));
  uint32_t wa[U][K], wb[U][K];
  uint32_t sa[U], sb[U];                             // row scales (fp16 bits), one per register
  load(t, wa, sa);
  wait_vmcnt<U * (K + 1)>();
  __syncthreads();
  auto pass = [&](uint32_t tt, const uint32_t (&w)[U][K], const uint32_t (&sc)[U]) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t slot = tt + u * blockDim.x;
      const uint32_t pair = slot >> 4;
      const uint32_t slice = pair / (uint32_t)d_out;
      const int row = (int)(pair - slice * (uint32_t)d_out);
      const int grp = (int)slice * 16 + (int)(slot & 15);
      if (slot >= nslot || grp >= G) continue;
      const int sh = 8 * (int)(slot & 3);
      float acc[8];
#pragma unroll
      for (int m = 0; m < K; ++m) fold_codeword(acc, cb8[m * 256 + ((w[u][m] >> sh) & 0xFFu)], m == 0);
      const float scale = f16_to_f32((uint16_t)sc[u]);
      float v[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        v[e] = acc[e] * scale;
        asm volatile("" : "+v"(v[e]));  // keep the binary32 product (see dequant_kernel)
      }
      store_group<OUT>(W, (size_t)row * d_in + (size_t)grp * 8, v);
    }
  };
  for (; t < nslot; t += 2 * stride) {
    load(t + stride, wb, sb);
    __builtin_amdgcn_sched_barrier(0);
    pass(t, wa, sa);
    if (t + stride >= nslot) break;
    load(t + 2 * stride, wa, sa);
    __builtin_amdgcn_sched_barrier(0);
    pass(t + stride, wb, sb);
  }
}

// 8-bit codes, 16-bit output (f16 or bf16), K = k planes: tiles of RT rows x GT groups (RT GT =
// 2048 or 4096 groups, 32 or 64 KiB of output), 512 threads. Thread t takes row t % RT of the tile
// and P = RT GT / 512 consecutive groups of it (part (t / RT) of the tile's GT / 16 slices): one
// P-byte code load per plane brings them, which it folds (same arithmetic and order as
// dequant8_kernel) into the tile in LDS, row-major, its 16-byte chunks XOR-swizzled by row so that
// both the column-wise writes and the row-wise reads hit every bank group. Then the waves write
// the tile row by row, 1 KiB contiguous per store instruction (measured: 64 rows x 256-byte
// pieces per instruction, the thread-per-group layout, is 20 % slower; rows written by one lane
// each, 4x slower). Tiles are numbered column tiles fastest, so the tiles in flight together
// cover whole rows of the output (a contiguous range of addresses). A workgroup walks its tiles
// with the grid's stride; the code words of its next tile are requested before the current one is
// folded.
namespace dq {
constexpr int kThreads = 512, kWaves = kThreads / 64;
}

// LDS writes of this wave complete, then a workgroup barrier (global loads stay in flight).
__device__ __forceinline__ void dq_lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);                  // lgkmcnt(0); vmcnt and expcnt at their maxima
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

template <int OUT, int K, int RT, int GT>
__global__ __launch_bounds__(dq::kThreads) void dequant8_tile_kernel(const unsigned char* codes, const uint16_t* codebooks,
                                                                    const uint16_t* scales, void* W, int d_out, int d_in,
                                                                    int G, int S, size_t plane_bytes) {
  static_assert(OUT == AQMB_F16 || OUT == AQMB_BF16, "16-bit outputs");
  static_assert(RT * GT == 4096 || RT * GT == 2048, "tile size");
  static_assert(GT >= 64 && (GT & (GT - 1)) == 0 && RT <= 64, "swizzle range");
  using namespace dq;
  constexpr int P = RT * GT / kThreads, kParts = 16 / P, ST = GT / 16, CP = GT / 64;
  // static LDS, codebooks first: their addresses fit the reads' offset field
  __shared__ struct {
    uint4 cb[K * 256];                                 // [K][256] codewords
    uint4 tile[RT * GT];                               // [RT rows][GT chunks of 16 bytes], swizzled
  } sm;
  uint4* cb8 = sm.cb;
  uint4* tile = sm.tile;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  for (int q = tid; q < K * 256; q += kThreads) cb8[q] = ((const uint4*)codebooks)[q];
  const int n_ct = (S + ST - 1) / ST, n_tiles = n_ct * ((d_out + RT - 1) / RT);
  const int rl = tid % RT, q = tid / RT, sl_t = q / kParts, part = q % kParts;   // row, slice, part of the slice
  uint2 c[K];
  uint32_t sc = 0;
  // code words (P bytes per plane) and row scale of tile t for this thread; tiles past the end
  // reload the last one, rows and slices past the layer reload its last row and slice (never stored)
  auto load = [&](int t) {
    const int tc = t < n_tiles ? t : n_tiles - 1;
    int row = (tc / n_ct) * RT + rl, sl = (tc % n_ct) * ST + sl_t;
    row = row < d_out ? row : d_out - 1;
    sl = sl < S ? sl : S - 1;
    sc = scales[row];
    const unsigned char* p = codes + ((size_t)sl * d_out + row) * 16 + part * P;
#pragma unroll
    for (int m = 0; m < K; ++m) {
      if constexpr (P == 8) c[m] = load_stream8(p + m * plane_bytes);
      else c[m] = make_uint2(__builtin_nontemporal_load((const uint32_t*)(p + m * plane_bytes)), 0u);
    }
  };
  int t = blockIdx.x;
  load(t);
  __syncthreads();
  for (; t < n_tiles; t += gridDim.x) {
    const int r0 = (t / n_ct) * RT, g0 = (t % n_ct) * GT;
    const float scale = f16_to_f32((uint16_t)sc);
    uint2 w[K];
#pragma unroll
    for (int m = 0; m < K; ++m) w[m] = c[m];
    load(t + gridDim.x);
#pragma unroll
    for (int jj = 0; jj < P; ++jj) {
      uint4 cw[K];
#pragma unroll
      for (int m = 0; m < K; ++m)
        cw[m] = *(const uint4*)((const char*)(cb8 + m * 256) + code_x16(jj < 4 ? w[m].x : w[m].y, jj & 3));
      float acc[8];
      if constexpr (K == 1) fold_codeword(acc, cw[0], true);
      else fold_first_two(acc, cw[0], cw[1]);
#pragma unroll
      for (int m = 2; m < K; ++m) fold_codeword(acc, cw[m], false);
      float v[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        v[e] = acc[e] * scale;
        asm volatile("" : "+v"(v[e]));  // keep the binary32 product (see dequant_kernel)
      }
      const uint4 o = OUT == AQMB_F16
                          ? make_uint4(pack_f16x2(v[0], v[1]), pack_f16x2(v[2], v[3]), pack_f16x2(v[4], v[5]), pack_f16x2(v[6], v[7]))
                          : make_uint4(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]), pack_bf16x2(v[4], v[5]),
                                       pack_bf16x2(v[6], v[7]));
      const int chunk = sl_t * 16 + part * P + jj;
      tile[rl * GT + (chunk ^ rl)] = o;
    }
    dq_lds_barrier();
    // P stores per wave: store j = wave P + i writes chunk part j % CP of tile row j / CP
#pragma unroll
    for (int i = 0; i < P; ++i) {
      const int j = wave * P + i, r = j / CP, ch = (j % CP) * 64 + lane, row = r0 + r, grp = g0 + ch;
      const uint4 o = tile[r * GT + (ch ^ r)];
      if (row < d_out && grp < G) store_stream16((uint16_t*)W + (size_t)row * d_in + (size_t)grp * 8, o.x, o.y, o.z, o.w);
    }
    dq_lds_barrier();                                   // the tile is read before the next one is written
  }
}

// Tile shape and grid. Layers with at most two 64 KiB tiles per compute unit: one tile per
// workgroup, as few rows and as many groups as the row length allows (8 x 512 for rows of 512
// groups or more: a workgroup writes whole rows, one contiguous range); measured on the 4096 x 4096
// layer, 8.6 / 8.8 / 9.5 / 10.0 us at k = 1..4 against 8.6 / 9.6 / 9.5 / 10.5 for 64 x 64 tiles.
// Larger layers: 32 x 64 tiles and two workgroups per compute unit, each walking its tiles (on the
// 11008 x 4096 layer 22 / 26 us at k = 1 / 4 against 25 / 29 for one 8 x 512 tile per workgroup).
template <int OUT, int K>
static void launch_dequant8_tile_k(const Layer& L, void* W, int n_cu, hipStream_t st) {
  const int d_out = L.d.d_out;
  auto n_tiles = [&](int rt, int gt) { return ((d_out + rt - 1) / rt) * ((L.S + gt / 16 - 1) / (gt / 16)); };
  auto go = [&](auto kern, int grid) {
    kern<<<(unsigned)std::min(grid, 65535), dq::kThreads, 0, st>>>(L.codes, L.codebooks, L.scales, W, d_out, L.d.d_in,
                                                                   L.G, L.S, L.plane_bytes);
  };
  if (n_cu > 0 && n_tiles(64, 64) > 2 * n_cu) {
    go(dequant8_tile_kernel<OUT, K, 32, 64>, std::min(n_tiles(32, 64), 2 * n_cu));
  } else if (L.G > 256) {
    go(dequant8_tile_kernel<OUT, K, 8, 512>, n_tiles(8, 512));
  } else if (L.G > 128) {
    go(dequant8_tile_kernel<OUT, K, 16, 256>, n_tiles(16, 256));
  } else if (L.G > 64) {
    go(dequant8_tile_kernel<OUT, K, 32, 128>, n_tiles(32, 128));
  } else {
    go(dequant8_tile_kernel<OUT, K, 64, 64>, n_tiles(64, 64));
  }
}

template <int OUT>
static void launch_dequant8_tile(const Layer& L, int k, void* W, int n_cu, hipStream_t st) {
  switch (k) {
    case 1: launch_dequant8_tile_k<OUT, 1>(L, W, n_cu, st); break;
    case 2: launch_dequant8_tile_k<OUT, 2>(L, W, n_cu, st); break;
    case 3: launch_dequant8_tile_k<OUT, 3>(L, W, n_cu, st); break;
    case 4: launch_dequant8_tile_k<OUT, 4>(L, W, n_cu, st); break;
    case 5: launch_dequant8_tile_k<OUT, 5>(L, W, n_cu, st); break;
    case 6: launch_dequant8_tile_k<OUT, 6>(L, W, n_cu, st); break;
    case 7: launch_dequant8_tile_k<OUT, 7>(L, W, n_cu, st); break;
    default: launch_dequant8_tile_k<OUT, 8>(L, W, n_cu, st); break;
  }
}

template <int OUT>
static void launch_dequant8(const Layer& L, int k, void* W, unsigned grid, hipStream_t st) {
  const size_t lds = (size_t)k * 256 * 16;
  auto go = [&](auto kern) {
    kern<<<grid, 256, lds, st>>>(L.codes, L.codebooks, L.scales, W, L.d.d_out, L.d.d_in, L.G, L.S, L.plane_bytes);
  };
  switch (k) {
    case 1: go(dequant8_kernel<OUT, 1>); break;
    case 2: go(dequant8_kernel<OUT, 2>); break;
    case 3: go(dequant8_kernel<OUT, 3>); break;
    case 4: go(dequant8_kernel<OUT, 4>); break;
    case 5: go(dequant8_kernel<OUT, 5>); break;
    case 6: go(dequant8_kernel<OUT, 6>); break;
    case 7: go(dequant8_kernel<OUT, 7>); break;
    default: go(dequant8_kernel<OUT, 8>); break;
  }
}

hipError_t launch_dequant(const Layer& L, int k, void* W, aqmb_dtype w_dtype, hipStream_t st) {
  const size_t nslot = (size_t)L.S * L.d.d_out * 16;
  if (L.d.code_bits == 8 && w_dtype != AQMB_F32 && nslot < ((size_t)1 << 30)) {
    if (w_dtype == AQMB_F16) launch_dequant8_tile<AQMB_F16>(L, k, W, L.n_cu, st);
    else launch_dequant8_tile<AQMB_BF16>(L, k, W, L.n_cu, st);
    return hipGetLastError();
  }
  if (L.d.code_bits == 8 && nslot < ((size_t)1 << 30)) {
    // fp32 output: one thread per group slot and pass; at most 2048 workgroups (eight per CU), so
    // large layers take several passes and the reads of one overlap the writes of another
    // (t + 2 * stride stays below 2^31)
    const unsigned grid = (unsigned)std::max<size_t>(1, std::min<size_t>((nslot + 255) / 256, 2048));
    launch_dequant8<AQMB_F32>(L, k, W, grid, st);
    return hipGetLastError();
  }
  // 16- and 4-bit codes (and 8-bit layers too large for 32-bit thread indices): one thread per group
  const size_t n = (size_t)L.S * L.d.d_out * L.J;
  const unsigned grid = (unsigned)std::min<size_t>((n + 1023) / 1024, 2048);
  const size_t lds = L.d.code_bits <= 8 ? ((size_t)k << L.d.code_bits) * 16 : 0;
  auto go = [&](auto kern) {
    kern<<<grid, 256, lds, st>>>(L.codes, L.codebooks, L.scales, W, L.d.d_out, L.d.d_in, L.G, L.S, k, L.plane_bytes);
  };
  auto pick = [&](auto f32, auto f16, auto bf16) {
    if (w_dtype == AQMB_F32) go(f32);
    else if (w_dtype == AQMB_F16) go(f16);
    else go(bf16);
  };
  if (L.d.code_bits == 8) pick(dequant_kernel<AQMB_F32, 8>, dequant_kernel<AQMB_F16, 8>, dequant_kernel<AQMB_BF16, 8>);
  else if (L.d.code_bits == 4) pick(dequant_kernel<AQMB_F32, 4>, dequant_kernel<AQMB_F16, 4>, dequant_kernel<AQMB_BF16, 4>);
  else pick(dequant_kernel<AQMB_F32, 16>, dequant_kernel<AQMB_F16, 16>, dequant_kernel<AQMB_BF16, 16>);
  return hipGetLastError();
}

}  // namespace aqmb
