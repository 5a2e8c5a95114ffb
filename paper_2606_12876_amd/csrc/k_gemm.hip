// Prefill GEMM: Y[n][i] = s_i * sum_t X[n][t] * Wb[i][t], where Wb is the unscaled
// reconstruction from the first k codebooks (binary32 left fold over planes), rounded to bf16,
// and the products run on the bf16 matrix cores (v_mfma_f32_32x32x16_bf16, fp32 accumulate).
//
// A workgroup computes a BM x BN tile of Y (256 tokens x 128 output rows; 128 x 128 or 128 x 64
// when larger tiles would leave compute units idle), walking
// d_in in steps of BK = 64 (four MFMA K-blocks of 16). CW + 4 waves share the four SIMDs in two
// roles, handing data over through LDS with one barrier per step:
//   - CW consumer waves (four, or eight on the 256 x 128 tile at k <= 2) each own a
//     BM/(CW/2) x 64 block of the tile (MFMA blocks of 32 x 32, fp32 accumulators in registers;
//     the same products in the same order for either CW). They also stream X: direct global->LDS loads (16 bytes
//     per lane, eight lanes per 128-byte row segment) fill a ring of X stages several steps
//     ahead, so X reaches LDS without passing through registers. Within a step the fragments
//     of K-block i + 1 are read from LDS while the MFMAs of block i run;
//   - four producer waves dequantize the next step's weight slab into a double-buffered LDS
//     buffer: per group, gather the k codewords from the codebooks held in LDS, fold them in
//     binary32 and round to bf16. Each producer wave streams its own code words into its own
//     LDS ring a few steps ahead with direct loads (8-bit codes: the 4 groups of its thread in one
//     word per plane; 4-bit codes: the step's 8 groups in one word per plane, of which the thread
//     takes its 4 nibbles).
// X stages are row-major with the eight 16-byte pieces of a row XOR-swizzled by (row / 2) mod 8:
// rows are 128 bytes, so two consecutive rows fill one 256-byte bank row, and any 16 consecutive
// rows of a fragment read (one LDS cycle's worth of 16-byte lanes) hit 16 distinct 16-byte slots. Weight slabs are stored in MFMA operand
// order (a 1 KiB chunk is one 32 x 16 fragment as the 64 lanes read it).
// Column blocks start their K walk at different steps, so the workgroups that share an XCD
// (and its L2) read different parts of their common X rows at any time. Row scales are applied
// to the fp32 accumulators in the epilogue.
//
// Loads that fill LDS directly are issued as inline assembly and awaited with explicit vmcnt
// waits before the barrier (or, for a wave's private code ring, before its own reads): the
// compiler cannot see that their destinations are disjoint and would otherwise serialise them.
// Every such load instruction is issued unconditionally (out-of-range rows and groups read a
// valid address and are masked later), so each wait counts a fixed number of loads.
#include <cstdlib>

#include "device.h"
#include "launch.h"

namespace aqmb {

namespace gemm {
constexpr int BM = 256, BN = 128, BK = 64;
template <int K> constexpr int x_depth() { return K <= 4 ? 3 : 2; }   // X stages (LDS budget)
template <int BMT> constexpr int x_stage() { return BMT * BK; }   // bf16 elements: BMT rows x 128 bytes
constexpr int kChunk = 512;                          // one weight fragment: 64 lanes x 8 bf16
template <int BNT> constexpr int slab_elems() { return (BNT / 32) * (BK / 16) * kChunk; }   // column blocks x 4 K-blocks
constexpr int kCodeDepth = 4;                        // steps of code words in flight per producer wave
typedef __attribute__((address_space(3))) void* lds_ptr;
}  // namespace gemm

#define AQMB_WAIT_VMCNT(n) __builtin_amdgcn_s_waitcnt(((n) & 15) | (((n) >> 4) << 14) | 0x70 | 0xF00)


// Direct global->LDS load of 4 bytes per lane: lane l's word lands at lds_base + 4 l.
__device__ __forceinline__ void load_lds4(const void* gptr, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dword %1, off"
               :: "s"(__builtin_amdgcn_readfirstlane(lds_base)), "v"(gptr) : "memory", "m0");
}

template <int K>
__device__ __forceinline__ uint4 fold_bf16(const uint4 (&c)[K]) {
  float w[8] = {f16lo(c[0].x), f16hi(c[0].x), f16lo(c[0].y), f16hi(c[0].y),
                f16lo(c[0].z), f16hi(c[0].z), f16lo(c[0].w), f16hi(c[0].w)};
#pragma unroll
  for (int m = 1; m < K; ++m) {
    w[0] = add_f16_lo(c[m].x, w[0]); w[1] = add_f16_hi(c[m].x, w[1]);
    w[2] = add_f16_lo(c[m].y, w[2]); w[3] = add_f16_hi(c[m].y, w[3]);
    w[4] = add_f16_lo(c[m].z, w[4]); w[5] = add_f16_hi(c[m].z, w[5]);
    w[6] = add_f16_lo(c[m].w, w[6]); w[7] = add_f16_hi(c[m].w, w[7]);
  }
  return make_uint4(pack_bf16x2(w[0], w[1]), pack_bf16x2(w[2], w[3]), pack_bf16x2(w[4], w[5]), pack_bf16x2(w[6], w[7]));
}

template <int K>
__device__ __forceinline__ uint4 dequant_group_bf16(const uint4* __restrict__ cbs, const uint32_t (&word)[K], int sh) {
  const uint4 c0 = cbs[(word[0] >> sh) & 0xFFu];
  float w[8] = {f16lo(c0.x), f16hi(c0.x), f16lo(c0.y), f16hi(c0.y), f16lo(c0.z), f16hi(c0.z), f16lo(c0.w), f16hi(c0.w)};
#pragma unroll
  for (int m = 1; m < K; ++m) {
    const uint4 c = cbs[m * 256 + ((word[m] >> sh) & 0xFFu)];
    w[0] = add_f16_lo(c.x, w[0]); w[1] = add_f16_hi(c.x, w[1]);
    w[2] = add_f16_lo(c.y, w[2]); w[3] = add_f16_hi(c.y, w[3]);
    w[4] = add_f16_lo(c.z, w[4]); w[5] = add_f16_hi(c.z, w[5]);
    w[6] = add_f16_lo(c.w, w[6]); w[7] = add_f16_hi(c.w, w[7]);
  }
  return make_uint4(pack_bf16x2(w[0], w[1]), pack_bf16x2(w[2], w[3]), pack_bf16x2(w[4], w[5]), pack_bf16x2(w[6], w[7]));
}

// CB = code bits: 8 (256 codewords per codebook) or 4 (16 codewords).
template <int K, int YDT, int CB, int BMT, int BNT, int CW = 4>
__global__ __launch_bounds__(64 * (CW + 4)) void gemm_kernel(const unsigned char* __restrict__ codes,
                                                              const uint16_t* __restrict__ codebooks,
                                                              const uint16_t* __restrict__ scales,
                                                              const uint16_t* __restrict__ X, void* __restrict__ Y,
                                                              int n_tokens, int d_out, int d_in, int G,
                                                              size_t plane_bytes, int n_tb, int n_cb) {
  using namespace gemm;
  constexpr int kDepth = x_depth<K>();
  constexpr int NCW = 1 << CB;
  constexpr int kXStage = x_stage<BMT>();
  constexpr int kThreads = 64 * (CW + 4);          // CW consumer waves, then 4 producer waves
  constexpr int MA = BMT / (CW / 2) / 32;          // 32-row MFMA blocks per consumer wave
  constexpr int NBB = BNT / 64;                    // 32-column MFMA blocks per consumer wave
  constexpr int kXLoads = BMT / (8 * CW);          // direct X loads per consumer wave and step
  constexpr int kRowsW = BMT / CW;                 // X rows loaded by each consumer wave
  constexpr int kSlab = slab_elems<BNT>();
  constexpr int QG = BNT / 32;                     // groups per producer thread and step
  extern __shared__ uint4 smem[];
  uint16_t* Xs = (uint16_t*)smem;                  // [kDepth][256 rows][8 swizzled 16-byte pieces]
  uint16_t* Bs = Xs + kDepth * kXStage;            // [2][4 col blocks][4 K-blocks][64 lanes][8]
  uint4* cbs = (uint4*)(Bs + 2 * kSlab);           // [K][NCW] codewords (fp16 x 8)
  uint32_t* cring = (uint32_t*)(cbs + K * NCW);     // [kCodeDepth][4 producer waves][K][64 lanes] code words

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform across the wave
  const int half = lane >> 5, r32 = lane & 31;
  const int tb = blockIdx.x % n_tb, cb = blockIdx.x / n_tb;
  const int n0 = tb * BMT, i0 = cb * BNT;
  const int nsteps = (d_in + BK - 1) / BK;
  const int s0 = (int)(((long long)cb * nsteps) / n_cb);
  auto step_of = [&](int seq) { int st = s0 + seq; return st >= nsteps ? st - nsteps : st; };

  for (int q = tid; q < K * NCW; q += kThreads) cbs[q] = ((const uint4*)codebooks)[q];

  if (wave >= CW) {
    // ------------------------------------------------------------------ producers
    const int p = tid - 64 * CW;
    const int col = p & (BNT - 1), gq = p / BNT;   // weight row; groups QG gq .. QG gq + QG - 1 of a step
    const bool col_ok = i0 + col < d_out;
    // Code words: each producer wave streams exactly the words its own lanes need (one 4-byte
    // word per plane holding this thread's groups of its column in the step) straight into its own
    // LDS ring, kCodeDepth steps ahead, and waits only for its own loads (no other wave reads
    // them). Exactly K loads per step per wave, so "step q's words are in" is a fixed vmcnt.
    const int pw = wave - CW;
    const int col_ld = col_ok ? i0 + col : d_out - 1;
    auto ring_base = [&](int seq) {
      return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void*)(cring + ((seq % kCodeDepth) * 4 + pw) * K * 64);
    };
    auto load_codes = [&](int seq) {
      const uint32_t base = ring_base(seq);
      if constexpr (CB == 8) {
        int j0 = step_of(seq) * (BK / 8) + ((QG * gq) & ~3);   // 4-aligned: one code word per plane
        if (j0 >= G) j0 = 0;                          // padding groups: any valid word, zeroed later
#pragma unroll
        for (int m = 0; m < K; ++m)
          load_lds4(codes + m * plane_bytes + ((size_t)(j0 >> 4) * d_out + col_ld) * 16 + (j0 & 15), base + m * 256);
      } else {                                        // groups 8 s .. 8 s + 7: one word of a 32-group slice
        int j0 = step_of(seq) * (BK / 8);
        if (j0 >= G) j0 = 0;
#pragma unroll
        for (int m = 0; m < K; ++m)
          load_lds4(codes + m * plane_bytes + ((size_t)(j0 >> 5) * d_out + col_ld) * 16 + ((j0 & 31) >> 1), base + m * 256);
      }
    };
    auto wait_codes = [&](int seq) {               // this wave's words of step seq are in LDS
      const int after = min(kCodeDepth - 1, nsteps - 1 - seq);
      if (after >= 3) AQMB_WAIT_VMCNT(3 * K);
      else if (after == 2) AQMB_WAIT_VMCNT(2 * K);
      else if (after == 1) AQMB_WAIT_VMCNT(K);
      else AQMB_WAIT_VMCNT(0);
    };
    auto produce = [&](int seq) {
      const int j0 = step_of(seq) * (BK / 8) + QG * gq;
      uint16_t* slab = Bs + (seq & 1) * kSlab;
      const uint32_t* words = cring + ((seq % kCodeDepth) * 4 + pw) * K * 64 + lane;
      uint32_t word[K];
#pragma unroll
      for (int m = 0; m < K; ++m) word[m] = words[m * 64];
      // all QG K codeword gathers first, then the folds
      uint4 cw[QG][K];
#pragma unroll
      for (int q = 0; q < QG; ++q)
#pragma unroll
        for (int m = 0; m < K; ++m) {
          const uint32_t code = CB == 8 ? (word[m] >> (8 * (((QG * gq) & 3) + q))) & 0xFFu
                                        : (word[m] >> (4 * (QG * gq + q))) & 15u;
          cw[q][m] = cbs[m * NCW + code];
        }
#pragma unroll
      for (int q = 0; q < QG; ++q) {
        const int g = QG * gq + q;                  // group within the step: K-block g / 2, half g % 2
        uint4 v = fold_bf16<K>(cw[q]);
        if (!col_ok || j0 + q >= G) v = make_uint4(0, 0, 0, 0);
        *(uint4*)(slab + ((col >> 5) * 4 + (g >> 1)) * kChunk + ((col & 31) + 32 * (g & 1)) * 8) = v;
      }
    };
    for (int d = 0; d < kCodeDepth && d < nsteps; ++d) load_codes(d);
    __syncthreads();                                 // codebooks staged
    wait_codes(0);
    produce(0);
    if (kCodeDepth < nsteps) load_codes(kCodeDepth);   // refills the slot of step 0
    for (int seq = 0; seq < nsteps; ++seq) {
      __syncthreads();                               // slab seq published; slab seq+1 free
      if (seq + 1 < nsteps) {
        wait_codes(seq + 1);
        produce(seq + 1);
        if (seq + 1 + kCodeDepth < nsteps) load_codes(seq + 1 + kCodeDepth);
      }
    }
    return;
  }

  // -------------------------------------------------------------------- consumers
  const int wm = wave >> 1, wn = wave & 1;          // BMT/(CW/2) x 64 block of the tile
  // X stage layout: row r's 16-byte piece kc (8 bf16 of K) sits at r * 128 + ((kc ^ ((r >> 1) & 7)) * 16)
  // bytes. A direct load covers 8 rows x 128 bytes (8 lanes per row, full cache lines); the
  // XOR keeps fragment reads (32 rows, one piece each) on distinct banks.
  auto load_x = [&](int seq) {
    const int k0 = step_of(seq) * BK;
    uint16_t* stage = Xs + (seq % kDepth) * kXStage;
    const int pos = lane & 7, rsub = lane >> 3;
    if (k0 + BK <= d_in) {
#pragma unroll
      for (int t = 0; t < kXLoads; ++t) {           // this wave's rows (BMT/4) wave .. + BMT/4 - 1
        const int r = wave * kRowsW + t * 8 + rsub;
        const int kc = pos ^ ((r >> 1) & 7);
        const int row = n0 + r < n_tokens ? n0 + r : n_tokens - 1;
        uint16_t* base = stage + (wave * kRowsW + t * 8) * BK;   // 1 KiB: 8 rows, written lane-ordered
        load_lds16(X + (size_t)row * d_in + k0 + kc * 8, (uint32_t)(uintptr_t)(lds_ptr)base);
      }
    } else {                                         // the ragged last step: zero past d_in
#pragma unroll
      for (int t = 0; t < kXLoads; ++t) {
        const int r = wave * kRowsW + t * 8 + rsub;
        const int kc = pos ^ ((r >> 1) & 7);
        const int row = n0 + r;
        uint16_t* base = stage + (wave * kRowsW + t * 8) * BK;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (row < n_tokens && k0 + kc * 8 < d_in) v = *(const uint4*)(X + (size_t)row * d_in + k0 + kc * 8);
        *(uint4*)(base + lane * 8) = v;
      }
    }
  };
  f32x16_t acc[MA][NBB];
#pragma unroll
  for (int a = 0; a < MA; ++a)
#pragma unroll
    for (int b = 0; b < NBB; ++b)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[a][b][e] = 0.f;

  struct Frags { bf16x8_t a[MA], b[NBB]; };
  auto read_frags = [&](const uint16_t* xst, const uint16_t* bsl, int i, Frags& f) {
#pragma unroll
    for (int b = 0; b < NBB; ++b) f.b[b] = *(const bf16x8_t*)(bsl + ((wn * NBB + b) * 4 + i) * kChunk + lane * 8);
    const int kc = 2 * i + half;
#pragma unroll
    for (int a = 0; a < MA; ++a) {
      const int r = wm * (BMT / (CW / 2)) + a * 32 + r32;
      f.a[a] = *(const bf16x8_t*)(xst + r * BK + ((kc ^ ((r >> 1) & 7)) * 8));
    }
  };
  auto mfmas = [&](const Frags& f) {
#pragma unroll
    for (int a = 0; a < MA; ++a)
#pragma unroll
      for (int b = 0; b < NBB; ++b) acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[a], f.b[b], acc[a][b], 0, 0, 0);
  };

  for (int seq = 0; seq < kDepth - 1 && seq < nsteps; ++seq) load_x(seq);
  __syncthreads();                                   // codebooks staged
  for (int seq = 0; seq < nsteps; ++seq) {
    {                                                // own X loads of step seq done
      const int after = min(kDepth - 2, nsteps - 1 - seq);   // later steps already issued
      if (after >= 1) AQMB_WAIT_VMCNT(kXLoads); else AQMB_WAIT_VMCNT(0);
    }
    __syncthreads();                                 // X stage seq and slab seq published
    if (seq + kDepth - 1 < nsteps) load_x(seq + kDepth - 1);
    const uint16_t* xst = Xs + (seq % kDepth) * kXStage;
    const uint16_t* bsl = Bs + (seq & 1) * kSlab;
    // K-blocks 0..3: the fragments of block i + 1 are read while block i's MFMAs run
    // (one read, one MFMA, alternating); a scheduling barrier closes each block so the compiler
    // cannot pull the next block's MFMAs (and their LDS waits) forward.
    Frags f0, f1;
    read_frags(xst, bsl, 0, f0);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      Frags& cur = (i & 1) ? f1 : f0;
      Frags& nxt = (i & 1) ? f0 : f1;
      if (i < 3) read_frags(xst, bsl, i + 1, nxt);
      mfmas(cur);
      if (i < 3) {
        __builtin_amdgcn_sched_group_barrier(0x100, MA + NBB, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, NBB * MA, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  }
#pragma unroll
  for (int b = 0; b < NBB; ++b) {
    const int col = i0 + wn * (BNT / 2) + b * 32 + r32;
    if (col >= d_out) continue;
    const float scale = f16_to_f32(scales[col]);
#pragma unroll
    for (int a = 0; a < MA; ++a) {
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int row = n0 + wm * (BMT / (CW / 2)) + a * 32 + 8 * (e >> 2) + 4 * half + (e & 3);
        if (row < n_tokens) OutT<YDT>::store(Y, (size_t)row * d_out + col, acc[a][b][e] * scale);
      }
    }
  }
}

// ---------------------------------------------------------------------------------------------
// Two-pass prefill GEMM (a caller-provided workspace, k >= 2 at large token counts). With the large
// tiles every column block of weights is dequantized once per token tile (eight times for 2048
// tokens), and at k >= 2 the producer waves' codeword gathers (one unreplicated LDS copy of the
// codebooks: the X ring leaves no room for replicas) outlast the matrix cores. Here the weights
// are reconstructed once, by the same fold and rounding, into the workspace, tiled in the order
// in which the MFMAs read them; a dense kernel then streams X and those tiles. Same products in
// the same order as gemm_kernel<., 256, 128>: the results are bit-identical.
//
// Workspace layout (bf16): chunk ((c32 * nsteps + s) * 4 + i), 512 values, holds weight rows
// 32 c32 .. 32 c32 + 31 and inputs 64 s + 16 i .. + 15 as the B fragment of one MFMA K-block:
// value 8 l + e is row 32 c32 + (l % 32), input 64 s + 16 i + 8 (l / 32) + e (zero past d_out and
// past d_in), which is also the order of a weight slab in gemm_kernel's LDS.
namespace gemm2 {
constexpr int kTileWaves = 4, kRep = 2;            // tiling pass: 4 waves, two codebook copies
constexpr int kWaves = 8, kThreads = 64 * kWaves;  // dense pass: 8 waves (two per SIMD)
constexpr int BM = 256, BN = 128, BK = 64, kDepth = 3;
constexpr int kXStage = BM * BK;                   // bf16 values: 256 rows x 128 bytes
constexpr int kSlab = (BN / 32) * 4 * gemm::kChunk;
constexpr int kStage = kXStage + kSlab;
}  // namespace gemm2

// Pass 1. A wave takes 32 weight rows and two K-steps (lane l: row l % 32, step l / 32), a
// workgroup 32 rows and 8 steps per item; the lane folds the 8 groups of its step and writes each
// one 16-byte piece (a wave's writes of one group are two 512-byte runs). Codebooks: two
// interleaved copies in LDS, lane parity choosing the copy.
template <int K, int CB>
__global__ __launch_bounds__(64 * gemm2::kTileWaves) void gemm_wtile_kernel(const unsigned char* __restrict__ codes,
                                                                          const uint16_t* __restrict__ codebooks,
                                                                          uint16_t* __restrict__ Wt, int d_out, int G,
                                                                          int nsteps, size_t plane_bytes, int n_c32) {
  using namespace gemm2;
  constexpr int NCW = 1 << CB;
  extern __shared__ uint4 cb_lds[];                // [K][NCW][kRep]
  for (int q = threadIdx.x; q < K * NCW; q += 64 * kTileWaves) {
    const uint4 v = ((const uint4*)codebooks)[q];
#pragma unroll
    for (int r = 0; r < kRep; ++r) cb_lds[q * kRep + r] = v;
  }
  __syncthreads();
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int rep = lane & (kRep - 1);
  constexpr int kSteps = 2 * kTileWaves;           // steps per item
  const int n_sc = (nsteps + kSteps - 1) / kSteps;
  const int items = n_c32 * n_sc;
  for (int it = blockIdx.x; it < items; it += gridDim.x) {
    const int c32 = it / n_sc;
    const int s = (it - c32 * n_sc) * kSteps + wave * 2 + (lane >> 5);
    if (s >= nsteps) continue;
    const int row = c32 * 32 + (lane & 31);
    const bool row_ok = row < d_out;
    const int rl = row_ok ? row : d_out - 1;
    uint32_t w[K][2];                              // the step's 8 codes of the row, per plane
#pragma unroll
    for (int m = 0; m < K; ++m) {
      if constexpr (CB == 8) {                     // 8 bytes of a 16-group slice
        const uint2 v = *(const uint2*)(codes + m * plane_bytes + ((size_t)((8 * s) >> 4) * d_out + rl) * 16 + ((8 * s) & 15));
        w[m][0] = v.x; w[m][1] = v.y;
      } else {                                     // 4 bytes (8 nibbles) of a 32-group slice
        w[m][0] = *(const uint32_t*)(codes + m * plane_bytes + ((size_t)((8 * s) >> 5) * d_out + rl) * 16 + (((8 * s) & 31) >> 1));
        w[m][1] = 0;
      }
    }
    uint16_t* dst = Wt + ((size_t)c32 * nsteps + s) * 4 * gemm::kChunk + (lane & 31) * 8;
#pragma unroll
    for (int g = 0; g < 8; ++g) {
      uint4 c[K];
#pragma unroll
      for (int m = 0; m < K; ++m) {
        const uint32_t code = CB == 8 ? (w[m][g >> 2] >> (8 * (g & 3))) & 0xFFu : (w[m][0] >> (4 * g)) & 15u;
        c[m] = cb_lds[(m * NCW + code) * kRep + rep];
      }
      uint4 v = fold_bf16<K>(c);
      if (!row_ok || 8 * s + g >= G) v = make_uint4(0, 0, 0, 0);
      const u32x4_t vv = {v.x, v.y, v.z, v.w};        // non-temporal: the tiles are read once, by the dense pass
      __builtin_nontemporal_store(vv, (u32x4_t*)(dst + (g >> 1) * gemm::kChunk + 32 * (g & 1) * 8));
    }
  }
}

// Pass 2: 256 x 128 output tiles, 8 waves (two per SIMD) of 64 tokens x 64 weight rows (2 x 2 MFMA
// blocks of 32 x 32), d_in in steps of 64 through a ring of three LDS stages, each holding the
// step's X rows (the swizzled layout of gemm_kernel) and its weight tile, both filled by direct
// global->LDS loads two steps ahead; one barrier per step. Column blocks start their K walk at the
// steps gemm_kernel uses. Workgroups are placed on XCDs (workgroup w runs on XCD w mod 8) in a
// grid of ga x gb blocks of token tiles x column blocks, so that the workgroups sharing weight
// tiles and X rows share an L2 (ga = 0: the plain order).
template <int YDT>
__global__ __launch_bounds__(gemm2::kThreads) void gemm_dense_kernel(const uint16_t* __restrict__ Wt,
                                                                    const uint16_t* __restrict__ scales,
                                                                    const uint16_t* __restrict__ X, void* __restrict__ Y,
                                                                    int n_tokens, int d_out, int d_in, int nsteps,
                                                                    int n_tb, int n_cb, int n_c32, int ga, int gb) {
  using namespace gemm2;
  constexpr int MA = 2, NBB = 2;                   // 32 x 32 blocks per wave: 2 token x 2 weight row
  constexpr int kXLoads = BM / (8 * kWaves), kWLoads = BN / (8 * kWaves), kLoads = kXLoads + kWLoads;
  constexpr int kRowsW = BM / kWaves;              // X rows loaded by each wave
  extern __shared__ uint4 smem2[];
  uint16_t* S = (uint16_t*)smem2;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int half = lane >> 5, r32 = lane & 31;
  int tb = blockIdx.x % n_tb, cb = blockIdx.x / n_tb;
  if (ga > 0) {
    const int xcd = blockIdx.x & 7, j = blockIdx.x >> 3, per_cb = n_cb / gb, per_tb = n_tb / ga;
    cb = per_cb * (xcd % gb) + j % per_cb;
    tb = per_tb * (xcd / gb) + j / per_cb;
  }
  const int n0 = tb * BM, i0 = cb * BN;
  const int s0 = (int)(((long long)cb * nsteps) / n_cb);
  auto step_of = [&](int seq) { int st = s0 + seq; return st >= nsteps ? st - nsteps : st; };

  auto load_stage = [&](int seq) {
    const int st = step_of(seq);
    const int k0 = st * BK;
    uint16_t* stage = S + (seq % kDepth) * kStage;
#pragma unroll
    for (int t = 0; t < kWLoads; ++t) {            // chunk c: column block c / 4, K-block c % 4
      const int c = wave * kWLoads + t;
      int c32 = i0 / 32 + (c >> 2);
      if (c32 >= n_c32) c32 = n_c32 - 1;           // rows past d_out: any valid tile, never stored
      load_lds16(Wt + (((size_t)c32 * nsteps + st) * 4 + (c & 3)) * gemm::kChunk + lane * 8,
                 lds_addr(stage + kXStage + c * gemm::kChunk));
    }
    const int pos = lane & 7, rsub = lane >> 3;
    if (k0 + BK <= d_in) {
#pragma unroll
      for (int t = 0; t < kXLoads; ++t) {
        const int r = wave * kRowsW + t * 8 + rsub;
        const int kc = pos ^ ((r >> 1) & 7);
        const int row = n0 + r < n_tokens ? n0 + r : n_tokens - 1;
        load_lds16(X + (size_t)row * d_in + k0 + kc * 8, lds_addr(stage + (wave * kRowsW + t * 8) * BK));
      }
    } else {                                       // the ragged last step: zero past d_in
#pragma unroll
      for (int t = 0; t < kXLoads; ++t) {
        const int r = wave * kRowsW + t * 8 + rsub;
        const int kc = pos ^ ((r >> 1) & 7);
        const int row = n0 + r;
        uint16_t* base = stage + (wave * kRowsW + t * 8) * BK;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (row < n_tokens && k0 + kc * 8 < d_in) v = *(const uint4*)(X + (size_t)row * d_in + k0 + kc * 8);
        *(uint4*)(base + lane * 8) = v;
      }
    }
  };
  const int wm = wave >> 1, wn = wave & 1;         // tokens 64 wm .., weight rows 64 wn ..
  f32x16_t acc[MA][NBB];
#pragma unroll
  for (int a = 0; a < MA; ++a)
#pragma unroll
    for (int b = 0; b < NBB; ++b)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[a][b][e] = 0.f;
  struct Frags { bf16x8_t a[MA], b[NBB]; };
  auto read_frags = [&](const uint16_t* xst, const uint16_t* bsl, int i, Frags& f) {
#pragma unroll
    for (int b = 0; b < NBB; ++b) f.b[b] = *(const bf16x8_t*)(bsl + ((wn * NBB + b) * 4 + i) * gemm::kChunk + lane * 8);
    const int kc = 2 * i + half;
#pragma unroll
    for (int a = 0; a < MA; ++a) {
      const int r = wm * 64 + a * 32 + r32;
      f.a[a] = *(const bf16x8_t*)(xst + r * BK + ((kc ^ ((r >> 1) & 7)) * 8));
    }
  };
  auto mfmas = [&](const Frags& f) {
#pragma unroll
    for (int a = 0; a < MA; ++a)
#pragma unroll
      for (int b = 0; b < NBB; ++b) acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[a], f.b[b], acc[a][b], 0, 0, 0);
  };
  for (int seq = 0; seq < kDepth - 1 && seq < nsteps; ++seq) load_stage(seq);
  for (int seq = 0; seq < nsteps; ++seq) {
    {                                              // own loads of step seq done (step seq + 1's may be out)
      const int after = min(kDepth - 2, nsteps - 1 - seq);
      if (after >= 1) wait_vmcnt<kLoads>(); else wait_vmcnt<0>();
    }
    __syncthreads();                               // stage seq published; stage seq - 1 free
    if (seq + kDepth - 1 < nsteps) load_stage(seq + kDepth - 1);
    const uint16_t* xst = S + (seq % kDepth) * kStage;
    const uint16_t* bsl = xst + kXStage;
    Frags f0, f1;
    read_frags(xst, bsl, 0, f0);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      Frags& cur = (i & 1) ? f1 : f0;
      Frags& nxt = (i & 1) ? f0 : f1;
      if (i < 3) read_frags(xst, bsl, i + 1, nxt);
      mfmas(cur);
      if (i < 3) {
        __builtin_amdgcn_sched_group_barrier(0x100, MA + NBB, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, NBB * MA, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  }
#pragma unroll
  for (int b = 0; b < NBB; ++b) {
    const int col = i0 + wn * 64 + b * 32 + r32;
    if (col >= d_out) continue;
    const float scale = f16_to_f32(scales[col]);
#pragma unroll
    for (int a = 0; a < MA; ++a) {
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int row = n0 + wm * 64 + a * 32 + 8 * (e >> 2) + 4 * half + (e & 3);
        if (row < n_tokens) OutT<YDT>::store(Y, (size_t)row * d_out + col, acc[a][b][e] * scale);
      }
    }
  }
}

template <int K, int CB, int BMT, int BNT, int CW>
static void launch_kcm(const Layer& L, const void* X, int n_tokens, void* Y, aqmb_dtype y_dtype, hipStream_t st) {
  using namespace gemm;
  constexpr int kDepth = x_depth<K>();
  const int n_tb = (n_tokens + BMT - 1) / BMT, n_cb = (L.d.d_out + BNT - 1) / BNT;
  const size_t lds = ((size_t)kDepth * x_stage<BMT>() + 2 * slab_elems<BNT>()) * 2 + (size_t)K * (1 << CB) * 16 +
                     (size_t)kCodeDepth * 4 * K * 64 * 4;
  const dim3 grid(n_tb * n_cb);
  if (y_dtype == AQMB_BF16)
    gemm_kernel<K, AQMB_BF16, CB, BMT, BNT, CW><<<grid, 64 * (CW + 4), lds, st>>>(
        L.codes, L.codebooks, L.scales, (const uint16_t*)X, Y, n_tokens, L.d.d_out, L.d.d_in, L.G, L.plane_bytes, n_tb, n_cb);
  else
    gemm_kernel<K, AQMB_F32, CB, BMT, BNT, CW><<<grid, 64 * (CW + 4), lds, st>>>(
        L.codes, L.codebooks, L.scales, (const uint16_t*)X, Y, n_tokens, L.d.d_out, L.d.d_in, L.G, L.plane_bytes, n_tb, n_cb);
}

// Tile shape: 0 = 256 tokens x 128 rows, 1 = 128 x 128, 2 = 128 x 64. Unless the caller names one,
// the shape with the least estimated time: rounds of workgroups (one workgroup per CU) times the
// shape's measured cost per workgroup relative to the largest tile (4096 x 4096 layer, one round:
// 1, 0.9, 0.6).
static int gemm_tile(const Layer& L, int n_tokens, int forced) {
  if (forced >= 0 && forced <= 2) return forced;
  const int bm[3] = {256, 128, 128}, bn[3] = {128, 128, 64};
  const double rel[3] = {1.0, 0.9, 0.6};
  const long long ncu = L.n_cu > 0 ? L.n_cu : 256;
  int best = 0;
  double best_t = 0;
  for (int c = 0; c < 3; ++c) {
    const long long wg = (long long)((n_tokens + bm[c] - 1) / bm[c]) * ((L.d.d_out + bn[c] - 1) / bn[c]);
    const double t = (double)((wg + ncu - 1) / ncu) * rel[c];
    if (c == 0 || t < best_t) { best = c; best_t = t; }
  }
  return best;
}

template <int K, int CB>
static void launch_kc(const Layer& L, const void* X, int n_tokens, void* Y, aqmb_dtype y_dtype, int tile,
                      hipStream_t st) {
  switch (gemm_tile(L, n_tokens, tile)) {
    // 256 x 128 tiles at k <= 2: eight consumer waves (two per SIMD, 64 x 64 each) beside the four
    // producers (2048 tokens, 4096 x 4096: 73.2 -> 72.0 us at k = 1, 79.9 -> 77.5 us at k = 2); from
    // k = 3, and on the smaller tiles, four consumer waves are faster
    case 0:
      if constexpr (K <= 2) launch_kcm<K, CB, 256, 128, 8>(L, X, n_tokens, Y, y_dtype, st);
      else launch_kcm<K, CB, 256, 128, 4>(L, X, n_tokens, Y, y_dtype, st);
      break;
    case 1: launch_kcm<K, CB, 128, 128, 4>(L, X, n_tokens, Y, y_dtype, st); break;
    default: launch_kcm<K, CB, 128, 64, 4>(L, X, n_tokens, Y, y_dtype, st); break;
  }
}

template <int K>
static void launch_k(const Layer& L, const void* X, int n_tokens, void* Y, aqmb_dtype y_dtype, int tile,
                     hipStream_t st) {
  if (L.d.code_bits == 4) launch_kc<K, 4>(L, X, n_tokens, Y, y_dtype, tile, st);
  else launch_kc<K, 8>(L, X, n_tokens, Y, y_dtype, tile, st);
}

hipError_t launch_gemm(const Layer& L, int k, const void* X, int n_tokens, void* Y, aqmb_dtype y_dtype, int tile,
                       hipStream_t st) {
  switch (k) {
    case 1: launch_k<1>(L, X, n_tokens, Y, y_dtype, tile, st); break;
    case 2: launch_k<2>(L, X, n_tokens, Y, y_dtype, tile, st); break;
    case 3: launch_k<3>(L, X, n_tokens, Y, y_dtype, tile, st); break;
    case 4: launch_k<4>(L, X, n_tokens, Y, y_dtype, tile, st); break;
    case 5: launch_k<5>(L, X, n_tokens, Y, y_dtype, tile, st); break;
    case 6: launch_k<6>(L, X, n_tokens, Y, y_dtype, tile, st); break;
    case 7: launch_k<7>(L, X, n_tokens, Y, y_dtype, tile, st); break;
    default: launch_k<8>(L, X, n_tokens, Y, y_dtype, tile, st); break;
  }
  return hipGetLastError();
}


// Workspace bytes of the two-pass GEMM (0: the path does not apply). It applies at k >= 3 with 4-
// or 8-bit codes where the library's choice is the 256 x 128 tiling with at least one workgroup
// per compute unit (the same per-output arithmetic as that tiling). At k <= 2 the one-pass kernel
// with eight consumer waves is as fast (2048 x 4096 x 4096, k = 2: 77.5 us against 80.1).
size_t gemm_two_pass_bytes(const Layer& L, int k, int n_tokens) {
  if (k < 3 || (L.d.code_bits != 8 && L.d.code_bits != 4)) return 0;
  if (gemm_tile(L, n_tokens, -1) != 0) return 0;
  const long long wg = (long long)((n_tokens + gemm2::BM - 1) / gemm2::BM) * ((L.d.d_out + gemm2::BN - 1) / gemm2::BN);
  if (wg < (L.n_cu > 0 ? L.n_cu : 256)) return 0;
  const size_t n_c32 = (L.d.d_out + 31) / 32, nsteps = (L.d.d_in + gemm2::BK - 1) / gemm2::BK;
  return n_c32 * nsteps * 4 * gemm::kChunk * 2;
}

template <int K, int CB>
static void launch_wtile(const Layer& L, uint16_t* Wt, int n_c32, int nsteps, hipStream_t st) {
  using namespace gemm2;
  const int items = n_c32 * ((nsteps + 2 * kTileWaves - 1) / (2 * kTileWaves));
  const int grid = items < 2048 ? items : 2048;
  const size_t lds = (size_t)K * (1 << CB) * kRep * 16;
  gemm_wtile_kernel<K, CB><<<grid, 64 * kTileWaves, lds, st>>>(L.codes, L.codebooks, Wt, L.d.d_out, L.G, nsteps,
                                                              L.plane_bytes, n_c32);
}

template <int K>
static void launch_wtile_k(const Layer& L, uint16_t* Wt, int n_c32, int nsteps, hipStream_t st) {
  if (L.d.code_bits == 4) launch_wtile<K, 4>(L, Wt, n_c32, nsteps, st);
  else launch_wtile<K, 8>(L, Wt, n_c32, nsteps, st);
}

hipError_t launch_gemm_two_pass(const Layer& L, int k, const void* X, int n_tokens, void* Y, aqmb_dtype y_dtype,
                                void* workspace, hipStream_t st) {
  using namespace gemm2;
  const int n_c32 = (L.d.d_out + 31) / 32, nsteps = (L.d.d_in + BK - 1) / BK;
  uint16_t* Wt = (uint16_t*)workspace;
  switch (k) {
    case 2: launch_wtile_k<2>(L, Wt, n_c32, nsteps, st); break;
    case 3: launch_wtile_k<3>(L, Wt, n_c32, nsteps, st); break;
    case 4: launch_wtile_k<4>(L, Wt, n_c32, nsteps, st); break;
    case 5: launch_wtile_k<5>(L, Wt, n_c32, nsteps, st); break;
    case 6: launch_wtile_k<6>(L, Wt, n_c32, nsteps, st); break;
    case 7: launch_wtile_k<7>(L, Wt, n_c32, nsteps, st); break;
    default: launch_wtile_k<8>(L, Wt, n_c32, nsteps, st); break;
  }
  const int n_tb = (n_tokens + BM - 1) / BM, n_cb = (L.d.d_out + BN - 1) / BN;
  // XCD blocks: token tiles in ga groups, column blocks in gb groups, ga * gb = 8
  int ga = 0, gb = 0;
  const int cand[4][2] = {{2, 4}, {1, 8}, {4, 2}, {8, 1}};
  for (const auto& c : cand)
    if (n_tb % c[0] == 0 && n_cb % c[1] == 0) { ga = c[0]; gb = c[1]; break; }
  const size_t lds = (size_t)kDepth * kStage * 2;
  const dim3 grid(n_tb * n_cb);
  if (y_dtype == AQMB_BF16)
    gemm_dense_kernel<AQMB_BF16><<<grid, kThreads, lds, st>>>(Wt, L.scales, (const uint16_t*)X, Y, n_tokens, L.d.d_out,
                                                             L.d.d_in, nsteps, n_tb, n_cb, n_c32, ga, gb);
  else
    gemm_dense_kernel<AQMB_F32><<<grid, kThreads, lds, st>>>(Wt, L.scales, (const uint16_t*)X, Y, n_tokens, L.d.d_out,
                                                            L.d.d_in, nsteps, n_tb, n_cb, n_c32, ga, gb);
  return hipGetLastError();
}

}  // namespace aqmb
