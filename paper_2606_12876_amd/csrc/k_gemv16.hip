// Decode GEMV of a layer with 16-bit codes (2^16-codeword codebooks, 1 MiB each):
//   y[b][i] = s_i * sum_j sum_{m<k} <x[b, group j], C_m[b_{ijm}]>
// (the section 5 reconstruction with B = 16: the notation of section 3.2 allows 2^B codewords
// for any B). A codebook is far larger than LDS, so every code costs one random 16-byte load of
// its codeword from global memory, served by the L2 cache of the XCD (each XCD's 4 MB L2 holds
// the codebooks in use); this gather rate, not HBM, bounds the kernel.
//
// One kernel, no partial sums in memory: a persistent workgroup of 1024 threads takes work items
// of 8 output rows (items blockIdx.x, blockIdx.x + gridDim.x, ...). Thread (wave w, lane l) owns
// row l % 8 of the item and 4 consecutive groups 4 h .. 4 h + 3 (h = l / 8 + 8 w) of every
// 512-group block of the row: one 8-byte half of a 16-byte code slice per plane, so the 16 lanes
// that share a slice read one full 128-byte line of 8 rows. The 128 threads of a row cover a
// block; longer rows take several blocks. A row's 128 partial sums are added in a fixed order
// (a butterfly over the wave's 8 lanes of the row, then the 16 waves in order through LDS), so
// results are reproducible.
//
// Loads are pipelined over units (item, block, chunk of up to 4 planes): while the codewords of
// unit v are in flight the code words of unit v + 2 are requested, and the gathers of unit v + 1
// are issued before the row reduction's barrier, so the L2 always has requests from every wave.
// Loads complete in order, so waiting for the gathers of unit v also finds the code words of
// unit v + 1 arrived.
//
// x: the batch tile's rows are staged in LDS as they are (fp16 or bf16 bits, zero past d_in), a
// whole row at once when it fits (otherwise one 512-group block at a time). fp16 x: products by
// v_dot2 (exact fp16 products, fp32 sums) chained over the planes; bf16 x: fp32 fused
// multiply-adds of exactly widened values. Code planes m >= k are never read.
#include "device.h"
#include "launch.h"

namespace aqmb {

namespace g16 {
constexpr int kThreads = 1024, kWaves = 16;
constexpr int kRows = 8;              // output rows per work item
constexpr int kBlock = 512;           // groups per block: 128 threads per row, 4 groups each
constexpr int kPlaneChunk = 4;        // planes per unit (a thread's gathers of a unit in registers)
constexpr size_t kLds = 160 * 1024;
}  // namespace g16

struct Gemv16Args {
  const unsigned char* codes;
  const uint16_t* codebooks;
  const uint16_t* scales;
  const uint16_t* x;
  void* y;
  size_t plane_bytes;
  int d_out, d_in, G, S, k, batch, y_dtype;
  int n_items;          // ceil(d_out / kRows)
  int n_blocks;         // ceil(G / kBlock)
  int n_pc;             // ceil(k / kPlaneChunk)
  int xchunk;           // blocks of x staged at once (n_blocks when the whole row fits)
};

// <x group, codeword>: fp16 x by exact fp16 products (v_dot2), bf16 x by fp32 fused multiply-adds.
template <int XDT>
__device__ __forceinline__ float g16_dot(uint4 xw, uint4 cw, float s) {
  if constexpr (XDT == AQMB_F16) {
    s = dot2_f16(xw.x, cw.x, s);
    s = dot2_f16(xw.y, cw.y, s);
    s = dot2_f16(xw.z, cw.z, s);
    return dot2_f16(xw.w, cw.w, s);
  } else {
    s = __builtin_fmaf(bf16lo(xw.x), f16lo(cw.x), s);
    s = __builtin_fmaf(bf16hi(xw.x), f16hi(cw.x), s);
    s = __builtin_fmaf(bf16lo(xw.y), f16lo(cw.y), s);
    s = __builtin_fmaf(bf16hi(xw.y), f16hi(cw.y), s);
    s = __builtin_fmaf(bf16lo(xw.z), f16lo(cw.z), s);
    s = __builtin_fmaf(bf16hi(xw.z), f16hi(cw.z), s);
    s = __builtin_fmaf(bf16lo(xw.w), f16lo(cw.w), s);
    return __builtin_fmaf(bf16hi(xw.w), f16hi(cw.w), s);
  }
}

// One unit's work: item, block and plane chunk.
struct G16Unit {
  int item, blk, pc;
};

__device__ __forceinline__ G16Unit g16_unit(const Gemv16Args& a, int v) {
  // v counts this workgroup's units: items blockIdx.x + gridDim.x * (v / per_item), then blocks,
  // then plane chunks
  const int per_item = a.n_blocks * a.n_pc;
  G16Unit u;
  u.item = blockIdx.x + gridDim.x * (v / per_item);
  const int r = v % per_item;
  u.blk = r / a.n_pc;
  u.pc = r % a.n_pc;
  return u;
}

// Code words of unit u for this thread: plane pc * KC + m of its half slice (8 bytes = 4 codes).
// Every thread issues the same loads, with no branch: planes >= k reload plane k - 1 (their
// products are skipped), slices past the row reload the last slice (their groups meet x = 0) and
// rows past d_out reload the last row (never stored).
template <int KC>
__device__ __forceinline__ void g16_load_codes(const Gemv16Args& a, const G16Unit& u, uint2 (&c)[KC]) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int h = (lane >> 3) + 8 * (tid >> 6);
  int slice = u.blk * (g16::kBlock / 8) + (h >> 1);
  slice = slice < a.S ? slice : a.S - 1;
  int row = u.item * g16::kRows + (lane & 7);
  row = row < a.d_out ? row : a.d_out - 1;
  const unsigned char* p = a.codes + ((size_t)slice * a.d_out + row) * 16 + (h & 1) * 8;
#pragma unroll
  for (int m = 0; m < KC; ++m) {
    const int plane = u.pc * KC + m < a.k ? u.pc * KC + m : a.k - 1;
    c[m] = load_stream8(p + (size_t)plane * a.plane_bytes);
  }
}

// Codewords of the 4 groups x KC planes of unit u (codes already in c).
template <int KC>
__device__ __forceinline__ void g16_gather(const Gemv16Args& a, const G16Unit& u, const uint2 (&c)[KC],
                                           uint4 (&w)[4][KC]) {
  const uint4* cb = (const uint4*)a.codebooks;
#pragma unroll
  for (int m = 0; m < KC; ++m) {
    const int plane = u.pc * KC + m < a.k ? u.pc * KC + m : a.k - 1;
    const uint4* book = cb + ((size_t)plane << 16);
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      const uint32_t word = jj < 2 ? c[m].x : c[m].y;
      const uint32_t code = (word >> (16 * (jj & 1))) & 0xFFFFu;
      w[jj][m] = book[code];
    }
  }
}

// Stage x rows b0 .. b0 + NB - 1, blocks blk0 .. blk0 + xchunk - 1, into xs ([NB][xchunk * 512]
// groups of 16 bytes); zero past d_in and past the batch.
template <int NB>
__device__ __forceinline__ void g16_stage_x(const Gemv16Args& a, uint4* xs, int b0, int blk0) {
  const int groups = a.xchunk * g16::kBlock;
  for (int q = threadIdx.x; q < NB * groups; q += g16::kThreads) {
    const int b = q / groups, jl = q % groups;
    const int j = blk0 * g16::kBlock + jl;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (b0 + b < a.batch && j < a.G) v = *(const uint4*)(a.x + (size_t)(b0 + b) * a.d_in + (size_t)j * 8);
    xs[q] = v;
  }
}

// LDS writes of this wave complete, then a workgroup barrier; global loads stay in flight (a
// __syncthreads() fence would also wait for the gathers and code words already requested).
__device__ __forceinline__ void g16_lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);                  // lgkmcnt(0); vmcnt and expcnt at their maxima
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

template <int KC, int NB, int XDT>
__global__ __launch_bounds__(g16::kThreads) void gemv_b16_kernel(Gemv16Args a) {
  extern __shared__ uint4 xs[];                         // [NB][xchunk * 512] x groups
  __shared__ float red[2][g16::kWaves][g16::kRows][NB];  // per-wave row sums, two items in turn
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = (lane >> 3) + 8 * wave;                // groups 4 h .. 4 h + 3 of each block
  const int my_items = a.n_items > (int)blockIdx.x ? (a.n_items - 1 - (int)blockIdx.x) / (int)gridDim.x + 1 : 0;
  const int nv = my_items * a.n_blocks * a.n_pc;        // this workgroup's units
  if (nv == 0) return;                                  // uniform: the whole workgroup leaves
  const int xgroups = a.xchunk * g16::kBlock;
  const bool restage = a.xchunk < a.n_blocks;
  int parity = 0;

  for (int b0 = 0; b0 < a.batch; b0 += NB) {
    if (!restage) {
      if (b0 > 0) g16_lds_barrier();                   // every wave is done with the previous tile's x
      g16_stage_x<NB>(a, xs, b0, 0);
      __syncthreads();
    }
    // Every load below is issued by every thread (unit indices past the last unit are clamped to
    // it: a repeated load, never used), so the number of loads in flight is the same on every path
    // and waiting for the codewords of unit v never waits for the code words requested after them.
    uint2 c1[KC], c2[KC];
    uint4 w[4][KC];
    {
      uint2 c0[KC];
      g16_load_codes<KC>(a, g16_unit(a, 0), c0);
      g16_load_codes<KC>(a, g16_unit(a, nv > 1 ? 1 : 0), c1);
      g16_gather<KC>(a, g16_unit(a, 0), c0, w);
    }
    float acc[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) acc[b] = 0.f;
    for (int v = 0; v < nv; ++v) {
      const G16Unit u = g16_unit(a, v);
      g16_load_codes<KC>(a, g16_unit(a, v + 2 < nv ? v + 2 : nv - 1), c2);
      if (restage && u.pc == 0 && u.blk % a.xchunk == 0) {
        g16_lds_barrier();                             // every wave is done with the previous chunk
        g16_stage_x<NB>(a, xs, b0, u.blk);
        g16_lds_barrier();
      }
      // dot products of unit v: x of the thread's 4 groups, each batch row, each plane below k
      const int jl = (u.blk % a.xchunk) * g16::kBlock + 4 * h;
      const int kc = a.k - u.pc * KC;                  // planes of this chunk that are used
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
#pragma unroll
        for (int b = 0; b < NB; ++b) {
          const uint4 xv = xs[b * xgroups + jl + jj];
          float s = acc[b];
#pragma unroll
          for (int m = 0; m < KC; ++m)
            if (m < kc) s = g16_dot<XDT>(xv, w[jj][m], s);
          acc[b] = s;
        }
      }
      // the next unit's gathers: its code words arrived before this unit's codewords
      g16_gather<KC>(a, g16_unit(a, v + 1 < nv ? v + 1 : v), c1, w);
#pragma unroll
      for (int m = 0; m < KC; ++m) c1[m] = c2[m];
      if (u.blk == a.n_blocks - 1 && u.pc == a.n_pc - 1) {
        // the item's last unit: row sums over the 8 lanes of the row in this wave, then the waves
#pragma unroll
        for (int b = 0; b < NB; ++b) {
          float s = acc[b];
          s += __shfl_xor(s, 8);
          s += __shfl_xor(s, 16);
          s += __shfl_xor(s, 32);
          acc[b] = 0.f;
          if (lane < g16::kRows) red[parity][wave][lane][b] = s;
        }
        g16_lds_barrier();
        if (tid < g16::kRows * NB) {
          const int r = tid % g16::kRows, b = tid / g16::kRows;
          const int row = u.item * g16::kRows + r;
          if (row < a.d_out && b0 + b < a.batch) {
            float sum = 0.f;
#pragma unroll
            for (int w2 = 0; w2 < g16::kWaves; ++w2) sum += red[parity][w2][r][b];
            const float val = sum * f16_to_f32(a.scales[row]);
            const size_t o = (size_t)(b0 + b) * a.d_out + row;
            if (a.y_dtype == AQMB_F16) OutT<AQMB_F16>::store(a.y, o, val);
            else if (a.y_dtype == AQMB_BF16) OutT<AQMB_BF16>::store(a.y, o, val);
            else OutT<AQMB_F32>::store(a.y, o, val);
          }
        }
        parity ^= 1;                                   // the next item writes the other half
      }
    }
  }
}

template <int KC, int NB, int XDT>
static hipError_t launch_g16(const Gemv16Args& a, int grid, size_t lds, hipStream_t st) {
  gemv_b16_kernel<KC, NB, XDT><<<grid, g16::kThreads, lds, st>>>(a);
  return hipGetLastError();
}

template <int NB, int XDT>
static hipError_t launch_g16_nb(const Gemv16Args& a, int grid, size_t lds, hipStream_t st) {
  switch (a.k < g16::kPlaneChunk ? a.k : g16::kPlaneChunk) {
    case 1: return launch_g16<1, NB, XDT>(a, grid, lds, st);
    case 2: return launch_g16<2, NB, XDT>(a, grid, lds, st);
    case 3: return launch_g16<3, NB, XDT>(a, grid, lds, st);
    default: return launch_g16<4, NB, XDT>(a, grid, lds, st);
  }
}

template <int XDT>
static hipError_t launch_g16_x(Gemv16Args a, int n_cu, hipStream_t st) {
  // batch tile: the whole batch when its x rows fit (a batch of 2..4 in a tile of 4, 5..16 in one
  // of 16), else tiles of 4 or 1; x chunk: the whole row when it fits, else one block
  const int nb = a.batch == 1 ? 1 : a.batch <= 4 ? 4 : 16;
  const size_t block_bytes = (size_t)g16::kBlock * 16;
  // x tile plus the static row sums (2 x 16 waves x 8 rows x tile floats) and a margin
  auto budget = [&](int t) { return g16::kLds - (size_t)2 * g16::kWaves * g16::kRows * t * 4 - 512; };
  auto lds_for = [&](int t, int chunk) { return (size_t)t * chunk * block_bytes; };
  int tile = nb, chunk = a.n_blocks;
  while (tile > 1 && lds_for(tile, chunk) > budget(tile)) tile = tile == 16 ? 4 : 1;
  if (lds_for(tile, chunk) > budget(tile)) chunk = (int)(budget(tile) / block_bytes);
  if (chunk >= a.n_blocks) chunk = a.n_blocks;
  a.xchunk = chunk;
  const int grid = a.n_items < n_cu ? a.n_items : n_cu;
  const size_t lds = lds_for(tile, chunk);
  if (tile == 1) return launch_g16_nb<1, XDT>(a, grid, lds, st);
  if (tile == 4) return launch_g16_nb<4, XDT>(a, grid, lds, st);
  return launch_g16_nb<16, XDT>(a, grid, lds, st);
}

hipError_t launch_gemv_b16(const Layer& L, int k, const void* x, aqmb_dtype x_dtype, int batch, void* y,
                           aqmb_dtype y_dtype, hipStream_t st) {
  Gemv16Args a{};
  a.codes = L.codes;
  a.codebooks = L.codebooks;
  a.scales = L.scales;
  a.x = (const uint16_t*)x;
  a.y = y;
  a.plane_bytes = L.plane_bytes;
  a.d_out = L.d.d_out;
  a.d_in = L.d.d_in;
  a.G = L.G;
  a.S = L.S;
  a.k = k;
  a.batch = batch;
  a.y_dtype = (int)y_dtype;
  a.n_items = (L.d.d_out + g16::kRows - 1) / g16::kRows;
  a.n_blocks = (L.G + g16::kBlock - 1) / g16::kBlock;
  a.n_pc = (k + g16::kPlaneChunk - 1) / g16::kPlaneChunk;
  const int n_cu = L.n_cu > 0 ? L.n_cu : 256;
  return x_dtype == AQMB_F16 ? launch_g16_x<AQMB_F16>(a, n_cu, st) : launch_g16_x<AQMB_BF16>(a, n_cu, st);
}

}  // namespace aqmb
