// Decode GEMV of layers with 8-bit codes (256-codeword codebooks):
//   y[b][i] = s_i * sum_j sum_{m<k} <x[b, group j], C_m[code(m,i,j)]>
// (section 5: the partial reconstruction from the first k codebooks, applied as a product).
//
// Direct gathers (gemv_cw_kernel and its persistent and multi-layer forms, the default at batch 1):
// the codebooks are replicated in LDS and every code costs one 16-byte codeword read and its dot
// product with x, accumulated per row; no partial sums leave the workgroup.
//
// Lookup tables (gemv_lut_kernel + gemv_reduce_kernel, chosen explicitly): a workgroup owns a
// chunk of rows and one slice (16 consecutive groups); for the slice's groups and every used plane
// m, LUT_m[j][c] = <x[b, group j], C_m[c]> is built once per workgroup (one codeword per thread,
// fp32 dot products of exact fp16 products), then every code byte costs one LDS read and one fp32
// add. Rows map to threads, so each thread's accumulators need no cross-lane reduction. Every
// row's sum over slices is a split-K reduction: each workgroup writes fp32 partial sums for its
// rows to caller-provided scratch and a second, small kernel adds the partials of all slices in
// slice order, applies the row scale and rounds once to the output dtype. The kernel boundary
// orders the two phases, and the result does not depend on scheduling.
//
// Code planes m >= k are never read.
#include "device.h"
#include "launch.h"

namespace aqmb {

constexpr int kThreads = 512;       // 8 waves: two per SIMD
constexpr int kRowsPerThread = 1;
constexpr int kRowsPerWG = kThreads * kRowsPerThread;
constexpr int kReduceThreads = 256;

// vmcnt(0) only (expcnt and lgkmcnt left at their maxima), gfx9 encoding.
#define AQMB_GEMV_WAIT_VMCNT0() __builtin_amdgcn_s_waitcnt(0x70 | 0xF00)

struct GemvArgs {
  const unsigned char* codes;
  const uint16_t* codebooks;
  const uint16_t* scales;
  const void* x;
  void* y;
  float* partials;     // [S][batch][d_out] (lookup-table kernel: caller's scratch)
  const void* zero_page;  // 1 KiB of zeros, never written
  size_t plane_bytes;
  int d_out, d_in, G, S, k, batch;
  int y_dtype;
  int nrep;            // codebook replicas in LDS (direct-gather kernel), a power of two
  int cb_shift;        // log2(nrep * 16): byte shift from a code to its codeword
  int n_cu;            // compute units (host side: the persistent grid)
};

size_t gemv_lut_scratch_bytes(const Layer& L, int batch) {
  return (size_t)L.S * batch * L.d.d_out * sizeof(float);   // [S][batch][d_out] partial sums
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

// Direct-gather GEMV for 8-bit codes: one kernel, no partial sums. A workgroup of 1024 threads
// owns 16 rows; the 64 threads of a row split its groups (thread `part` takes groups
// 512 u + 8 part .. + 7 for u = 0 .. UB - 1), gather each code's codeword from the codebooks held
// in LDS and accumulate <x_group, codeword> in fp32 (dot products of exact fp16 products).
// A row's 64 partial sums are added in a fixed order (two shuffles, then the 16 waves through
// LDS), so results are reproducible.
// The codebooks are stored nrep times in LDS, interleaved so that codeword c of replica r sits
// at (c * nrep + r) * 16 bytes: lane l reads replica l % nrep, which spreads the random 16-byte
// reads of a wave over nrep bank groups instead of colliding at random.
// x is staged in LDS once per batch tile of NB rows by direct global->LDS loads, each row padded
// with zeros (read from the layer's zero page) up to the padded group
// count, so the group loops need no bounds tests: padding groups have code 0 and x = 0.
// Issue order: x, then the codebooks, then every code word the thread needs (all planes, all
// blocks, addresses clamped into the layer so that each thread issues the same loads). Code
// words are read once, with a streaming (nontemporal) hint that keeps them from evicting the
// codebooks and x, which every workgroup re-reads. Loads
// complete in order, so the codebook replication waits for the codebook only while the code
// planes stream in from HBM, and with one batch row the gather of plane m waits only for plane m.
namespace cw {
constexpr int kThreads = 1024, kRows = 16, kParts = 64, kWaves = kThreads / 64;
__host__ __device__ inline size_t row_stride(int S) {   // bytes per staged x row, whole KiB
  return ((size_t)S * 16 * 16 + 1023) / 1024 * 1024;
}
}

constexpr int kCwMaxBlocks = 4;   // 512-group blocks per row held in registers: d_in <= 16384

// Paired codebook layout of the batch-1 direct gathers (when it fits next to x): 64 KiB regions
// of 256 rows of 256 bytes; row c of region p holds 8 copies of C_2p[c] in its first 128 bytes and
// 8 copies of C_2p+1[c] in the second, and a plane without a partner (odd k) has a region of 16
// copies. A 16-byte LDS gather by 16 lanes is free of bank conflicts only when the lanes hit the
// 16 distinct 16-byte units of a 256-byte bank row; with 8 interleaved copies of one book lanes l
// and l + 8 share a copy and collide whenever their codewords have the same parity. Here each
// instruction of a pair's two gathers has lanes 0..7 in one half and lanes 8..15 in the other, each
// on its own copy: the 16 lanes cover the 16 units whatever the codes, in the LDS of 8 copies.
constexpr uint32_t kCwRegion = 256 * 256;

// LDS address of a codeword in the paired layout, one v_perm_b32: byte 1 is the code (byte j of the
// code word w: rows of 256 bytes), bytes 0, 2 and 3 come from `base` (the lane's 16-byte unit in the
// row, plus the LDS address of the region, a multiple of 64 KiB: the codebooks open the kernels'
// LDS, which holds no static variables, so their address is 0).
__device__ __forceinline__ uint32_t cw_pair_addr(uint32_t w, uint32_t base, int j) {
  return __builtin_amdgcn_perm(w, base, 0x03020000u | ((4u + (uint32_t)j) << 8));
}
__device__ __forceinline__ uint4 cw_lds_read16(uint32_t addr) {
  const u32x4_t v = *(const __attribute__((address_space(3))) u32x4_t*)(uintptr_t)addr;
  return make_uint4(v.x, v.y, v.z, v.w);
}

// <x group, codeword> of fp16 values added to s (a group's running sum over the planes).
__device__ __forceinline__ float group_dot_acc(uint4 xw, uint4 cw, float s) {
  s = dot2_f16(xw.x, cw.x, s);
  s = dot2_f16(xw.y, cw.y, s);
  s = dot2_f16(xw.z, cw.z, s);
  return dot2_f16(xw.w, cw.w, s);
}

// The gather-and-reduce part shared by the direct-gather kernels. For this thread's row and part,
// gather the codewords of its groups (code words in `code`: UB blocks x K planes, already
// requested), dot them with the NB staged x rows, reduce each row in a fixed order (a butterfly
// over the wave's parts, then the waves in order), scale by `scale` (the row's, loaded by the
// caller with the code words) and store y rows b0 .. b0 + NB - 1 (those below `batch`) of output
// row `row`. `red` is reused: the caller separates calls with a barrier.
// The staged x holds fp16 values: the input itself, or (XS) bf16 input converted by
// cw_convert_own_bf16 to x / scl[group] (scl rows of rstride / 16 floats). A group's dot products
// are chained over the planes into one partial sum (independent chains, one v_dot2 per code word
// pair), which is then added to the row's accumulator (XS: multiplied by the group's scale).
// `after_gathers` runs in each wave once its own gathers are done, before the row reduction's
// barrier (the multi-layer kernel writes the next layer's replicas there).
struct CwNothing {
  __device__ void operator()() const {}
};
// x of a thread's 8 groups (and, for bf16 x, their scales) held in registers by kernels that run
// several row blocks or layers on one x (one batch row, rows of one 512-group block), so that the
// staged x is read from LDS once per workgroup instead of once per block.
struct CwXReg {
  uint4 x[8];
  float s[8];
};
template <bool XS>
__device__ __forceinline__ void cw_load_xreg(const uint16_t* xs, const float* scl, int Gp, CwXReg& xr) {
  const int j0 = ((int)threadIdx.x >> 4) * 8;
  const bool ok = j0 < Gp;                                 // parts past the padded groups: never used
#pragma unroll
  for (int jj = 0; jj < 8; ++jj) xr.x[jj] = ok ? *(const uint4*)((const char*)xs + (size_t)(j0 + jj) * 16) : make_uint4(0, 0, 0, 0);
#pragma unroll
  for (int jj = 0; jj < 8; ++jj) xr.s[jj] = XS && ok ? scl[j0 + jj] : 0.f;
}
template <int K, int NB, int UB, bool XS, bool PL, bool XR = false, typename After = CwNothing>
__device__ __forceinline__ void cw_tile(const uint2 (&code)[UB][K], const uint4* cb_rep, const uint16_t* xs,
                                        size_t rstride, int Gp, int cb_shift, uint32_t rep_off,
                                        float (&red)[cw::kWaves][cw::kRows][NB], int b0, int batch, int row,
                                        bool row_ok, float scale, void* y, int d_out, int y_dtype,
                                        const float* scl, const CwXReg& xr, const After& after_gathers = After()) {
  static_assert(!XR || (NB == 1 && UB == 1), "x in registers: one batch row, one block per row");
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int rw = lane & 15, part = tid >> 4;
  const uint32_t cb_stride = 1u << cb_shift;
  static_assert(!PL || NB == 1, "the paired layout serves one batch row");
  float acc[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) acc[b] = 0.f;
#pragma unroll
  for (int u = 0; u < UB; ++u) {
    const int j0 = u * 512 + part * 8;
    if (j0 >= Gp) continue;                                // past the padded groups (short rows)
    const char* xrow = (const char*)xs + (size_t)j0 * 16;
    if constexpr (NB == 1) {
      // plane-major: x for the 8 groups in registers, 8 independent gathers per plane
      uint4 xg[8];
#pragma unroll
      for (int jj = 0; jj < 8; ++jj) xg[jj] = XR ? xr.x[jj] : *(const uint4*)(xrow + jj * 16);
      float t[8];                                          // per-group sums over the planes
#pragma unroll
      for (int jj = 0; jj < 8; ++jj) t[jj] = 0.f;
      if constexpr (PL) {
        // paired layout: rows 0..7 of the block take plane 2p from their own copy in the first
        // half of the codeword's row and plane 2p + 1 from the second half, rows 8..15 the other
        // way round in each instruction; a group's sum adds the pair in the order of its first
        // instruction (fixed per row, so results are reproducible)
        const bool upper = (lane & 8) != 0;
        const uint32_t r8 = (uint32_t)(lane & 7) * 16 + (upper ? 128u : 0u);
#pragma unroll
        for (int pp = 0; pp < K / 2; ++pp) {
          uint2 ca = code[u][2 * pp], cb = code[u][2 * pp + 1];
          asm volatile("" : "+v"(ca), "+v"(cb));
          const uint2 w0 = upper ? cb : ca, w1 = upper ? ca : cb;
          const uint32_t rb = lds_addr(cb_rep) + ((uint32_t)pp << 16);   // region base (low 16 bits zero)
          const uint32_t b0 = r8 | rb, b1 = (r8 ^ 128u) | rb;
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {                 // four groups at a time: 8 gathers in flight
            uint4 g0[4], g1[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              g0[q] = cw_lds_read16(cw_pair_addr(hh ? w0.y : w0.x, b0, q));
              g1[q] = cw_lds_read16(cw_pair_addr(hh ? w1.y : w1.x, b1, q));
            }
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              t[4 * hh + q] = group_dot_acc(xg[4 * hh + q], g0[q], t[4 * hh + q]);
              t[4 * hh + q] = group_dot_acc(xg[4 * hh + q], g1[q], t[4 * hh + q]);
            }
          }
        }
        if constexpr (K & 1) {                             // the plane without a partner: 16 copies
          uint2 cm = code[u][K - 1];
          asm volatile("" : "+v"(cm));
          const uint32_t bl = (uint32_t)(lane & 15) * 16 | (lds_addr(cb_rep) + ((uint32_t)(K / 2) << 16));
          uint4 g[8];
#pragma unroll
          for (int jj = 0; jj < 8; ++jj) g[jj] = cw_lds_read16(cw_pair_addr(jj < 4 ? cm.x : cm.y, bl, jj & 3));
#pragma unroll
          for (int jj = 0; jj < 8; ++jj) t[jj] = group_dot_acc(xg[jj], g[jj], t[jj]);
        }
      } else {
        // the same order of planes per group as the paired layout (rows 8..15 of the block take
        // each complete pair in the other order), so both layouts give identical results
        const bool upper = (lane & 8) != 0;
#pragma unroll
      for (int m = 0; m < K; ++m) {
        // plane m's code word is awaited here, not earlier (the empty asm keeps its unpacking
        // from being hoisted above the gathers of the previous planes)
        const bool sw = upper && m < 2 * (K / 2);
        uint2 cm = code[u][m];
        if (m < 2 * (K / 2)) {                             // a complete pair (known after unrolling)
          uint2 co = code[u][m ^ 1];
          asm volatile("" : "+v"(cm), "+v"(co));           // values, so that the pick is a select of registers
          cm = upper ? co : cm;
        } else {
          asm volatile("" : "+v"(cm));
        }
        const uint32_t base = (uint32_t)((sw ? m ^ 1 : m) * 256) * cb_stride + rep_off;
        uint4 cw[8];
#pragma unroll
        for (int jj = 0; jj < 8; ++jj) {
          const uint32_t word = jj < 4 ? cm.x : cm.y;
          const uint32_t c = (word >> (8 * (jj & 3))) & 0xFFu;
          cw[jj] = *(const uint4*)((const char*)cb_rep + (c << cb_shift) + base);
        }
#pragma unroll
        for (int jj = 0; jj < 8; ++jj) t[jj] = group_dot_acc(xg[jj], cw[jj], t[jj]);
      }
      }
      if constexpr (XS) {                                  // the group scales, read once the sums are done
        float xsc[8];
        if constexpr (XR) {
#pragma unroll
          for (int jj = 0; jj < 8; ++jj) xsc[jj] = xr.s[jj];
        } else {
          const float4 s0 = *(const float4*)(scl + j0), s1 = *(const float4*)(scl + j0 + 4);
          xsc[0] = s0.x; xsc[1] = s0.y; xsc[2] = s0.z; xsc[3] = s0.w;
          xsc[4] = s1.x; xsc[5] = s1.y; xsc[6] = s1.z; xsc[7] = s1.w;
        }
#pragma unroll
        for (int jj = 0; jj < 8; ++jj) acc[0] = __builtin_fmaf(t[jj], xsc[jj], acc[0]);
      } else {
#pragma unroll
        for (int jj = 0; jj < 8; ++jj) acc[0] += t[jj];
      }
    } else {
      // group-major: the NB x vectors of a group are read once and used for every plane
#pragma unroll
      for (int jj = 0; jj < 8; ++jj) {
        uint4 xg[NB];
        float t[NB], xsc[NB];
#pragma unroll
        for (int b = 0; b < NB; ++b) {
          xg[b] = *(const uint4*)(xrow + b * rstride + jj * 16);
          if constexpr (XS) xsc[b] = scl[(size_t)b * (rstride / 16) + j0 + jj];
          t[b] = 0.f;
        }
#pragma unroll
        for (int m = 0; m < K; ++m) {
          const uint32_t word = jj < 4 ? code[u][m].x : code[u][m].y;
          const uint32_t c = (word >> (8 * (jj & 3))) & 0xFFu;
          const uint4 cwv = *(const uint4*)((const char*)cb_rep + (c << cb_shift) + (uint32_t)(m * 256) * cb_stride + rep_off);
#pragma unroll
          for (int b = 0; b < NB; ++b) t[b] = group_dot_acc(xg[b], cwv, t[b]);
        }
#pragma unroll
        for (int b = 0; b < NB; ++b) {
          if constexpr (XS) acc[b] = __builtin_fmaf(t[b], xsc[b], acc[b]);
          else acc[b] += t[b];
        }
      }
    }
  }
  after_gathers();
  // row sum: lanes rw, rw + 16, rw + 32, rw + 48 of the wave, then the 16 waves in order
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    float v = acc[b];
    v += __shfl_xor(v, 16);
    v += __shfl_xor(v, 32);
    acc[b] = v;
  }
  if (lane < 16) {
#pragma unroll
    for (int b = 0; b < NB; ++b) red[wave][rw][b] = acc[b];
  }
  __syncthreads();
  if (wave == 0 && lane < 16 && row_ok) {
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      if (b0 + b < batch) {
        float sum = 0.f;
#pragma unroll
        for (int w = 0; w < cw::kWaves; ++w) sum += red[w][rw][b];
        const size_t o = (size_t)(b0 + b) * d_out + row;
        const float v = sum * scale;
        if (y_dtype == AQMB_F16) OutT<AQMB_F16>::store(y, o, v);
        else if (y_dtype == AQMB_BF16) OutT<AQMB_BF16>::store(y, o, v);
        else OutT<AQMB_F32>::store(y, o, v);
      }
    }
  }
}

// Write this thread's codebook word (codeword q = tid, q < K * 256) to its nrep replicas. Write i
// goes to replica (i + q / (16 / nrep)) % nrep: the 16 threads that share a 256-byte bank row
// write 16 distinct 16-byte slots of it, so the stores do not collide.
template <int K>
__device__ __forceinline__ void cw_replicate(uint4* cb_rep, uint4 cbv, int nrep, int cb_shift) {
  const int q = threadIdx.x;
  if (q < K * 256) {
    const int rot = q >> (8 - cb_shift);                   // q / (16 / nrep); cb_shift = log2(16 nrep)
    for (int i = 0; i < nrep; ++i) cb_rep[q * nrep + ((i + rot) & (nrep - 1))] = cbv;
  }
}

// The per-wave row sums of the direct-gather kernels sit in dynamic LDS after the x tile and its
// group scales (the codebooks stay at LDS address 0, where codeword offsets are addresses): `sets`
// buffers of kWaves x kRows x NB floats.
template <int NB, int SETS = 1>
__device__ __forceinline__ float (&cw_red(const float* scl, size_t rstride, bool bf16))[SETS][cw::kWaves][cw::kRows][NB] {
  char* p = (char*)scl + (bf16 ? (size_t)NB * rstride / 4 : 0);
  return *reinterpret_cast<float (*)[SETS][cw::kWaves][cw::kRows][NB]>(p);
}
__host__ __device__ inline size_t cw_red_bytes(int nb, int sets = 1) { return (size_t)sets * cw::kWaves * cw::kRows * nb * 4; }

// The codebook word that replication slot q (a thread, q < K * 256) loads for the paired layout:
// slots of a pair region alternate between its two planes, so that the 16 lanes of a write
// cover the 16 units of a row.
template <int K>
__device__ __forceinline__ int cw_pair_word(int q) {
  if (q < (K / 2) * 512) return (2 * (q >> 9) + (q & 1)) * 256 + ((q & 511) >> 1);
  return q;
}

// This thread's codebook word (slot q = tid) into the paired layout: 8 copies in its half of
// codeword c's row of a pair region, or 16 copies in the lone plane's region; write i of slot q
// goes to unit (i + c) % 8 of its half (% 16 for the lone plane), so no two of a write's 16 lanes
// share a bank.
template <int K>
__device__ __forceinline__ void cw_replicate_paired(uint4* cb_rep, uint4 v) {
  const int q = threadIdx.x;
  char* base = (char*)cb_rep;
  if (q < (K / 2) * 512) {
    const int c = (q & 511) >> 1, half = q & 1;
    char* row = base + (q >> 9) * kCwRegion + c * 256 + half * 128;
    for (int i = 0; i < 8; ++i) *(uint4*)(row + ((i + c) & 7) * 16) = v;
  } else if (q < K * 256) {
    const int c = q - (K / 2) * 512;
    char* row = base + (K / 2) * kCwRegion + c * 256;
    for (int i = 0; i < 16; ++i) *(uint4*)(row + ((i + c) & 15) * 16) = v;
  }
}

template <int K, bool PL>
__device__ __forceinline__ uint4 cw_first_word(const uint16_t* codebooks) {
  const int q = (int)threadIdx.x % (K * 256);              // K * 256 <= 1024 codewords
  return ((const uint4*)codebooks)[PL ? cw_pair_word<K>(q) : q];
}

template <int K, bool PL>
__device__ __forceinline__ void cw_replicate_any(uint4* cb_rep, uint4 cbv, int nrep, int cb_shift) {
  if constexpr (PL) cw_replicate_paired<K>(cb_rep, cbv);
  else cw_replicate<K>(cb_rep, cbv, nrep, cb_shift);
}

// uint4 words of LDS the replicated codebooks take.
template <int K, bool PL>
__device__ __forceinline__ int cw_rep_words(int nrep) {
  return PL ? ((K + 1) / 2) * (int)(kCwRegion / 16) : K * 256 * nrep;
}

// x rows b0 .. b0 + NB - 1 into LDS by direct loads; elements past d_in (and rows past `batch`)
// read zeros from the zero page.
template <int NB>
__device__ __forceinline__ void cw_stage_x(const void* x, const void* zero_page, int b0, int batch, int d_in,
                                           size_t rstride, uint32_t xs_base) {
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
  const int nch = (int)(rstride / 1024);
  for (int q = wave; q < NB * nch; q += cw::kWaves) {
    const int b = q / nch, ch = q % nch;
    const int e = ch * 512 + lane * 8;                     // element offset in the row
    const void* src = (b0 + b < batch && e < d_in) ? (const void*)((const uint16_t*)x + (size_t)(b0 + b) * d_in + e)
                                                   : zero_page;
    load_lds16(src, xs_base + (uint32_t)(b * rstride + (size_t)ch * 1024));
  }
}

// bf16 x -> fp16, one power-of-two scale per 8-value group: this thread converts in place the
// 16-byte groups its own cw_stage_x loads brought in (so no barrier is needed before it; the
// caller's barrier publishes the result) and writes the group's scale 2^e to scl. e puts the
// group's largest magnitude in [2^14, 2^15), where a bf16 value (8 significant bits) is exact in
// fp16; only values below 2^-29 of the group maximum fall in the fp16 subnormal range and are
// rounded, to a multiple of 2^-39 of it (far below the rounding of the fp32 sums). The fp16 dot
// products then apply and cw_tile multiplies each group's sum by its scale.
template <int NB>
__device__ __forceinline__ void cw_convert_own_bf16(uint16_t* xs, float* scl, size_t rstride) {
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
  const int nch = (int)(rstride / 1024);
  for (int q = wave; q < NB * nch; q += cw::kWaves) {
    const int b = q / nch, ch = q % nch;
    const int g = ch * 64 + lane;                          // group of the row (the one this lane loaded)
    char* p = (char*)xs + (size_t)b * rstride + (size_t)g * 16;
    const uint4 v = *(const uint4*)p;
    uint32_t w[4] = {v.x, v.y, v.z, v.w};
    uint32_t e = 0;                                        // largest exponent field (bf16 subnormals: 0)
#pragma unroll
    for (int h = 0; h < 4; ++h) e = max(e, max((w[h] >> 7) & 0xFFu, (w[h] >> 23) & 0xFFu));
    const int sh = (int)e - 141;                           // (e - 127) - 14
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      const _Float16 lo = (_Float16)ldexpf(bf16lo(w[h]), -sh);
      const _Float16 hi = (_Float16)ldexpf(bf16hi(w[h]), -sh);
      w[h] = (uint32_t)__builtin_bit_cast(uint16_t, lo) | ((uint32_t)__builtin_bit_cast(uint16_t, hi) << 16);
    }
    *(uint4*)p = make_uint4(w[0], w[1], w[2], w[3]);
    scl[(size_t)b * (rstride / 16) + g] = ldexpf(1.0f, sh);
  }
}

// An execution barrier between the workgroup's small loads (x, codebook words, row scales) and its
// code words: a CU's vector memory requests leave in order, so without it the waves that start
// last queue their codebook word behind the other waves' code words, which stream from HBM, and
// the codebook replication (which every gather waits for) waits for them. Measured on the
// 4096 x 4096 layer, batch 1: 6.2 to 5.5 us at k = 4.
__device__ __forceinline__ void cw_small_loads_first() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// This thread's code words (UB blocks x K planes) of row `rowc`: 8 groups per (block, plane),
// streaming loads, addresses clamped so that every thread issues the same loads.
template <int K, int UB>
__device__ __forceinline__ void cw_load_codes(uint2 (&code)[UB][K], const unsigned char* codes, size_t plane_bytes,
                                              int d_out, int rowc, int Gp) {
  const int part = threadIdx.x >> 4;
#pragma unroll
  for (int u = 0; u < UB; ++u) {
    int j0 = u * 512 + part * 8;
    j0 = j0 < Gp ? j0 : Gp - 8;                            // unused blocks reload a valid word
#pragma unroll
    for (int m = 0; m < K; ++m)
      code[u][m] = load_stream8(codes + m * plane_bytes + ((size_t)(j0 >> 4) * d_out + rowc) * 16 + (j0 & 8));
  }
}

template <int K, int NB, int XDT, int UB, bool PL>
__global__ __launch_bounds__(cw::kThreads) __attribute__((amdgpu_waves_per_eu(4, 4)))
void gemv_cw_kernel(GemvArgs a) {
  extern __shared__ uint4 smem_cw[];
  const int nrep = a.nrep;
  uint4* cb_rep = smem_cw;                               // [K][256][nrep] codewords, or PL regions
  uint16_t* xs = (uint16_t*)(cb_rep + cw_rep_words<K, PL>(nrep));   // [NB][row_stride] x tile
  constexpr bool kXS = XDT == AQMB_BF16;                   // bf16 x: converted to fp16 per group
  const int tid = threadIdx.x, lane = tid & 63;
  const int rw = lane & 15;
  const int row = blockIdx.x * cw::kRows + rw;
  const bool row_ok = row < a.d_out;
  const int rowc = row_ok ? row : a.d_out - 1;
  const int Gp = a.S * 16;                                 // padded groups per row
  const size_t rstride = cw::row_stride(a.S);
  const uint32_t xs_base = lds_addr(xs);
  const uint32_t rep_off = (uint32_t)(lane % nrep) * 16;

  cw_stage_x<NB>(a.x, a.zero_page, 0, a.batch, a.d_in, rstride, xs_base);
  asm volatile("" ::: "memory");
  const uint4 cbv = cw_first_word<K, PL>(a.codebooks);
  asm volatile("" ::: "memory");
  const uint16_t sbits = a.scales[rowc];                   // the row scale, needed only at the end
  cw_small_loads_first();
  uint2 code[UB][K];
  cw_load_codes<K, UB>(code, a.codes, a.plane_bytes, a.d_out, rowc, Gp);
  wait_vmcnt<UB * K + 1>();                                // x and the codebook word are in (older than the scale and codes)
  float* scl = (float*)((char*)xs + NB * rstride);         // bf16 x: [NB][rstride / 16] group scales
  float (&red)[cw::kWaves][cw::kRows][NB] = cw_red<NB>(scl, rstride, kXS)[0];   // per-wave row sums
  if constexpr (kXS) cw_convert_own_bf16<NB>(xs, scl, rstride);
  cw_replicate_any<K, PL>(cb_rep, cbv, nrep, a.cb_shift);
  __syncthreads();

  // The first batch tile is peeled out of the loop so that its waits for the code planes are exact.
  const float scale = f16_to_f32(sbits);
  CwXReg xr_unused;
  cw_tile<K, NB, UB, kXS, PL>(code, cb_rep, xs, rstride, Gp, a.cb_shift, rep_off, red, 0, a.batch, row, row_ok,
                              scale, a.y, a.d_out, a.y_dtype, scl, xr_unused);
  for (int b0 = NB; b0 < a.batch; b0 += NB) {
    __syncthreads();                                       // the previous tile's reads of xs are done
    cw_stage_x<NB>(a.x, a.zero_page, b0, a.batch, a.d_in, rstride, xs_base);
    wait_vmcnt<0>();
    if constexpr (kXS) cw_convert_own_bf16<NB>(xs, scl, rstride);
    __syncthreads();
    cw_tile<K, NB, UB, kXS, PL>(code, cb_rep, xs, rstride, Gp, a.cb_shift, rep_off, red, b0, a.batch, row, row_ok,
                                scale, a.y, a.d_out, a.y_dtype, scl, xr_unused);
  }
}

// Layers with more 16-row blocks than compute units (e.g. 11008 rows): one persistent workgroup
// per CU walks the row blocks blockIdx.x, blockIdx.x + gridDim.x, ... (rows of at most 512
// groups, one batch tile). x is staged and the codebooks replicated once; the code words of the
// next block are requested before the current block is gathered (two register sets in turn), so
// a block costs its gathers, not a workgroup's start-up, load latency and replica writes. Same
// arithmetic and reduction order as gemv_cw_kernel.
template <int K, int NB, int XDT, bool PL>
__global__ __launch_bounds__(cw::kThreads) __attribute__((amdgpu_waves_per_eu(4, 4)))
void gemv_cw_persist_kernel(GemvArgs a) {
  constexpr int UB = 1;
  extern __shared__ uint4 smem_cw[];
  const int nrep = a.nrep;
  uint4* cb_rep = smem_cw;                               // [K][256][nrep] codewords, or PL regions
  uint16_t* xs = (uint16_t*)(cb_rep + cw_rep_words<K, PL>(nrep));   // [NB][row_stride] x tile
  constexpr bool kXS = XDT == AQMB_BF16;                   // bf16 x: converted to fp16 per group
  const int tid = threadIdx.x, lane = tid & 63;
  const int rw = lane & 15;
  const int Gp = a.S * 16;
  const size_t rstride = cw::row_stride(a.S);
  const uint32_t xs_base = lds_addr(xs);
  const uint32_t rep_off = (uint32_t)(lane % nrep) * 16;
  const int n_rb = (a.d_out + cw::kRows - 1) / cw::kRows;
  float* scl = (float*)((char*)xs + NB * rstride);         // bf16 x: [NB][rstride / 16] group scales
  float (&red)[cw::kWaves][cw::kRows][NB] = cw_red<NB>(scl, rstride, kXS)[0];   // per-wave row sums

  CwXReg xr;                                               // batch 1: x of this thread's groups, for every block
  auto load_block = [&](int rb, uint32_t& sbits, uint2 (&code)[UB][K]) {
    const int row = rb * cw::kRows + rw;
    const int rowc = row < a.d_out ? row : a.d_out - 1;
    sbits = a.scales[rowc];
    cw_load_codes<K, UB>(code, a.codes, a.plane_bytes, a.d_out, rowc, Gp);
  };
  auto run_block = [&](int rb, uint32_t sbits, const uint2 (&code)[UB][K]) {
    const int row = rb * cw::kRows + rw;
    cw_tile<K, NB, UB, kXS, PL, NB == 1>(code, cb_rep, xs, rstride, Gp, a.cb_shift, rep_off, red, 0, a.batch, row,
                                         row < a.d_out, f16_to_f32((uint16_t)sbits), a.y, a.d_out, a.y_dtype, scl, xr);
  };

  int rb = blockIdx.x;                                     // the grid never exceeds the block count
  cw_stage_x<NB>(a.x, a.zero_page, 0, a.batch, a.d_in, rstride, xs_base);
  asm volatile("" ::: "memory");
  const uint4 cbv = cw_first_word<K, PL>(a.codebooks);
  asm volatile("" ::: "memory");
  uint32_t sa, sb;
  uint2 ca[UB][K], cb[UB][K];
  cw_small_loads_first();
  load_block(rb, sa, ca);
  wait_vmcnt<UB * K + 1>();                                // x and the codebook word are in
  if constexpr (kXS) cw_convert_own_bf16<NB>(xs, scl, rstride);
  cw_replicate_any<K, PL>(cb_rep, cbv, nrep, a.cb_shift);
  __syncthreads();
  if constexpr (NB == 1) cw_load_xreg<kXS>(xs, scl, Gp, xr);
  for (;;) {
    int nrb = rb + (int)gridDim.x;
    load_block(nrb < n_rb ? nrb : rb, sb, cb);            // past the last block: a harmless reload
    run_block(rb, sa, ca);
    if (nrb >= n_rb) break;
    rb = nrb;
    __syncthreads();                                       // wave 0 has read the previous row sums
    nrb = rb + (int)gridDim.x;
    load_block(nrb < n_rb ? nrb : rb, sa, ca);
    run_block(rb, sb, cb);
    if (nrb >= n_rb) break;
    rb = nrb;
    __syncthreads();
  }
}

// ------------------------------------------------------------------ several layers, one launch
// Layers that share the input x (fused projections such as q/k/v or gate/up): one persistent
// workgroup per 16-row block walks through the layers that have that block. x is staged once;
// the replicas of the next layer's codebooks are written right after the reduction barrier of
// the current one (every wave has finished its gathers by then; wave 0 still reads only the row
// sums), and one more barrier publishes them;
// while a layer's codewords are gathered, the codebook word and code words of the next layer are
// already on their way (two register sets used in turn), so a layer costs its gathers and the
// replica writes of its codebooks, not a launch and the load latency. Results are those of one
// aqmb_gemv call per layer (same arithmetic, same reduction order).
struct GemvMultiLayer {
  const unsigned char* codes;
  const uint16_t* codebooks;
  const uint16_t* scales;
  void* y;
  size_t plane_bytes;
  int d_out;
  int row_blocks;                                          // ceil(d_out / 16)
};

struct GemvMultiArgs {
  GemvMultiLayer L[AQMB_MAX_MULTI];
  const void* x;
  const void* zero_page;
  int n_layers, d_in, S, batch, y_dtype, nrep, cb_shift;
};

template <int K, int NB, int XDT, int UB, bool DB, bool PL>
__global__ __launch_bounds__(cw::kThreads) __attribute__((amdgpu_waves_per_eu(4, 4)))
void gemv_cw_multi_kernel(GemvMultiArgs a) {
  extern __shared__ uint4 smem_cw[];
  const int nrep = a.nrep;
  // DB: two replica sets (and two row-sum buffers) in turn. Each wave writes the next layer's
  // replicas into the idle set as soon as its own gathers of the current layer are done; the
  // row reduction's barrier then separates those writes from the next layer's gathers, and no
  // barrier of its own is needed. A set (or buffer) is written again two layers later, after a
  // barrier that every wave reaches only once it has finished reading it.
  const int rep_words = cw_rep_words<K, PL>(nrep);
  uint4* rep[2] = {smem_cw, smem_cw + (DB ? rep_words : 0)};
  uint16_t* xs = (uint16_t*)(smem_cw + (DB ? 2 : 1) * rep_words);
  const int tid = threadIdx.x, lane = tid & 63;
  const int rw = lane & 15;
  const int row = blockIdx.x * cw::kRows + rw;
  const int Gp = a.S * 16;
  const size_t rstride = cw::row_stride(a.S);
  const uint32_t xs_base = lds_addr(xs);
  const uint32_t rep_off = (uint32_t)(lane % nrep) * 16;
  // next layer (after l) that has this workgroup's row block, or -1 (uniform)
  auto next_layer = [&](int l) {
    for (int j = l + 1; j < a.n_layers; ++j)
      if ((int)blockIdx.x < a.L[j].row_blocks) return j;
    return -1;
  };
  // the layer's codebook word (first) and row scale; its code words
  auto load_small = [&](int l, uint4& cbv, uint32_t& sbits) {
    cbv = cw_first_word<K, PL>(a.L[l].codebooks);
    asm volatile("" ::: "memory");                        // the codebook word goes out first
    const int d_out = a.L[l].d_out;
    sbits = a.L[l].scales[row < d_out ? row : d_out - 1];
  };
  auto load_codes = [&](int l, uint2 (&code)[UB][K]) {
    const int d_out = a.L[l].d_out;
    cw_load_codes<K, UB>(code, a.L[l].codes, a.L[l].plane_bytes, d_out, row < d_out ? row : d_out - 1, Gp);
  };
  // the layer's codebook word (first), row scale and code words
  auto load_layer = [&](int l, uint4& cbv, uint32_t& sbits, uint2 (&code)[UB][K]) {
    load_small(l, cbv, sbits);
    load_codes(l, code);
  };
  constexpr bool kXS = XDT == AQMB_BF16;                   // bf16 x: converted to fp16 per group, once
  float* scl = (float*)((char*)xs + NB * rstride);         // [NB][rstride / 16] group scales
  float (&red)[DB ? 2 : 1][cw::kWaves][cw::kRows][NB] = cw_red<NB, DB ? 2 : 1>(scl, rstride, kXS);   // row sums
  int buf = 0;                                             // the replica set and row-sum buffer in use
  // batch 1: x of this thread's groups in registers for every layer (not with bf16 x at k = 2 in
  // two paired replica sets, where they would not fit)
  constexpr bool kXR = NB == 1 && UB == 1 && !(XDT == AQMB_BF16 && K == 2 && DB && PL);
  CwXReg xr;
  // layer l from replica set `buf`; with DB and a next layer, its replicas (word cbn) go to the
  // other set once this wave's gathers are done
  auto run_layer = [&](int l, uint32_t sbits, const uint2 (&code)[UB][K], bool next, const uint4& cbn) {
    const int d_out = a.L[l].d_out;
    auto after = [&]() {
      if constexpr (DB) {
        if (next) {
          wait_vmcnt<UB * K + 1>();                        // the next codebook word is in
          cw_replicate_any<K, PL>(rep[buf ^ 1], cbn, nrep, a.cb_shift);
        }
      }
    };
    cw_tile<K, NB, UB, kXS, PL, kXR>(code, rep[buf], xs, rstride, Gp, a.cb_shift, rep_off,
                                                    red[DB ? buf : 0], 0, a.batch, row, row < d_out,
                                                    f16_to_f32((uint16_t)sbits), a.L[l].y, d_out, a.y_dtype, scl, xr,
                                                    after);
  };
  // after layer `cur` (its reduction barrier passed): make `nxt` current
  auto switch_to = [&](const uint4& cbn) {
    if constexpr (DB) {
      buf ^= 1;
    } else {
      wait_vmcnt<UB * K + 1>();                            // the next codebook word is in
      cw_replicate_any<K, PL>(rep[0], cbn, nrep, a.cb_shift);
      __syncthreads();
    }
  };

  int cur = next_layer(-1);                                // the grid never exceeds the largest layer
  cw_stage_x<NB>(a.x, a.zero_page, 0, a.batch, a.d_in, rstride, xs_base);
  asm volatile("" ::: "memory");
  uint4 cba, cbb;
  uint32_t sa, sb;
  uint2 ca[UB][K], cb[UB][K];
  load_small(cur, cba, sa);
  cw_small_loads_first();
  load_codes(cur, ca);
  wait_vmcnt<UB * K + 1>();                                // x and the codebook word are in
  if constexpr (kXS) cw_convert_own_bf16<NB>(xs, scl, rstride);
  cw_replicate_any<K, PL>(rep[0], cba, nrep, a.cb_shift);
  __syncthreads();
  if constexpr (kXR) cw_load_xreg<kXS>(xs, scl, Gp, xr);
  for (;;) {
    int nxt = next_layer(cur);
    load_layer(nxt >= 0 ? nxt : cur, cbb, sb, cb);         // without a next layer: a harmless reload
    run_layer(cur, sa, ca, nxt >= 0, cbb);                 // its reduction barrier: all gathers done
    if (nxt < 0) break;
    switch_to(cbb);
    cur = nxt;
    nxt = next_layer(cur);
    load_layer(nxt >= 0 ? nxt : cur, cba, sa, ca);
    run_layer(cur, sb, cb, nxt >= 0, cba);
    if (nxt < 0) break;
    switch_to(cba);
    cur = nxt;
  }
}

// LDS bytes of the direct-gather kernel: replicated codebooks plus the x tile (plus one float
// per staged group for bf16 x).
static size_t cw_lds(int K, int nb, int S, int nrep, bool bf16) {
  const size_t xt = (size_t)nb * cw::row_stride(S);
  return (size_t)K * 256 * nrep * 16 + xt + (bf16 ? xt / 4 : 0);
}

// Replicas per codebook: as many as fit next to the x tile (LDS holds 160 KiB per workgroup).
// Sixteen (allowed by the caller) let every 16 lanes of a wave gather without bank conflicts (a
// codeword's 16 copies span the 64 banks): half the LDS cycles of eight copies per gather, for
// twice the replica writes; they fit for k <= 2.
static int cw_nrep(int K, int nb, int S, bool bf16, bool allow16 = false) {
  const size_t budget = 160 * 1024 - (size_t)cw::kWaves * cw::kRows * 4 * nb - 512;  // minus the row sums
  if (allow16 && cw_lds(K, nb, S, 16, bf16) <= budget) return 16;
  for (int r : {8, 4})
    if (cw_lds(K, nb, S, r, bf16) <= budget) return r;
  return 0;
}
static int cw_shift(int nrep) { return nrep == 16 ? 8 : nrep == 8 ? 7 : 6; }

// LDS bytes with the paired layout (batch 1): (k + 1) / 2 regions plus the x tile; `sets`
// replica sets (the multi-layer kernel's double buffering).
static size_t cw_lds_paired(int K, int S, bool bf16, int sets = 1) {
  const size_t xt = cw::row_stride(S);
  return (size_t)sets * ((K + 1) / 2) * kCwRegion + xt + (bf16 ? xt / 4 : 0);
}
static size_t cw_budget(int nb, int sets = 1) {   // LDS left next to the row sums
  return 160 * 1024 - (size_t)sets * cw::kWaves * cw::kRows * 4 * nb - 512;
}

static int cw_nb(int batch) { return batch == 1 ? 1 : batch == 2 ? 2 : 4; }
static int cw_blocks(int S) { return (S * 16 + 511) / 512; }

template <int K, int NB, int XDT>
static hipError_t launch_cw_nb(GemvArgs a, hipStream_t st) {
  const int n_rb = (a.d_out + cw::kRows - 1) / cw::kRows;
  // Sixteen replicas where a workgroup gathers at least two 512-group blocks (long rows, or a
  // persistent workgroup with two or more row blocks): there the halved gather cost repays the
  // extra replica writes (batch 1: 11008 x 4096, k = 1: 6.62 -> 5.95 us; 4096 x 11008, k = 2:
  // 7.98 -> 7.47 us; one block of 4096 x 4096 gains nothing).
  const bool many = cw_blocks(a.S) >= 2 || (a.n_cu > 0 && n_rb >= 2 * a.n_cu);
  a.nrep = cw_nrep(K, NB, a.S, XDT == AQMB_BF16, many);
  if (a.nrep == 0) return hipErrorInvalidValue;  // x tile does not fit: caller uses another path
  a.cb_shift = cw_shift(a.nrep);
  const dim3 grid(n_rb);
  const bool persist = cw_blocks(a.S) == 1 && a.batch <= NB && n_rb > a.n_cu && a.n_cu > 0;   // one workgroup per CU
  if constexpr (NB == 1) {
    // the paired layout from k = 3, and at k = 2 on rows of one 512-group block (where the
    // interleaved copies measured faster: 4096 x 11008, k = 2, 16 copies: 7.05 against 7.28 us;
    // paired elsewhere: 4096 x 4096, k = 3: 5.01 -> 4.70 us, k = 4: 5.70 -> 5.23 us; 11008 x
    // 4096, k = 4: 11.6 -> 10.9 us)
    const size_t lds = cw_lds_paired(K, a.S, XDT == AQMB_BF16);
    if ((K >= 3 || (K == 2 && cw_blocks(a.S) == 1)) && lds <= cw_budget(NB)) {
      if (persist) gemv_cw_persist_kernel<K, NB, XDT, true><<<dim3(a.n_cu), cw::kThreads, lds + cw_red_bytes(NB), st>>>(a);
      else if (cw_blocks(a.S) == 1) gemv_cw_kernel<K, NB, XDT, 1, true><<<grid, cw::kThreads, lds + cw_red_bytes(NB), st>>>(a);
      else gemv_cw_kernel<K, NB, XDT, kCwMaxBlocks, true><<<grid, cw::kThreads, lds + cw_red_bytes(NB), st>>>(a);
      return hipGetLastError();
    }
  }
  const size_t lds = cw_lds(K, NB, a.S, a.nrep, XDT == AQMB_BF16);
  if (persist) gemv_cw_persist_kernel<K, NB, XDT, false><<<dim3(a.n_cu), cw::kThreads, lds + cw_red_bytes(NB), st>>>(a);
  else if (cw_blocks(a.S) == 1) gemv_cw_kernel<K, NB, XDT, 1, false><<<grid, cw::kThreads, lds + cw_red_bytes(NB), st>>>(a);
  else gemv_cw_kernel<K, NB, XDT, kCwMaxBlocks, false><<<grid, cw::kThreads, lds + cw_red_bytes(NB), st>>>(a);
  return hipGetLastError();
}

template <int K, int XDT>
static hipError_t launch_cw(const GemvArgs& a, hipStream_t st) {
  if (a.batch == 1) return launch_cw_nb<K, 1, XDT>(a, st);
  if (a.batch == 2) return launch_cw_nb<K, 2, XDT>(a, st);
  return launch_cw_nb<K, 4, XDT>(a, st);         // batch 3..16: tiles of 4 rows
}

// The direct-gather kernel covers k <= 4 and d_in <= 16384 (the code words of a thread's
// groups stay in registers); the matrix-core and lookup-table kernels take the other shapes.
static bool cw_fits(int K, int batch, int S, bool bf16) {
  return K <= 4 && cw_blocks(S) <= kCwMaxBlocks && cw_nrep(K, cw_nb(batch), S, bf16) > 0;
}

bool gemv_cw_fits(const Layer& L, int k, int batch, aqmb_dtype x_dtype) {
  return L.d.code_bits == 8 && cw_fits(k, batch, L.S, x_dtype == AQMB_BF16);
}

template <int K, int XDT>
static void launch_lut(const GemvArgs& a, dim3 grid, hipStream_t st) {
  const size_t lds = (size_t)K * 16 * 256 * sizeof(float);  // K * JH * 256 * BT floats, JH * BT = 16
  if (a.batch == 1) gemv_lut_kernel<K, 1, XDT><<<grid, kThreads, lds, st>>>(a);
  else if (a.batch == 2) gemv_lut_kernel<K, 2, XDT><<<grid, kThreads, lds, st>>>(a);
  else gemv_lut_kernel<K, 4, XDT><<<grid, kThreads, lds, st>>>(a);
}

template <int XDT>
static hipError_t launch_cw_any(const GemvArgs& a, hipStream_t st) {
  switch (a.k) {
    case 1: return launch_cw<1, XDT>(a, st);
    case 2: return launch_cw<2, XDT>(a, st);
    case 3: return launch_cw<3, XDT>(a, st);
    case 4: return launch_cw<4, XDT>(a, st);
    default: return hipErrorInvalidValue;       // not reached: cw_fits requires k <= 4
  }
}

template <int XDT>
static void launch_lut_k(const GemvArgs& a, dim3 grid, hipStream_t st) {
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

static GemvArgs gemv_args(const Layer& L, int k, const void* x, int batch, void* y, aqmb_dtype y_dtype) {
  GemvArgs a{};
  a.codes = L.codes;
  a.codebooks = L.codebooks;
  a.scales = L.scales;
  a.x = x;
  a.y = y;
  a.zero_page = L.zero_page();
  a.partials = nullptr;
  a.plane_bytes = L.plane_bytes;
  a.d_out = L.d.d_out;
  a.d_in = L.d.d_in;
  a.G = L.G;
  a.S = L.S;
  a.k = k;
  a.batch = batch;
  a.y_dtype = (int)y_dtype;
  a.n_cu = L.n_cu;
  return a;
}

hipError_t launch_gemv_cw(const Layer& L, int k, const void* x, aqmb_dtype x_dtype, int batch, void* y,
                          aqmb_dtype y_dtype, hipStream_t st) {
  if (!gemv_cw_fits(L, k, batch, x_dtype)) return hipErrorInvalidValue;   // the caller checks first
  const GemvArgs a = gemv_args(L, k, x, batch, y, y_dtype);
  return x_dtype == AQMB_F16 ? launch_cw_any<AQMB_F16>(a, st) : launch_cw_any<AQMB_BF16>(a, st);
}

hipError_t launch_gemv_lut(const Layer& L, int k, const void* x, aqmb_dtype x_dtype, int batch, void* y,
                           aqmb_dtype y_dtype, float* scratch, hipStream_t st) {
  GemvArgs a = gemv_args(L, k, x, batch, y, y_dtype);
  a.partials = scratch;
  const dim3 grid((L.d.d_out + kRowsPerWG - 1) / kRowsPerWG, L.S);
  if (x_dtype == AQMB_F16) launch_lut_k<AQMB_F16>(a, grid, st);
  else launch_lut_k<AQMB_BF16>(a, grid, st);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int items = batch * ((L.d.d_out + 3) / 4);
  gemv_reduce_kernel<<<(items + 63) / 64, kReduceThreads, 0, st>>>(a);
  return hipGetLastError();
}

template <int K, int NB, int XDT>
static hipError_t launch_multi_nb(GemvMultiArgs a, int grid, hipStream_t st) {
  a.nrep = cw_nrep(K, NB, a.S, XDT == AQMB_BF16);
  a.cb_shift = cw_shift(a.nrep);
  const size_t lds = cw_lds(K, NB, a.S, a.nrep, XDT == AQMB_BF16);
  // two replica sets when they fit (k <= 2, one 512-group block, rows of at most 512 groups)
  const size_t lds2 = lds + (size_t)K * 256 * a.nrep * 16;
  const size_t budget = 160 * 1024 - (size_t)2 * cw::kWaves * cw::kRows * 4 * NB - 512;
  // the paired layout at even k, where it fits (16 layers of 4096 x 4096 per launch, k = 2:
  // 2.40 -> 2.11 us per layer, k = 4: 3.99 -> 3.75 us); at odd k the lone plane's 16 copies cost
  // more replica writes per layer than its conflict-free gathers save (k = 1: 1.62 -> 2.28 us;
  // k = 3: 3.15 -> 3.72 us). Both layouts give identical results.
  if constexpr (NB == 1 && K % 2 == 0) {
    const bool bf = XDT == AQMB_BF16;
    if constexpr (K <= 2) {
      const size_t p2 = cw_lds_paired(K, a.S, bf, 2);
      if (cw_blocks(a.S) == 1 && p2 <= cw_budget(NB, 2)) {
        gemv_cw_multi_kernel<K, NB, XDT, 1, true, true><<<grid, cw::kThreads, p2 + cw_red_bytes(NB, 2), st>>>(a);
        return hipGetLastError();
      }
    }
    const size_t p1 = cw_lds_paired(K, a.S, bf);
    if (p1 <= cw_budget(NB)) {
      if (cw_blocks(a.S) == 1) gemv_cw_multi_kernel<K, NB, XDT, 1, false, true><<<grid, cw::kThreads, p1 + cw_red_bytes(NB), st>>>(a);
      else gemv_cw_multi_kernel<K, NB, XDT, kCwMaxBlocks, false, true><<<grid, cw::kThreads, p1 + cw_red_bytes(NB), st>>>(a);
      return hipGetLastError();
    }
  }
  if constexpr (K <= 2) {
    if (cw_blocks(a.S) == 1 && lds2 <= budget) {
      gemv_cw_multi_kernel<K, NB, XDT, 1, true, false><<<grid, cw::kThreads, lds2 + cw_red_bytes(NB, 2), st>>>(a);
      return hipGetLastError();
    }
  }
  if (cw_blocks(a.S) == 1) {
    gemv_cw_multi_kernel<K, NB, XDT, 1, false, false><<<grid, cw::kThreads, lds + cw_red_bytes(NB), st>>>(a);
  } else {
    gemv_cw_multi_kernel<K, NB, XDT, kCwMaxBlocks, false, false><<<grid, cw::kThreads, lds + cw_red_bytes(NB), st>>>(a);
  }
  return hipGetLastError();
}

template <int K, int XDT>
static hipError_t launch_multi_k(const GemvMultiArgs& a, int grid, hipStream_t st) {
  if (a.batch == 1) return launch_multi_nb<K, 1, XDT>(a, grid, st);
  if (a.batch == 2) return launch_multi_nb<K, 2, XDT>(a, grid, st);
  return launch_multi_nb<K, 4, XDT>(a, grid, st);  // batch 3..4: one tile of 4 rows
}

template <int XDT>
static hipError_t launch_multi_x(const GemvMultiArgs& a, int k, int grid, hipStream_t st) {
  switch (k) {
    case 1: return launch_multi_k<1, XDT>(a, grid, st);
    case 2: return launch_multi_k<2, XDT>(a, grid, st);
    case 3: return launch_multi_k<3, XDT>(a, grid, st);
    default: return launch_multi_k<4, XDT>(a, grid, st);   // k <= 4 checked by the caller
  }
}

hipError_t launch_gemv_multi(const Layer* const* Ls, int n, int k, const void* x, aqmb_dtype x_dtype, int batch,
                             void* const* ys, aqmb_dtype y_dtype, hipStream_t st) {
  // One launch when every layer takes the direct-gather path in a single batch tile (8-bit codes,
  // k <= 4, batch <= 4) and, for rows of more than 512 groups, k = 1 (two layers' code words for
  // several blocks do not fit in registers beyond one plane); otherwise the layers are launched
  // one after another.
  const Layer& L0 = *Ls[0];
  bool one = batch <= 4 && cw_fits(k, batch, L0.S, x_dtype == AQMB_BF16) && (cw_blocks(L0.S) == 1 || k == 1);
  for (int i = 0; i < n && one; ++i) one = Ls[i]->d.code_bits == 8;
  if (!one) {
    for (int i = 0; i < n; ++i) {
      hipError_t e = launch_gemv_cw(*Ls[i], k, x, x_dtype, batch, ys[i], y_dtype, st);
      if (e != hipSuccess) return e;
    }
    return hipSuccess;
  }
  GemvMultiArgs a{};
  int grid = 0;
  for (int i = 0; i < n; ++i) {
    const Layer& L = *Ls[i];
    a.L[i].codes = L.codes;
    a.L[i].codebooks = L.codebooks;
    a.L[i].scales = L.scales;
    a.L[i].y = ys[i];
    a.L[i].plane_bytes = L.plane_bytes;
    a.L[i].d_out = L.d.d_out;
    a.L[i].row_blocks = (L.d.d_out + cw::kRows - 1) / cw::kRows;
    grid = a.L[i].row_blocks > grid ? a.L[i].row_blocks : grid;
  }
  a.x = x;
  a.zero_page = L0.zero_page();
  a.n_layers = n;
  a.d_in = L0.d.d_in;
  a.S = L0.S;
  a.batch = batch;
  a.y_dtype = (int)y_dtype;
  return x_dtype == AQMB_F16 ? launch_multi_x<AQMB_F16>(a, k, grid, st) : launch_multi_x<AQMB_BF16>(a, k, grid, st);
}

}  // namespace aqmb
