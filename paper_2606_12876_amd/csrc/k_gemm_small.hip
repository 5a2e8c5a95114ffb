// Prefill GEMM for small token counts (8- and 4-bit codes): Y[n][i] = s_i sum_t X[n][t] Wb_k[i][t], with
// Wb_k = RNE_bf16(binary32 left fold of C_m[b_{ijm}] over m < k), bf16 matrix cores, fp32 sums:
// the arithmetic of the large-tile GEMM, on a tiling that keeps every CU busy when n is small.
//
// A workgroup of 8 waves owns 16 weight rows and one pass of up to 16 NA tokens (grid: row blocks
// x passes). The waves take interleaved runs of four K-steps of 32 inputs (a run is the 16 groups
// of one code slice: one 16-byte load per plane). In a K-step lane l stands for weight row l % 16
// and group l / 16: it gathers that group's codeword of every plane from codebooks replicated in
// LDS, folds them in binary32 and rounds the sum to bf16: that is its B fragment of
// v_mfma_f32_16x16x32_bf16, used for the NA token blocks of the pass (A fragments straight from X:
// lane l holds 8 values of token l % 16 of the block; tokens past n read zeros). The 8 waves'
// partial tiles are added in wave order, scaled once and rounded once.
#include "device.h"
#include "launch.h"

namespace aqmb {

namespace gs {
constexpr int kThreads = 512, kWaves = 8, kRows = 16;
template <int K, int CB> struct Rep {                       // codebook replicas in LDS
  // 16-codeword codebooks fill the LDS banks once: one copy reads without conflicts
  static constexpr int kNrep = CB == 4 ? 1 : K <= 6 ? 4 : 2;
  static constexpr int kShift = kNrep == 4 ? 6 : kNrep == 2 ? 5 : 4;
};
typedef __bf16 b16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
}  // namespace gs

struct GemmSmallArgs {
  const unsigned char* codes;
  const uint16_t* codebooks;
  const uint16_t* scales;
  const uint16_t* X;          // [n][d_in] bf16
  void* Y;                    // [n][d_out]
  const void* zero_page;      // >= 16 zero bytes
  size_t plane_bytes;
  int d_out, d_in, G, n, y_dtype;
};

template <int K, int NA>
struct GsRun {
  uint4 xa[4][NA];
  uint4 c[K];
};

// CB = code bits (8: a run is one 16-byte slice; 4: a run is half a slice, 8 bytes).
template <int K, int NA, int CB>
__global__ __launch_bounds__(gs::kThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void gemm_small_kernel(GemmSmallArgs a) {
  using namespace gs;
  constexpr int kNrep = Rep<K, CB>::kNrep, kShift = Rep<K, CB>::kShift, NCW = 1 << CB;
  extern __shared__ uint4 smem_gs[];
  uint4* cb_rep = smem_gs;                                   // [K][NCW][kNrep] codewords
  f32x4_t* red = (f32x4_t*)(smem_gs + K * NCW * kNrep);      // [kWaves][NA][64] partial tiles
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int col = lane & 15, kc = lane >> 4;
  const int row0 = blockIdx.x * kRows;
  const int rowc = row0 + col < a.d_out ? row0 + col : a.d_out - 1;
  const int t0 = blockIdx.y * 16 * NA;                       // first token of the pass
  const int n_runs = (a.G + 15) / 16;                        // 16-group runs (4-bit slices hold two)
  const uint32_t rep_off = (uint32_t)(lane & (kNrep - 1)) * 16;

  // Loads of run r (past the end: the last run again, never used).
  auto load_run = [&](int r, GsRun<K, NA>& R) {
    const int rc = r < n_runs ? r : n_runs - 1;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int e = rc * 128 + j * 32 + kc * 8;
#pragma unroll
      for (int na = 0; na < NA; ++na) {
        const int t = t0 + na * 16 + col;
        const void* src = (t < a.n && e < a.d_in) ? (const void*)(a.X + (size_t)t * a.d_in + e) : a.zero_page;
        R.xa[j][na] = *(const uint4*)src;
      }
    }
#pragma unroll
    for (int m = 0; m < K; ++m) {
      if constexpr (CB == 8) {
        R.c[m] = load_stream16(a.codes + m * a.plane_bytes + ((size_t)rc * a.d_out + rowc) * 16);
      } else {                                               // groups 16 rc .. + 15: half of slice rc / 2
        const uint2 h = load_stream8(a.codes + m * a.plane_bytes + ((size_t)(rc >> 1) * a.d_out + rowc) * 16 + (rc & 1) * 8);
        R.c[m] = make_uint4(h.x, h.y, 0u, 0u);
      }
    }
  };

  // When each thread replicates at most one codeword, that word is requested ahead of the runs
  // (a CU's requests leave in order and the replication waits for it), with an execution barrier
  // between every wave's codebook request and the code words.
  constexpr bool kPre = K * NCW <= kThreads;
  uint4 v0 = make_uint4(0, 0, 0, 0);
  if constexpr (kPre) {
    v0 = ((const uint4*)a.codebooks)[tid < K * NCW ? tid : 0];
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  }
  GsRun<K, NA> ra, rb;
  int r = wave;
  load_run(r, ra);
  load_run(r + kWaves, rb);
  for (int q = tid; q < K * NCW; q += kThreads) {
    const uint4 v = kPre ? v0 : ((const uint4*)a.codebooks)[q];
    const int rot = q >> (8 - kShift);
#pragma unroll
    for (int i = 0; i < kNrep; ++i) cb_rep[q * kNrep + ((i + rot) & (kNrep - 1))] = v;
  }
  __syncthreads();

  f32x4_t acc[NA];
#pragma unroll
  for (int na = 0; na < NA; ++na) acc[na] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  auto compute = [&](const GsRun<K, NA>& R) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      // the weight group: binary32 left fold of the k codewords, rounded once to bf16
      float w[8];
#pragma unroll
      for (int m = 0; m < K; ++m) {
        uint32_t code;
        if constexpr (CB == 8) {
          const uint32_t word = j == 0 ? R.c[m].x : j == 1 ? R.c[m].y : j == 2 ? R.c[m].z : R.c[m].w;
          code = (word >> (8 * kc)) & 0xFFu;
        } else {                                             // nibble 4 j + kc of the run's 8 bytes
          const uint32_t word = j < 2 ? R.c[m].x : R.c[m].y;
          code = (word >> (4 * (4 * (j & 1) + kc))) & 15u;
        }
        const uint4 cw = *(const uint4*)((const char*)cb_rep + (((uint32_t)(m * NCW) + code) << kShift) + rep_off);
        const uint32_t u[4] = {cw.x, cw.y, cw.z, cw.w};
#pragma unroll
        for (int h = 0; h < 4; ++h) {
          if (m == 0) {
            w[2 * h] = f16lo(u[h]);
            w[2 * h + 1] = f16hi(u[h]);
          } else {
            w[2 * h] = w[2 * h] + f16lo(u[h]);
            w[2 * h + 1] = w[2 * h + 1] + f16hi(u[h]);
          }
        }
      }
      gs::b16x8_t b;
#pragma unroll
      for (int t = 0; t < 8; ++t) b[t] = (__bf16)w[t];      // round to nearest even
#pragma unroll
      for (int na = 0; na < NA; ++na)
        acc[na] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(gs::b16x8_t, R.xa[j][na]), b, acc[na], 0, 0, 0);
    }
  };
  for (; r < n_runs; r += 2 * kWaves) {
    compute(ra);
    if (r + kWaves >= n_runs) break;
    if (r + 2 * kWaves < n_runs) load_run(r + 2 * kWaves, ra);
    compute(rb);
    if (r + 3 * kWaves < n_runs) load_run(r + 3 * kWaves, rb);
  }
  // Partial tiles in wave order; element e of lane l is token 4 (l / 16) + e of its block,
  // weight row l % 16. Wave w adds token blocks w, w + 8, ... over the 8 waves.
#pragma unroll
  for (int na = 0; na < NA; ++na) red[(wave * NA + na) * 64 + lane] = acc[na];
  __syncthreads();
  const int row = row0 + col;
  for (int na = wave; na < NA; na += kWaves) {
    f32x4_t sum = red[na * 64 + lane];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) sum += red[(w * NA + na) * 64 + lane];
    if (row < a.d_out) {
      const float scale = f16_to_f32(a.scales[row]);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int t = t0 + na * 16 + 4 * kc + e;
        if (t < a.n) {
          const size_t o = (size_t)t * a.d_out + row;
          const float v = sum[e] * scale;
          if (a.y_dtype == AQMB_BF16) OutT<AQMB_BF16>::store(a.Y, o, v);
          else OutT<AQMB_F32>::store(a.Y, o, v);
        }
      }
    }
  }
}

template <int K, int NA, int CB>
static hipError_t launch_small(const GemmSmallArgs& a, hipStream_t st) {
  const size_t lds = (size_t)K * (1 << CB) * 16 * gs::Rep<K, CB>::kNrep + (size_t)gs::kWaves * NA * 64 * 16;
  const dim3 grid((a.d_out + gs::kRows - 1) / gs::kRows, (a.n + 16 * NA - 1) / (16 * NA));
  gemm_small_kernel<K, NA, CB><<<grid, gs::kThreads, lds, st>>>(a);
  return hipGetLastError();
}

template <int K, int CB>
static hipError_t launch_small_cb(const GemmSmallArgs& a, hipStream_t st) {
  if (a.n <= 16) return launch_small<K, 1, CB>(a, st);
  if (a.n <= 32) return launch_small<K, 2, CB>(a, st);
  return launch_small<K, 4, CB>(a, st);
}

template <int K>
static hipError_t launch_small_k(const GemmSmallArgs& a, int code_bits, hipStream_t st) {
  return code_bits == 4 ? launch_small_cb<K, 4>(a, st) : launch_small_cb<K, 8>(a, st);
}

hipError_t launch_gemm_small(const Layer& L, int k, const void* X, int n_tokens, void* Y, aqmb_dtype y_dtype,
                             hipStream_t st) {
  GemmSmallArgs a{};
  a.codes = L.codes;
  a.codebooks = L.codebooks;
  a.scales = L.scales;
  a.X = (const uint16_t*)X;
  a.Y = Y;
  a.zero_page = L.zero_page();
  a.plane_bytes = L.plane_bytes;
  a.d_out = L.d.d_out;
  a.d_in = L.d.d_in;
  a.G = L.G;
  a.n = n_tokens;
  a.y_dtype = (int)y_dtype;
  const int cb = L.d.code_bits;
  switch (k) {
    case 1: return launch_small_k<1>(a, cb, st);
    case 2: return launch_small_k<2>(a, cb, st);
    case 3: return launch_small_k<3>(a, cb, st);
    case 4: return launch_small_k<4>(a, cb, st);
    case 5: return launch_small_k<5>(a, cb, st);
    case 6: return launch_small_k<6>(a, cb, st);
    case 7: return launch_small_k<7>(a, cb, st);
    default: return launch_small_k<8>(a, cb, st);
  }
}

}  // namespace aqmb
