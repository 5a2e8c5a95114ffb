// Code search by beam search (Appendix C, code optimisation; Alg. 1 updates the assignments b by
// beam search), for codebooks of 256 (8-bit codes) or 16 (4-bit codes) codewords: for every group
// (row i, group j) of a dense weight matrix, the tuple
// (c_0, ..., c_{k-1}) of codewords of codebooks 0..k-1 that minimises the group's squared error
// ||w - s_i sum_m C_m[c_m]||^2 is searched stage by stage, keeping the `beam` best partial tuples.
//
// Every decision is taken in binary32 in one stated order (the reference implements the same):
// S_m[c][t] = s_i * C_m[c][t] (two fp16 values: exact); the residual of a kept tuple is
// r = w - S_0[c_0] - S_1[c_1] - ... (each subtraction rounded); a candidate (kept tuple, c) at
// stage m has d_t = fl(r_t - S_m[c][t]) and error e = fl(...fl(fl(d_0 d_0) + fl(d_1 d_1)) ... +
// fl(d_7 d_7)), added left to right, no fused multiply-add. Candidates are ordered by e, equal e
// by the tuple (lexicographically); the `beam` first are kept, at the last stage the first one.
//
// One lane per group; a workgroup takes up to 256 consecutive groups of one row (one scale). The fp16 codebooks
// stay in LDS; for the stage being searched their scaled binary32 codewords are written to LDS
// and every lane reads codeword c at the same time (broadcast). Each lane keeps its beam as
// residuals in registers and the new beam as a sorted list of (e, key), key = (rank of the parent
// tuple among the kept tuples in lexicographic order) * 256 + c, which orders equal errors by
// the tuple. The kept tuples' residuals are rebuilt from their codes by the same subtraction
// chain, so they are bit-identical to the candidate's d.
#include "device.h"
#include "launch.h"

namespace aqmb {

namespace beam {
constexpr int kThreads = 256;
}  // namespace beam

struct BeamArgs {
  const uint16_t* W;          // [d_out][d_in] fp16
  const uint16_t* codebooks;  // [>= k][256][8] fp16
  const uint16_t* scales;     // [d_out] fp16
  unsigned char* codes;       // [k][d_out][G]
  float* errors;              // [d_out][G] or null
  int d_out, d_in, G, k;
};

namespace {

__device__ __forceinline__ bool before(float e, uint32_t key, float e2, uint32_t key2) {
  return e < e2 || (e == e2 && key < key2);
}

// Error of candidate codeword sc (scaled) against residual r, in the stated order.
__device__ __forceinline__ float cand_error(const float (&r)[8], const float4& s0, const float4& s1) {
#pragma clang fp contract(off)
  const float d0 = r[0] - s0.x, d1 = r[1] - s0.y, d2 = r[2] - s0.z, d3 = r[3] - s0.w;
  const float d4 = r[4] - s1.x, d5 = r[5] - s1.y, d6 = r[6] - s1.z, d7 = r[7] - s1.w;
  float e = d0 * d0;
  e = e + d1 * d1;
  e = e + d2 * d2;
  e = e + d3 * d3;
  e = e + d4 * d4;
  e = e + d5 * d5;
  e = e + d6 * d6;
  e = e + d7 * d7;
  return e;
}

// Insert (e, key) into the list (le, lk)[0..B-1], ascending by (e, key), dropping the last entry.
// Walking up from the end, each entry takes its upper neighbour while the new one belongs above
// it, then the new one; written as selects so that the list stays in registers.
template <int B>
__device__ __forceinline__ void insert(float (&le)[B], uint32_t (&lk)[B], float e, uint32_t key) {
  bool placed = false;
#pragma unroll
  for (int q = B - 1; q >= 0; --q) {
    const int up = q > 0 ? q - 1 : 0;
    const bool go_up = q > 0 && before(e, key, le[up], lk[up]);
    const float ne = placed ? le[q] : (go_up ? le[up] : e);
    const uint32_t nk = placed ? lk[q] : (go_up ? lk[up] : key);
    le[q] = ne;
    lk[q] = nk;
    placed = placed || !go_up;
  }
}

}  // namespace

// NCW = codewords per codebook (256 for 8-bit codes, 16 for 4-bit codes).
template <int B, int NCW>
__global__ __launch_bounds__(beam::kThreads) void beam_kernel(BeamArgs a) {
  __shared__ float4 sc[NCW][2];         // scaled codewords of the stage being searched
  extern __shared__ uint4 cb_dyn[];     // fp16 codebooks 0..k-1: [k][NCW] 16-byte codewords
  uint4 (*cb)[NCW] = (uint4 (*)[NCW])cb_dyn;
  const int n_chunks = (a.G + beam::kThreads - 1) / beam::kThreads;
  const int tid = threadIdx.x, i = blockIdx.x / n_chunks, j = (blockIdx.x % n_chunks) * beam::kThreads + tid;
  const bool ok = j < a.G;
  const int jc = ok ? j : a.G - 1;
  const float s = f16_to_f32(a.scales[i]);
  if (tid < NCW)
    for (int m = 0; m < a.k; ++m) cb[m][tid] = ((const uint4*)a.codebooks)[m * NCW + tid];

  float w[8];
  {
    const uint4 wr = *(const uint4*)(a.W + (size_t)i * a.d_in + (size_t)jc * 8);
    const uint32_t u[4] = {wr.x, wr.y, wr.z, wr.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      w[2 * q] = f16lo(u[q]);
      w[2 * q + 1] = f16hi(u[q]);
    }
  }
  // The kept tuples: residuals, codes (byte m = c_m), lexicographic ranks.
  float r[B][8];
  uint32_t lo[B], hi[B], rank[B];
#pragma unroll
  for (int p = 0; p < B; ++p) {
#pragma unroll
    for (int t = 0; t < 8; ++t) r[p][t] = w[t];
    lo[p] = hi[p] = rank[p] = 0;
  }
  int n_par = 1;                        // stage 0 extends the single empty tuple
  float best_e = 0.f;

  for (int m = 0; m < a.k; ++m) {
    __syncthreads();                    // codebooks written; previous stage done with sc
    if (tid < NCW) {
      const uint4 v = cb[m][tid];
      const uint32_t u[4] = {v.x, v.y, v.z, v.w};
      float x[8];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        x[2 * q] = s * f16lo(u[q]);     // exact: a product of two fp16 values
        x[2 * q + 1] = s * f16hi(u[q]);
      }
      sc[tid][0] = make_float4(x[0], x[1], x[2], x[3]);
      sc[tid][1] = make_float4(x[4], x[5], x[6], x[7]);
    }
    __syncthreads();
    const bool last = m == a.k - 1;
    float le[B];
    uint32_t lk[B];
#pragma unroll
    for (int q = 0; q < B; ++q) {
      le[q] = __builtin_inff();
      lk[q] = 0xFFFFFFFFu;
    }
    if (last) {
      // Only the best candidate is kept.
      for (int c = 0; c < NCW; ++c) {
        const float4 s0 = sc[c][0], s1 = sc[c][1];
#pragma unroll
        for (int p = 0; p < B; ++p) {
          if (p < n_par) {
            const float e = cand_error(r[p], s0, s1);
            const uint32_t key = (rank[p] << 8) | (uint32_t)c;
            const bool bt = before(e, key, le[0], lk[0]);
            le[0] = bt ? e : le[0];
            lk[0] = bt ? key : lk[0];
          }
        }
      }
    } else {
      for (int c = 0; c < NCW; ++c) {
        const float4 s0 = sc[c][0], s1 = sc[c][1];
#pragma unroll
        for (int p = 0; p < B; ++p) {
          if (p < n_par) {
            const float e = cand_error(r[p], s0, s1);
            const uint32_t key = (rank[p] << 8) | (uint32_t)c;
            if (before(e, key, le[B - 1], lk[B - 1])) insert<B>(le, lk, e, key);
          }
        }
      }
    }
    // New kept tuples: codes from the parent (the kept tuple whose rank is key >> 8) plus c.
    const int n_new = last ? 1 : B;
    uint32_t nlo[B], nhi[B], nrank[B];
#pragma unroll
    for (int q = 0; q < B; ++q) {
      const uint32_t pr = lk[q] >> 8, c = lk[q] & 0xFFu;
      uint32_t plo = 0, phi = 0;
#pragma unroll
      for (int p = 0; p < B; ++p)
      {
        const bool hit = rank[p] == pr && p < n_par;
        plo = hit ? lo[p] : plo;
        phi = hit ? hi[p] : phi;
      }
      if (m < 4) plo |= c << (8 * m); else phi |= c << (8 * (m - 4));
      nlo[q] = plo;
      nhi[q] = phi;
      uint32_t rk = 0;                  // rank among the new tuples: order of (parent rank, c) = key
#pragma unroll
      for (int q2 = 0; q2 < B; ++q2) rk += (q2 < n_new && lk[q2] < lk[q]) ? 1u : 0u;
      nrank[q] = rk;
    }
    best_e = le[0];
#pragma unroll
    for (int q = 0; q < B; ++q) {
      lo[q] = nlo[q];
      hi[q] = nhi[q];
      rank[q] = nrank[q];
    }
    n_par = n_new;
    if (!last) {
      // Residuals of the kept tuples, by the subtraction chain w - S_0[c_0] - ... - S_m[c_m].
#pragma unroll
      for (int q = 0; q < B; ++q) {
#pragma unroll
        for (int t = 0; t < 8; ++t) r[q][t] = w[t];
        for (int mm = 0; mm <= m; ++mm) {
          const uint32_t c = ((mm < 4 ? lo[q] : hi[q]) >> (8 * (mm & 3))) & 0xFFu;
          const uint4 v = cb[mm][c];
          const uint32_t u[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
          for (int h = 0; h < 4; ++h) {
#pragma clang fp contract(off)
            r[q][2 * h] = r[q][2 * h] - s * f16lo(u[h]);
            r[q][2 * h + 1] = r[q][2 * h + 1] - s * f16hi(u[h]);
          }
        }
      }
    }
  }
  if (ok) {
    const size_t plane = (size_t)a.d_out * a.G, o = (size_t)i * a.G + j;
    for (int m = 0; m < a.k; ++m)
      a.codes[m * plane + o] = (unsigned char)(((m < 4 ? lo[0] : hi[0]) >> (8 * (m & 3))) & 0xFFu);
    if (a.errors) a.errors[o] = best_e;
  }
}

// ------------------------------------------------------------------ data-aware objective
// The weighted search (the WMSE of §2.2 restricted to each group's diagonal block H = H_jj of
// X X^T / n, symmetric): the error of a candidate is d^T H d, d = w - s_i sum_m C_m[c_m]. With r
// the kept tuple's residual and C the unscaled candidate codeword it is evaluated in binary32 as
//   b_t = sum_u fl(H_tu r_u), A = sum_t fl(r_t b_t)                  (per kept tuple)
//   Q = sum_t fl(C_t q_t), q_t = sum_u fl(H_tu C_u)                  (per codeword)
//   T = sum_t fl(C_t b_t), e = fl(fl(A - fl(fl(2 s) T)) + fl(fl(s s) Q))   (per candidate)
// every sum left to right, no fused multiply-add (the reference implements the same order).
// H differs between groups and is shared by all rows, so a workgroup takes one group j of 256
// rows (one lane per row): H is uniform (scalar registers), Q is computed once per codeword and
// stage by the workgroup, and a candidate costs 8 products and 11 other operations, about what
// the squared error costs. Decisions, tie-breaks and residuals as in beam_kernel.
struct BeamWeightedArgs {
  const uint16_t* W;          // [d_out][d_in] fp16
  const uint16_t* codebooks;  // [>= k][NCW][8] fp16
  const uint16_t* scales;     // [d_out] fp16
  const float* H;             // [G][8][8] fp32, symmetric blocks
  unsigned char* codes;       // [k][d_out][G]
  float* errors;              // [d_out][G] or null
  int d_out, d_in, G, k;
};

namespace {
// fl(sum_u fl(h_u v_u)), u = 0..7 left to right
__device__ __forceinline__ float dot8(const float (&h)[8], const float (&v)[8]) {
#pragma clang fp contract(off)
  float acc = h[0] * v[0];
#pragma unroll
  for (int u = 1; u < 8; ++u) acc = acc + h[u] * v[u];
  return acc;
}
}  // namespace

template <int B, int NCW>
__global__ __launch_bounds__(beam::kThreads) void beam_weighted_kernel(BeamWeightedArgs a) {
#pragma clang fp contract(off)
  __shared__ float cwf[NCW][8];         // unscaled codewords of the stage being searched
  __shared__ float cq[NCW];             // their C^T H C
  extern __shared__ uint4 cb_dyn[];     // fp16 codebooks 0..k-1: [k][NCW] 16-byte codewords
  uint4 (*cb)[NCW] = (uint4 (*)[NCW])cb_dyn;
  const int n_rchunks = (a.d_out + beam::kThreads - 1) / beam::kThreads;
  const int tid = threadIdx.x;
  const int j = blockIdx.x / n_rchunks;                    // the group (uniform)
  const int i = (blockIdx.x % n_rchunks) * beam::kThreads + tid;
  const bool ok = i < a.d_out;
  const int ic = ok ? i : a.d_out - 1;
  float H[8][8];                                           // uniform: scalar loads
#pragma unroll
  for (int t = 0; t < 8; ++t)
#pragma unroll
    for (int u = 0; u < 8; ++u) H[t][u] = a.H[(size_t)j * 64 + t * 8 + u];
  const float s = f16_to_f32(a.scales[ic]);
  const float two_s = 2.0f * s, ss = s * s;                // exact for an fp16 scale
  if (tid < NCW)
    for (int m = 0; m < a.k; ++m) cb[m][tid] = ((const uint4*)a.codebooks)[m * NCW + tid];

  float w[8];
  {
    const uint4 wr = *(const uint4*)(a.W + (size_t)ic * a.d_in + (size_t)j * 8);
    const uint32_t u[4] = {wr.x, wr.y, wr.z, wr.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      w[2 * q] = f16lo(u[q]);
      w[2 * q + 1] = f16hi(u[q]);
    }
  }
  // The kept tuples: b = H r and A = r^T b of their residuals r, codes (byte m = c_m), ranks.
  float bv[B][8], A[B];
  uint32_t lo[B], hi[B], rank[B];
  auto set_parent = [&](int p, const float (&r)[8]) {
#pragma unroll
    for (int t = 0; t < 8; ++t) bv[p][t] = dot8(H[t], r);
    A[p] = dot8(r, bv[p]);
  };
#pragma unroll
  for (int p = 0; p < B; ++p) {
    set_parent(p, w);
    lo[p] = hi[p] = rank[p] = 0;
  }
  int n_par = 1;                        // stage 0 extends the single empty tuple
  float best_e = 0.f;

  for (int m = 0; m < a.k; ++m) {
    __syncthreads();                    // codebooks written; previous stage done with cwf, cq
    if (tid < NCW) {
      const uint4 v = cb[m][tid];
      const uint32_t u[4] = {v.x, v.y, v.z, v.w};
      float c[8];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        c[2 * q] = f16lo(u[q]);
        c[2 * q + 1] = f16hi(u[q]);
      }
      float hc[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        hc[t] = dot8(H[t], c);
        cwf[tid][t] = c[t];
      }
      cq[tid] = dot8(c, hc);
    }
    __syncthreads();
    const bool last = m == a.k - 1;
    float le[B];
    uint32_t lk[B];
#pragma unroll
    for (int q = 0; q < B; ++q) {
      le[q] = __builtin_inff();
      lk[q] = 0xFFFFFFFFu;
    }
    for (int c = 0; c < NCW; ++c) {
      float cv[8];
      const float4 c0 = *(const float4*)&cwf[c][0], c1 = *(const float4*)&cwf[c][4];
      cv[0] = c0.x; cv[1] = c0.y; cv[2] = c0.z; cv[3] = c0.w;
      cv[4] = c1.x; cv[5] = c1.y; cv[6] = c1.z; cv[7] = c1.w;
      const float sq = ss * cq[c];
#pragma unroll
      for (int p = 0; p < B; ++p) {
        if (p < n_par) {
          const float T = dot8(cv, bv[p]);
          const float e = (A[p] - two_s * T) + sq;
          const uint32_t key = (rank[p] << 8) | (uint32_t)c;
          if (last) {
            const bool bt = before(e, key, le[0], lk[0]);
            le[0] = bt ? e : le[0];
            lk[0] = bt ? key : lk[0];
          } else if (before(e, key, le[B - 1], lk[B - 1])) {
            insert<B>(le, lk, e, key);
          }
        }
      }
    }
    // New kept tuples: codes from the parent (the kept tuple whose rank is key >> 8) plus c.
    const int n_new = last ? 1 : B;
    uint32_t nlo[B], nhi[B], nrank[B];
#pragma unroll
    for (int q = 0; q < B; ++q) {
      const uint32_t pr = lk[q] >> 8, c = lk[q] & 0xFFu;
      uint32_t plo = 0, phi = 0;
#pragma unroll
      for (int p = 0; p < B; ++p) {
        const bool hit = rank[p] == pr && p < n_par;
        plo = hit ? lo[p] : plo;
        phi = hit ? hi[p] : phi;
      }
      if (m < 4) plo |= c << (8 * m); else phi |= c << (8 * (m - 4));
      nlo[q] = plo;
      nhi[q] = phi;
      uint32_t rk = 0;
#pragma unroll
      for (int q2 = 0; q2 < B; ++q2) rk += (q2 < n_new && lk[q2] < lk[q]) ? 1u : 0u;
      nrank[q] = rk;
    }
    best_e = le[0];
#pragma unroll
    for (int q = 0; q < B; ++q) {
      lo[q] = nlo[q];
      hi[q] = nhi[q];
      rank[q] = nrank[q];
    }
    n_par = n_new;
    if (!last) {
      // Residuals of the kept tuples by the subtraction chain w - S_0[c_0] - ... - S_m[c_m], then
      // their b = H r and A = r^T b.
#pragma unroll
      for (int q = 0; q < B; ++q) {
        float r[8];
#pragma unroll
        for (int t = 0; t < 8; ++t) r[t] = w[t];
        for (int mm = 0; mm <= m; ++mm) {
          const uint32_t c = ((mm < 4 ? lo[q] : hi[q]) >> (8 * (mm & 3))) & 0xFFu;
          const uint4 v = cb[mm][c];
          const uint32_t u[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
          for (int h = 0; h < 4; ++h) {
            r[2 * h] = r[2 * h] - s * f16lo(u[h]);
            r[2 * h + 1] = r[2 * h + 1] - s * f16hi(u[h]);
          }
        }
        set_parent(q, r);
      }
    }
  }
  if (ok) {
    const size_t plane = (size_t)a.d_out * a.G, o = (size_t)i * a.G + j;
    for (int m = 0; m < a.k; ++m)
      a.codes[m * plane + o] = (unsigned char)(((m < 4 ? lo[0] : hi[0]) >> (8 * (m & 3))) & 0xFFu);
    if (a.errors) a.errors[o] = best_e;
  }
}

template <int B>
static hipError_t launch_beam_weighted_b(const BeamWeightedArgs& a, int ncw, hipStream_t st) {
  const int grid = ((a.d_out + beam::kThreads - 1) / beam::kThreads) * a.G;   // validated below 2^31
  if (ncw == 16) beam_weighted_kernel<B, 16><<<grid, beam::kThreads, (size_t)a.k * 16 * 16, st>>>(a);
  else beam_weighted_kernel<B, 256><<<grid, beam::kThreads, (size_t)a.k * 256 * 16, st>>>(a);
  return hipGetLastError();
}

hipError_t launch_beam_search_weighted(const aqmb_desc& d, int k, int beam_width, const void* W,
                                       const uint16_t* codebooks, const uint16_t* scales, const float* H,
                                       unsigned char* codes, float* errors, hipStream_t st) {
  BeamWeightedArgs a{};
  a.W = (const uint16_t*)W;
  a.codebooks = codebooks;
  a.scales = scales;
  a.H = H;
  a.codes = codes;
  a.errors = errors;
  a.d_out = d.d_out;
  a.d_in = d.d_in;
  a.G = d.d_in / d.group_size;
  a.k = k;
  const int ncw = 1 << d.code_bits;
  switch (beam_width) {
    case 1: return launch_beam_weighted_b<1>(a, ncw, st);
    case 2: return launch_beam_weighted_b<2>(a, ncw, st);
    case 3: return launch_beam_weighted_b<3>(a, ncw, st);
    case 4: return launch_beam_weighted_b<4>(a, ncw, st);
    case 5: return launch_beam_weighted_b<5>(a, ncw, st);
    case 6: return launch_beam_weighted_b<6>(a, ncw, st);
    case 7: return launch_beam_weighted_b<7>(a, ncw, st);
    case 8: return launch_beam_weighted_b<8>(a, ncw, st);
    case 9: return launch_beam_weighted_b<9>(a, ncw, st);
    case 10: return launch_beam_weighted_b<10>(a, ncw, st);
    case 11: return launch_beam_weighted_b<11>(a, ncw, st);
    case 12: return launch_beam_weighted_b<12>(a, ncw, st);
    case 13: return launch_beam_weighted_b<13>(a, ncw, st);
    case 14: return launch_beam_weighted_b<14>(a, ncw, st);
    case 15: return launch_beam_weighted_b<15>(a, ncw, st);
    default: return launch_beam_weighted_b<16>(a, ncw, st);
  }
}

template <int B>
static hipError_t launch_beam_b(const BeamArgs& a, int ncw, hipStream_t st) {
  const int grid = ((a.G + beam::kThreads - 1) / beam::kThreads) * a.d_out;   // validated below 2^31
  if (ncw == 16) beam_kernel<B, 16><<<grid, beam::kThreads, (size_t)a.k * 16 * 16, st>>>(a);
  else beam_kernel<B, 256><<<grid, beam::kThreads, (size_t)a.k * 256 * 16, st>>>(a);
  return hipGetLastError();
}

hipError_t launch_beam_search(const aqmb_desc& d, int k, int beam_width, const void* W, const uint16_t* codebooks,
                              const uint16_t* scales, unsigned char* codes, float* errors, hipStream_t st) {
  BeamArgs a{};
  a.W = (const uint16_t*)W;
  a.codebooks = codebooks;
  a.scales = scales;
  a.codes = codes;
  a.errors = errors;
  a.d_out = d.d_out;
  a.d_in = d.d_in;
  a.G = d.d_in / d.group_size;
  a.k = k;
  const int ncw = 1 << d.code_bits;
  switch (beam_width) {
    case 1: return launch_beam_b<1>(a, ncw, st);
    case 2: return launch_beam_b<2>(a, ncw, st);
    case 3: return launch_beam_b<3>(a, ncw, st);
    case 4: return launch_beam_b<4>(a, ncw, st);
    case 5: return launch_beam_b<5>(a, ncw, st);
    case 6: return launch_beam_b<6>(a, ncw, st);
    case 7: return launch_beam_b<7>(a, ncw, st);
    case 8: return launch_beam_b<8>(a, ncw, st);
    case 9: return launch_beam_b<9>(a, ncw, st);
    case 10: return launch_beam_b<10>(a, ncw, st);
    case 11: return launch_beam_b<11>(a, ncw, st);
    case 12: return launch_beam_b<12>(a, ncw, st);
    case 13: return launch_beam_b<13>(a, ncw, st);
    case 14: return launch_beam_b<14>(a, ncw, st);
    case 15: return launch_beam_b<15>(a, ncw, st);
    default: return launch_beam_b<16>(a, ncw, st);
  }
}

}  // namespace aqmb
