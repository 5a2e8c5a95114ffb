// Decode GEMV on the matrix cores (8- and 4-bit codes, any batch up to 16): y[b][i] = s_i sum_j sum_{m<k}
// <x[b, group j], C_m[b_{ijm}]>, the per-plane products computed by v_mfma_f32_16x16x32 with the
// batch in the 16 rows of the A operand and 16 weight rows in the columns of the B operand.
//
// A workgroup of 16 waves owns 16 weight rows; the waves take interleaved runs of 4 K-steps of 32
// inputs (a run is 16 groups: one 16-byte code slice per plane, or half of a 4-bit slice). In a K-step lane l
// of a wave stands for weight row l % 16 and group l / 16 of the step: it gathers that group's
// codeword of every plane from the codebooks replicated in LDS, which is the B fragment of that
// plane's MFMA as it is (8 fp16 values of one row and group). The A fragment is x: lane l holds 8
// values of batch row l % 16 (rows past the batch are never stored). So every code costs one
// codeword gather, as at batch 1, and the dot products run on the matrix cores whatever the batch.
// Products are exact: fp16 x by the fp16 codeword directly; bf16 x either converted to fp16 times
// a power of two per batch row and run (values far below the row's maximum truncated), or
// multiplied by the codeword split exactly into two bf16 parts (see mg_split).
// Sums are fp32. The 16 waves' partial tiles are added in a fixed order (a tree over the waves),
// scaled once and rounded once, so results are reproducible.
#include <type_traits>

#include "device.h"
#include "launch.h"

namespace aqmb {

namespace mg {
constexpr int kThreads = 1024, kWaves = 16, kRows = 16;
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 b16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
}  // namespace mg

struct GemvMmaArgs {
  const unsigned char* codes;
  const uint16_t* codebooks;
  const uint16_t* scales;
  const uint16_t* x;
  void* y;
  const void* zero_page;      // >= 16 zero bytes
  size_t plane_bytes;
  int d_out, d_in, G, batch, y_dtype, nrep, cb_shift;
  int n_cu;                   // compute units (host side: the persistent grid)
};


// A run: 4 consecutive K-steps = 16 groups (8-bit codes: one 16-byte code slice; 4-bit codes:
// half of a 32-group slice, 8 bytes). Per lane: NX 16-byte pieces of x (below) and the run's code
// bytes of its weight row, per plane.
//
// x of a run is NX loads. Load t puts in lane L = 16 kc + R u + b (R = 4 NX rows per load,
// u < 4 / NX) the 8 values of batch row b at inputs 32 j + 8 kc of the run, j = t (4 / NX) + u.
// The A fragment of step j (lane 16 kc + b: row b, inputs 32 j + 8 kc) is then load j / (4 / NX)
// shifted down by R (j % (4 / NX)) lanes within each row of 16 lanes (a DPP row shift). Lanes of
// rows R and up take other rows' values: those rows of the product are never stored. One load per
// run for batch <= 4, two for batch <= 8, four (no shift) above.
//
// At k >= 2 (4-bit codes: k >= 3; at k = 2 the nibble packing costs more than the load it saves)
// the codes are loaded four planes at a time: lane 16 m + r of load t holds the run's
// codes of plane 4 t + m for weight row r (8-bit: the 16-byte slice; 4-bit: its 8-byte half).
// Before use, each lane packs the codes of group 4 j + q (j = 0..3) into dword q (8-bit: byte j;
// 4-bit: nibble j), and a transpose across the rows of 16 lanes (swaps of lane halves and of row
// pairs) leaves in lane 16 kc + r, dword m, the codes that lane uses from plane 4 t + m. So a run
// costs ceil(k / 4) code loads instead of k.
template <int K, int CB> constexpr bool mg_codes_t() { return CB == 8 ? K >= 2 : K >= 3; }
template <int K, int CB> constexpr int mg_code_loads() { return mg_codes_t<K, CB>() ? (K + 3) / 4 : K; }

template <int K, int CB, int NX>
struct MgRun {
  uint4 xa[NX];
  typename std::conditional<CB == 8, uint4, uint2>::type c[mg_code_loads<K, CB>()];
  // bf16 x converted in place: the factor 2^sh of the batch row of each of this lane's four
  // accumulator elements (set with the conversion, kept while the set holds the same x)
  float f[4];
};

// Loads of run r of weight row rowc (r clamped to the last run: a reload, never used): x of the
// run in the layout above (zeros past d_in, past the batch, and for dummy runs; skipped when
// with_x is false and R already holds it), and slice r of the row in every plane. With kSwap
// (four-plane loads feeding the paired gathers), the lanes of weight rows 8..15 load the planes
// of each pair in swapped order (plane 4 t + (m ^ 1) in place of 4 t + m), so that every lane
// finds the plane of its own half (slot 0 of the pair's gathers) in the pair's first dword.
template <int K, int CB, int NX, bool kSwap = false>
__device__ __forceinline__ void mg_load_run(const GemvMmaArgs& a, int r, int rowc, bool xok, MgRun<K, CB, NX>& R,
                                            bool with_x = true) {
  constexpr int kRowsX = 4 * NX, kPer = 4 / NX;              // batch rows per load, steps per load
  const int lane = threadIdx.x & 63, kc = lane >> 4;
  const int b = lane & (kRowsX - 1), u = (lane & 15) / kRowsX;
  const int n_runs = (a.G + 15) / 16;
  const int rc = r < n_runs ? r : n_runs - 1;
  if (with_x) {
#pragma unroll
    for (int t = 0; t < NX; ++t) {
      const int e = rc * 128 + (t * kPer + u) * 32 + kc * 8;
      const void* src = (xok && b < a.batch && e < a.d_in) ? (const void*)(a.x + (size_t)b * a.d_in + e) : a.zero_page;
      R.xa[t] = *(const uint4*)src;
    }
  }
  if constexpr (mg_codes_t<K, CB>()) {
#pragma unroll
    for (int t = 0; t < mg_code_loads<K, CB>(); ++t) {
      const int q = kSwap && (lane & 8) ? kc ^ 1 : kc;
      const int m = 4 * t + q < K ? 4 * t + q : K - 1;       // rows past the last plane reload it (unused)
      if constexpr (CB == 8) R.c[t] = load_stream16(a.codes + m * a.plane_bytes + ((size_t)rc * a.d_out + rowc) * 16);
      else R.c[t] = load_stream8(a.codes + m * a.plane_bytes + ((size_t)(rc >> 1) * a.d_out + rowc) * 16 + (rc & 1) * 8);
    }
  } else {
#pragma unroll
    for (int m = 0; m < K; ++m) {
      if constexpr (CB == 8) R.c[m] = load_stream16(a.codes + m * a.plane_bytes + ((size_t)rc * a.d_out + rowc) * 16);
      else R.c[m] = load_stream8(a.codes + m * a.plane_bytes + ((size_t)(rc >> 1) * a.d_out + rowc) * 16 + (rc & 1) * 8);
    }
  }
}

// When every thread replicates at most one codeword (K * NCW <= 1024), that word is requested
// ahead of the wave's run loads, so the replication waits for it only. (With more codewords per
// thread the runs' registers leave no room to hold it.) No barrier orders these small loads ahead
// of the other waves' run loads: with one or two loads per run it cost more than it saved.
template <int K, int CB> constexpr bool mg_preload() { return K * (1 << CB) <= mg::kThreads; }

// Paired codebook layout (8-bit codes; the default wherever it fits). A random 16-byte gather by
// 16 lanes is conflict-free only if the 16 lanes hit 16 different 16-byte units of the 64 banks;
// with 8 interleaved copies of one codebook, lanes l and l + 8 use the same copy and collide when
// their codewords have the same parity (half the time: 8 instead of 4 LDS cycles per gather).
// Here the codebooks are stored in 64 KiB regions of 256 rows of 256 bytes, row c holding, for a
// pair of planes (2p, 2p + 1), 8 copies of plane 2p's codeword c in its first 128 bytes and 8
// copies of plane 2p + 1's codeword c in the second. A pair of planes is gathered in two
// instructions: in the first, lanes with (l % 16) < 8 read their plane-2p codeword (bytes
// 0..127 of its row, copy l % 8) and lanes with (l % 16) >= 8 their plane-(2p + 1) codeword (bytes
// 128..255), in the second the other way round, so the 16 lanes always cover the 16 units: no
// conflicts, whatever the codes, and no more LDS than 8 copies. A plane without a partner (odd k)
// has a region of 16 copies. The split bf16 form pairs a plane's high and low parts. Each MFMA
// then takes codewords of two planes in its two halves of weight rows (columns 0..7 and 8..15),
// and the two MFMAs of a pair add both planes to every column (in a different order for the two
// halves: fixed, so results are reproducible). Regions: ceil(k / 2), or k in the split form.
template <int K, bool kSplit> constexpr int mg_regions() { return kSplit ? K : (K + 1) / 2; }
template <int K, int CB, bool kSplit> constexpr bool mg_paired() { return CB == 8 && mg_regions<K, kSplit>() <= 2; }
// Paired gathers of plane pairs (fp16 codewords, k >= 2: always four-plane code loads): the code
// loads swap each pair's planes in the lanes of rows 8..15 (mg_load_run's kSwap).
template <int K, int CB, bool kSplit> constexpr bool mg_swap_pairs() { return mg_paired<K, CB, kSplit>() && !kSplit && K >= 2; }
constexpr uint32_t kMgRegion = 256 * 256;                    // bytes per region

// The codebook word (index m * NCW + c) that replication slot q copies: in the paired layout
// slots of a pair region alternate between its two planes, so that the 16 lanes of a replica
// write also cover the 16 units of a row.
template <int K, int CB, bool kSplit>
__device__ __forceinline__ int mg_rep_word(int q) {
  if constexpr (mg_paired<K, CB, kSplit>() && !kSplit) {
    if (q < (K / 2) * 512) return (2 * (q >> 9) + (q & 1)) * 256 + ((q & 511) >> 1);
  }
  return q;
}

template <int K, int CB, bool kSplit>
__device__ __forceinline__ uint4 mg_first_word(const GemvMmaArgs& a) {
  if constexpr (!mg_preload<K, CB>()) return make_uint4(0, 0, 0, 0);
  const int q = (int)threadIdx.x < K * (1 << CB) ? (int)threadIdx.x : 0;
  return ((const uint4*)a.codebooks)[mg_rep_word<K, CB, kSplit>(q)];
}

// bf16 x takes one of two forms. Converted (mg_bf16_to_f16): x becomes fp16 times a power of two
// per batch row and run (exact but for values far below the row's maximum), one gather and one
// fp16 MFMA per code, at the price of the conversion (NX registers per lane and run). Split
// (exact): every codeword is split once, when copied into LDS, into a bf16 high part (RNE) and a
// bf16 low part (the remainder, at most 3 significant bits): two gathers and two bf16 MFMAs per
// code, no conversion. The split form is kept where the planes are too few to repay the
// conversion (measured crossovers: k = 1 at batch <= 4, k <= 2 above). The persistent kernel (P)
// converts each run's x once for all its blocks, so there the conversion wins from k = 2 at every
// batch (11008 x 4096, k = 2: batch 8 11.95 -> 11.37 us, batch 16 13.74 -> 12.73 us).
template <int K, int XDT, int NX, bool P = false>
constexpr bool mg_split_p() { return XDT == AQMB_BF16 && K < (P ? 2 : (NX == 1 ? 2 : 3)); }
template <int K, int XDT, int NX>
constexpr bool mg_split() { return mg_split_p<K, XDT, NX, false>(); }

// Codebook word q (q < K * NCW) into its nrep replicas (split form: a book of high and a book of
// low parts); v0 is word threadIdx.x, already loaded.
template <int K, int CB, bool kSplit>
__device__ __forceinline__ void mg_replicate(const GemvMmaArgs& a, uint4* cb_rep, uint4 v0) {
  using namespace mg;
  constexpr int NCW = 1 << CB;
  if constexpr (mg_paired<K, CB, kSplit>()) {
    // write i of slot q goes to unit (i + c) % 8 of its half row (16 units for a lone plane), so
    // the 16 lanes of a write cover a row's 16 units
    char* base = (char*)cb_rep;
    for (int q = threadIdx.x; q < K * NCW; q += kThreads) {
      const uint4 v = mg_preload<K, CB>() ? v0 : ((const uint4*)a.codebooks)[mg_rep_word<K, CB, kSplit>(q)];
      if constexpr (!kSplit) {
        if (q < (K / 2) * 512) {                             // a pair region: 8 copies in its half
          const int c = (q & 511) >> 1, half = q & 1;
          char* row = base + (q >> 9) * kMgRegion + c * 256 + half * 128;
          for (int i = 0; i < 8; ++i) *(uint4*)(row + ((i + c) & 7) * 16) = v;
        } else {                                             // the plane without a partner: 16 copies
          const int c = q - (K / 2) * 512;
          char* row = base + (K / 2) * kMgRegion + c * 256;
          for (int i = 0; i < 16; ++i) *(uint4*)(row + ((i + c) & 15) * 16) = v;
        }
      } else {                                               // region m: high parts, then low parts
        const f16x8_t cv = __builtin_bit_cast(f16x8_t, v);
        b16x8_t hi, lo;
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          const float cf = (float)cv[t];
          hi[t] = (__bf16)cf;                                // round to nearest even
          lo[t] = (__bf16)(cf - (float)hi[t]);               // exact: at most 3 significant bits
        }
        const uint4 vh = __builtin_bit_cast(uint4, hi), vl = __builtin_bit_cast(uint4, lo);
        const int c = q & (NCW - 1);
        // slots with c % 16 < 8 write their high part first, the others their low part, so the
        // 16 lanes of each write cover both halves of a row
        const bool sw = (c & 8) != 0;
        const uint4 va = sw ? vl : vh, vb = sw ? vh : vl;
        char* row = base + (q >> 8) * kMgRegion + c * 256;
        const int ha = sw ? 128 : 0, hb = 128 - ha;
        for (int i = 0; i < 8; ++i) *(uint4*)(row + ha + ((i + c) & 7) * 16) = va;
        for (int i = 0; i < 8; ++i) *(uint4*)(row + hb + ((i + c) & 7) * 16) = vb;
      }
    }
    return;
  }
  for (int q = threadIdx.x; q < K * NCW; q += kThreads) {
    const uint4 v = mg_preload<K, CB>() ? v0 : ((const uint4*)a.codebooks)[q];
    const int rot = q >> (8 - a.cb_shift);
    if constexpr (!kSplit) {
      for (int i = 0; i < a.nrep; ++i) cb_rep[q * a.nrep + ((i + rot) & (a.nrep - 1))] = v;
    } else {
      const f16x8_t c = __builtin_bit_cast(f16x8_t, v);
      b16x8_t hi, lo;
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const float cf = (float)c[t];
        hi[t] = (__bf16)cf;                                  // round to nearest even
        lo[t] = (__bf16)(cf - (float)hi[t]);                 // exact: at most 3 significant bits
      }
      const uint4 vh = __builtin_bit_cast(uint4, hi), vl = __builtin_bit_cast(uint4, lo);
      for (int i = 0; i < a.nrep; ++i) {
        cb_rep[q * a.nrep + ((i + rot) & (a.nrep - 1))] = vh;
        cb_rep[(K * NCW + q) * a.nrep + ((i + rot) & (a.nrep - 1))] = vl;
      }
    }
  }
}

// Lane i of each row of 16 lanes takes lane i + S of the row (S = 0: the value itself).
template <int S>
__device__ __forceinline__ uint4 mg_row_shift(uint4 v) {
  if constexpr (S == 0) {
    return v;
  } else {
    return make_uint4((uint32_t)__builtin_amdgcn_mov_dpp((int)v.x, 0x100 + S, 0xF, 0xF, false),
                      (uint32_t)__builtin_amdgcn_mov_dpp((int)v.y, 0x100 + S, 0xF, 0xF, false),
                      (uint32_t)__builtin_amdgcn_mov_dpp((int)v.z, 0x100 + S, 0xF, 0xF, false),
                      (uint32_t)__builtin_amdgcn_mov_dpp((int)v.w, 0x100 + S, 0xF, 0xF, false));
  }
}

// Code dwords of a four-plane load (layout above MgRun): dword m of the result holds the lane's
// codes of plane 4 t + m, the code of step j in byte j (8-bit) or nibble j (4-bit).
__device__ __forceinline__ void mg_rows_transpose(uint32_t (&d)[4]);
__device__ __forceinline__ void mg_codes_transpose(uint4 v, uint32_t (&d)[4]) {
  // byte q of each slice word (group 4 j + q) into dword q, a 4 x 4 byte transpose in two rounds
  // of byte selections (v_perm_b32: selector bytes 0..3 pick bytes of the second source, 4..7 of
  // the first): (x, y) and (z, w) interleaved by byte pairs, then the pairs joined
  const uint32_t xy01 = __builtin_amdgcn_perm(v.y, v.x, 0x05010400u);   // x0 y0 x1 y1
  const uint32_t xy23 = __builtin_amdgcn_perm(v.y, v.x, 0x07030602u);   // x2 y2 x3 y3
  const uint32_t zw01 = __builtin_amdgcn_perm(v.w, v.z, 0x05010400u);   // z0 w0 z1 w1
  const uint32_t zw23 = __builtin_amdgcn_perm(v.w, v.z, 0x07030602u);   // z2 w2 z3 w3
  d[0] = __builtin_amdgcn_perm(zw01, xy01, 0x05040100u);                 // x0 y0 z0 w0
  d[1] = __builtin_amdgcn_perm(zw01, xy01, 0x07060302u);                 // x1 y1 z1 w1
  d[2] = __builtin_amdgcn_perm(zw23, xy23, 0x05040100u);
  d[3] = __builtin_amdgcn_perm(zw23, xy23, 0x07060302u);
  mg_rows_transpose(d);
}
__device__ __forceinline__ void mg_codes_transpose(uint2 v, uint32_t (&d)[4]) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {                              // nibble 4 j + q of the 8 bytes: dword j / 2, bits 16 (j % 2) + 4 q
    const uint32_t a = (v.x >> (4 * q)) & 0x000F000Fu, b = (v.y >> (4 * q)) & 0x000F000Fu;
    d[q] = (a & 0xFu) | ((a >> 12) & 0xF0u) | ((b & 0xFu) << 8) | ((b >> 4) & 0xF000u);
  }
  mg_rows_transpose(d);
}

// d[q] of lane 16 m + r -> d[m] of lane 16 q + r (a 4 x 4 transpose of dwords and rows of 16 lanes).
__device__ __forceinline__ void mg_rows_transpose(uint32_t (&d)[4]) {
  // rows 2, 3 of d0 / d1 <-> rows 0, 1 of d2 / d3, then rows 1, 3 of d0 / d2 <-> rows 0, 2 of d1 / d3
  auto s02 = __builtin_amdgcn_permlane32_swap(d[0], d[2], false, false);
  auto s13 = __builtin_amdgcn_permlane32_swap(d[1], d[3], false, false);
  auto s01 = __builtin_amdgcn_permlane16_swap(s02[0], s13[0], false, false);
  auto s23 = __builtin_amdgcn_permlane16_swap(s02[1], s13[1], false, false);
  d[0] = s01[0]; d[1] = s01[1]; d[2] = s23[0]; d[3] = s23[1];
}

// bf16 x of a run as fp16 times a power of two per batch row: the exponent shift that puts the
// row's largest magnitude over the run's 128 inputs in [2^14, 2^15) (the rule of the
// direct-gather kernel's per-group conversion). Every lane computes the shift of the batch row it
// loaded (its largest exponent field e, then the maximum over the lanes that hold the same row:
// the same position in the other rows of 16 lanes and, for NX < 4, positions 4 NX apart within
// the row) and converts its own values. For 30 <= e <= 254 the conversion is integer arithmetic
// on the bit patterns (two values per 32-bit word): the exponent field lowered by e - 29 with the
// mantissa's 7 bits moved to fp16's 10, so a value is exact unless it lies below 2^-28 of the
// row maximum, where it is truncated (error below 2^-29 of the maximum); rows past the batch (never
// stored) take it too. Other rows (a maximum below 2^-97, Inf or NaN) are converted by ldexp and
// round-to-nearest-even, as in the direct-gather kernel. Returns the lane's shift: its values were
// multiplied by 2^-sh.
typedef unsigned short mg_u16x2 __attribute__((ext_vector_type(2)));
template <int NX>
__device__ __forceinline__ int mg_bf16_to_f16(uint4 (&xa)[NX], int batch) {
  // magnitudes (sign bits cleared): their largest 16-bit pattern holds the largest exponent field
  uint32_t mag[NX][4];
  mg_u16x2 ex = {0, 0};
#pragma unroll
  for (int t = 0; t < NX; ++t) {
    const uint32_t w[4] = {xa[t].x, xa[t].y, xa[t].z, xa[t].w};
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      mag[t][h] = w[h] & 0x7FFF7FFFu;
      ex = __builtin_elementwise_max(ex, __builtin_bit_cast(mg_u16x2, mag[t][h]));
    }
  }
  uint32_t e = (uint32_t)max(ex.x, ex.y) >> 7;
  const auto r32 = __builtin_amdgcn_permlane32_swap(e, e, false, false);   // rows 0, 1 <-> rows 2, 3
  e = max(r32[0], r32[1]);
  const auto r16 = __builtin_amdgcn_permlane16_swap(e, e, false, false);   // rows 0, 2 <-> rows 1, 3
  e = max(r16[0], r16[1]);
  if constexpr (NX == 1) e = max(e, (uint32_t)__builtin_amdgcn_mov_dpp((int)e, 0x124, 0xF, 0xF, false));  // row_ror:4
  if constexpr (NX <= 2) e = max(e, (uint32_t)__builtin_amdgcn_mov_dpp((int)e, 0x128, 0xF, 0xF, false));  // row_ror:8
  const int sh = (int)e - 141;                               // (e - 127) - 14
  const int row = (int)(threadIdx.x & 63) & (4 * NX - 1);   // the batch row this lane loaded
  if ((e >= 30 && e <= 254) || row >= batch) {
    const uint32_t d = (uint32_t)max((int)e - 29, 1) << 7;
    const mg_u16x2 dd = {(unsigned short)d, (unsigned short)d};
#pragma unroll
    for (int t = 0; t < NX; ++t) {
      uint32_t w[4] = {xa[t].x, xa[t].y, xa[t].z, xa[t].w};
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        mg_u16x2 v = __builtin_elementwise_sub_sat(__builtin_bit_cast(mg_u16x2, mag[t][h]), dd);
        v = v << (unsigned short)3;
        w[h] = (w[h] & 0x80008000u) | __builtin_bit_cast(uint32_t, v);
      }
      xa[t] = make_uint4(w[0], w[1], w[2], w[3]);
    }
    return sh;
  }
#pragma unroll
  for (int t = 0; t < NX; ++t) {
    uint32_t w[4] = {xa[t].x, xa[t].y, xa[t].z, xa[t].w};
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      const _Float16 lo = (_Float16)ldexpf(bf16lo(w[h]), -sh);
      const _Float16 hi = (_Float16)ldexpf(bf16hi(w[h]), -sh);
      w[h] = (uint32_t)__builtin_bit_cast(uint16_t, lo) | ((uint32_t)__builtin_bit_cast(uint16_t, hi) << 16);
    }
    xa[t] = make_uint4(w[0], w[1], w[2], w[3]);
  }
  return sh;
}

// The A fragment of step J (layout above MgRun).
template <int NX, int J>
__device__ __forceinline__ uint4 mg_x_step(const uint4 (&xa)[NX]) {
  constexpr int kPer = 4 / NX;
  return mg_row_shift<4 * NX * (J % kPer)>(xa[J / kPer]);
}

// The MFMAs of one run. Step j of a run: group 4 j + kc of the run (8-bit codes: byte 4 j + kc of
// the plane's slice word; 4-bit codes: nibble 4 j + kc of its 8 bytes).
// With bf16 x in the converted form, `convert` says whether R holds x as loaded: it is then
// converted in place (R.xa, with the row factors R.f), so a register set that keeps its run's x
// for several blocks (the persistent kernel) converts it, and fetches the factors, once.
template <int K, int XDT, int CB, int NX, bool P = false>
__device__ __forceinline__ void mg_compute(const GemvMmaArgs& a, const uint4* cb_rep, uint32_t rep_off,
                                           MgRun<K, CB, NX>& R, mg::f32x4_t (&acc)[4], bool convert = true) {
  using namespace mg;
  constexpr int NCW = 1 << CB;
  const int lane = threadIdx.x & 63, kc = lane >> 4;
  constexpr bool kSplit = mg_split_p<K, XDT, NX, P>(), kConv = XDT == AQMB_BF16 && !kSplit;
  if constexpr (kConv) {
    if (convert) {
      const int sh = mg_bf16_to_f16<NX>(R.xa, a.batch);
      // element e of this lane's accumulators is batch row 4 kc + e, whose shift lane 4 kc + e
      // computed: its factor 2^sh (a normal or subnormal float: -141 <= sh <= 113)
      const int f = __float_as_int(ldexpf(1.0f, sh));
#pragma unroll
      for (int e = 0; e < 4; ++e) R.f[e] = __int_as_float(__builtin_amdgcn_ds_bpermute((4 * kc + e) * 4, f));
    }
  }
  uint4 xa[NX];
#pragma unroll
  for (int t = 0; t < NX; ++t) xa[t] = R.xa[t];
  const uint4 xs[4] = {mg_x_step<NX, 0>(xa), mg_x_step<NX, 1>(xa), mg_x_step<NX, 2>(xa), mg_x_step<NX, 3>(xa)};
  // bf16 x: the run's products go to two fresh sums (steps j and j + 2 share one), scaled by each
  // batch row's 2^sh at the end; otherwise to the four steps' accumulators
  f32x4_t run[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) run[j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  f32x4_t (&dst)[4] = kConv ? run : acc;
  constexpr int kDst = kConv ? 1 : 3;                        // accumulator of step j: j & kDst
  constexpr int kCT = mg_codes_t<K, CB>() ? 4 * mg_code_loads<K, CB>() : 1;
  uint32_t cd[kCT];
  if constexpr (mg_codes_t<K, CB>()) {
#pragma unroll
    for (int t = 0; t < mg_code_loads<K, CB>(); ++t) {
      uint32_t d[4];
      mg_codes_transpose(R.c[t], d);
#pragma unroll
      for (int q = 0; q < 4; ++q) cd[4 * t + q] = d[q];
    }
  }
  if constexpr (mg_paired<K, CB, kSplit>()) {
    // Codeword addresses in one v_perm_b32 each: byte 1 is the code (a byte of the run's code
    // word), bytes 0, 2 and 3 come from a per-lane base (the lane's 16-byte unit in the 256-byte
    // row, plus the LDS address of the region, a multiple of 64 KiB: the codebooks open the
    // kernel's LDS, which holds no static variables).
    const bool upper = (lane & 8) != 0;                       // weight rows 8..15 of the tile
    const uint32_t r8 = (uint32_t)(lane & 7) * 16 + (upper ? 128u : 0u);   // slot 0: own half
    const uint32_t lds0 = lds_addr(cb_rep);
    const uint32_t kcsel = 0x03020000u | ((4u + (uint32_t)kc) << 8);      // byte kc of a slice word
    // the word holding the code of plane m for step j (this lane's weight row and group), and the
    // selector of its byte
    auto word_of = [&](int m, int j) -> uint32_t {
      if constexpr (mg_codes_t<K, CB>()) return cd[m];
      else return j == 0 ? R.c[m].x : j == 1 ? R.c[m].y : j == 2 ? R.c[m].z : R.c[m].w;
    };
    auto sel_of = [&](int j) -> uint32_t {
      if constexpr (mg_codes_t<K, CB>()) return 0x03020000u | ((4u + (uint32_t)j) << 8);
      else return kcsel;
    };
    auto read = [&](uint32_t addr) -> uint4 {
      const u32x4_t v = *(const __attribute__((address_space(3))) u32x4_t*)(uintptr_t)addr;
      return make_uint4(v.x, v.y, v.z, v.w);
    };
    // The run's codeword reads, listed in the order their MFMAs consume them, are issued kAhead
    // ahead of those MFMAs (scheduling groups: kAhead reads, then one MFMA and one read in turn),
    // so the LDS latency of a gather is not paid before every product; consecutive MFMAs go to
    // the steps' accumulators in turn. Each accumulator still adds its products in the same
    // order (pair by pair, slot 0 then slot 1).
    constexpr int kReads = kSplit ? 2 * K * 4 : (K / 2) * 8 + (K & 1) * 4;
    constexpr int kAhead = kReads < 4 ? kReads : 4;
    uint4 wv[kReads];
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (!kSplit) {
#pragma unroll
      for (int pp = 0; pp < K / 2; ++pp) {
        const uint32_t rb = lds0 + ((uint32_t)pp << 16);
        const uint32_t b0 = r8 | rb, b1 = (r8 ^ 128u) | rb;
        // slot 0: the plane of the lane's own half, in the pair's first code dword (the loads
        // swapped the pair's planes in rows 8..15), slot 1 the other
        static_assert(K < 2 || (mg_swap_pairs<K, CB, kSplit>() && mg_codes_t<K, CB>()), "pairs come from swapped four-plane loads");
        const uint32_t w0 = cd[2 * pp], w1 = cd[2 * pp + 1];
#pragma unroll
        for (int j = 0; j < 4; ++j) wv[pp * 8 + j] = read(__builtin_amdgcn_perm(w0, b0, sel_of(j)));
#pragma unroll
        for (int j = 0; j < 4; ++j) wv[pp * 8 + 4 + j] = read(__builtin_amdgcn_perm(w1, b1, sel_of(j)));
      }
      if constexpr (K & 1) {                                 // the plane without a partner: 16 copies
        const uint32_t bl = (uint32_t)(lane & 15) * 16 | (lds0 + ((uint32_t)(K / 2) << 16));
#pragma unroll
        for (int j = 0; j < 4; ++j) wv[(K / 2) * 8 + j] = read(__builtin_amdgcn_perm(word_of(K - 1, j), bl, sel_of(j)));
      }
#pragma unroll
      for (int pp = 0; pp < K / 2; ++pp)
#pragma unroll
        for (int q = 0; q < 8; ++q)                          // slot q / 4 of step q % 4
          dst[q & kDst] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8_t, xs[q & 3]),
                                                                 __builtin_bit_cast(f16x8_t, wv[pp * 8 + q]), dst[q & kDst], 0, 0, 0);
      if constexpr (K & 1) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
          dst[j & kDst] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8_t, xs[j]),
                                                                 __builtin_bit_cast(f16x8_t, wv[(K / 2) * 8 + j]), dst[j & kDst], 0, 0, 0);
      }
    } else {
#pragma unroll
      for (int m = 0; m < K; ++m) {
        const uint32_t bm = r8 | (lds0 + ((uint32_t)m << 16));
        uint32_t a0[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) a0[j] = __builtin_amdgcn_perm(word_of(m, j), bm, sel_of(j));
#pragma unroll
        for (int j = 0; j < 4; ++j) wv[m * 8 + j] = read(a0[j]);             // high (rows 0..7) or low part
#pragma unroll
        for (int j = 0; j < 4; ++j) wv[m * 8 + 4 + j] = read(a0[j] ^ 128u);  // the other part
      }
#pragma unroll
      for (int m = 0; m < K; ++m)
#pragma unroll
        for (int q = 0; q < 8; ++q)
          acc[q & 3] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(b16x8_t, xs[q & 3]),
                                                               __builtin_bit_cast(b16x8_t, wv[m * 8 + q]), acc[q & 3], 0, 0, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x100, kAhead, 0);
#pragma unroll
    for (int t = kAhead; t < kReads; ++t) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, kAhead, 0);
    __builtin_amdgcn_sched_barrier(0);
  } else {
#pragma unroll
  for (int m = 0; m < K; ++m) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      uint32_t code;
      if constexpr (mg_codes_t<K, CB>()) {
        code = CB == 8 ? (cd[m] >> (8 * j)) & 0xFFu : (cd[m] >> (4 * j)) & 15u;
      } else if constexpr (CB == 8) {
        const uint32_t word = j == 0 ? R.c[m].x : j == 1 ? R.c[m].y : j == 2 ? R.c[m].z : R.c[m].w;
        code = (word >> (8 * kc)) & 0xFFu;
      } else {
        const uint32_t word = j < 2 ? R.c[m].x : R.c[m].y;
        code = (word >> (4 * (4 * (j & 1) + kc))) & 15u;
      }
      const uint32_t off = (((uint32_t)(m * NCW) + code) << a.cb_shift) + rep_off;
      const uint4 cw = *(const uint4*)((const char*)cb_rep + off);
      if constexpr (!kSplit) {
        dst[j & kDst] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8_t, xs[j]),
                                                               __builtin_bit_cast(f16x8_t, cw), dst[j & kDst], 0, 0, 0);
      } else {
        const uint4 cl = *(const uint4*)((const char*)cb_rep + ((uint32_t)(K * NCW) << a.cb_shift) + off);
        const b16x8_t xb = __builtin_bit_cast(b16x8_t, xs[j]);
        acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xb, __builtin_bit_cast(b16x8_t, cw), acc[j], 0, 0, 0);
        acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xb, __builtin_bit_cast(b16x8_t, cl), acc[j], 0, 0, 0);
      }
    }
  }
  }
  if constexpr (kConv) {
    // each batch row's sum scaled by its factor inside the add: one rounding, as after an exact
    // scaling
    const f32x4_t t = run[0] + run[1];
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[0][e] = fmaf(t[e], R.f[e], acc[0][e]);
  }
}

// Partial tiles of the 16 waves summed in a fixed order, scaled once and rounded once, for the 16
// weight rows from row0. Element e of lane l of a tile is batch row 4 (l / 16) + e, weight row
// l % 16; read as floats, a tile holds 256 outputs, output o = 4 l + e. The four waves of group
// grp (threads 256 grp .. 256 grp + 255; t = tid % 256) each read the 16 partials of output t (all
// requested at once), add them in a fixed tree, scale and store; a persistent workgroup rotates
// the group from block to block, so the extra work does not fall on the same waves at every
// block end. sbits is the scale of weight row row0 + (t / 4) % 16. Ends with the partial tiles
// read by the group (the caller separates two calls with a barrier).
__device__ __forceinline__ int mg_out_row(int t) { return (t >> 2) & 15; }
__device__ __forceinline__ bool mg_in_group(int grp) { return ((int)threadIdx.x >> 8) == grp; }
__device__ __forceinline__ void mg_reduce_store(const GemvMmaArgs& a, mg::f32x4_t* red, const mg::f32x4_t (&acc)[4],
                                                int row0, uint16_t sbits, int grp = 0) {
  using namespace mg;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  red[wave * 64 + lane] = (acc[0] + acc[1]) + (acc[2] + acc[3]);
  __syncthreads();
  const int t = tid & 255;
  const int b = 4 * (t >> 6) + (t & 3);                      // batch row of output t
  const int row = row0 + mg_out_row(t);
  if (mg_in_group(grp) && b < a.batch && row < a.d_out) {
    const float* rf = (const float*)red + t;
    float p[kWaves];
#pragma unroll
    for (int w = 0; w < kWaves; ++w) p[w] = rf[w * 256];
#pragma unroll
    for (int h = 1; h < kWaves; h *= 2)                      // pairs, then pairs of pairs, ...
#pragma unroll
      for (int w = 0; w < kWaves; w += 2 * h) p[w] += p[w + h];
    const float v = p[0] * f16_to_f32(sbits);
    const size_t off = (size_t)b * a.d_out + row;
    if (a.y_dtype == AQMB_F16) OutT<AQMB_F16>::store(a.y, off, v);
    else if (a.y_dtype == AQMB_BF16) OutT<AQMB_BF16>::store(a.y, off, v);
    else OutT<AQMB_F32>::store(a.y, off, v);
  }
}

// 16-row block blk of a layer (the body of a one-block workgroup).
template <int K, int XDT, int CB, int NX>
__device__ __forceinline__ void mg_one_block(const GemvMmaArgs& a, int blk) {
  using namespace mg;
  constexpr bool kSpl = mg_split<K, XDT, NX>();
  constexpr int kBooks = kSpl ? 2 : 1;                       // fp16 codewords, or bf16 high and low parts
  extern __shared__ uint4 smem_mg[];
  uint4* cb_rep = smem_mg;                                   // paired regions, or [kBooks][K][NCW][nrep] codewords
  f32x4_t* red = (f32x4_t*)(smem_mg + (mg_paired<K, CB, kSpl>() ? mg_regions<K, kSpl>() * (kMgRegion / 16)
                                                                 : kBooks * K * (1 << CB) * a.nrep));   // [kWaves][64] partial tiles
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int col = lane & 15;                                 // weight row in the block
  const int row0 = blk * kRows;
  const int rowc = row0 + col < a.d_out ? row0 + col : a.d_out - 1;
  const int n_runs = (a.G + 15) / 16;                        // code slices per row
  const uint32_t rep_off = (uint32_t)(lane & (a.nrep - 1)) * 16;

  // The wave's runs are wave, wave + 16, ...; the first two are requested before the codebooks are
  // replicated into LDS (a 4096-wide row has 32 runs: two per wave).
  MgRun<K, CB, NX> ra, rb;
  int r = wave;
  const uint4 w0 = mg_first_word<K, CB, kSpl>(a);
  const int srow = row0 + mg_out_row(tid);                   // the row this thread stores, if any
  const uint16_t sbits = tid < 256 ? a.scales[srow < a.d_out ? srow : a.d_out - 1] : 0;
  constexpr bool kSw = mg_swap_pairs<K, CB, kSpl>();
  mg_load_run<K, CB, NX, kSw>(a, r, rowc, true, ra);
  mg_load_run<K, CB, NX, kSw>(a, r + kWaves, rowc, true, rb);
  mg_replicate<K, CB, kSpl>(a, cb_rep, w0);
  __syncthreads();

  f32x4_t acc[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) acc[j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  // Two register sets in turn: the loads of the wave's run after next are requested while it
  // computes one.
  for (; r < n_runs; r += 2 * kWaves) {
    mg_compute<K, XDT, CB, NX>(a, cb_rep, rep_off, ra, acc);
    if (r + kWaves >= n_runs) break;
    if (r + 2 * kWaves < n_runs) mg_load_run<K, CB, NX, kSw>(a, r + 2 * kWaves, rowc, true, ra);
    mg_compute<K, XDT, CB, NX>(a, cb_rep, rep_off, rb, acc);
    if (r + 3 * kWaves < n_runs) mg_load_run<K, CB, NX, kSw>(a, r + 3 * kWaves, rowc, true, rb);
  }
  mg_reduce_store(a, red, acc, row0, sbits);
}

template <int K, int XDT, int CB, int NX>
__global__ __launch_bounds__(mg::kThreads) __attribute__((amdgpu_waves_per_eu(4, 4)))
void gemv_mma_kernel(GemvMmaArgs a) {
  mg_one_block<K, XDT, CB, NX>(a, (int)blockIdx.x);
}

// Several layers on one input (same d_in, code width and k): one launch over the row blocks of
// all of them, workgroup w running block w - first[l] of the layer l with first[l] <= w <
// first[l + 1], exactly as a one-block workgroup of that layer's own launch.
struct GemvMmaMultiArgs {
  GemvMmaArgs L[AQMB_MAX_MULTI];
  int first[AQMB_MAX_MULTI + 1];
  int n;
};
static_assert(sizeof(GemvMmaMultiArgs) <= 4096, "kernel arguments are limited to 4 KiB");

template <int K, int XDT, int CB, int NX>
__global__ __launch_bounds__(mg::kThreads) __attribute__((amdgpu_waves_per_eu(4, 4)))
void gemv_mma_multi_kernel(GemvMmaMultiArgs m) {
  int l = 0;
  while (l + 1 < m.n && (int)blockIdx.x >= m.first[l + 1]) ++l;
  mg_one_block<K, XDT, CB, NX>(m.L[l], (int)blockIdx.x - m.first[l]);
}

// Layers with more 16-row blocks than compute units: one persistent workgroup per CU walks the
// row blocks blockIdx.x, blockIdx.x + gridDim.x, ... with the codebooks replicated once. Each
// wave takes the same per = ceil(n_runs / 16) runs of every block (wave, wave + 16, ...; runs past
// the row are dummies: x reads zeros) as one flat sequence of items over its blocks, two items
// ahead in two register sets, so the next block's first runs are in flight while a block ends
// (partial tiles reduced as in gemv_mma_kernel; same arithmetic and order).
template <int K, int XDT, int CB, int NX>
__global__ __launch_bounds__(mg::kThreads) __attribute__((amdgpu_waves_per_eu(4, 4)))
void gemv_mma_persist_kernel(GemvMmaArgs a) {
  using namespace mg;
  constexpr bool kSpl = mg_split_p<K, XDT, NX, true>();
  constexpr int kBooks = kSpl ? 2 : 1;                       // fp16 codewords, or bf16 high and low parts
  extern __shared__ uint4 smem_mg[];
  uint4* cb_rep = smem_mg;                                   // paired regions, or [kBooks][K][NCW][nrep] codewords
  f32x4_t* red = (f32x4_t*)(smem_mg + (mg_paired<K, CB, kSpl>() ? mg_regions<K, kSpl>() * (kMgRegion / 16)
                                                                 : kBooks * K * (1 << CB) * a.nrep));   // [2][kWaves][64] partial tiles
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int col = lane & 15;
  const int n_runs = (a.G + 15) / 16;
  const int n_rb = (a.d_out + kRows - 1) / kRows;
  const int per = (n_runs + kWaves - 1) / kWaves;            // items per block, the same for every wave
  const int nb = (n_rb - (int)blockIdx.x + (int)gridDim.x - 1) / (int)gridDim.x;   // this workgroup's blocks
  const int n_items = per * nb;
  const uint32_t rep_off = (uint32_t)(lane & (a.nrep - 1)) * 16;

  // item i: block blockIdx.x + (i / per) gridDim.x, run wave + (i % per) 16 (items past the end:
  // the last item again, never used). Even items go to register set ra, odd ones to rb; with at
  // most two runs per wave and block (rows of at most 32 runs) a set always holds the same run, so
  // its x is loaded once, with the first block.
  auto load_item = [&](int i, MgRun<K, CB, NX>& R) {
    const int ic = i < n_items ? i : n_items - 1;
    const int row = ((int)blockIdx.x + (ic / per) * (int)gridDim.x) * kRows + col;
    const int r = wave + (ic % per) * kWaves;
    mg_load_run<K, CB, NX, mg_swap_pairs<K, CB, kSpl>()>(a, r, row < a.d_out ? row : a.d_out - 1, r < n_runs, R,
                                                        i < 2 || per > 2);
  };
  auto block_row0 = [&](int i) {                             // first row of the block of item i
    return ((int)blockIdx.x + ((i < n_items ? i : n_items - 1) / per) * (int)gridDim.x) * kRows;
  };
  // The scale of the row this thread stores (in the block's reducing group), requested a block ahead.
  auto group_of = [&](int i) { return ((i < n_items ? i : n_items - 1) / per) & 3; };   // the block's reducing waves
  auto scale_of = [&](int i) -> uint16_t {
    const int row = block_row0(i) + mg_out_row(tid & 255);
    return mg_in_group(group_of(i)) ? a.scales[row < a.d_out ? row : a.d_out - 1] : 0;
  };
  uint16_t sbits;
  f32x4_t acc[4];
  // Two partial-tile buffers in turn: block b's tiles are read (by threads < 256) while the other
  // waves go on to block b + 1; block b + 2 writes the buffer again only after block b + 1's
  // barrier, which every thread reaches after its reads of block b.
  auto end_block = [&](int i) {                              // item i closed its block
    mg_reduce_store(a, red + ((i / per) & 1) * (kWaves * 64), acc, block_row0(i), sbits, group_of(i));
    sbits = scale_of(i + 1);
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  };

  MgRun<K, CB, NX> ra, rb;
  const uint4 w0 = mg_first_word<K, CB, kSpl>(a);
  sbits = scale_of(0);
  load_item(0, ra);
  // the codebook replication waits only for the codebook word and the first item's loads; the
  // second item's loads queue behind the replica writes
  mg_replicate<K, CB, kSpl>(a, cb_rep, w0);
  load_item(1, rb);
  __syncthreads();
#pragma unroll
  for (int j = 0; j < 4; ++j) acc[j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  for (int i = 0; i < n_items; i += 2) {
    mg_compute<K, XDT, CB, NX, true>(a, cb_rep, rep_off, ra, acc, i < 2 || per > 2);   // x loaded with the item
    load_item(i + 2, ra);
    if ((i + 1) % per == 0) end_block(i);
    if (i + 1 >= n_items) break;
    mg_compute<K, XDT, CB, NX, true>(a, cb_rep, rep_off, rb, acc, i < 2 || per > 2);
    load_item(i + 3, rb);
    if ((i + 2) % per == 0) end_block(i + 1);
  }
}

// 16-codeword codebooks (4-bit codes) fill the LDS banks once: one copy reads without conflicts.
// (mm: several layers in one launch; a is then mm->L[0].)
template <int K, int XDT, int CB, int NX>
static hipError_t launch_mma_knx(GemvMmaArgs a, GemvMmaMultiArgs* mm, hipStream_t st) {
  const int n_rb = (a.d_out + mg::kRows - 1) / mg::kRows;
  const bool persist = !mm && n_rb > a.n_cu && a.n_cu > 0;   // one workgroup per CU walks the blocks
  const bool split = persist ? mg_split_p<K, XDT, NX, true>() : mg_split<K, XDT, NX>();
  // partial tiles: one buffer, two in the persistent kernel
  const size_t red = (size_t)(persist ? 2 : 1) * mg::kWaves * 64 * 16, book = (size_t)(split ? 2 : 1) * K * (1 << CB) * 16;
  const size_t budget = 160 * 1024 - 1024 - red;
  const bool paired = persist ? mg_paired<K, CB, mg_split_p<K, XDT, NX, true>()>()
                              : mg_paired<K, CB, mg_split<K, XDT, NX>()>();
  const int regions = persist ? mg_regions<K, mg_split_p<K, XDT, NX, true>()>() : mg_regions<K, mg_split<K, XDT, NX>()>();
  // otherwise (k > 4; k > 2 split): as many interleaved copies per codebook as fit
  a.nrep = CB == 4 ? 1 : paired ? 8 : book * 8 <= budget ? 8 : book * 4 <= budget ? 4 : 2;
  a.cb_shift = a.nrep == 8 ? 7 : a.nrep == 4 ? 6 : a.nrep == 2 ? 5 : 4;
  const size_t lds = (paired ? (size_t)regions * kMgRegion : book * a.nrep) + red;
  if (mm) {
    for (int l = 0; l < mm->n; ++l) {
      mm->L[l].nrep = a.nrep;
      mm->L[l].cb_shift = a.cb_shift;
    }
    gemv_mma_multi_kernel<K, XDT, CB, NX><<<dim3(mm->first[mm->n]), mg::kThreads, lds, st>>>(*mm);
    return hipGetLastError();
  }
  if (persist) gemv_mma_persist_kernel<K, XDT, CB, NX><<<dim3(a.n_cu), mg::kThreads, lds, st>>>(a);
  else gemv_mma_kernel<K, XDT, CB, NX><<<dim3(n_rb), mg::kThreads, lds, st>>>(a);
  return hipGetLastError();
}

// x loads per run: batch rows in groups of 4 per 16-lane row (see MgRun).
template <int K, int XDT, int CB>
static hipError_t launch_mma_kc(const GemvMmaArgs& a, GemvMmaMultiArgs* mm, hipStream_t st) {
  if (a.batch <= 4) return launch_mma_knx<K, XDT, CB, 1>(a, mm, st);
  if (a.batch <= 8) return launch_mma_knx<K, XDT, CB, 2>(a, mm, st);
  return launch_mma_knx<K, XDT, CB, 4>(a, mm, st);
}

template <int K, int XDT>
static hipError_t launch_mma_k(const GemvMmaArgs& a, GemvMmaMultiArgs* mm, int code_bits, hipStream_t st) {
  return code_bits == 4 ? launch_mma_kc<K, XDT, 4>(a, mm, st) : launch_mma_kc<K, XDT, 8>(a, mm, st);
}

template <int XDT>
static hipError_t launch_mma_x(const GemvMmaArgs& a, GemvMmaMultiArgs* mm, int k, int cb, hipStream_t st) {
  switch (k) {
    case 1: return launch_mma_k<1, XDT>(a, mm, cb, st);
    case 2: return launch_mma_k<2, XDT>(a, mm, cb, st);
    case 3: return launch_mma_k<3, XDT>(a, mm, cb, st);
    case 4: return launch_mma_k<4, XDT>(a, mm, cb, st);
    case 5: return launch_mma_k<5, XDT>(a, mm, cb, st);
    case 6: return launch_mma_k<6, XDT>(a, mm, cb, st);
    case 7: return launch_mma_k<7, XDT>(a, mm, cb, st);
    default: return launch_mma_k<8, XDT>(a, mm, cb, st);
  }
}

static GemvMmaArgs mma_args(const Layer& L, const void* x, int batch, void* y, aqmb_dtype y_dtype) {
  GemvMmaArgs a{};
  a.codes = L.codes;
  a.codebooks = L.codebooks;
  a.scales = L.scales;
  a.x = (const uint16_t*)x;
  a.y = y;
  a.zero_page = L.zero_page();
  a.plane_bytes = L.plane_bytes;
  a.d_out = L.d.d_out;
  a.d_in = L.d.d_in;
  a.G = L.G;
  a.batch = batch;
  a.y_dtype = (int)y_dtype;
  a.n_cu = L.n_cu;
  return a;
}

hipError_t launch_gemv_mma(const Layer& L, int k, const void* x, aqmb_dtype x_dtype, int batch, void* y,
                           aqmb_dtype y_dtype, hipStream_t st) {
  const GemvMmaArgs a = mma_args(L, x, batch, y, y_dtype);
  const int cb = L.d.code_bits;
  return x_dtype == AQMB_F16 ? launch_mma_x<AQMB_F16>(a, nullptr, k, cb, st) : launch_mma_x<AQMB_BF16>(a, nullptr, k, cb, st);
}

hipError_t launch_gemv_mma_multi(const Layer* const* Ls, int n, int k, const void* x, aqmb_dtype x_dtype, int batch,
                                 void* const* ys, aqmb_dtype y_dtype, hipStream_t st) {
  GemvMmaMultiArgs m{};
  m.n = n;
  m.first[0] = 0;
  for (int l = 0; l < n; ++l) {
    m.L[l] = mma_args(*Ls[l], x, batch, ys[l], y_dtype);
    m.first[l + 1] = m.first[l] + (Ls[l]->d.d_out + mg::kRows - 1) / mg::kRows;
  }
  const int cb = Ls[0]->d.code_bits;
  return x_dtype == AQMB_F16 ? launch_mma_x<AQMB_F16>(m.L[0], &m, k, cb, st)
                             : launch_mma_x<AQMB_BF16>(m.L[0], &m, k, cb, st);
}

}  // namespace aqmb
