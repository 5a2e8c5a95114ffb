// Distortion of every prefix level in one pass (8- or 4-bit codes) (the quantity the training loop of Drop-by-Drop
// evaluates after each new codebook, section 5 and Alg. 1, with the weighted MSE of section 2.2,
// Eq. wmse-task): for k = 1..M,
//   D^(k) = ||(W - W^(k)) X||_F^2 / (d_out n),  W^(k)[i, j g + t] = s_i sum_{m<k} C_m[b_{ijm}][t],
// with the n calibration inputs given as rows X^T = [n][d_in].
//
// For an output tile (samples x weight rows) the kernel accumulates, over d_in, the dense product
// P = X^T W^T and one product per code plane, Q_m = X^T C_m[b_m]^T (unscaled). Then
//   R_k = P - s_i (Q_0 + ... + Q_{k-1}),   D^(k) = sum of R_k^2 / (d_out n).
// W, X and the codebooks are fp16 and the products run on the fp16 matrix cores
// (v_mfma_f32_32x32x16_f16): every product of two fp16 values is exact in the fp32 accumulator,
// so the only roundings are those of the fp32 sums, of s_i Q and of the differences.
//
// Work item: kTok = 32 NA samples x 128 weight rows. Each of the four waves owns 32 rows (one
// MFMA column block) and all NA sample blocks, so the B fragment of a row block (a W piece or a
// codeword) feeds NA MFMAs. d_in is walked in steps of 64 (four K-blocks of 16 = eight groups),
// with the loads of the next kPre steps in flight while a step computes:
//   - the kTok x 64 slice of X is staged in LDS (direct loads into kPre + 1 buffers, swizzled
//     so that the 32 rows of an A fragment read hit distinct banks) and read by all four waves;
//   - the W pieces come from global memory into registers (16 bytes per lane and K-block),
//     together with the code bytes (8 bytes = 8 groups per plane), in kPre + 1 register sets;
//   - the B fragment of plane m is the codeword itself: lane l of a K-block needs the 8 values of
//     one group of one row, i.e. C_m[code], gathered from codebooks replicated in LDS.
// Each lane keeps fp64 sums of R_k^2 over its outputs; each workgroup writes its sums and a
// second kernel adds them in a fixed order, so the result does not depend on scheduling.
#include <mutex>
#include <type_traits>

#include "device.h"
#include "launch.h"

namespace aqmb {

namespace dist {
constexpr int kThreads = 256;                // four waves
constexpr int kRows = 128;                   // weight rows per work item (32 per wave)
constexpr int kStep = 64;                    // d_in per step: four K-blocks of 16 = eight groups
constexpr int kPre = 2;                      // steps whose loads are in flight ahead of the computed one
constexpr int kBufs = kPre + 1;              // X buffers and register sets
constexpr int kMaxGrid = 256;                // one workgroup per CU; each loops over work items
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
// CB = code bits: 8 (256 codewords, replicated) or 4 (16 codewords: they fill the LDS banks once,
// so one copy is read without conflicts).
template <int M, int CB> struct Cfg {
  // 32-sample blocks per wave (accumulators: 16 NA (M+1)); M = 6 with 4-bit codes takes one (with
  // two, its registers overflow)
  static constexpr int NA = M <= 5 || (M == 6 && CB == 8) ? 2 : 1;
  static constexpr int kTok = 32 * NA;
  static constexpr int NCW = 1 << CB;
  static constexpr int kNrep = CB == 4 ? 1 : M <= 4 ? 8 : 4;   // codebook replicas in LDS
  static constexpr int kShift = kNrep == 8 ? 7 : kNrep == 4 ? 6 : 4;   // log2(16 kNrep)
  static constexpr size_t kCbBytes = (size_t)M * NCW * kNrep * 16;
  static constexpr size_t kXBytes = (size_t)kTok * kStep * 2;  // one X stage
  static constexpr size_t kLds = kCbBytes + kBufs * kXBytes;
  static constexpr int kLoads = NA + 4 + M;                    // loads per wave per step
};
// One step's operands in registers: the W pieces of the four K-blocks and 8 code bytes per plane.
// (8-bit codes: 8 code bytes per plane; 4-bit codes: one 4-byte word of 8 nibbles per plane.)
template <int M, int CB> struct Frag {
  f16x8_t w[4];
  typename std::conditional<CB == 8, uint2, uint32_t>::type c[M];
};
}  // namespace dist

size_t distortion_scratch_bytes() { return (size_t)dist::kMaxGrid * 8 * sizeof(double); }

// Scratch of the allocation-free entry point: one per-workgroup sum slot for each of the at most
// kMaxGrid workgroups and 8 levels (16 KiB per device, held until the process ends). Host code
// never passes the array's name to a kernel: its device address, looked up once per device with
// hipGetSymbolAddress while that device is current, is what the kernels receive. Every call on a
// device shares that device's copy, so calls that overlap on one device race. Nothing in it needs
// clearing: each workgroup writes its slots before the final sum reads them.
static __device__ __align__(256) double scratch[dist::kMaxGrid * 8];
constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static double* g_scratch_ptr[kMaxDevices];

hipError_t distortion_static_scratch(int device, double** out, size_t* bytes) {
  *out = nullptr;
  *bytes = sizeof(scratch);
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[device]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[device] = (double*)p;
  }
  *out = g_scratch_ptr[device];
  return hipSuccess;
}

struct DistArgs {
  const unsigned char* codes;
  const uint16_t* codebooks;
  const uint16_t* scales;
  const uint16_t* W;      // [d_out][d_in] fp16
  const uint16_t* X;      // [n][d_in] fp16
  double* partials;       // [gridDim.x][8]
  const void* zero_page;  // >= 16 zero bytes
  size_t plane_bytes;
  int d_out, d_in, n, n_rb, n_items;
};

template <int M, int CB>
__global__ __launch_bounds__(dist::kThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void distortion_kernel(DistArgs a) {
  using namespace dist;
  using C = Cfg<M, CB>;
  constexpr int NA = C::NA, kTok = C::kTok, kNrep = C::kNrep, kShift = C::kShift, kLoads = C::kLoads;
  constexpr int NCW = C::NCW;
  extern __shared__ uint4 smem_d[];
  uint4* cbr = smem_d;                                          // [M][NCW][kNrep] codewords
  char* xs = (char*)smem_d + C::kCbBytes;                       // [kBufs][kTok][128 bytes]
  __shared__ double red[4][M];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = lane >> 5, r32 = lane & 31;
  const int nsteps = (a.d_in + kStep - 1) / kStep;

  // Codebooks, replicated: replica r of codeword q (= m * NCW + c) at slot q * kNrep + r. The
  // writers of one store instruction are rotated so that 16 consecutive q fill a bank row.
  for (int q = tid; q < M * NCW; q += kThreads) {
    const uint4 v = ((const uint4*)a.codebooks)[q];
    const int rot = q >> (8 - kShift);
#pragma unroll
    for (int i = 0; i < kNrep; ++i) cbr[q * kNrep + ((i + rot) & (kNrep - 1))] = v;
  }
  const char* cbase = (const char*)cbr + (lane & (kNrep - 1)) * 16;   // this lane's replica

  double part[M];
#pragma unroll
  for (int m = 0; m < M; ++m) part[m] = 0.0;

  for (int item = blockIdx.x; item < a.n_items; item += gridDim.x) {
    const int rb = item % a.n_rb, t0 = (item / a.n_rb) * kTok;
    const int row = rb * kRows + wave * 32 + r32;
    const bool row_ok = row < a.d_out;
    const int rowc = row_ok ? row : a.d_out - 1;

    // X stage of step st into buffer buf: 16-byte slot q of the stage holds sample q / 8,
    // piece (q % 8) ^ ((sample / 2) % 8) of the step's 128 bytes (two 128-byte sample rows share
    // a bank row, so the 32 samples an A fragment reads land on distinct banks). Each wave loads
    // NA runs of 64 slots. Past d_in (and past the last step) the zero page is loaded.
    auto stage_x = [&](int st, int buf) {
#pragma unroll
      for (int j = 0; j < NA; ++j) {
        const int q = (wave * NA + j) * 64 + lane, smp = q >> 3;
        const int piece = (q & 7) ^ ((smp >> 1) & 7);
        const int t = t0 + smp, k = st * kStep + piece * 8;
        const void* src = (t < a.n && k < a.d_in) ? (const void*)(a.X + (size_t)t * a.d_in + k) : a.zero_page;
        load_lds16(src, lds_addr(xs + buf * C::kXBytes + (wave * NA + j) * 1024));
      }
    };
    // W pieces (K-block kb: values 16 kb + 8 h .. + 7 of the step) and the code bytes of groups
    // 8 st .. 8 st + 7 of this lane's row (one 8-byte half of a 16-group slice). Past the last
    // step the last one is loaded again (never used), so every step issues the same loads.
    auto load_w = [&](int st, Frag<M, CB>& f, int kb) {
      const int stc = st < nsteps ? st : nsteps - 1;
      int k = stc * kStep + kb * 16 + h * 8;
      k = k < a.d_in ? k : 0;                                  // only meets zero X
      f.w[kb] = *(const f16x8_t*)(a.W + (size_t)rowc * a.d_in + k);
    };
    auto load_codes = [&](int st, Frag<M, CB>& f) {
      const int g0 = (st < nsteps ? st : nsteps - 1) * 8;
#pragma unroll
      for (int m = 0; m < M; ++m) {
        if constexpr (CB == 8)
          f.c[m] = *(const uint2*)(a.codes + m * a.plane_bytes + ((size_t)(g0 >> 4) * a.d_out + rowc) * 16 + (g0 & 8));
        else
          f.c[m] = *(const uint32_t*)(a.codes + m * a.plane_bytes + ((size_t)(g0 >> 5) * a.d_out + rowc) * 16 + ((g0 & 31) >> 1));
      }
    };
    // The loads of one step, issued in three parts (with the MFMAs of K-blocks 0, 1, 2 of the step
    // kPre earlier), kLoads in all.
    auto issue_part = [&](int st, int buf, Frag<M, CB>& f, int part) {
      if (part == 0) { stage_x(st, buf); load_w(st, f, 0); load_w(st, f, 1); }
      if (part == 1) { load_w(st, f, 2); load_w(st, f, 3); }
      if (part == 2) load_codes(st, f);
    };

    f32x16_t acc[M + 1][NA];
#pragma unroll
    for (int s = 0; s <= M; ++s)
#pragma unroll
      for (int na = 0; na < NA; ++na)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[s][na][e] = 0.f;

    // For each K-block: NA A fragments from the X stage and M codewords gathered from the
    // codebooks. No lane is masked: past d_in the staged X is zero, so whatever W piece or
    // codeword sits in the B operand there contributes nothing (W and the codebooks are finite).
    struct Ops { f16x8_t xa[NA]; f16x8_t bq[M]; };
    auto read_ops = [&](int buf, const Frag<M, CB>& f, int kb, Ops& o) {
      const char* xst = xs + buf * C::kXBytes;
      const int piece = kb * 2 + h;                            // = group of the step
#pragma unroll
      for (int na = 0; na < NA; ++na) {
        const int smp = na * 32 + r32;
        o.xa[na] = *(const f16x8_t*)(xst + smp * 128 + ((piece ^ ((smp >> 1) & 7)) << 4));
      }
#pragma unroll
      for (int m = 0; m < M; ++m) {
        uint32_t code;
        if constexpr (CB == 8) {
          const uint32_t word = kb < 2 ? f.c[m].x : f.c[m].y;
          code = (word >> (16 * (kb & 1) + 8 * h)) & 0xFFu;
        } else {                                               // nibble `piece` of the step's word
          code = (f.c[m] >> (4 * piece)) & 15u;
        }
        o.bq[m] = *(const f16x8_t*)(cbase + ((uint32_t)(m * NCW + code) << kShift));
      }
    };

    // Software pipeline over steps (j = st % kBufs selects X buffer and register set):
    //   K-block kb of step st: read the operands of the next K-block, issue part kb of the loads of
    //   step st + kPre, then the MFMAs of kb. Before the MFMAs of K-block 3 each wave waits for its
    //   loads of step st + 1 and the workgroup synchronises (every wave's X slots of step st + 1
    //   are in; every wave has read step st's operands, whose buffer the loads issued during step
    //   st + 1 overwrite), and K-block 0 of step st + 1 is read: the MFMA stream never waits for
    //   the first reads of a step.
    Frag<M, CB> f[kBufs];
    Ops o[2];
#pragma unroll
    for (int j = 0; j < kPre; ++j)
#pragma unroll
      for (int part = 0; part < 3; ++part) issue_part(j, j, f[j], part);
    wait_vmcnt<(kPre - 1) * kLoads>();
    __syncthreads();
    read_ops(0, f[0], 0, o[0]);

    auto step = [&](int st, int j) {                           // j = st % kBufs, a constant
      const int jn = (j + 1) % kBufs, jl = (j + kPre) % kBufs;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        if (kb < 3) {
          read_ops(j, f[j], kb + 1, o[(kb + 1) & 1]);
          issue_part(st + kPre, jl, f[jl], kb);
        } else {
          wait_vmcnt<(kPre - 1) * kLoads>();                   // this wave's loads of step st + 1
          __syncthreads();
          read_ops(jn, f[jn], 0, o[0]);                        // past the last step: unused
        }
        __builtin_amdgcn_sched_barrier(0);
        const Ops& c = o[kb & 1];
#pragma unroll
        for (int na = 0; na < NA; ++na)
          acc[0][na] = __builtin_amdgcn_mfma_f32_32x32x16_f16(c.xa[na], f[j].w[kb], acc[0][na], 0, 0, 0);
#pragma unroll
        for (int m = 0; m < M; ++m)
#pragma unroll
          for (int na = 0; na < NA; ++na)
            acc[m + 1][na] = __builtin_amdgcn_mfma_f32_32x32x16_f16(c.xa[na], c.bq[m], acc[m + 1][na], 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
      }
    };
    // Whole rounds of kBufs steps, then the last nsteps % kBufs steps: a loop body without
    // skipped steps lets the compiler see when each register set was loaded.
    int st0 = 0;
    for (; st0 + kBufs <= nsteps; st0 += kBufs) {
#pragma unroll
      for (int j = 0; j < kBufs; ++j) step(st0 + j, j);
    }
#pragma unroll
    for (int j = 0; j < kBufs - 1; ++j)
      if (st0 + j < nsteps) step(st0 + j, j);
    // R_k = P - s (Q_0 + ... + Q_{k-1}) for each output (sample t, row), summed squared over the
    // outputs inside the matrix. Element e of an accumulator is sample 8 (e / 4) + 4 h + e % 4 of
    // its block, row r32 of the wave's block.
    const float sc = f16_to_f32(a.scales[rowc]);
#pragma unroll
    for (int na = 0; na < NA; ++na) {
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int t = t0 + na * 32 + 8 * (e >> 2) + 4 * h + (e & 3);
        const bool ok = row_ok && t < a.n;
        float r = acc[0][na][e];
#pragma unroll
        for (int m = 0; m < M; ++m) {
          r -= sc * acc[m + 1][na][e];
          if (ok) part[m] += (double)r * (double)r;
        }
      }
    }
    wait_vmcnt<0>();                                           // loads past the last step
    __syncthreads();                                           // X buffers are restaged next item
  }
  // Workgroup sums in a fixed order: butterfly within each wave, then waves 0..3.
#pragma unroll
  for (int m = 0; m < M; ++m) {
    double v = part[m];
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
    if (lane == 0) red[wave][m] = v;
  }
  __syncthreads();
  if (tid < M) a.partials[(size_t)blockIdx.x * 8 + tid] = ((red[0][tid] + red[1][tid]) + red[2][tid]) + red[3][tid];
}

// D[m] = (sum of the workgroup sums) / (d_out n): thread b loads workgroup b's sums, then a tree
// with a fixed pairing (b + half into b) adds them, so the result does not depend on scheduling.
__global__ __launch_bounds__(dist::kMaxGrid) void distortion_reduce_kernel(const double* partials, int grid, int M,
                                                                          double inv, double* D) {
  __shared__ double s[8][dist::kMaxGrid];
  const int b = threadIdx.x;
#pragma unroll
  for (int m = 0; m < 8; ++m) s[m][b] = (b < grid && m < M) ? partials[(size_t)b * 8 + m] : 0.0;
  __syncthreads();
  for (int half = dist::kMaxGrid / 2; half >= 1; half >>= 1) {
    if (b < half)
#pragma unroll
      for (int m = 0; m < 8; ++m) s[m][b] += s[m][b + half];
    __syncthreads();
  }
  if (b < M) D[b] = s[b][0] * inv;
}

template <int M, int CB>
static hipError_t launch_dist_mc(DistArgs& a, hipStream_t st, int* grid_out) {
  using C = dist::Cfg<M, CB>;
  a.n_rb = (a.d_out + dist::kRows - 1) / dist::kRows;
  a.n_items = a.n_rb * ((a.n + C::kTok - 1) / C::kTok);
  const int grid = a.n_items < dist::kMaxGrid ? a.n_items : dist::kMaxGrid;
  static_assert(C::kLds <= 160 * 1024 - 512, "LDS budget");
  distortion_kernel<M, CB><<<grid, dist::kThreads, C::kLds, st>>>(a);
  *grid_out = grid;
  return hipGetLastError();
}

template <int M>
static hipError_t launch_dist_m(DistArgs& a, int code_bits, hipStream_t st, int* grid_out) {
  return code_bits == 4 ? launch_dist_mc<M, 4>(a, st, grid_out) : launch_dist_mc<M, 8>(a, st, grid_out);
}

hipError_t launch_distortion(const Layer& L, const void* W, const void* X, int n, double* D, double* scratch,
                             hipStream_t st) {
  DistArgs a{};
  a.codes = L.codes;
  a.codebooks = L.codebooks;
  a.scales = L.scales;
  a.W = (const uint16_t*)W;
  a.X = (const uint16_t*)X;
  a.partials = scratch;                            // [grid][8], every slot written before it is read
  a.zero_page = L.zero_page();
  a.plane_bytes = L.plane_bytes;
  a.d_out = L.d.d_out;
  a.d_in = L.d.d_in;
  a.n = n;
  int grid = 0;
  hipError_t e;
  switch (L.resident) {                            // the resident levels
    case 1: e = launch_dist_m<1>(a, L.d.code_bits, st, &grid); break;
    case 2: e = launch_dist_m<2>(a, L.d.code_bits, st, &grid); break;
    case 3: e = launch_dist_m<3>(a, L.d.code_bits, st, &grid); break;
    case 4: e = launch_dist_m<4>(a, L.d.code_bits, st, &grid); break;
    case 5: e = launch_dist_m<5>(a, L.d.code_bits, st, &grid); break;
    case 6: e = launch_dist_m<6>(a, L.d.code_bits, st, &grid); break;
    case 7: e = launch_dist_m<7>(a, L.d.code_bits, st, &grid); break;
    default: e = launch_dist_m<8>(a, L.d.code_bits, st, &grid); break;
  }
  if (e != hipSuccess) return e;
  distortion_reduce_kernel<<<1, dist::kMaxGrid, 0, st>>>(a.partials, grid, L.resident,
                                             1.0 / ((double)L.d.d_out * (double)n), D);
  return hipGetLastError();
}

}  // namespace aqmb
