// Adapter weight gradients (FourTune Sec. 3.2, the gradients after Eq. 3):
//   dB = (X A)^T G      dB[j,n] = sum_m xa[m,j]  G[m,n]
//   dA = X^T (G B^T)    dA[k,j] = sum_m X[m,k]   gbt[m,j]
// Both are sums over the token axis m of a skinny fp32 factor L[m, j]
// (r columns) times a wide bf16 tensor V[m, c].  The reduction axis is the
// row axis of both operands in memory, so 64-row stages of both are copied to
// LDS as stored and the MFMA operands are gathered from there: V with the
// transposing 16-bit LDS read, L with 32-bit reads, split into two bf16 terms
// (hi + lo) so that its ~16 leading bits take part.
//
// Workgroup = 4 waves over 256 output columns (two 32-column tiles per wave,
// sharing each hi/lo split of L) and one chunk of the token axis.  With several chunks each one stores its fp32 partial in a
// workspace and a reduction kernel sums them in a fixed order.  Stages move through an LDS
// ring with buffer loads that write LDS directly, one or two stages ahead of
// the one on the matrix cores.  The two k-halves of an MFMA take the even and
// odd rows of a 16-row step, which keeps the 32-bit L reads conflict-free.
// dB's tile has j on the MFMA rows (A = L) and dA's has j on the columns
// (B = L), so both store contiguous runs in their output layout.
#include <mutex>

#include "ft_device.h"
#include "ft_kernels.h"

namespace ft {

constexpr int LG_WC = 256;                    // output columns per workgroup
constexpr int LG_BM = 64;                     // token rows per stage
constexpr int LG_VROW = LG_WC * 2;            // bytes per V row in LDS
constexpr int LG_VBYTES = LG_BM * LG_VROW;    // 32 KB

template <int RTJ>
struct LoraGeom {
  static constexpr int LROW = RTJ * 128;                  // bytes per L row (RTJ*32 fp32)
  static constexpr int LBYTES = LG_BM * LROW;
  static constexpr int SLOT = LG_VBYTES + LBYTES;
  static constexpr int NS = RTJ == 1 ? 3 : 2;             // ring slots
  static constexpr int PD = NS - 1;                       // stages in flight ahead
  static_assert(PD == 1 || PD == 2, "the prologue issues stages 0 and 1 and the waits allow one stage outstanding");
  static constexpr int V_LOADS = LG_VBYTES / 1024 / 4;    // per wave per stage
  static constexpr int L_LOADS = LBYTES / 1024 / 4;
  static constexpr int LOADS = V_LOADS + L_LOADS;
};

struct LoraJob {
  const float* L;       // [rows, ld] fp32; columns [0, r) used
  const uint16_t* V;    // [rows, C] bf16
  float* out;
  int C;
  int out_rows_are_j;   // 1: out[j * C + c] (dB);  0: out[c * r + j] (dA)
  int ncg;              // column groups of LG_WC
  uint32_t v_bytes;     // rows * C * 2  (< 2^31)
  uint32_t l_bytes;     // rows * ld * 4 (< 2^31)
  size_t part_off;      // offset of this output within a workspace part (floats)
};

// 16-byte chunk swizzle of a V row (32 chunks): rows 0..7 of a group spread
// their chunks over 16 positions.
__device__ __forceinline__ int lg_swz(int row, int chunk) { return chunk ^ ((row & 7) << 1); }

// One workgroup's share: output columns [c0, c0 + LG_WC) of `job` over token
// rows [mbeg, mend).  DB selects the operand roles and the store layout.
template <int RTJ, bool DB>
__device__ __forceinline__ void lora_tile(const LoraJob& job, uint8_t* lds, int c0, int mbeg, int mend, int ld, int r,
                                          float* part, int accumulate) {
  using G = LoraGeom<RTJ>;
  const int nst = (mend - mbeg + LG_BM - 1) / LG_BM;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const v4i rv = rsrc_words(job.V, job.v_bytes);
  const v4i rl = rsrc_words(job.L, job.l_bytes);
  const uint32_t lds0 = lds_addr(lds);

  // Per-lane DMA sources.  V load i of this wave fills LDS bytes
  // [1024 (8 wave + i), +1024) of the stage's V area: rows 2(8 wave + i) + lane/32,
  // physical chunk lane%32 holding logical chunk lg_swz(row, lane%32).
  int v_row[G::V_LOADS];
  uint32_t v_src[G::V_LOADS];
#pragma unroll
  for (int i = 0; i < G::V_LOADS; i++) {
    const int row = 2 * (G::V_LOADS * wave + i) + (lane >> 5);
    const int c = c0 + 8 * lg_swz(row, lane & 31);
    v_row[i] = row;
    v_src[i] = c < job.C ? (uint32_t)(row * job.C + c) * 2u : kOobOffset;
  }
  int l_row[G::L_LOADS];
  uint32_t l_src[G::L_LOADS];
#pragma unroll
  for (int i = 0; i < G::L_LOADS; i++) {
    const int byte = 1024 * (G::L_LOADS * wave + i) + 16 * lane;
    const int row = byte / G::LROW, q = (byte % G::LROW) / 16;
    l_row[i] = row;
    l_src[i] = 4 * q < r ? (uint32_t)(row * ld + 4 * q) * 4u : kOobOffset;
  }

  auto issue = [&](int s) {
    const int m0 = mbeg + s * LG_BM;
    const uint32_t slot = lds0 + (uint32_t)((s % G::NS) * G::SLOT);
    const uint32_t vs = (uint32_t)m0 * (uint32_t)job.C * 2u, ls = (uint32_t)m0 * (uint32_t)ld * 4u;
#pragma unroll
    for (int i = 0; i < G::V_LOADS; i++)
      dma16(rv, slot + 1024 * (G::V_LOADS * wave + i), m0 + v_row[i] < mend ? v_src[i] : kOobOffset, vs);
#pragma unroll
    for (int i = 0; i < G::L_LOADS; i++)
      dma16(rl, slot + LG_VBYTES + 1024 * (G::L_LOADS * wave + i), m0 + l_row[i] < mend ? l_src[i] : kOobOffset, ls);
  };

  // LDS read offsets within a slot.  V: source lane (jj, qq) of 16-lane group
  // g16 reads row 2 jj + h (+8 for the second read, +16 per k-step) at
  // logical column 64 wave + 32 t2 + 16 (g16 & 1) + 4 qq for column tile t2.
  // L: lane (j, h) reads rows 2e + h (+16 per k-step) of column j.
  const int g16 = lane >> 4, i16 = lane & 15, jj = i16 >> 2, qq = i16 & 3, h = g16 >> 1;
  const int vr0 = 2 * jj + h;
  uint32_t v_rd[2];
#pragma unroll
  for (int t2 = 0; t2 < 2; t2++) {
    const int vcol = 64 * wave + 32 * t2 + 16 * (g16 & 1) + 4 * qq;
    v_rd[t2] = (uint32_t)(vr0 * LG_VROW + lg_swz(vr0, vcol >> 3) * 16 + (vcol & 7) * 2);
  }
  const uint32_t l_rd = (uint32_t)(LG_VBYTES + h * G::LROW + 4 * (lane & 31));

  v16f acc[RTJ][2];
#pragma unroll
  for (int t = 0; t < RTJ; t++) acc[t][0] = acc[t][1] = v16f{};

  issue(0);
  if (G::PD > 1 && nst > 1) issue(1);
#pragma unroll 1
  for (int s = 0; s < nst; s++) {
    if (G::PD > 1 && s + 1 < nst) wait_vm<G::LOADS>();
    else wait_vm<0>();
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");  // no LDS read moves above the barrier
    if (s + G::PD < nst) issue(s + G::PD);

    // All of the stage's fragments are read first and the MFMAs follow: with
    // one wave per SIMD nothing else hides an LDS round trip, so the reads
    // must not be interleaved with the arithmetic that consumes them.
    const FT_LDS uint8_t* sb = (const FT_LDS uint8_t*)lds + (s % G::NS) * G::SLOT;
    v8bf vf[4][2];
    float lv[4][RTJ][8];
#pragma unroll
    for (int ks = 0; ks < 4; ks++) {
#pragma unroll
      for (int t2 = 0; t2 < 2; t2++) {
        const FT_LDS uint8_t* vp = sb + v_rd[t2] + ks * 16 * LG_VROW;
        vf[ks][t2] = make_v8bf(lds_read_tr16(vp), lds_read_tr16(vp + 8 * LG_VROW));
      }
#pragma unroll
      for (int t = 0; t < RTJ; t++) {
        const FT_LDS float* lp = (const FT_LDS float*)(sb + l_rd + ks * 16 * G::LROW + t * 128);
#pragma unroll
        for (int e = 0; e < 4; e++) {
          lv[ks][t][2 * e] = lp[4 * e * (G::LROW / 4)];
          lv[ks][t][2 * e + 1] = lp[(4 * e + 2) * (G::LROW / 4)];
        }
      }
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int ks = 0; ks < 4; ks++) {
#pragma unroll
      for (int t = 0; t < RTJ; t++) {
        v4i hi, lo;
#pragma unroll
        for (int e = 0; e < 4; e++) {
          uint32_t hp, lq;
          split_bf16x2(lv[ks][t][2 * e], lv[ks][t][2 * e + 1], hp, lq);
          hi[e] = (int)hp;
          lo[e] = (int)lq;
        }
        const v8bf ah = __builtin_bit_cast(v8bf, hi), al = __builtin_bit_cast(v8bf, lo);
#pragma unroll
        for (int t2 = 0; t2 < 2; t2++) {
          if constexpr (DB) acc[t][t2] = mfma_bf16_32x32x16(ah, vf[ks][t2], acc[t][t2]);
          else acc[t][t2] = mfma_bf16_32x32x16(vf[ks][t2], ah, acc[t][t2]);
        }
#pragma unroll
        for (int t2 = 0; t2 < 2; t2++) {
          if constexpr (DB) acc[t][t2] = mfma_bf16_32x32x16(al, vf[ks][t2], acc[t][t2]);
          else acc[t][t2] = mfma_bf16_32x32x16(vf[ks][t2], al, acc[t][t2]);
        }
      }
    }
  }

  // acc[t]: lane l, element v -> tile row 8(v/4) + 4h + v%4, tile column l%32.
  // dB: rows are j (t*32 + row), columns c;  dA: rows are c, columns j.
  const int l32 = lane & 31;
#pragma unroll
  for (int t = 0; t < RTJ; t++)
#pragma unroll
    for (int t2 = 0; t2 < 2; t2++)
#pragma unroll
      for (int v = 0; v < 16; v++) {
        const int tr = 8 * (v >> 2) + 4 * h + (v & 3);
        const int j = DB ? t * 32 + tr : t * 32 + l32;
        const int c = c0 + 64 * wave + 32 * t2 + (DB ? l32 : tr);
        if (j < r && c < job.C) {
          const size_t idx = DB ? (size_t)j * job.C + c : (size_t)c * r + j;
          if (part) part[job.part_off + idx] = acc[t][t2][v];
          else job.out[idx] = accumulate ? job.out[idx] + acc[t][t2][v] : acc[t][t2][v];
        }
      }
}

// parts: nmch workspace parts of part_len floats, or NULL when one chunk covers
// the token axis (outputs written directly, added to when accumulate).
template <int RTJ>
__global__ __launch_bounds__(256) void k_lora_grads(LoraJob jb0, LoraJob jb1, int M, int ld, int r, int mchunk,
                                                    int nmch, float* parts, size_t part_len, int accumulate) {
  __shared__ __attribute__((aligned(16))) uint8_t lds[LoraGeom<RTJ>::NS * LoraGeom<RTJ>::SLOT];
  int b = blockIdx.x;
  const int n0 = jb0.ncg * nmch;
  const bool second = b >= n0;
  if (second) b -= n0;
  const LoraJob& job = second ? jb1 : jb0;
  const int cg = b % job.ncg, mc = b / job.ncg;
  const int mbeg = mc * mchunk, mend = min(M, mbeg + mchunk);
  float* part = parts ? parts + (size_t)mc * part_len : nullptr;
  if (job.out_rows_are_j) lora_tile<RTJ, true>(job, lds, cg * LG_WC, mbeg, mend, ld, r, part, accumulate);
  else lora_tile<RTJ, false>(job, lds, cg * LG_WC, mbeg, mend, ld, r, part, accumulate);
}

// Token chunking: the fewest rounds of workgroups that keep at least 90 % of
// the CUs busy (one round at the QKV and MLP shapes; two for the single-
// stream shapes, where one round of 96 column groups left a quarter of the
// CUs idle: 18432 x (3072 + 21504) 268-287 -> 249-275 us).  Every ring takes
// more than half of LDS (96 KB or more), so a CU holds one workgroup.
static void lg_geometry(int rows, int K, int N, int r, int& nmch, int& mchunk) {
  const int rtj = (r + 31) / 32;
  const int slot_bytes = LG_VBYTES + LG_BM * rtj * 128, ns = rtj == 1 ? 3 : 2;
  const int slots = (2 * ns * slot_bytes <= 160 * 1024 ? 2 : 1) * 256;
  const int ncg = (N + LG_WC - 1) / LG_WC + (K + LG_WC - 1) / LG_WC;
  const int mblocks = (rows + LG_BM - 1) / LG_BM;
  nmch = std::max(1, std::min(mblocks, slots / ncg));
  for (int k = 1; k <= 4; k++) {
    const int c = std::min(mblocks, k * slots / ncg);
    if (c >= 1 && (double)ncg * c >= 0.9 * k * slots) {
      nmch = c;
      break;
    }
  }
  mchunk = ((mblocks + nmch - 1) / nmch) * LG_BM;
  nmch = (rows + mchunk - 1) / mchunk;
}

// Token windows small enough that every buffer stays below 2 GiB, so the
// out-of-range offset used for masked lanes is beyond every buffer.
static size_t lg_window(int M, int K, int N, int ld) {
  const size_t lim = (size_t)1 << 31;
  const size_t seg = std::min(lim / ((size_t)std::max(K, N) * 2), lim / ((size_t)ld * 4));
  return std::min((size_t)M, seg / LG_BM * LG_BM);
}

size_t lora_grads_workspace(int M, int K, int N, int ld, int r) {
  if (M == 0) return 0;
  const size_t seg = lg_window(M, K, N, ld);
  if (seg == 0) return 0;
  int nmch, mchunk;
  lg_geometry((int)seg, K, N, r, nmch, mchunk);   // the first window has the most chunks
  return nmch > 1 ? (size_t)nmch * r * ((size_t)N + K) * sizeof(float) : 0;
}

hipError_t launch_lora_grads(const uint16_t* x, int M, int K, const uint16_t* dy, int N, const float* xa,
                             const float* dyb, int ld, int r, float* dA, float* dB, bool accumulate, float* ws,
                             hipStream_t st) {
  if (M == 0)  // empty sums: zeros (a reduction over no parts), or nothing to add
    return accumulate ? hipSuccess : launch_reduce_parts(nullptr, 0, (size_t)r * N, dB, (size_t)K * r, dA, false, st);
  const size_t seg = lg_window(M, K, N, ld);
  if (seg == 0) return hipErrorInvalidValue;
  const size_t part_len = (size_t)r * ((size_t)N + K);
  for (size_t m0 = 0; m0 < (size_t)M; m0 += seg) {
    const int rows = (int)std::min(seg, (size_t)M - m0);
    const bool acc = accumulate || m0 > 0;
    const LoraJob jobB{xa + m0 * ld, dy + m0 * N, dB, N, 1, (N + LG_WC - 1) / LG_WC,
                       (uint32_t)((size_t)rows * N * 2), (uint32_t)((size_t)rows * ld * 4), 0};
    const LoraJob jobA{dyb + m0 * ld, x + m0 * K, dA, K, 0, (K + LG_WC - 1) / LG_WC,
                       (uint32_t)((size_t)rows * K * 2), (uint32_t)((size_t)rows * ld * 4), (size_t)r * N};
    int nmch, mchunk;
    lg_geometry(rows, K, N, r, nmch, mchunk);
    float* parts = nmch > 1 ? ws : nullptr;
    const unsigned grid = (unsigned)((jobB.ncg + jobA.ncg) * nmch);
    switch ((r + 31) / 32) {
      case 1: k_lora_grads<1><<<grid, 256, 0, st>>>(jobB, jobA, rows, ld, r, mchunk, nmch, parts, part_len, acc); break;
      case 2: k_lora_grads<2><<<grid, 256, 0, st>>>(jobB, jobA, rows, ld, r, mchunk, nmch, parts, part_len, acc); break;
      case 3: k_lora_grads<3><<<grid, 256, 0, st>>>(jobB, jobA, rows, ld, r, mchunk, nmch, parts, part_len, acc); break;
      default: k_lora_grads<4><<<grid, 256, 0, st>>>(jobB, jobA, rows, ld, r, mchunk, nmch, parts, part_len, acc); break;
    }
    hipError_t e = hipGetLastError();
    if (e == hipSuccess && parts) e = launch_reduce_parts(parts, nmch, (size_t)r * N, dB, (size_t)K * r, dA, acc, st);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// ------------------------------------------------ allocation-free variant
// Scratch for callers that cannot allocate (code under graph capture, tight
// serving loops): the token-chunk partials live in this file-scope array,
// which every GPU the library runs on holds until the process ends.  Host
// code never passes `scratch` itself (its host-side name is not a device
// address): the device address comes from hipGetSymbolAddress, looked up once
// per device with that device current and kept per device.
static __device__ __align__(256) float scratch[kLoraScratchBytes / sizeof(float)];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
float* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

hipError_t lora_grads_scratch(float** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = (float*)p;
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace ft
