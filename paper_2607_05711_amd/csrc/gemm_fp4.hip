// Block-scaled FP4 GEMM for the triple-branch linear (gfx950).
//
// Forward (FourTune Eq. 2):   Y  = DQ(Xq) DQ(Wq)^T + P U + bias
// Backward (Eq. 3):           dX = DQ(Gq) DQ(Wq)   + Qp D^T
// The backward reads the forward's weight codes and 32x32 scales in
// transposed order (Sec. 3.2): the weight tile is staged in LDS as stored
// ([n][k], two codes per byte) and the B operand is gathered with the
// nibble-transposing LDS read, so no transposed or re-quantized weight copy
// exists.  The low-rank term is folded into the same fp32 accumulators in
// the epilogue (Sec. 3.3) with bf16 MFMAs, P split into two bf16 terms.
//
// Workgroup: 256 threads = 4 waves in a 2x2 grid; tile 256x256 outputs,
// each wave 128x128 = 4x4 MFMA tiles of 32x32 (256 fp32 accumulators per
// lane).  Reduction staged 256 elements (128 bytes of codes per row) at a
// time, double-buffered through LDS with a 16-byte row pad, loads for stage
// s+1 in flight while stage s runs on the matrix cores.
#include <type_traits>

#include "ft_device.h"
#include "ft_kernels.h"

namespace ft {

constexpr int GB = 256;                 // output tile edge (rows and columns)
constexpr int GK = 256;                 // reduction elements per stage
constexpr int GROW = GK / 2;            // bytes of codes per tile row per stage
constexpr int GSTRIDE = GROW + 16;      // padded LDS row stride (bytes)
constexpr int GTILE = GB * GSTRIDE;     // bytes per operand tile per stage

template <bool BWD, bool OUT_F32>
__global__ __launch_bounds__(256, 1) void k_gemm_fp4_generic(const uint8_t* __restrict__ A, const uint8_t* __restrict__ As,
                                                     const uint8_t* __restrict__ Wq, const uint8_t* __restrict__ Ws,
                                                     int M, int N, int K, const float* __restrict__ P, int R,
                                                     const uint16_t* __restrict__ LR,
                                                     const uint16_t* __restrict__ bias, void* __restrict__ out) {
  __shared__ __attribute__((aligned(16))) uint8_t lds[2 * 2 * GTILE];

  // Output is [M, NO]; the reduction runs over KR.
  const int NO = BWD ? K : N;
  const int KR = BWD ? N : K;
  const int lda = KR >> 1;              // bytes per row of A codes
  const int nkb = KR >> 5;              // scale blocks per row of A
  const int ldw = K >> 1;               // bytes per row of W codes
  const int nwkb = K >> 5;              // scale columns of W

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r32 = lane & 31, h = lane >> 5, g16 = lane >> 4, t16 = lane & 15;
  const int wm = wave >> 1, wn = wave & 1;
  const int m0 = blockIdx.y * GB, n0 = blockIdx.x * GB;

  // ---- global -> register staging (8 x 16 bytes per operand per thread)
  uint4 ra[8], rb[8];
  uint32_t sa_n[4], sb_n[4];

  auto load_stage = [&](int s) {
    const int kbyte0 = s * GROW;  // byte offset along the reduction in A rows
#pragma unroll
    for (int i = 0; i < 8; i++) {
      const int c = tid + 256 * i, row = c >> 3, col = (c & 7) * 16;
      const int gm = min(m0 + row, M - 1);
      ra[i] = (kbyte0 + col < lda) ? *(const uint4*)(A + (size_t)gm * lda + kbyte0 + col) : make_uint4(0, 0, 0, 0);
      if constexpr (!BWD) {
        const int gn = min(n0 + row, N - 1);
        rb[i] = (kbyte0 + col < ldw) ? *(const uint4*)(Wq + (size_t)gn * ldw + kbyte0 + col) : make_uint4(0, 0, 0, 0);
      } else {
        // W rows are the reduction index n; columns are output k (two per byte)
        const int gn = s * GK + row;
        const int kb = (n0 >> 1) + col;
        rb[i] = (gn < N && kb < ldw) ? *(const uint4*)(Wq + (size_t)gn * ldw + kb) : make_uint4(0, 0, 0, 0);
      }
    }
    // scales for stage s: byte kk of the word = k-step kk (64 elements), block 2kk + h
    const int kb0 = s * (GK / 32);
#pragma unroll
    for (int i = 0; i < 4; i++) {
      const int gm = min(m0 + wm * 128 + i * 32 + r32, M - 1);
      uint32_t w = 0;
#pragma unroll
      for (int kk = 0; kk < 4; kk++) {
        const int kb = kb0 + 2 * kk + h;
        const uint32_t b = kb < nkb ? As[(size_t)gm * nkb + kb] : 127u;
        w |= b << (8 * kk);
      }
      sa_n[i] = w;
    }
#pragma unroll
    for (int j = 0; j < 4; j++) {
      uint32_t w = 0;
      const int col = n0 + wn * 128 + j * 32;  // first output column of the MFMA tile
#pragma unroll
      for (int kk = 0; kk < 4; kk++) {
        const int kb = kb0 + 2 * kk + h;        // reduction block
        uint32_t b = 127u;
        if (kb < (KR >> 5)) {
          if constexpr (!BWD) b = Ws[(size_t)(min(col, N - 32) >> 5) * nwkb + kb];
          else b = Ws[(size_t)kb * nwkb + (min(col, K - 32) >> 5)];
        }
        w |= b << (8 * kk);
      }
      sb_n[j] = w;
    }
  };

  auto store_stage = [&](int buf) {
    uint8_t* la = lds + buf * 2 * GTILE;
    uint8_t* lb = la + GTILE;
#pragma unroll
    for (int i = 0; i < 8; i++) {
      const int c = tid + 256 * i, row = c >> 3, col = (c & 7) * 16;
      *(uint4*)(la + row * GSTRIDE + col) = ra[i];
      *(uint4*)(lb + row * GSTRIDE + col) = rb[i];
    }
  };

  v16f acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; i++)
#pragma unroll
    for (int j = 0; j < 4; j++) acc[i][j] = v16f{};

  const int nst = (KR + GK - 1) / GK;
  uint32_t sa[4], sb[4];
  load_stage(0);
  store_stage(0);
#pragma unroll
  for (int i = 0; i < 4; i++) { sa[i] = sa_n[i]; sb[i] = sb_n[i]; }
  __syncthreads();

#pragma unroll 1
  for (int s = 0; s < nst; s++) {
    const int cur = s & 1;
    if (s + 1 < nst) load_stage(s + 1);
    const uint8_t* la = lds + cur * 2 * GTILE;
    const uint8_t* lb = la + GTILE;
#pragma unroll
    for (int kk = 0; kk < 4; kk++) {
      v4i af[4], bf[4];
#pragma unroll
      for (int i = 0; i < 4; i++)
        af[i] = *(const v4i*)(la + (wm * 128 + i * 32 + r32) * GSTRIDE + (2 * kk + h) * 16);
#pragma unroll
      for (int j = 0; j < 4; j++) {
        if constexpr (!BWD) {
          bf[j] = *(const v4i*)(lb + (wn * 128 + j * 32 + r32) * GSTRIDE + (2 * kk + h) * 16);
        } else {
          const int row = kk * 64 + 32 * h + t16;
          const int byte = wn * 64 + j * 16 + 8 * (g16 & 1);
          const v2i lo = lds_read_tr4((const FT_LDS void*)(lb + row * GSTRIDE + byte));
          const v2i hi = lds_read_tr4((const FT_LDS void*)(lb + (row + 16) * GSTRIDE + byte));
          bf[j] = v4i{lo[0], lo[1], hi[0], hi[1]};
        }
      }
#pragma unroll
      for (int i = 0; i < 4; i++)
#pragma unroll
        for (int j = 0; j < 4; j++) {
          if (kk == 0) acc[i][j] = mfma_fp4_32x32x64<0>(af[i], bf[j], acc[i][j], (int)sa[i], (int)sb[j]);
          if (kk == 1) acc[i][j] = mfma_fp4_32x32x64<1>(af[i], bf[j], acc[i][j], (int)sa[i], (int)sb[j]);
          if (kk == 2) acc[i][j] = mfma_fp4_32x32x64<2>(af[i], bf[j], acc[i][j], (int)sa[i], (int)sb[j]);
          if (kk == 3) acc[i][j] = mfma_fp4_32x32x64<3>(af[i], bf[j], acc[i][j], (int)sa[i], (int)sb[j]);
        }
    }
    if (s + 1 < nst) store_stage(cur ^ 1);
#pragma unroll
    for (int i = 0; i < 4; i++) { sa[i] = sa_n[i]; sb[i] = sb_n[i]; }
    __syncthreads();
  }

  // ---- epilogue: low-rank up-projection into the same accumulators
  for (int jb = 0; jb < R; jb += 16) {
    v8bf ahi[4], alo[4], bv[4];
#pragma unroll
    for (int i = 0; i < 4; i++) {
      const int gm = min(m0 + wm * 128 + i * 32 + r32, M - 1);
      const float4* pp = (const float4*)(P + (size_t)gm * R + jb + 8 * h);
      const float4 p0 = pp[0], p1 = pp[1];
      const float pv[8] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
      uint32_t hh[8], ll[8];
#pragma unroll
      for (int e = 0; e < 8; e++) split_bf16(pv[e], hh[e], ll[e]);
      ahi[i] = pack_v8bf(hh);
      alo[i] = pack_v8bf(ll);
    }
#pragma unroll
    for (int j = 0; j < 4; j++) {
      const int gc = min(n0 + wn * 128 + j * 32 + r32, NO - 1);
      if constexpr (!BWD) {
        uint32_t u[8];
#pragma unroll
        for (int e = 0; e < 8; e++) u[e] = LR[(size_t)(jb + 8 * h + e) * N + gc];
        bv[j] = pack_v8bf(u);
      } else {
        bv[j] = __builtin_bit_cast(v8bf, *(const v4i*)(LR + (size_t)gc * R + jb + 8 * h));
      }
    }
#pragma unroll
    for (int i = 0; i < 4; i++)
#pragma unroll
      for (int j = 0; j < 4; j++) {
        acc[i][j] = mfma_bf16_32x32x16(ahi[i], bv[j], acc[i][j]);
        acc[i][j] = mfma_bf16_32x32x16(alo[i], bv[j], acc[i][j]);
      }
  }

  // ---- bias and store
#pragma unroll
  for (int j = 0; j < 4; j++) {
    const int gc = n0 + wn * 128 + j * 32 + r32;
    const bool col_ok = gc < NO;
    float bb = 0.0f;
    if constexpr (!BWD) {
      if (bias && col_ok) bb = bf16_to_f32(bias[gc]);
    }
#pragma unroll
    for (int i = 0; i < 4; i++) {
#pragma unroll
      for (int v = 0; v < 16; v++) {
        const int gr = m0 + wm * 128 + i * 32 + 8 * (v >> 2) + 4 * h + (v & 3);
        if (col_ok && gr < M) {
          const float y = acc[i][j][v] + bb;
          if constexpr (OUT_F32) ((float*)out)[(size_t)gr * NO + gc] = y;
          else ((uint16_t*)out)[(size_t)gr * NO + gc] = (uint16_t)f32_to_bf16_rne(y);
        }
      }
    }
  }
}


// ============================================================== fast path
// Pipelined kernel for reduction lengths that are multiples of 128 (and, for
// the backward, K a multiple of 128).  Stages of work move through a 2-slot
// LDS ring filled by buffer loads that write LDS directly; rows past the
// matrix edge read as zeros through the buffer range check, so tiles need no
// branches.
//
// Stage kinds:
//   FP4 stage: 256 reduction elements, so that each tile row of a stage is one
//     whole 128-byte line: what the loads cost follows the number of lines
//     they touch more than their bytes.  Slot = A tile [256 rows][128 B] +
//     W tile (forward [256 n][128 B]; backward [256 reduction rows][128 B],
//     read with the nibble-transposing LDS read) + the stage's E8M0 scales.
//     When the reduction length is an odd multiple of 128, the upper half of
//     the last stage reads as zeros.
//   Low-rank stage (after the FP4 stages): 32 columns of the up-projection.
//     Slot = P chunk [256 rows][32 fp32] + U chunk (forward, [32 j][256 n]
//     bf16) or D chunk (backward, [256 k][32 j] bf16).  P is split into two
//     bf16 terms in registers; its product lands in the same accumulators.
// An FP4 stage runs as four k-steps of 16 MFMAs per wave (a low-rank stage
// as two of 32), each carrying the LDS reads of the next.  The loads of stage
// s+2 start right after the barrier that publishes stage s+1 (the slot of
// stage s is free from then on) and spread over k-step 3 of stage s and
// k-steps 0 and 1 of stage s+1, one load per two MFMAs at most: a load that
// fills LDS holds its wave for about one MFMA's time when the four waves
// issue loads back to back, much less when they are spaced.  The barrier
// before the last k-step of stage s+1 publishes stage s+2.
// The finished tile is staged through LDS for coalesced stores.

constexpr int PK = 256;                  // reduction elements per FP4 stage
constexpr int PROW = PK / 2;             // bytes per tile row per stage (one line)
constexpr int SLOT = 68 * 1024;          // bytes per ring slot
constexpr int NSLOT = 2;
constexpr int OFF_B = 32 * 1024;         // W tile / U / D chunk within a slot
constexpr int OFF_SA = 64 * 1024;        // A scales: 256 rows x 8 bytes
// With the reduction length a multiple of 512, the A scales of stages 2q and
// 2q+1 (16 contiguous bytes per row) load together into a ring of their own:
// one 16-byte load per row touches half the lines of two 8-byte ones.
constexpr int OFF_SAP = 2 * 68 * 1024;   // after the two slots
constexpr int SAP_SLOT = 256 * 16;       // bytes per stage pair; a third slot takes loads that do not apply
constexpr int OFF_SB = 66 * 1024;        // W scales: 4 waves x 256 bytes
constexpr int LR_COLS = 32;              // up-projection columns per low-rank stage

// Stage kinds, and a compile-time tag for the pipeline bodies.
enum { SK_NONE = 0, SK_FP4 = 1, SK_LR = 2 };
template <int V> struct IC { static constexpr int value = V; };

// 16-byte chunk swizzles: 64-byte rows (4 chunks) and 128-byte rows (8 chunks)
__device__ __forceinline__ int swz64(int r) { return ((r >> 1) ^ (r >> 2)) & 3; }
__device__ __forceinline__ int swz128(int r) { return (r & 7) ^ ((r >> 3) & 1); }

// Workgroup id -> output tile.  Consecutive ids go to different XCDs, so each
// XCD gets a contiguous range of tiles; within it tiles run in groups of 4
// tile-rows, which keeps their A rows and W columns together in that XCD's L2.
__device__ __forceinline__ void tile_coords(int bid, int tiles_m, int tiles_n, int& mt, int& nt) {
  const int T = tiles_m * tiles_n;
  int t = bid;
  if (T % 8 == 0) t = (bid & 7) * (T >> 3) + (bid >> 3);
  constexpr int GM = 4;
  const int gsize = GM * tiles_n;
  const int g = t / gsize, first = g * GM;
  const int gm = min(GM, tiles_m - first);
  const int w = t - g * gsize;
  mt = first + w % gm;
  nt = w / gm;
}

template <bool BWD, bool OUT_F32, int EPI, bool SAP>
__global__ __launch_bounds__(256, 1) void k_gemm_fp4_pipe(const uint8_t* __restrict__ A, const uint8_t* __restrict__ As,
                                                          const uint8_t* __restrict__ Wq, const uint8_t* __restrict__ Ws,
                                                          int M, int N, int K, const float* __restrict__ P, int R,
                                                          const uint16_t* __restrict__ LR,
                                                          const uint16_t* __restrict__ bias, void* __restrict__ out,
                                                          int tiles_m, int tiles_n, GemmEpilogue ep) {
  static_assert(OFF_SAP == NSLOT * SLOT, "pair ring follows the slots");
  __shared__ __attribute__((aligned(16))) uint8_t lds[NSLOT * SLOT + (SAP ? 3 * SAP_SLOT : 0)];

  const int NO = BWD ? K : N;
  const int KR = BWD ? N : K;
  const int lda = KR >> 1, nkb = KR >> 5, ldw = K >> 1, nwkb = K >> 5;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: keeps LDS bases in SGPRs
  const int r32 = lane & 31, h = lane >> 5, g16 = lane >> 4, t16 = lane & 15;
  const int wm = wave >> 1, wn = wave & 1;
  int mt, nt;
  tile_coords(blockIdx.x, tiles_m, tiles_n, mt, nt);
  const int m0 = mt * GB, n0 = nt * GB;

  const v4i ra = rsrc_words(A, (uint32_t)M * lda);
  const v4i rw = rsrc_words(Wq, (uint32_t)N * ldw);
  const v4i ras = rsrc_words(As, (uint32_t)M * nkb);
  const v4i rws = rsrc_words(Ws, (uint32_t)(N >> 5) * nwkb);
  const v4i rp = rsrc_words(P, (uint32_t)M * R * 4);
  const v4i rl = rsrc_words(LR, (uint32_t)(BWD ? K : N) * R * 2);
  const uint32_t lds0 = lds_addr(lds);

  const int nst = (KR + PK - 1) / PK;            // FP4 stages
  const int nfull = KR / PK;                     // ... of which whole (the last may be half)
  const bool half_last = nfull != nst;
  const int nlr = (R + LR_COLS - 1) / LR_COLS, total = nst + nlr;
  const bool half_lr = (R % LR_COLS) != 0;       // the last low-rank stage has 16 columns

  // Accumulator tiles are computed transposed (W fragment as MFMA operand A):
  // lane (r32, h) of tile acc[i][j] holds output row wm*128 + 32i + r32 and,
  // in element 4q + e, column wn*128 + 32j + 8q + 4h + e.

  // ---------------- per-lane load geometry (constant over stages)
  // Each buffer load takes a per-lane byte offset (rows outside the matrix
  // hold kOobOffset, which reads zeros) plus a uniform per-stage offset that
  // stays inside the row of every valid lane.
  // 128-byte-row tiles (A, W, P chunk): instruction u of this wave fills rows
  // wave*64 + 8u + [0,8); lane L -> row + L/8 and physical chunk L%8, which
  // holds logical chunk (L%8) ^ swz128(row) = c8 ^ (u & 1).
  const int r8 = lane >> 3;
  const int c8 = (lane & 7) ^ r8;
  const bool upper = (c8 & 4) != 0;              // logical chunks 4..7 (the upper half of a stage)
  uint32_t a_base[8], w_base[8];
#pragma unroll
  for (int u = 0; u < 8; u++) {
    const int r = wave * 64 + 8 * u + r8;
    const int c = c8 ^ (u & 1);
    a_base[u] = (m0 + r < M) ? (uint32_t)(m0 + r) * lda + c * 16 : kOobOffset;
    if constexpr (!BWD) {
      w_base[u] = (n0 + r < N) ? (uint32_t)(n0 + r) * ldw + c * 16 : kOobOffset;
    } else {
      // reduction row r of the stage; the tile's 256 output columns are 128 bytes of it
      const int byte = (n0 >> 1) + c * 16;
      w_base[u] = (byte < ldw) ? (uint32_t)r * ldw + byte : kOobOffset;
    }
  }
  // A scales: instruction v of wave w stages rows wave*64 + 32v + L/2, dword
  // L%2 (blocks 4(L%2)..+3 of the stage) at OFF_SA + 8*row + 4(L%2).
  uint32_t sa_base[2];
#pragma unroll
  for (int v = 0; v < 2; v++) {
    const int r = m0 + wave * 64 + 32 * v + (lane >> 1);
    sa_base[v] = (r < M) ? (uint32_t)r * nkb + 4 * (lane & 1) : kOobOffset;
  }
  // stage pairs: lane L of wave w loads row w*64 + L (16 bytes) into the pair ring
  const uint32_t sap_base = (m0 + wave * 64 + lane < M) ? (uint32_t)(m0 + wave * 64 + lane) * nkb : kOobOffset;
  // W scales (lanes 0..3 of each wave, two 8-byte rows per wave):
  //   forward: 32-column block 2w + L/2 of the tile, dword L%2 of the stage;
  //   backward: reduction block 2w + L/2 of the stage, dword L%2 (column
  //   blocks 4(L%2)..+3 of the tile).
  // Row b lands at OFF_SB + (b/2)*256 + (b%2)*8 (each wave writes its own 256 bytes).
  uint32_t sb_base = kOobOffset;
  if (lane < 4) {
    const int b = 2 * wave + (lane >> 1), d = lane & 1;
    if constexpr (!BWD) {
      const int nb = (n0 >> 5) + b;
      if (nb < (N >> 5)) sb_base = (uint32_t)nb * nwkb + 4 * d;
    } else {
      const int kb = (n0 >> 5) + 4 * d;
      if (kb < nwkb) sb_base = (uint32_t)b * nwkb + kb;
    }
  }
  auto slot_of = [&](int t) { return (uint32_t)((t & (NSLOT - 1)) * SLOT); };
  auto kind_of = [&](int u) { return u >= total ? SK_NONE : (u < nst ? SK_FP4 : SK_LR); };

  // ---------------- stage loads (LDS destinations and per-stage offsets are uniform)
  // One load at a time, so that loads can sit between MFMAs.  hf: the stage
  // is a half one (FP4: upper 128 reduction elements; low-rank: 16 columns),
  // whose missing part reads as zeros.
  // FP4 stage u, part 1: loads v < 8 fill A-tile rows wave*64 + 8v + [0,8);
  // v = 8, 9 stage A-scale rows wave*64 + 32(v-8) + [0,32).
  // SAP: the scales of stage pair (u, u+1), u even; go = false sends zeros
  // to the spare slot instead (no branch).
  auto pair_load = [&](int u, bool go) {
    dma16(ras, lds0 + OFF_SAP + (go ? ((u >> 1) & 1) : 2) * SAP_SLOT + wave * 1024, go ? sap_base : kOobOffset,
          (uint32_t)(u >> 1) * 16);
  };
  // (SAP: load 8 of an even stage brings the scales of the stage pair.)
  auto fp4_part1_one = [&](int u, int v, bool hf) {
    const uint32_t slot = lds0 + slot_of(u);
    if (v < 8) {
      dma16(ra, slot + (wave * 64 + 8 * v) * PROW, (hf && upper) ? kOobOffset : a_base[v], (uint32_t)u * PROW);
    } else if constexpr (SAP) {
      if (v == 8 && (u & 1) == 0) pair_load(u, true);
    } else {
      dma4(ras, slot + OFF_SA + (wave * 64 + 32 * (v - 8)) * 8, (hf && (lane & 1)) ? kOobOffset : sa_base[v - 8],
           (uint32_t)u * 8);
    }
  };
  // FP4 stage u, part 2: loads v < 8 fill W-tile rows wave*64 + 8v + [0,8);
  // v = 8 stages this wave's two W-scale rows.
  auto fp4_part2_one = [&](int u, int v, bool hf) {
    const uint32_t slot = lds0 + slot_of(u);
    if constexpr (!BWD) {
      if (v < 8)
        dma16(rw, slot + OFF_B + (wave * 64 + 8 * v) * PROW, (hf && upper) ? kOobOffset : w_base[v],
              (uint32_t)u * PROW);
      else
        dma4(rws, slot + OFF_SB + wave * 256, (hf && (lane & 1)) ? kOobOffset : sb_base, (uint32_t)u * 8);
    } else {
      // rows 128..255 of a half stage (waves 2, 3) are past the matrix
      const bool off = hf && wave >= 2;
      if (v < 8)
        dma16(rw, slot + OFF_B + (wave * 64 + 8 * v) * 128, off ? kOobOffset : w_base[v], (uint32_t)u * PK * ldw);
      else
        dma4(rws, slot + OFF_SB + wave * 256, off ? kOobOffset : sb_base, (uint32_t)u * 8 * nwkb);
    }
  };
  // Low-rank stage u (chunk q = u - nst), part 1, load v < 8: rows wave*64 +
  // 8v + [0,8) of the P chunk [256 rows][32 fp32], laid out like the A tile.
  auto lr_part1_one = [&](int u, int v, bool hf) {
    const uint32_t slot = lds0 + slot_of(u);
    const int q = u - nst;
    const int r = m0 + wave * 64 + 8 * v + r8;
    const uint32_t off = (r < M && !(hf && upper)) ? (uint32_t)r * R * 4 + (c8 ^ (v & 1)) * 16 : kOobOffset;
    dma16(rp, slot + (wave * 64 + 8 * v) * 128, off, (uint32_t)q * 128);
  };
  // Low-rank stage u, part 2, load v < 4 (instruction ins = 4 wave + v):
  //   forward U chunk [32 j][256 n] (512-byte rows): rows 2 ins, 2 ins + 1;
  //     lane L -> row + L/32, chunk (L%32) ^ (2*(row&3));
  //   backward D chunk [256 k][32 j] (64-byte rows): rows 16 ins + [0,16);
  //     lane L -> row + L/4, chunk (L%4) ^ swz64(row).
  auto lr_part2_one = [&](int u, int v, bool hf) {
    const uint32_t slot = lds0 + slot_of(u);
    const int q = u - nst;
    const int ins = 4 * wave + v;
    if constexpr (!BWD) {
      // rows 16..31 of a half chunk (waves 2, 3) are past U
      const int j = 2 * ins + (lane >> 5);
      const int c = (lane & 31) ^ (2 * (j & 3));
      const uint32_t off =
          (n0 + c * 8 < N && !(hf && wave >= 2)) ? (uint32_t)j * N * 2 + (uint32_t)(n0 + c * 8) * 2 : kOobOffset;
      dma16(rl, slot + OFF_B + ins * 1024, off, (uint32_t)q * 32 * N * 2);
    } else {
      // columns 16..31 of a half chunk (logical chunks 2, 3) are past D's rows
      const int k = 16 * ins + (lane >> 2);
      const int c = (lane & 3) ^ swz64(k);
      const uint32_t off = (n0 + k < K && !(hf && (c & 2))) ? (uint32_t)(n0 + k) * R * 2 + c * 16 : kOobOffset;
      dma16(rl, slot + OFF_B + ins * 1024, off, (uint32_t)q * 64);
    }
  };
  auto issue_part1 = [&](int u) {
    if (u >= total) return;
    if (u < nst) {
      const bool hf = half_last && u == nst - 1;
#pragma unroll
      for (int v = 0; v < 10; v++) fp4_part1_one(u, v, hf);
    } else {
      const bool hf = half_lr && u == total - 1;
#pragma unroll
      for (int v = 0; v < 8; v++) lr_part1_one(u, v, hf);
    }
  };
  auto issue_part2 = [&](int u) {
    if (u >= total) return;
    if (u < nst) {
      const bool hf = half_last && u == nst - 1;
#pragma unroll
      for (int v = 0; v < 9; v++) fp4_part2_one(u, v, hf);
    } else {
      const bool hf = half_lr && u == total - 1;
#pragma unroll
      for (int v = 0; v < 4; v++) lr_part2_one(u, v, hf);
    }
  };
  // Loads of either part for a stage of any kind, as one fixed instruction
  // sequence whose operands are picked by the (uniform) kind: the tail of the
  // tile runs without branches between its MFMAs.  A load a kind does not
  // have reads zeros (kOobOffset) into a part of the slot that kind leaves
  // unused; a stage past the end reads zeros into its free slot.  The
  // choices are made once per stage (bitwise logic: no branches).
  constexpr uint32_t SPARE = 48 * 1024;   // unused by low-rank stages: 4 waves x 1 KB
  struct StageSel { uint32_t slot; int u, q; bool fp, lr, hf; };
  auto stage_sel = [&](int u) {
    StageSel t;
    const int k = kind_of(u);
    t.u = u;
    t.q = u - nst;
    t.slot = lds0 + slot_of(u);
    t.fp = k == SK_FP4;
    t.lr = k == SK_LR;
    t.hf = t.lr ? (half_lr & (u == total - 1)) : (half_last & (u == nst - 1));
    return t;
  };
  auto any_part1_one = [&](const StageSel& t, int v) {
    if (v < 8) {
      const int r = m0 + wave * 64 + 8 * v + r8;
      const uint32_t p_off = (r < M) ? (uint32_t)r * R * 4 + (c8 ^ (v & 1)) * 16 : kOobOffset;
      const bool zero = !(t.fp | t.lr) | (t.hf & upper);
      const uint32_t off = zero ? kOobOffset : (t.lr ? p_off : a_base[v]);
      dma16(t.lr ? rp : ra, t.slot + (wave * 64 + 8 * v) * 128, off,
            t.lr ? (uint32_t)t.q * 128 : (uint32_t)t.u * PROW);
    } else if constexpr (SAP) {
      if (v == 8) pair_load(t.u, t.fp & ((t.u & 1) == 0));
    } else {
      const bool zero = !t.fp | (t.hf & ((lane & 1) != 0));
      dma4(ras, t.slot + OFF_SA + (wave * 64 + 32 * (v - 8)) * 8, zero ? kOobOffset : sa_base[v - 8],
           (uint32_t)t.u * 8);
    }
  };
  auto any_part2_one = [&](const StageSel& t, int v) {
    // zero halves of a half stage: forward W upper chunks; backward W rows of waves 2, 3
    const bool w_cut = BWD ? (t.hf & (wave >= 2)) : (t.hf & upper);
    if (v < 8) {
      const uint32_t w_off = (t.fp & !w_cut) ? w_base[v] : kOobOffset;
      const uint32_t w_dst = t.slot + OFF_B + (wave * 64 + 8 * v) * PROW;
      const uint32_t w_so = BWD ? (uint32_t)t.u * PK * ldw : (uint32_t)t.u * PROW;
      if (v < 4) {
        const int ins = 4 * wave + v;
        uint32_t l_off, l_so;
        if constexpr (!BWD) {
          // rows 16..31 of a half chunk (waves 2, 3) are past U
          const int j = 2 * ins + (lane >> 5);
          const int c = (lane & 31) ^ (2 * (j & 3));
          const bool ok = (n0 + c * 8 < N) & !(t.hf & (wave >= 2));
          l_off = ok ? (uint32_t)j * N * 2 + (uint32_t)(n0 + c * 8) * 2 : kOobOffset;
          l_so = (uint32_t)t.q * 32 * N * 2;
        } else {
          // columns 16..31 of a half chunk (logical chunks 2, 3) are past D's rows
          const int kk = 16 * ins + (lane >> 2);
          const int c = (lane & 3) ^ swz64(kk);
          const bool ok = (n0 + kk < K) & !(t.hf & ((c & 2) != 0));
          l_off = ok ? (uint32_t)(n0 + kk) * R * 2 + c * 16 : kOobOffset;
          l_so = (uint32_t)t.q * 64;
        }
        dma16(t.lr ? rl : rw, t.lr ? t.slot + OFF_B + ins * 1024 : w_dst, t.lr ? l_off : w_off,
              t.lr ? l_so : w_so);
      } else {
        dma16(rw, t.lr ? t.slot + SPARE + wave * 1024 : w_dst, w_off, w_so);
      }
    } else {
      const bool s_cut = BWD ? (t.hf & (wave >= 2)) : (t.hf & ((lane & 1) != 0));
      dma4(rws, t.slot + OFF_SB + wave * 256, (t.fp & !s_cut) ? sb_base : kOobOffset,
           BWD ? (uint32_t)t.u * 8 * nwkb : (uint32_t)t.u * 8);
    }
  };
  // Every load this wave issued has landed and its own LDS reads are done;
  // after the barrier the same holds for all waves.
  auto publish_all = [&]() {
    __builtin_amdgcn_s_waitcnt(0x0070);   // vmcnt(0) lgkmcnt(0)
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");        // no LDS read moves above the barrier
  };

  // ---------------- fragment reads
  const int sw_r = swz128(r32);                     // rows ... + r32 of 128-byte-row tiles
  const int sw_t = swz128(t16);                     // rows ... + t16 of the backward W tile
  const int sw_d = swz64(r32);                      // rows ... + r32 of the backward D chunk
  const uint32_t psel = h ? 0x07050301u : 0x06040200u;   // bytes h, h+2, h+4, h+6 of a dword pair

  // Per-lane LDS read offsets within a slot, one per k-step (a fragment read
  // is then one address add plus an immediate offset).
  uint32_t rd_a[4], rd_b[4], rd_t[4];
#pragma unroll
  for (int kk = 0; kk < 4; kk++) {
    rd_a[kk] = (wm * 128 + r32) * PROW + (((2 * kk + h) ^ sw_r) << 4);
    rd_b[kk] = OFF_B + (wn * 128 + r32) * PROW + (((2 * kk + h) ^ sw_r) << 4);
  }
#pragma unroll
  for (int j = 0; j < 4; j++)   // + kk * 64 rows for k-step kk
    rd_t[j] = OFF_B + (32 * h + t16) * 128 + (((wn * 4 + j) ^ sw_t) << 4) + 8 * (g16 & 1);
  const uint32_t rd_sa = OFF_SA + (wm * 128 + r32) * 8;

  struct Fp4Frag { v4i a[4], b[4]; };
  // Fragment q of k-step kk: q < 4 -> A row tile q; q >= 4 -> W tile q - 4
  // (backward: its two transposing halves are fragments 4 + 2j and 5 + 2j).
  constexpr int FRAG_READS = BWD ? 12 : 8;
  auto read_one = [&](int t, int kk, int q, Fp4Frag& f) {
    const uint8_t* slot = lds + slot_of(t);
    if (q < 4) {
      f.a[q] = *(const v4i*)(slot + rd_a[kk] + q * 32 * PROW);
    } else if constexpr (!BWD) {
      f.b[q - 4] = *(const v4i*)(slot + rd_b[kk] + (q - 4) * 32 * PROW);
    } else {
      const int j = (q - 4) >> 1, half = (q - 4) & 1;
      const v2i v = lds_read_tr4((const FT_LDS void*)(slot + rd_t[j] + (kk * 64 + half * 16) * 128));
      if (half == 0) { f.b[j][0] = v[0]; f.b[j][1] = v[1]; }
      else { f.b[j][2] = v[0]; f.b[j][3] = v[1]; }
    }
  };
  // Raw scale words of a stage (8 blocks per row or column block); turned
  // into MFMA scale operands (one byte per k-step) only when the stage's
  // MFMAs are about to issue.
  struct ScaleRaw { uint32_t a[8], b[8]; };
  auto read_scales_a = [&](int t, ScaleRaw& r) {
    const uint8_t* base = SAP ? lds + OFF_SAP + ((t >> 1) & 1) * SAP_SLOT + (wm * 128 + r32) * 16 + (t & 1) * 8
                              : lds + slot_of(t) + rd_sa;
#pragma unroll
    for (int i = 0; i < 4; i++) {
      const v2i d = *(const v2i*)(base + i * (SAP ? 512 : 256));
      r.a[2 * i] = (uint32_t)d[0];
      r.a[2 * i + 1] = (uint32_t)d[1];
    }
  };
  auto read_scales_b = [&](const uint8_t* slot, ScaleRaw& r) {
    if constexpr (!BWD) {
#pragma unroll
      for (int j = 0; j < 4; j++) {   // 32-column block b = wn*4 + j
        const int b = wn * 4 + j;
        const v2i d = *(const v2i*)(slot + OFF_SB + (b >> 1) * 256 + (b & 1) * 8);
        r.b[2 * j] = (uint32_t)d[0];
        r.b[2 * j + 1] = (uint32_t)d[1];
      }
    } else {
#pragma unroll
      for (int kk = 0; kk < 4; kk++)   // reduction block 2kk + h, column blocks wn*4 .. +3
        r.b[kk] = *(const uint32_t*)(slot + OFF_SB + kk * 256 + h * 8 + wn * 4);
    }
  };
  auto scale_ops = [&](const ScaleRaw& r, uint32_t (&sa)[4], uint32_t (&sb)[4]) {
#pragma unroll
    for (int i = 0; i < 4; i++) sa[i] = __builtin_amdgcn_perm(r.a[2 * i + 1], r.a[2 * i], psel);
#pragma unroll
    for (int j = 0; j < 4; j++) {
      if constexpr (!BWD) {
        sb[j] = __builtin_amdgcn_perm(r.b[2 * j + 1], r.b[2 * j], psel);
      } else {
        sb[j] = __builtin_amdgcn_perm(r.b[1], r.b[0], 0x0c0c0400u | (j << 8) | j) |
                __builtin_amdgcn_perm(r.b[3], r.b[2], 0x04000c0cu | (j << 24) | (j << 16));
      }
    }
  };

  v16f acc[4][4];

  // Low-rank fragments, one 16-column half c of a stage at a time: the raw
  // LDS words (P fp32, U or D bf16), and the MFMA operands made from them
  // (each P pair split into bf16 hi + lo).
  struct LrRaw { v4i p[4][2]; v4i b[4]; };
  struct LrOps { v4i hi[4], lo[4]; };
  const int jj = t16 >> 2, qq = t16 & 3;
  // Read q of half c of low-rank stage t: q < 8 -> P row tile q/2, dwords
  // 4(q%2)..+3 of the lane's eight; then the U / D fragment of each column
  // tile (forward: two transposing reads of 4 rows each).
  constexpr int LR_READS = BWD ? 12 : 16;
  auto lr_read_one = [&](int t, int c, int q, LrRaw& f) {
    const uint8_t* slot = lds + slot_of(t);
    if (q < 8) {
      const int i = q >> 1, e = q & 1;
      f.p[i][e] = *(const v4i*)(slot + (wm * 128 + i * 32 + r32) * 128 + (((4 * c + 2 * h + e) ^ sw_r) << 4));
    } else if constexpr (!BWD) {
      const int j = (q - 8) >> 1, half = (q - 8) & 1;
      const int n = wn * 128 + j * 32 + 16 * (g16 & 1) + 4 * qq;
      const int row = 16 * c + 8 * h + jj + 4 * half;
      const int byte = ((((n >> 3) ^ (2 * (row & 3))) << 4)) + ((n >> 2) & 1) * 8;
      const v2i v = __builtin_bit_cast(v2i, lds_read_tr16((const FT_LDS void*)(slot + OFF_B + row * 512 + byte)));
      f.b[j][2 * half] = v[0];
      f.b[j][2 * half + 1] = v[1];
    } else {
      const int j = q - 8;
      const int k = wn * 128 + j * 32 + r32;
      f.b[j] = *(const v4i*)(slot + OFF_B + k * 64 + (((2 * c + h) ^ sw_d) << 4));
    }
  };
  // Split pair e (fp32 elements 2e, 2e+1) of row tile i into bf16 hi + lo.
  auto lr_split = [&](const LrRaw& f, int i, int e, LrOps& o) {
    const v4i x = f.p[i][e >> 1];
    uint32_t hp, lp;
    split_bf16x2(__int_as_float(x[2 * (e & 1)]), __int_as_float(x[2 * (e & 1) + 1]), hp, lp);
    o.hi[i][e] = (int)hp;
    o.lo[i][e] = (int)lp;
  };
  // MFMA m of a low-rank half: m < 16 -> hi terms of tile (m/4, m%4), then the
  // lo terms in the same order (no accumulator is used twice in a row).
  auto lr_mfma = [&](int m, const LrRaw& f, const LrOps& o) {
    const int i = (m >> 2) & 3, j = m & 3;
    const v4i a = m < 16 ? o.hi[i] : o.lo[i];
    acc[i][j] = mfma_bf16_32x32x16(__builtin_bit_cast(v8bf, f.b[j]), __builtin_bit_cast(v8bf, a), acc[i][j]);
  };

  // ---------------- pipeline
  // Stage u: A-tile rows 0..3 of each wave's 8 and the A scales ("part 1a")
  // issued in iteration u-2 after its barrier; A-tile rows 4..7 and the W
  // tile and scales in iteration u-1 (k-steps 0 and 1).  Stage 0 and part 1a
  // of stage 1 start here.
  issue_part1(0);
  issue_part2(0);
  // Bias of this lane's columns (forward): four bf16 per (j, q), loaded
  // behind stage 0 so that the two latencies overlap.  Buffer loads without
  // branches: columns past N (and a missing bias, an empty buffer) read zeros.
  uint2 bias4[4][4];
  {
    const __amdgpu_buffer_rsrc_t rb = make_rsrc(bias, bias ? (uint32_t)N * 2 : 0u);
#pragma unroll
    for (int j = 0; j < 4; j++)
#pragma unroll
      for (int q = 0; q < 4; q++) {
        bias4[j][q] = make_uint2(0u, 0u);
        if constexpr (!BWD) {
          const int gc = n0 + wn * 128 + j * 32 + 8 * q + 4 * h;
          const v2i b = __builtin_amdgcn_raw_buffer_load_b64(rb, gc < N ? (uint32_t)gc * 2 : kOobOffset, 0, 0);
          bias4[j][q] = make_uint2((uint32_t)b[0], (uint32_t)b[1]);
        }
      }
  }
  if (1 < total) {
    if (1 < nst) {
      const bool hf = half_last && 1 == nst - 1;
#pragma unroll
      for (int v = 0; v < 4; v++) fp4_part1_one(1, v, hf);
      fp4_part1_one(1, 8, hf);
      fp4_part1_one(1, 9, hf);
    } else {
      const bool hf = half_lr && 1 == total - 1;
#pragma unroll
      for (int v = 0; v < 4; v++) lr_part1_one(1, v, hf);
    }
  }
  // Accumulators start at the bias (forward): every output's sum begins with
  // its bias term, in both output precisions.
#pragma unroll
  for (int i = 0; i < 4; i++)
#pragma unroll
    for (int j = 0; j < 4; j++)
#pragma unroll
      for (int q = 0; q < 4; q++) {
        acc[i][j][4 * q + 0] = bf16_to_f32(bias4[j][q].x & 0xFFFFu);
        acc[i][j][4 * q + 1] = bf16_to_f32(bias4[j][q].x >> 16);
        acc[i][j][4 * q + 2] = bf16_to_f32(bias4[j][q].y & 0xFFFFu);
        acc[i][j][4 * q + 3] = bf16_to_f32(bias4[j][q].y >> 16);
      }
  // stage 0 landed; part 1a of stage 1 (4 tile loads, plus 2 scale loads
  // without paired A scales: stage 1's pair loaded with stage 0) may stay in flight
  switch (1 >= total ? 0 : (1 < nst && !SAP ? 6 : 4)) {
    case 4: wait_vm<4>(); break;
    case 6: wait_vm<6>(); break;
    default: wait_vm<0>(); break;
  }
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
  Fp4Frag f0, f1;
  ScaleRaw sr;
  uint32_t sa[4], sb[4];
  LrRaw ga, gb;   // the two halves of a low-rank stage
#pragma unroll
  for (int q = 0; q < FRAG_READS; q++) read_one(0, 0, q, f0);
  read_scales_a(0, sr);
  read_scales_b(lds + slot_of(0), sr);
  scale_ops(sr, sa, sb);

  // One FP4 iteration.  ANY = 0: stages s+1 and s+2 are whole FP4 stages;
  // ANY = 1: they may be of any kind (their loads pick operands by kind, and
  // the reads of stage s+1 as FP4 fragments are simply unused when it is
  // not).  Every other instruction sits between two MFMAs (one wave per SIMD:
  // the matrix pipe only stays busy if nothing waits in front of the next
  // MFMA):
  //   k-step 0 carries the reads of k-step 1, A-tile rows 4..7 and W-tile
  //   rows 0..3 of stage s+1;
  //   k-step 1 carries the reads of k-step 2, W-tile rows 4..7 and the W
  //   scales of stage s+1;
  //   k-step 2 carries the reads of k-step 3;
  //   the barrier publishes stage s+1 and frees the slot of stage s;
  //   k-step 3 carries the reads of stage s+1's k-step 0 and scales, part 1a
  //   of stage s+2 (A-tile rows 0..3, A scales), and the scale operands of
  //   stage s+1.
  // PAR (whole stages only): the parity of s, which decides whether k-step 3
  // loads a pair of A-scale stages (SAP).
  auto fp4_body = [&](int s, auto anyc, auto parc) {
    constexpr bool ANY = decltype(anyc)::value != 0;
    constexpr int PAR = decltype(parc)::value;
    const StageSel t2 = stage_sel(s + 1), t1 = stage_sel(s + 2);
    const uint8_t* nslot = lds + slot_of(s + 1);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int m = 0; m < 16; m++) {
      const int i = m >> 2, j = m & 3;
      acc[i][j] = mfma_fp4_32x32x64<0>(f0.b[j], f0.a[i], acc[i][j], (int)sb[j], (int)sa[i]);
      if (m < FRAG_READS) read_one(s, 1, m, f1);
      if ((m & 3) == 0) {
        const int v = 4 + (m >> 2);
        if constexpr (ANY) any_part1_one(t2, v);
        else fp4_part1_one(s + 1, v, false);
      } else if ((m & 3) == 2) {
        const int v = m >> 2;
        if constexpr (ANY) any_part2_one(t2, v);
        else fp4_part2_one(s + 1, v, false);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int m = 0; m < 16; m++) {
      const int i = m >> 2, j = m & 3;
      acc[i][j] = mfma_fp4_32x32x64<1>(f1.b[j], f1.a[i], acc[i][j], (int)sb[j], (int)sa[i]);
      if (m < FRAG_READS) read_one(s, 2, m, f0);
      if ((m & 3) == 0 || m == 2) {
        const int v = m == 2 ? 8 : 4 + (m >> 2);
        if constexpr (ANY) any_part2_one(t2, v);
        else fp4_part2_one(s + 1, v, false);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int m = 0; m < 16; m++) {
      const int i = m >> 2, j = m & 3;
      acc[i][j] = mfma_fp4_32x32x64<2>(f0.b[j], f0.a[i], acc[i][j], (int)sb[j], (int)sa[i]);
      if (m < FRAG_READS) read_one(s, 3, m, f1);
      __builtin_amdgcn_sched_barrier(0);
    }
    publish_all();
    __builtin_amdgcn_sched_barrier(0);
    uint32_t nsa[4], nsb[4];
#pragma unroll
    for (int m = 0; m < 16; m++) {
      const int i = m >> 2, j = m & 3;
      acc[i][j] = mfma_fp4_32x32x64<3>(f1.b[j], f1.a[i], acc[i][j], (int)sb[j], (int)sa[i]);
      if (m < FRAG_READS) read_one(s + 1, 0, m, f0);
      if (m == FRAG_READS - 4) read_scales_a(s + 1, sr);
      if (m == FRAG_READS - 2) read_scales_b(nslot, sr);
      if ((m & 3) == 0 || m == 2 || m == 6) {
        const int v = m == 2 ? 8 : m == 6 ? 9 : m >> 2;
        if constexpr (ANY) {
          any_part1_one(t1, v);
        } else if constexpr (SAP) {
          if (v < 8) fp4_part1_one(s + 2, v, false);
          else if (v == 8 && PAR == 0) pair_load(s + 2, true);
        } else {
          fp4_part1_one(s + 2, v, false);
        }
      }
      if (m == 15) scale_ops(sr, nsa, nsb);
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int q = 0; q < 4; q++) { sa[q] = nsa[q]; sb[q] = nsb[q]; }
  };

  // One low-rank iteration (stage s >= nst, its first half in ga):
  //   half 0: 32 MFMAs carrying the hi/lo splits of its row tiles 1..3, the
  //   reads of half 1, and P rows 4..7 and the U / D chunk of stage s+1;
  //   the barrier publishes stage s+1 and frees the slot of stage s;
  //   half 1: likewise, carrying part 1a of stage s+2 (P rows 0..3) and the
  //   reads of stage s+1's first half (unused past the last stage).
  // P2 / P1: stage s+1 / s+2 exists (no loads are issued for stages past
  // the end).  The second half of a 16-column last stage reads as zeros and
  // adds zeros.
  auto lr_body = [&](int s, auto p2c, auto p1c) {
    constexpr bool P2 = decltype(p2c)::value != 0, P1 = decltype(p1c)::value != 0;
    const StageSel t2 = stage_sel(s + 1), t1 = stage_sel(s + 2);
    LrOps o;
#pragma unroll
    for (int e = 0; e < 4; e++) lr_split(ga, 0, e, o);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int m = 0; m < 32; m++) {
      lr_mfma(m, ga, o);
      if (m < 12) lr_split(ga, (m >> 2) + 1, m & 3, o);
      if (m >= 16 && m - 16 < LR_READS) lr_read_one(s, 1, m - 16, gb);
      if constexpr (P2) {
        if ((m & 3) == 0 && m < 16) any_part1_one(t2, 4 + (m >> 2));
        else if ((m & 3) == 2 && m < 16) any_part2_one(t2, m >> 2);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    publish_all();
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int e = 0; e < 4; e++) lr_split(gb, 0, e, o);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int m = 0; m < 32; m++) {
      lr_mfma(m, gb, o);
      if (m < 12) lr_split(gb, (m >> 2) + 1, m & 3, o);
      if constexpr (P1) { if ((m & 3) == 0 && m < 16) any_part1_one(t1, m >> 2); }
      if (m >= 16 && m - 16 < LR_READS) lr_read_one(s + 1, 0, m - 16, ga);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  int s = 0;
  // stages s+1, s+2 whole FP4 stages: the loop the tile spends most time in
  // (two stages per trip: the parity of s is known in each body)
#pragma unroll 1
  for (; s + 3 < nfull; s += 2) {
    fp4_body(s, IC<0>{}, IC<0>{});
    fp4_body(s + 1, IC<0>{}, IC<1>{});
  }
  if (s + 2 < nfull) fp4_body(s++, IC<0>{}, IC<0>{});
#pragma unroll 1
  for (; s < nst; s++) fp4_body(s, IC<1>{}, IC<0>{});
  if (nlr > 0) {
#pragma unroll
    for (int q = 0; q < LR_READS; q++) lr_read_one(nst, 0, q, ga);
#pragma unroll 1
    for (; s < total - 2; s++) lr_body(s, IC<1>{}, IC<1>{});
    if (s < total - 1) lr_body(s++, IC<1>{}, IC<0>{});
    lr_body(s++, IC<0>{}, IC<0>{});
  }

  // ---------------- epilogue: convert, store
  const int orow0 = m0 + wm * 128, ocol0 = n0 + wn * 128;   // this wave's 128x128 block
  if constexpr (OUT_F32) {
#pragma unroll
    for (int i = 0; i < 4; i++) {
      const int gr = orow0 + 32 * i + r32;
#pragma unroll
      for (int j = 0; j < 4; j++)
#pragma unroll
        for (int q = 0; q < 4; q++) {
          const int gc = ocol0 + 32 * j + 8 * q + 4 * h;
          if (gr < M && gc < NO)
            *(float4*)((float*)out + (size_t)gr * NO + gc) =
                make_float4(acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]);
        }
    }
  } else if constexpr (EPI == EPI_PLAIN) {
    // Four passes of 32 rows.  The wave stages the pass's rows in LDS as bf16
    // (each lane writes its four-column runs, converted in pairs), then reads
    // them back as 16-byte row segments for coalesced buffer stores (rows or
    // columns past the edge get an out-of-range offset).
    __syncthreads();  // all waves are done with the ring
    constexpr int SROW = 128 * 2 + 16;                 // staged row stride (bytes)
    uint8_t* stg = lds + wave * (32 * SROW);
    const __amdgpu_buffer_rsrc_t ro = make_rsrc(out, (uint32_t)M * NO * 2);
#pragma unroll
    for (int i = 0; i < 4; i++) {
#pragma unroll
      for (int j = 0; j < 4; j++)
#pragma unroll
        for (int q = 0; q < 4; q++) {
          const v2f x01 = {acc[i][j][4 * q + 0], acc[i][j][4 * q + 1]};
          const v2f x23 = {acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
          *(v2i*)(stg + r32 * SROW + (32 * j + 8 * q + 4 * h) * 2) =
              v2i{(int)__builtin_bit_cast(uint32_t, __builtin_convertvector(x01, v2bf)),
                  (int)__builtin_bit_cast(uint32_t, __builtin_convertvector(x23, v2bf))};
        }
      __builtin_amdgcn_s_waitcnt(0xc07f);  // the wave reads back only its own rows
      v4i seg[8];
#pragma unroll
      for (int it = 0; it < 8; it++) seg[it] = *(const v4i*)(stg + (4 * it + (lane >> 4)) * SROW + (lane & 15) * 16);
#pragma unroll
      for (int it = 0; it < 8; it++) {
        const int gr = orow0 + 32 * i + 4 * it + (lane >> 4), gc = ocol0 + 8 * (lane & 15);
        const uint32_t off = (gr < M && gc < NO) ? ((uint32_t)gr * NO + gc) * 2 : kOobOffset;
        __builtin_amdgcn_raw_buffer_store_b128(seg[it], ro, off, 0, kStoreNT);
      }
    }
  } else {
    // ---- MLP epilogues (Sec. 3.3, MLP fusion): the output feeds the next
    // linear directly.
    //   EPI_GELU  (FC1 forward):  z = bf16(acc) (saved), h = bf16(GELU(z)),
    //                             h quantized in 1x32 blocks, FC2's down-
    //                             projection partial h . D2 over this tile.
    //   EPI_DGELU (FC2 backward-input): dz = bf16(acc * GELU'(z)) with the
    //                             fp32 acc (dH) unrounded, dz quantized, FC1's
    //                             partial dz . U1^T over this tile.
    // Four passes of 32 rows per wave; in each the wave stages its rows in LDS
    // (bf16 z, or fp32 dH), reads them back as 8-column row segments (a lane
    // quad holds one 32-column block), writes the outputs and the block codes,
    // puts the bf16 result back in place, and multiplies its 32x128 rows with
    // the staged projection slice.  The two waves sharing rows add their
    // partials through LDS; one stores them.
    constexpr bool G = EPI == EPI_GELU;
    constexpr int SROW = G ? 128 * 2 + 16 : 128 * 4 + 16;   // staged row stride (bytes)
    constexpr int STG = 32 * SROW;
    constexpr int PS1 = 64 + 16;                            // EPI_GELU slice [256 n][R2 <= 64]: halfwords per row
    constexpr int PS2 = 256 + 8;                            // EPI_DGELU slice [R2 <= 64][256 k]: halfwords per row
    constexpr int PSLICE = G ? 256 * PS1 * 2 : 64 * PS2 * 2;
    uint8_t* stg = lds + wave * STG;
    uint16_t* ps = (uint16_t*)(lds + 4 * STG);
    // This wave's E8M0 codes (128 rows x 4 blocks) and E2M1 codes (128 rows
    // x 64 bytes), written out once after the passes.
    uint8_t* sbuf = lds + 4 * STG + PSLICE + wave * 512;
    uint8_t* qbuf = lds + 4 * STG + PSLICE + 4 * 512 + wave * (128 * 64);
    static_assert(4 * STG + PSLICE + 4 * 512 + 4 * 128 * 64 <= NSLOT * SLOT, "epilogue LDS");
    // After the passes and the code flush, the projection partials of the two
    // waves that share rows are added through four [128 rows][64] fp32
    // regions at the start of LDS.
    const int R2 = ep.R2;
    const int tn = nt;
    // The projection slice: rows n0..n0+255 of D2 [NO, R2], or columns
    // n0..n0+255 of U1 [R2, NO]; zeros outside.  EPI_DGELU has registers to
    // spare: it issues its slice loads, and the first pass's z loads, before
    // the barrier that frees the ring, so they overlap the wait for the other
    // waves.  In EPI_GELU, holding the slice across the barrier would spill,
    // so each of its loads is written to LDS as it arrives, after the barrier.
    const __amdgpu_buffer_rsrc_t r_y = make_rsrc(ep.y, (uint32_t)M * NO * 2);
    const __amdgpu_buffer_rsrc_t r_z = make_rsrc(G ? (const void*)ep.z_out : (const void*)ep.z_in, (uint32_t)M * NO * 2);
    const __amdgpu_buffer_rsrc_t r_q = make_rsrc(ep.q, (uint32_t)M * (NO / 2));
    const int g16 = lane >> 4, t16 = lane & 15, jj = t16 >> 2, qq = t16 & 3;
    const int rt2 = (R2 + 31) >> 5;
    // EPI_DGELU: the z segments of pass i are loaded at the start of pass
    // i - 1, ahead of that pass's stores, so that waiting for them waits
    // only for the stores of pass i - 2 (loads and stores retire in order).
    // Issuing all passes' loads at once made every CU load its whole z tile
    // in one burst at the start of the epilogue.
    v4i zpre[2][8];
    auto load_z = [&](int i, v4i (&zd)[8]) {
#pragma unroll
      for (int it = 0; it < 8; it++) {
        const int gr = orow0 + 32 * i + 4 * it + g16, gc = ocol0 + 8 * t16;
        zd[it] = __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(
            r_z, (gr < M && gc < NO) ? ((uint32_t)gr * NO + gc) * 2 : kOobOffset, 0, 0));
      }
    };
    uint4 pv[8];
    if constexpr (!G) {
      if (R2 > 0) {
#pragma unroll
        for (int u = 0; u < 8; u++) {
          const int sl = tid + 256 * u, rr = sl >> 5, cc = (sl & 31) * 8;
          pv[u] = make_uint4(0, 0, 0, 0);
          if (rr < R2 && n0 + cc < NO) pv[u] = *(const uint4*)(ep.proj + (size_t)rr * NO + n0 + cc);
        }
      }
      load_z(0, zpre[0]);
    }
    __syncthreads();  // all waves are done with the ring
    if (R2 > 0) {
      if constexpr (G) {
        // all eight loads in flight at once, then the LDS writes (left to
        // itself the compiler waited for each load before the next); rows and
        // columns outside read zeros
        const __amdgpu_buffer_rsrc_t rp = make_rsrc(ep.proj, (uint32_t)NO * R2 * 2);
        v4i v[8];
#pragma unroll
        for (int u = 0; u < 8; u++) {
          const int sl = tid + 256 * u, rr = sl >> 3, cc = (sl & 7) * 8;
          v[u] = __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(
              rp, (n0 + rr < NO && cc < R2) ? ((uint32_t)(n0 + rr) * R2 + cc) * 2 : kOobOffset, 0, 0));
        }
#pragma unroll
        for (int u = 0; u < 8; u++) {
          const int sl = tid + 256 * u;
          *(v4i*)(ps + (sl >> 3) * PS1 + (sl & 7) * 8) = v[u];
        }
      } else {
#pragma unroll
        for (int u = 0; u < 8; u++) {
          const int sl = tid + 256 * u;
          *(uint4*)(ps + (sl >> 5) * PS2 + (sl & 31) * 8) = pv[u];
        }
      }
    }
    __syncthreads();
#pragma unroll   // acc[i] must be indexed by constants
    for (int i = 0; i < 4; i++) {
      if constexpr (!G) {
        if (i + 1 < 4) load_z(i + 1, zpre[(i + 1) & 1]);
      }
      // 1) stage this pass's 32 rows
#pragma unroll
      for (int j = 0; j < 4; j++)
#pragma unroll
        for (int q = 0; q < 4; q++) {
          const int col = 32 * j + 8 * q + 4 * h;
          if constexpr (G) {
            const v2f x01 = {acc[i][j][4 * q + 0], acc[i][j][4 * q + 1]};
            const v2f x23 = {acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
            *(v2i*)(stg + r32 * SROW + col * 2) =
                v2i{(int)__builtin_bit_cast(uint32_t, __builtin_convertvector(x01, v2bf)),
                    (int)__builtin_bit_cast(uint32_t, __builtin_convertvector(x23, v2bf))};
          } else {
            *(float4*)(stg + r32 * SROW + col * 4) =
                make_float4(acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]);
          }
        }
      __builtin_amdgcn_s_waitcnt(0xc07f);
      // 2) row segments: outputs, block codes, bf16 result back in place
#pragma unroll
      for (int it = 0; it < 8; it++) {
        const int rl = 4 * it + g16, seg = t16;
        const int gr = orow0 + 32 * i + rl, gc = ocol0 + 8 * seg;
        const bool inb = gr < M && gc < NO;
        const uint32_t off2 = inb ? ((uint32_t)gr * NO + gc) * 2 : kOobOffset;
        uint8_t* srow = stg + rl * SROW;
        uint32_t w[4];
        if constexpr (G) {
          const v4i zb = *(const v4i*)(srow + seg * 16);
          __builtin_amdgcn_raw_buffer_store_b128(zb, r_z, off2, 0, kStoreNT);
#pragma unroll
          for (int e = 0; e < 4; e++) {
            const v2f hv = {gelu_tanh(bf16_to_f32((uint32_t)zb[e] & 0xFFFFu)), gelu_tanh(bf16_to_f32((uint32_t)zb[e] >> 16))};
            w[e] = __builtin_bit_cast(uint32_t, __builtin_convertvector(hv, v2bf));
          }
        } else {
          const float4 d0 = *(const float4*)(srow + seg * 32), d1 = *(const float4*)(srow + seg * 32 + 16);
          const v4i zb = zpre[i & 1][it];
          const float dh[8] = {d0.x, d0.y, d0.z, d0.w, d1.x, d1.y, d1.z, d1.w};
#pragma unroll
          for (int e = 0; e < 4; e++) {
            const v2f dv = {dh[2 * e] * gelu_tanh_grad(bf16_to_f32((uint32_t)zb[e] & 0xFFFFu)),
                            dh[2 * e + 1] * gelu_tanh_grad(bf16_to_f32((uint32_t)zb[e] >> 16))};
            w[e] = __builtin_bit_cast(uint32_t, __builtin_convertvector(dv, v2bf));
          }
        }
        const v4i wv = {(int)w[0], (int)w[1], (int)w[2], (int)w[3]};
        __builtin_amdgcn_raw_buffer_store_b128(wv, r_y, off2, 0, kStoreNT);
        *(v4i*)(srow + seg * 16) = wv;   // bf16 result in place (for the projection)
        uint32_t sc;
        const uint32_t codes = quad_quantize8(w, sc);
        *(uint32_t*)(qbuf + (32 * i + rl) * 64 + seg * 4) = codes;
        sbuf[(32 * i + rl) * 4 + (seg >> 2)] = (uint8_t)sc;   // the quad's four lanes write the same code
      }
      if (R2 == 0) continue;
      __builtin_amdgcn_s_waitcnt(0xc07f);
      // 3) projection of the pass's 32 rows over this wave's 128 columns, into
      //    the pass's first two accumulator tiles (read out in step 1)
      //    Both 32-column slice tiles are always used (the slice holds zeros
      //    past R2), and the fragments of k-step ks + 1 are read while the
      //    MFMAs of k-step ks run.
      acc[i][0] = v16f{};
      acc[i][1] = v16f{};
      auto frag = [&](int ks, v8bf& a, v8bf (&b)[2]) {
        a = __builtin_bit_cast(v8bf, *(const v4i*)(stg + r32 * SROW + (16 * ks + 8 * h) * 2));
        const int kloc = wn * 128 + 16 * ks + 8 * h;      // column within the workgroup's 256
#pragma unroll
        for (int t = 0; t < 2; t++) {
          if constexpr (G) {
            const uint16_t* base = ps + (kloc + jj) * PS1 + 32 * t + 16 * (g16 & 1) + 4 * qq;
            b[t] = make_v8bf(lds_read_tr16((const FT_LDS void*)base), lds_read_tr16((const FT_LDS void*)(base + 4 * PS1)));
          } else {
            b[t] = __builtin_bit_cast(v8bf, *(const v4i*)(ps + (32 * t + r32) * PS2 + kloc));
          }
        }
      };
      v8bf fa[2], fb[2][2];
      frag(0, fa[0], fb[0]);
#pragma unroll
      for (int ks = 0; ks < 8; ks++) {
        if (ks + 1 < 8) frag(ks + 1, fa[(ks + 1) & 1], fb[(ks + 1) & 1]);
#pragma unroll
        for (int t = 0; t < 2; t++) acc[i][t] = mfma_bf16_32x32x16(fa[ks & 1], fb[ks & 1][t], acc[i][t]);
      }
    }
    // E2M1 codes: 16 bytes (32 columns) of a row per lane, all reads first,
    // then branch-free stores (outside rows and columns dropped)
    {
      v4i cq[8];
#pragma unroll
      for (int q = 0; q < 8; q++) cq[q] = *(const v4i*)(qbuf + (16 * q + (lane >> 2)) * 64 + 16 * (lane & 3));
#pragma unroll
      for (int q = 0; q < 8; q++) {
        const int gr = orow0 + 16 * q + (lane >> 2), c = lane & 3;
        __builtin_amdgcn_raw_buffer_store_b128(
            cq[q], r_q, (gr < M && ocol0 + 32 * c < NO) ? (uint32_t)gr * (NO / 2) + (ocol0 / 2) + 16 * c : kOobOffset, 0, kStoreNT);
      }
    }
    // E8M0 codes: each lane writes rows lane and lane + 64 of the wave's 128,
    // four blocks (one dword) per row when aligned and inside the matrix
    const bool s_al = ((NO >> 5) & 3) == 0 && ocol0 + 128 <= NO;
#pragma unroll
    for (int k = 0; k < 2; k++) {
      const int rr = lane + 64 * k, gr = orow0 + rr;
      const uint32_t v = *(const uint32_t*)(sbuf + rr * 4);
      if (gr < M) {
        uint8_t* d = ep.s + (size_t)gr * (NO >> 5) + (ocol0 >> 5);
        if (s_al) {
          *(uint32_t*)d = v;
        } else {
#pragma unroll
          for (int b = 0; b < 4; b++)
            if (ocol0 + 32 * b < NO) d[b] = (uint8_t)(v >> (8 * b));
        }
      }
    }
    if (R2 > 0) {
      // 4) the two waves with the same rows (wn = 0, 1) add their partials,
      //    all passes at once: each wave stores its own in a 32 KB region
      //    (the code buffers are flushed, so all of LDS is free), and after
      //    one barrier each wave adds the two partials of half of its rows
      //    and stores the sums as 16-byte segments
      static_assert(4 * 128 * 64 * 4 <= NSLOT * SLOT, "combine regions");
      __syncthreads();   // every wave is done with the passes' LDS and its code buffers
      float* mine = (float*)lds + (2 * wn + wm) * (128 * 64);
#pragma unroll
      for (int i = 0; i < 4; i++)
#pragma unroll
        for (int t = 0; t < 2; t++)
#pragma unroll
          for (int v = 0; v < 16; v++)
            mine[(32 * i + 8 * (v >> 2) + 4 * h + (v & 3)) * 64 + 32 * t + r32] = acc[i][t][v];
      __syncthreads();
      // all reads first, then branch-free stores (rows past M and columns
      // past R2 go to an offset past the buffer, which drops them)
      const float* c0 = (const float*)lds + wm * (128 * 64);          // the wn = 0 partial
      const float* c1 = (const float*)lds + (2 + wm) * (128 * 64);    // the wn = 1 partial
      float* dst = tiles_n > 1 ? ep.parts + (size_t)tn * M * R2 : ep.parts;
      const __amdgpu_buffer_rsrc_t rdst = make_rsrc(dst, (uint32_t)M * R2 * 4);
      const int j = 4 * (lane & 15);
      v4f sum[16];
#pragma unroll
      for (int q = 0; q < 16; q++) {
        const int rr = 64 * wn + 4 * q + (lane >> 4);
        sum[q] = *(const v4f*)(c1 + rr * 64 + j) + *(const v4f*)(c0 + rr * 64 + j);
      }
#pragma unroll
      for (int q = 0; q < 16; q++) {
        const int gr = orow0 + 64 * wn + 4 * q + (lane >> 4);
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4i, sum[q]), rdst,
                                               (j < R2 && gr < M) ? ((uint32_t)gr * R2 + j) * 4 : kOobOffset, 0, 0);
      }
    }
  }
}

hipError_t launch_gemm_fp4(bool bwd, const uint8_t* a, const uint8_t* as, const uint8_t* wq, const uint8_t* ws,
                           int M, int N, int K, const float* P, int R, const uint16_t* lr,
                           const uint16_t* bias, void* out, bool out_f32, hipStream_t st) {
  const int NO = bwd ? K : N;
  const int KR = bwd ? N : K;
  const int tm = (M + GB - 1) / GB, tn = (NO + GB - 1) / GB;
  // buffer ranges are 32-bit: the pipelined kernel takes operands below 2 GiB
  const bool small = (size_t)M * KR / 2 < (1u << 31) && (size_t)N * K / 2 < (1u << 31) &&
                     (size_t)M * (R > 0 ? R : 1) * 4 < (1u << 31) && (size_t)M * NO * 2 < (1u << 31);
  if (KR % 128 == 0 && K % 128 == 0 && small) {
    const unsigned grid = (unsigned)(tm * tn);
    const GemmEpilogue none{};
    const uint16_t* b = bwd ? nullptr : bias;
    // A scales in stage pairs when the reduction length is a multiple of 512
#define FT_PIPE(BW, F32, SP) \
  k_gemm_fp4_pipe<BW, F32, EPI_PLAIN, SP><<<grid, 256, 0, st>>>(a, as, wq, ws, M, N, K, P, R, lr, b, out, tm, tn, none)
    if (KR % 512 == 0) {
      if (!bwd) { if (out_f32) FT_PIPE(false, true, true); else FT_PIPE(false, false, true); }
      else { if (out_f32) FT_PIPE(true, true, true); else FT_PIPE(true, false, true); }
    } else {
      if (!bwd) { if (out_f32) FT_PIPE(false, true, false); else FT_PIPE(false, false, false); }
      else { if (out_f32) FT_PIPE(true, true, false); else FT_PIPE(true, false, false); }
    }
#undef FT_PIPE
    return hipGetLastError();
  }
  dim3 grid(tn, tm);
  if (!bwd) {
    if (out_f32) k_gemm_fp4_generic<false, true><<<grid, 256, 0, st>>>(a, as, wq, ws, M, N, K, P, R, lr, bias, out);
    else k_gemm_fp4_generic<false, false><<<grid, 256, 0, st>>>(a, as, wq, ws, M, N, K, P, R, lr, bias, out);
  } else {
    if (out_f32) k_gemm_fp4_generic<true, true><<<grid, 256, 0, st>>>(a, as, wq, ws, M, N, K, P, R, lr, nullptr, out);
    else k_gemm_fp4_generic<true, false><<<grid, 256, 0, st>>>(a, as, wq, ws, M, N, K, P, R, lr, nullptr, out);
  }
  return hipGetLastError();
}

static bool pipe_ok(bool bwd, int M, int N, int K, int R) {
  const int NO = bwd ? K : N, KR = bwd ? N : K;
  return KR % 128 == 0 && K % 128 == 0 && (size_t)M * KR / 2 < (1u << 31) && (size_t)N * K / 2 < (1u << 31) &&
         (size_t)M * (R > 0 ? R : 1) * 4 < (1u << 31) && (size_t)M * NO * 2 < (1u << 31);
}

bool gemm_fp4_fused_supported(bool bwd, int M, int N, int K, int R, int R2) {
  return pipe_ok(bwd, M, N, K, R) && R2 >= 0 && R2 <= 64 && R2 % 16 == 0 &&
         (size_t)M * (R2 > 0 ? R2 : 1) * 4 < (1u << 31);
}

int gemm_fp4_col_tiles(int NO) { return (NO + GB - 1) / GB; }

hipError_t launch_gemm_fp4_fused(bool bwd, const uint8_t* a, const uint8_t* as, const uint8_t* wq, const uint8_t* ws,
                                 int M, int N, int K, const float* P, int R, const uint16_t* lr, const uint16_t* bias,
                                 const GemmEpilogue& ep, float* proj_out, hipStream_t st) {
  const int NO = bwd ? K : N;
  const int tm = (M + GB - 1) / GB, tn = (NO + GB - 1) / GB;
  const unsigned grid = (unsigned)(tm * tn);
  const bool sap = (bwd ? N : K) % 512 == 0;   // A scales in stage pairs
  if (!bwd) {
    if (sap) k_gemm_fp4_pipe<false, false, EPI_GELU, true><<<grid, 256, 0, st>>>(a, as, wq, ws, M, N, K, P, R, lr, bias, nullptr, tm, tn, ep);
    else k_gemm_fp4_pipe<false, false, EPI_GELU, false><<<grid, 256, 0, st>>>(a, as, wq, ws, M, N, K, P, R, lr, bias, nullptr, tm, tn, ep);
  } else {
    if (sap) k_gemm_fp4_pipe<true, false, EPI_DGELU, true><<<grid, 256, 0, st>>>(a, as, wq, ws, M, N, K, P, R, lr, nullptr, nullptr, tm, tn, ep);
    else k_gemm_fp4_pipe<true, false, EPI_DGELU, false><<<grid, 256, 0, st>>>(a, as, wq, ws, M, N, K, P, R, lr, nullptr, nullptr, tm, tn, ep);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || ep.R2 == 0 || tn == 1) return e;
  return launch_reduce_parts(ep.parts, tn, (size_t)M * ep.R2, proj_out, 0, nullptr, false, st);
}

}  // namespace ft
