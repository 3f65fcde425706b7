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
// the backward, K a multiple of 128).  Every stage of work moves through a
// 4-slot LDS ring with buffer loads that write LDS directly; rows past the
// matrix edge read as zeros through the buffer range check, so tiles need no
// branches.  Three stages are in flight while one runs on the matrix cores.
//
// Stage kinds:
//   FP4 stage: 128 reduction elements.  Slot = A tile [256 rows][64 B] +
//     W tile (forward [256 n][64 B]; backward [128 n][128 B], read with the
//     nibble-transposing LDS read) + the stage's E8M0 scales.
//   Low-rank stage (after the FP4 stages): 16 columns of the up-projection.
//     Slot = P chunk [256 rows][16 fp32] + U chunk (forward, [16 j][256 n]
//     bf16) or D chunk (backward, [256 k][16 j] bf16).  P is split into two
//     bf16 terms in registers; its product lands in the same accumulators.
// Within a stage, the barrier that publishes the next stage sits between the
// two k-steps, so the next stage's first fragments load under the current
// MFMAs.  The finished tile is staged through LDS for coalesced stores.

constexpr int PK = 128;                  // reduction elements per FP4 stage
constexpr int PROW = PK / 2;             // bytes per A-tile row per stage
constexpr int SLOT = 36 * 1024;          // bytes per ring slot
constexpr int NSLOT = 4;
constexpr int OFF_B = 16 * 1024;         // W tile / U / D chunk within a slot
constexpr int OFF_SA = 32 * 1024;        // A scales: 256 rows x 4 bytes
constexpr int OFF_SB = 33 * 1024;        // W scales: 4 waves x 256 bytes
constexpr int LOADS_FP4 = 10;            // buffer loads per wave per FP4 stage
constexpr int LOADS_LR = 6;              // ... per low-rank stage

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

template <bool BWD, bool OUT_F32, int EPI>
__global__ __launch_bounds__(256, 1) void k_gemm_fp4_pipe(const uint8_t* __restrict__ A, const uint8_t* __restrict__ As,
                                                          const uint8_t* __restrict__ Wq, const uint8_t* __restrict__ Ws,
                                                          int M, int N, int K, const float* __restrict__ P, int R,
                                                          const uint16_t* __restrict__ LR,
                                                          const uint16_t* __restrict__ bias, void* __restrict__ out,
                                                          int tiles_m, int tiles_n, GemmEpilogue ep) {
  __shared__ __attribute__((aligned(16))) uint8_t lds[NSLOT * SLOT];

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

  const int nst = KR / PK, nlr = R / 16, total = nst + nlr;

  // Accumulator tiles are computed transposed (W fragment as MFMA operand A):
  // lane (r32, h) of tile acc[i][j] holds output row wm*128 + 32i + r32 and,
  // in element 4q + e, column wn*128 + 32j + 8q + 4h + e.
  // Bias of this lane's columns (forward): four bf16 per (j, q), loaded first.
  uint2 bias4[4][4];
#pragma unroll
  for (int j = 0; j < 4; j++)
#pragma unroll
    for (int q = 0; q < 4; q++) {
      bias4[j][q] = make_uint2(0u, 0u);
      if constexpr (!BWD) {
        const int gc = n0 + wn * 128 + j * 32 + 8 * q + 4 * h;
        if (bias && gc < N) bias4[j][q] = *(const uint2*)(bias + gc);
      }
    }

  // ---------------- per-lane load geometry (constant over stages)
  // Each buffer load takes a per-lane byte offset (constant over stages; rows
  // outside the matrix hold kOobOffset, which reads zeros) plus a uniform
  // per-stage offset.
  // 64-byte-row tiles (A, forward W, P chunk): instruction i of this wave
  // fills rows wave*64 + 16i + [0,16); lane L -> row + L/4, chunk (L%4)^swz64.
  const int r64 = wave * 64 + (lane >> 2);
  const int c64 = (lane & 3) ^ swz64(lane >> 2);
  uint32_t a_base[4], w_base[4], p_base[4];
#pragma unroll
  for (int i = 0; i < 4; i++) {
    const int r = r64 + 16 * i;
    a_base[i] = (m0 + r < M) ? (uint32_t)(m0 + r) * lda + c64 * 16 : kOobOffset;
    p_base[i] = (m0 + r < M) ? (uint32_t)(m0 + r) * R * 4 + c64 * 16 : kOobOffset;
    w_base[i] = kOobOffset;
    if constexpr (!BWD) w_base[i] = (n0 + r < N) ? (uint32_t)(n0 + r) * ldw + c64 * 16 : kOobOffset;
  }
  // backward W tile: 128 reduction rows x 128 bytes; instruction i fills rows
  // wave*32 + 8i + [0,8); lane L -> row + L/8, chunk (L%8) ^ swz128(row).
  const int rb128 = wave * 32 + (lane >> 3);
  const int cb128 = (lane & 7) ^ swz128(lane >> 3);
  uint32_t wt_base[4];
#pragma unroll
  for (int i = 0; i < 4; i++) {
    const int byte = (n0 >> 1) + ((cb128 ^ (i & 1)) * 16);
    wt_base[i] = (byte < ldw) ? (uint32_t)(rb128 + 8 * i) * ldw + byte : kOobOffset;
  }
  // scales: wave w stages A-scale dwords of tile rows 64w + lane; W scales:
  //   forward: lanes 0,1 of wave w fetch 32-column blocks 2w, 2w+1 of the tile;
  //   backward: lanes 0,1 of wave w fetch W-scale row (stage*4 + w), blocks 4*lane..+3.
  const uint32_t sa_base = (m0 + wave * 64 + lane < M) ? (uint32_t)(m0 + wave * 64 + lane) * nkb : kOobOffset;
  uint32_t sb_base = kOobOffset;
  if (lane < 2) {
    if constexpr (!BWD) {
      const int nb = (n0 >> 5) + 2 * wave + lane;
      if (nb < (N >> 5)) sb_base = (uint32_t)nb * nwkb;
    } else {
      const int kb = (n0 >> 5) + 4 * lane;
      if (kb < (K >> 5)) sb_base = (uint32_t)wave * nwkb + kb;
    }
  }
  // low-rank chunk geometry
  //   forward U chunk [16 j][256 n] (512-byte rows): instruction i fills rows
  //     2i, 2i+1 (waves 0..3 own instructions 2w, 2w+1); lane L -> row + L/32,
  //     chunk (L%32) ^ (2*(row&3)).
  //   backward D chunk [256 k][16 j] (32-byte rows): instruction i fills rows
  //     32i + [0,32) (waves own 2w, 2w+1); lane L -> row + L/2, half (L%2)^((row>>2)&1).
  uint32_t l_base[2];
#pragma unroll
  for (int i = 0; i < 2; i++) {
    const int ins = 2 * wave + i;
    if constexpr (!BWD) {
      const int j = 2 * ins + (lane >> 5);
      const int c = (lane & 31) ^ (2 * (j & 3));
      l_base[i] = (n0 + c * 8 < N) ? (uint32_t)j * N * 2 + (uint32_t)(n0 + c * 8) * 2 : kOobOffset;
    } else {
      const int k = 32 * ins + (lane >> 1);
      const int c = (lane & 1) ^ ((k >> 2) & 1);
      l_base[i] = (n0 + k < K) ? (uint32_t)(n0 + k) * R * 2 + c * 16 : kOobOffset;
    }
  }

  auto slot_of = [&](int t) { return (uint32_t)((t & (NSLOT - 1)) * SLOT); };

  // ---------------- stage loads (LDS destinations and per-stage offsets are uniform)
  auto issue_fp4 = [&](int t) {
    const uint32_t slot = lds0 + slot_of(t);
    const uint32_t sa_off = (uint32_t)t * PROW;
#pragma unroll
    for (int i = 0; i < 4; i++) dma16(ra, slot + (wave * 64 + 16 * i) * PROW, a_base[i], sa_off);
#pragma unroll
    for (int i = 0; i < 4; i++) {
      if constexpr (!BWD) dma16(rw, slot + OFF_B + (wave * 64 + 16 * i) * PROW, w_base[i], sa_off);
      else dma16(rw, slot + OFF_B + (wave * 32 + 8 * i) * 128, wt_base[i], (uint32_t)t * PK * ldw);
    }
    dma4(ras, slot + OFF_SA + wave * 256, sa_base, (uint32_t)t * 4);
    if constexpr (!BWD) dma4(rws, slot + OFF_SB + wave * 256, sb_base, (uint32_t)t * 4);
    else dma4(rws, slot + OFF_SB + wave * 256, sb_base, (uint32_t)t * 4 * nwkb);
  };
  auto issue_lr = [&](int t) {
    const uint32_t slot = lds0 + slot_of(t);
    const int q = t - nst;
#pragma unroll
    for (int i = 0; i < 4; i++) dma16(rp, slot + (wave * 64 + 16 * i) * 64, p_base[i], (uint32_t)q * 64);
#pragma unroll
    for (int i = 0; i < 2; i++)
      dma16(rl, slot + OFF_B + (2 * wave + i) * 1024, l_base[i], BWD ? (uint32_t)q * 32 : (uint32_t)q * 16 * N * 2);
  };
  auto issue = [&](int t) {
    if (t >= total) return;
    if (t < nst) issue_fp4(t);
    else issue_lr(t);
  };

  // Loads one wave issues for stage u (0 past the end).
  auto loads_of = [&](int u) { return u >= total ? 0 : (u < nst ? LOADS_FP4 : LOADS_LR); };
  // Wait until at most n of this wave's loads are outstanding, then barrier:
  // with n = the loads issued after stage u, stage u is in LDS for every wave.
  auto publish = [&](int n) {
    switch (n) {
      case 0: wait_vm<0>(); break;
      case LOADS_LR: wait_vm<LOADS_LR>(); break;
      case LOADS_FP4: wait_vm<LOADS_FP4>(); break;
      case 2 * LOADS_LR: wait_vm<2 * LOADS_LR>(); break;
      case LOADS_FP4 + LOADS_LR: wait_vm<LOADS_FP4 + LOADS_LR>(); break;
      default: wait_vm<2 * LOADS_FP4>(); break;
    }
    // plain barrier: the LDS data it publishes was written by buffer loads,
    // whose completion the vmcnt wait above already covers
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");     // no LDS read moves above the barrier
  };

  // ---------------- fragment reads
  const int sw_a = swz64(r32);                      // rows ... + r32 of 64-byte-row tiles
  const int sw_t = (t16 & 7) ^ ((t16 >> 3) & 1);    // rows ... + t16 of the backward W tile
  const uint32_t psel = h ? 0x0301u : 0x0200u;      // result bytes 0,1 = scale bytes h, h+2 of a dword

  // Per-lane LDS read offsets within a slot, one set per k-step (a fragment
  // read is then one address add plus an immediate offset).
  uint32_t rd_a[2], rd_b[2], rd_t[2][4];
#pragma unroll
  for (int kk = 0; kk < 2; kk++) {
    rd_a[kk] = (wm * 128 + r32) * PROW + (((2 * kk + h) ^ sw_a) << 4);
    rd_b[kk] = OFF_B + (wn * 128 + r32) * PROW + (((2 * kk + h) ^ sw_a) << 4);
#pragma unroll
    for (int j = 0; j < 4; j++)
      rd_t[kk][j] = OFF_B + (kk * 64 + 32 * h + t16) * 128 + (((wn * 4 + j) ^ sw_t) << 4) + 8 * (g16 & 1);
  }
  const uint32_t rd_sa = OFF_SA + (wm * 128 + r32) * 4;
  const uint32_t rd_sbt = OFF_SB + h * 256 + wn * 4;     // backward W-scale rows h (+2)

  struct Fp4Frag { v4i a[4], b[4]; };
  auto read_fp4 = [&](int t, int kk, Fp4Frag& f) {
    const uint8_t* slot = lds + slot_of(t);
    const uint8_t* pa = slot + rd_a[kk];
#pragma unroll
    for (int i = 0; i < 4; i++) f.a[i] = *(const v4i*)(pa + i * 32 * PROW);
    if constexpr (!BWD) {
      const uint8_t* pb = slot + rd_b[kk];
#pragma unroll
      for (int j = 0; j < 4; j++) f.b[j] = *(const v4i*)(pb + j * 32 * PROW);
    } else {
#pragma unroll
      for (int j = 0; j < 4; j++) {
        const uint8_t* pt = slot + rd_t[kk][j];
        const v2i lo = lds_read_tr4((const FT_LDS void*)pt);
        const v2i hi = lds_read_tr4((const FT_LDS void*)(pt + 16 * 128));
        f.b[j] = v4i{lo[0], lo[1], hi[0], hi[1]};
      }
    }
  };
  // Single-fragment reads, for interleaving with the MFMAs one at a time.
  // Fragment q of a k-step: q < 4 -> A row tile q; q >= 4 -> W tile q - 4
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
      const v2i v = lds_read_tr4((const FT_LDS void*)(slot + rd_t[kk][j] + half * 16 * 128));
      if (half == 0) { f.b[j][0] = v[0]; f.b[j][1] = v[1]; }
      else { f.b[j][2] = v[0]; f.b[j][3] = v[1]; }
    }
  };
  // Raw scale words of a stage; turned into MFMA scale operands (one byte per
  // k-step) only when the stage's MFMAs are about to issue.
  struct ScaleRaw { uint32_t a[4], b[4]; };
  auto read_scales = [&](int t, ScaleRaw& r) {
    const uint8_t* slot = lds + slot_of(t);
#pragma unroll
    for (int i = 0; i < 4; i++) r.a[i] = *(const uint32_t*)(slot + rd_sa + i * 128);
    if constexpr (!BWD) {
#pragma unroll
      for (int j = 0; j < 4; j++) {  // 32-column block wn*4 + j, staged by wave (wn*4+j)/2
        r.b[j] = *(const uint32_t*)(slot + OFF_SB + (wn * 2 + (j >> 1)) * 256 + (j & 1) * 4);
      }
    } else {
      // rows 2kk + h of this stage's W-scale block (staged by wave 2kk+h), column blocks wn*4 + j
      r.b[0] = *(const uint32_t*)(slot + rd_sbt);
      r.b[1] = *(const uint32_t*)(slot + rd_sbt + 512);
    }
  };
  auto scale_ops = [&](const ScaleRaw& r, uint32_t (&sa)[4], uint32_t (&sb)[4]) {
#pragma unroll
    for (int i = 0; i < 4; i++) sa[i] = __builtin_amdgcn_perm(0u, r.a[i], psel);
#pragma unroll
    for (int j = 0; j < 4; j++) {
      if constexpr (!BWD) sb[j] = __builtin_amdgcn_perm(0u, r.b[j], psel);
      else sb[j] = __builtin_amdgcn_perm(r.b[1], r.b[0], 0x0c0c0400u | (j << 8) | j);
    }
  };

  struct LrFrag { v4i p[4][2]; v8bf b[4]; };
  const int jj = t16 >> 2, qq = t16 & 3;
  auto read_lr = [&](int t, LrFrag& f) {
    const uint8_t* slot = lds + slot_of(t);
#pragma unroll
    for (int i = 0; i < 4; i++) {
      const uint8_t* row = slot + (wm * 128 + i * 32 + r32) * 64;
      f.p[i][0] = *(const v4i*)(row + (((2 * h) ^ sw_a) << 4));
      f.p[i][1] = *(const v4i*)(row + (((2 * h + 1) ^ sw_a) << 4));
    }
#pragma unroll
    for (int j = 0; j < 4; j++) {
      if constexpr (!BWD) {
        const int n = wn * 128 + j * 32 + 16 * (g16 & 1) + 4 * qq;
        const int row0 = 8 * h + jj;
        const int byte0 = ((((n >> 3) ^ (2 * (row0 & 3))) << 4)) + ((n >> 2) & 1) * 8;
        const v4s lo = lds_read_tr16((const FT_LDS void*)(slot + OFF_B + row0 * 512 + byte0));
        const int row1 = row0 + 4;
        const int byte1 = ((((n >> 3) ^ (2 * (row1 & 3))) << 4)) + ((n >> 2) & 1) * 8;
        const v4s hi = lds_read_tr16((const FT_LDS void*)(slot + OFF_B + row1 * 512 + byte1));
        f.b[j] = make_v8bf(lo, hi);
      } else {
        const int k = wn * 128 + j * 32 + r32;
        f.b[j] = __builtin_bit_cast(v8bf, *(const v4i*)(slot + OFF_B + k * 32 + ((h ^ ((k >> 2) & 1)) << 4)));
      }
    }
  };

  v16f acc[4][4];

  auto mfma_fp4_step = [&](int kk, const Fp4Frag& f, const uint32_t (&sa)[4], const uint32_t (&sb)[4]) {
#pragma unroll
    for (int i = 0; i < 4; i++)
#pragma unroll
      for (int j = 0; j < 4; j++) {
        if (kk == 0) acc[i][j] = mfma_fp4_32x32x64<0>(f.b[j], f.a[i], acc[i][j], (int)sb[j], (int)sa[i]);
        else acc[i][j] = mfma_fp4_32x32x64<1>(f.b[j], f.a[i], acc[i][j], (int)sb[j], (int)sa[i]);
      }
  };
  auto mfma_lr_step = [&](const LrFrag& f) {
    v8bf ahi[4], alo[4];
#pragma unroll
    for (int i = 0; i < 4; i++) {
      const v4i x0 = f.p[i][0], x1 = f.p[i][1];
      const int xs[8] = {x0[0], x0[1], x0[2], x0[3], x1[0], x1[1], x1[2], x1[3]};
      v4i hh, ll;
#pragma unroll
      for (int e = 0; e < 4; e++) {
        uint32_t hp, lp;
        split_bf16x2(__int_as_float(xs[2 * e]), __int_as_float(xs[2 * e + 1]), hp, lp);
        hh[e] = (int)hp;
        ll[e] = (int)lp;
      }
      ahi[i] = __builtin_bit_cast(v8bf, hh);
      alo[i] = __builtin_bit_cast(v8bf, ll);
    }
#pragma unroll
    for (int i = 0; i < 4; i++)
#pragma unroll
      for (int j = 0; j < 4; j++) {
        acc[i][j] = mfma_bf16_32x32x16(f.b[j], ahi[i], acc[i][j]);
        acc[i][j] = mfma_bf16_32x32x16(f.b[j], alo[i], acc[i][j]);
      }
  };

  // ---------------- pipeline
  // Stage t's slot is refilled (with stage t+4) in iteration t+1, after that
  // iteration's barrier; every wave passed its own wait for the reads of slot t
  // (the wait at the top of iteration t+1) before arriving there.
  issue(0);
  issue(1);
  issue(2);
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
  publish(loads_of(1) + loads_of(2));
  Fp4Frag f0, f1;
  ScaleRaw sr;
  read_fp4(0, 0, f0);
  read_scales(0, sr);

  // One FP4 iteration.  STEADY: stages t+1..t+3 are FP4 stages, so the body is
  // branch-free with constant wait counts, and every other instruction is
  // placed between two MFMAs (one wave per SIMD: the matrix pipe only stays
  // busy if nothing else waits in front of the next MFMA):
  //   k-step 0 (16 MFMAs on f0) carries the reads of this stage's k-step 1;
  //   then the barrier that publishes stage t+1;
  //   k-step 1 (16 MFMAs on f1) carries the reads of stage t+1's k-step 0 and
  //   scales, the loads of stage t+3, and the scale operands of stage t+1.
  uint32_t sa[4], sb[4];
  scale_ops(sr, sa, sb);
  auto fp4_iter_steady = [&](int t) {
    const uint8_t* nslot = lds + slot_of(t + 1);
    const uint32_t dslot = lds0 + slot_of(t + 3);
    const uint32_t a_off = (uint32_t)(t + 3) * PROW;
    const uint32_t wt_off = (uint32_t)(t + 3) * PK * ldw;
    const uint32_t s_off = (uint32_t)(t + 3) * 4;
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int m = 0; m < 16; m++) {
      const int i = m >> 2, j = m & 3;
      acc[i][j] = mfma_fp4_32x32x64<0>(f0.b[j], f0.a[i], acc[i][j], (int)sb[j], (int)sa[i]);
      if (m < FRAG_READS) read_one(t, 1, m, f1);
      __builtin_amdgcn_sched_barrier(0);
    }
    wait_vm<LOADS_FP4>();                // stage t+1 landed; stage t+2 may stay in flight
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
    uint32_t nsa[4], nsb[4];
#pragma unroll
    for (int m = 0; m < 16; m++) {
      const int i = m >> 2, j = m & 3;
      acc[i][j] = mfma_fp4_32x32x64<1>(f1.b[j], f1.a[i], acc[i][j], (int)sb[j], (int)sa[i]);
      // reads of stage t+1: fragments in slots 0..FRAG_READS-1, then scales
      if (m < FRAG_READS) read_one(t + 1, 0, m, f0);
      if (m == FRAG_READS - 4 || (BWD && m == 12)) {
        if (m == FRAG_READS - 4) {
#pragma unroll
          for (int q = 0; q < 4; q++) sr.a[q] = *(const uint32_t*)(nslot + rd_sa + q * 128);
        }
        if (!BWD || m == 12) {
          if constexpr (!BWD) {
#pragma unroll
            for (int q = 0; q < 4; q++)
              sr.b[q] = *(const uint32_t*)(nslot + OFF_SB + (wn * 2 + (q >> 1)) * 256 + (q & 1) * 4);
          } else {
            sr.b[0] = *(const uint32_t*)(nslot + rd_sbt);
            sr.b[1] = *(const uint32_t*)(nslot + rd_sbt + 512);
          }
        }
      }
      // loads of stage t+3: A tile rows in slots 0..3, W tile in 4..7, scales in 8, 9
      if (m < 4) dma16(ra, dslot + (wave * 64 + 16 * m) * PROW, a_base[m], a_off);
      else if (m < 8) {
        if constexpr (!BWD) dma16(rw, dslot + OFF_B + (wave * 64 + 16 * (m - 4)) * PROW, w_base[m - 4], a_off);
        else dma16(rw, dslot + OFF_B + (wave * 32 + 8 * (m - 4)) * 128, wt_base[m - 4], wt_off);
      } else if (m == 8) {
        dma4(ras, dslot + OFF_SA + wave * 256, sa_base, s_off);
      } else if (m == 9) {
        if constexpr (!BWD) dma4(rws, dslot + OFF_SB + wave * 256, sb_base, s_off);
        else dma4(rws, dslot + OFF_SB + wave * 256, sb_base, s_off * nwkb);
      }
      // scale operands of stage t+1 once its scale words are in registers
      if (m == 15) scale_ops(sr, nsa, nsb);
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int q = 0; q < 4; q++) { sa[q] = nsa[q]; sb[q] = nsb[q]; }
  };

  // Remaining FP4 iterations (the last three stages): loads may run out, so
  // waits and issues follow the stage kinds.
  auto fp4_iter = [&](int t) {
    read_fp4(t, 1, f1);
    __builtin_amdgcn_sched_barrier(0);
    mfma_fp4_step(0, f0, sa, sb);
    __builtin_amdgcn_sched_barrier(0);
    publish(loads_of(t + 2));
    issue(t + 3);
    if (t + 1 < nst) {
      read_fp4(t + 1, 0, f0);
      read_scales(t + 1, sr);
    }
    __builtin_amdgcn_sched_barrier(0);
    mfma_fp4_step(1, f1, sa, sb);
    __builtin_amdgcn_sched_barrier(0);
    if (t + 1 < nst) scale_ops(sr, sa, sb);
  };
  int t = 0;
#pragma unroll 1
  for (; t + 3 < nst; t++) fp4_iter_steady(t);
#pragma unroll 1
  for (; t < nst; t++) fp4_iter(t);
  if (nlr > 0) {
    LrFrag g;
    read_lr(nst, g);
#pragma unroll 1
    for (int t = nst; t < total; t++) {
      __builtin_amdgcn_s_waitcnt(0xc07f);  // this wave's reads of slot t-1 are done
      publish(loads_of(t + 2));
      issue(t + 3);
      LrFrag gn;
      if (t + 1 < total) read_lr(t + 1, gn);
      __builtin_amdgcn_sched_barrier(0);
      mfma_lr_step(g);
      __builtin_amdgcn_sched_barrier(0);
      g = gn;
    }
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
        __builtin_amdgcn_raw_buffer_store_b128(seg[it], ro, off, 0, 0);
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
    float* comb = (float*)(lds + 4 * STG + PSLICE);          // [2 buffers][2 pairs][32 rows][64]
    const int R2 = ep.R2;
    const int tn = nt;
    __syncthreads();  // all waves are done with the ring
    if (R2 > 0) {
      // stage the projection slice: rows n0..n0+255 of D2 [NO, R2], or
      // columns n0..n0+255 of U1 [R2, NO]; zeros outside
#pragma unroll
      for (int u = 0; u < 8; u++) {
        const int sl = tid + 256 * u;
        uint4 v = make_uint4(0, 0, 0, 0);
        if constexpr (G) {
          const int rr = sl >> 3, cc = (sl & 7) * 8;
          if (n0 + rr < NO && cc < R2) v = *(const uint4*)(ep.proj + (size_t)(n0 + rr) * R2 + cc);
          *(uint4*)(ps + rr * PS1 + cc) = v;
        } else {
          const int rr = sl >> 5, cc = (sl & 31) * 8;
          if (rr < R2 && n0 + cc < NO) v = *(const uint4*)(ep.proj + (size_t)rr * NO + n0 + cc);
          *(uint4*)(ps + rr * PS2 + cc) = v;
        }
      }
    }
    __syncthreads();
    const __amdgpu_buffer_rsrc_t r_y = make_rsrc(ep.y, (uint32_t)M * NO * 2);
    const __amdgpu_buffer_rsrc_t r_z = make_rsrc(G ? (const void*)ep.z_out : (const void*)ep.z_in, (uint32_t)M * NO * 2);
    const __amdgpu_buffer_rsrc_t r_q = make_rsrc(ep.q, (uint32_t)M * (NO / 2));
    const int g16 = lane >> 4, t16 = lane & 15, jj = t16 >> 2, qq = t16 & 3;
    const int rt2 = (R2 + 31) >> 5;
    // EPI_DGELU: every z segment this lane needs, loaded before the first
    // store (a load waited for after stores would wait for those stores too)
    v4i zpre[4][8];
    if constexpr (!G) {
#pragma unroll
      for (int i = 0; i < 4; i++)
#pragma unroll
        for (int it = 0; it < 8; it++) {
          const int gr = orow0 + 32 * i + 4 * it + g16, gc = ocol0 + 8 * t16;
          zpre[i][it] = __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(
              r_z, (gr < M && gc < NO) ? ((uint32_t)gr * NO + gc) * 2 : kOobOffset, 0, 0));
        }
    }
#pragma unroll   // acc[i] must be indexed by constants
    for (int i = 0; i < 4; i++) {
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
      if constexpr (!G) {
        if (i == 0) wait_vm<0>();   // z arrived (no store issued yet)
      }
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
          __builtin_amdgcn_raw_buffer_store_b128(zb, r_z, off2, 0, 0);
#pragma unroll
          for (int e = 0; e < 4; e++) {
            const v2f hv = {gelu_tanh(bf16_to_f32((uint32_t)zb[e] & 0xFFFFu)), gelu_tanh(bf16_to_f32((uint32_t)zb[e] >> 16))};
            w[e] = __builtin_bit_cast(uint32_t, __builtin_convertvector(hv, v2bf));
          }
        } else {
          const float4 d0 = *(const float4*)(srow + seg * 32), d1 = *(const float4*)(srow + seg * 32 + 16);
          const v4i zb = zpre[i][it];
          const float dh[8] = {d0.x, d0.y, d0.z, d0.w, d1.x, d1.y, d1.z, d1.w};
#pragma unroll
          for (int e = 0; e < 4; e++) {
            const v2f dv = {dh[2 * e] * gelu_tanh_grad(bf16_to_f32((uint32_t)zb[e] & 0xFFFFu)),
                            dh[2 * e + 1] * gelu_tanh_grad(bf16_to_f32((uint32_t)zb[e] >> 16))};
            w[e] = __builtin_bit_cast(uint32_t, __builtin_convertvector(dv, v2bf));
          }
        }
        const v4i wv = {(int)w[0], (int)w[1], (int)w[2], (int)w[3]};
        __builtin_amdgcn_raw_buffer_store_b128(wv, r_y, off2, 0, 0);
        *(v4i*)(srow + seg * 16) = wv;   // bf16 result in place (for the projection)
        uint32_t sc;
        const uint32_t codes = quad_quantize8(w, sc);
        __builtin_amdgcn_raw_buffer_store_b32((int)codes, r_q, inb ? (uint32_t)gr * (NO / 2) + gc / 2 : kOobOffset, 0, 0);
        if (inb && (lane & 3) == 0) ep.s[(size_t)gr * (NO / 32) + gc / 32] = (uint8_t)sc;
      }
      if (R2 == 0) continue;
      __builtin_amdgcn_s_waitcnt(0xc07f);
      // 3) projection of the pass's 32 rows over this wave's 128 columns
      v16f pacc[2] = {v16f{}, v16f{}};
#pragma unroll
      for (int ks = 0; ks < 8; ks++) {
        const v8bf a = __builtin_bit_cast(v8bf, *(const v4i*)(stg + r32 * SROW + (16 * ks + 8 * h) * 2));
        const int kloc = wn * 128 + 16 * ks + 8 * h;      // column within the workgroup's 256
#pragma unroll
        for (int t = 0; t < 2; t++) {
          if (t >= rt2) break;
          v8bf b;
          if constexpr (G) {
            const uint16_t* base = ps + (kloc + jj) * PS1 + 32 * t + 16 * (g16 & 1) + 4 * qq;
            b = make_v8bf(lds_read_tr16((const FT_LDS void*)base), lds_read_tr16((const FT_LDS void*)(base + 4 * PS1)));
          } else {
            b = __builtin_bit_cast(v8bf, *(const v4i*)(ps + (32 * t + r32) * PS2 + kloc));
          }
          pacc[t] = mfma_bf16_32x32x16(a, b, pacc[t]);
        }
      }
      // 4) the two waves with these rows (wn = 0, 1) add their partials
      float* cb = comb + ((i & 1) * 2 + wm) * (32 * 64);
      if (wn == 1) {
#pragma unroll
        for (int t = 0; t < 2; t++)
#pragma unroll
          for (int v = 0; v < 16; v++) cb[(8 * (v >> 2) + 4 * h + (v & 3)) * 64 + 32 * t + r32] = pacc[t][v];
      }
      __syncthreads();
      if (wn == 0) {
        float* dst = tiles_n > 1 ? ep.parts + (size_t)tn * M * R2 : ep.parts;
#pragma unroll
        for (int t = 0; t < 2; t++)
#pragma unroll
          for (int v = 0; v < 16; v++) {
            const int rr = 8 * (v >> 2) + 4 * h + (v & 3), j = 32 * t + r32;
            const int gr = orow0 + 32 * i + rr;
            if (j < R2 && gr < M) dst[(size_t)gr * R2 + j] = pacc[t][v] + cb[rr * 64 + j];
          }
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
  if (KR % PK == 0 && K % 128 == 0 && small) {
    const unsigned grid = (unsigned)(tm * tn);
    const GemmEpilogue none{};
    if (!bwd) {
      if (out_f32) k_gemm_fp4_pipe<false, true, EPI_PLAIN><<<grid, 256, 0, st>>>(a, as, wq, ws, M, N, K, P, R, lr, bias, out, tm, tn, none);
      else k_gemm_fp4_pipe<false, false, EPI_PLAIN><<<grid, 256, 0, st>>>(a, as, wq, ws, M, N, K, P, R, lr, bias, out, tm, tn, none);
    } else {
      if (out_f32) k_gemm_fp4_pipe<true, true, EPI_PLAIN><<<grid, 256, 0, st>>>(a, as, wq, ws, M, N, K, P, R, lr, nullptr, out, tm, tn, none);
      else k_gemm_fp4_pipe<true, false, EPI_PLAIN><<<grid, 256, 0, st>>>(a, as, wq, ws, M, N, K, P, R, lr, nullptr, out, tm, tn, none);
    }
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
  return KR % PK == 0 && K % 128 == 0 && (size_t)M * KR / 2 < (1u << 31) && (size_t)N * K / 2 < (1u << 31) &&
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
  if (!bwd) k_gemm_fp4_pipe<false, false, EPI_GELU><<<grid, 256, 0, st>>>(a, as, wq, ws, M, N, K, P, R, lr, bias, nullptr, tm, tn, ep);
  else k_gemm_fp4_pipe<true, false, EPI_DGELU><<<grid, 256, 0, st>>>(a, as, wq, ws, M, N, K, P, R, lr, nullptr, nullptr, tm, tn, ep);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || ep.R2 == 0 || tn == 1) return e;
  return launch_reduce_parts(ep.parts, tn, (size_t)M * ep.R2, proj_out, 0, nullptr, false, st);
}

}  // namespace ft
