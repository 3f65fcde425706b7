// Block-wise MXFP4 quantization kernels (gfx950).
//
// k_quant_rows: 1x32 blocks along rows of a bf16 matrix (activations X and
// gradients G, FourTune Sec. 3.1 dynamic quantization), fused with the
// low-rank down-projection of the same rows (Sec. 3.3, LoRA fusion: the
// stabilizer and adapter branches share the input, so one pass reads it once).
// Workgroups cover one column chunk, or (MC) a few consecutive ones with
// the projection slice re-staged between them; their partial projections
// are summed by k_reduce_parts.
// k_quant_rows_fr: the same for a [cols, R] projection with whole rows per
// workgroup, which adds its partial projections itself.
// k_quant_tiles: 32x32 tiles of the frozen weight (Sec. 3.2), offline.
#include "ft_device.h"
#include "ft_kernels.h"

namespace ft {

// ---------------------------------------------------------------- rows
// Workgroup = WAVES waves over 32*WAVES rows x CW columns (x cpw chunks with
// MC); wave w owns rows
// [row0 + 32w, +32).  The wave walks its columns in steps of 64.  Loads are
// row-contiguous: load q of a step brings rows 8q..8q+7, lane l taking
// elements [8(l%8), +8) of row 8q + l/8, so every 8 lanes read one whole
// 128-byte line.  A 32-element block then sits in 4 neighbouring lanes, which
// reduce its absmax with two quad-permute DPP moves and each convert their 8
// elements.  For the projection the wave writes the step's bf16 values to a
// private LDS tile and reads them back in the MFMA operand layout (lane =
// row), so the 32x32x16 bf16 MFMAs see the natural reduction order.
//
// proj chunk staged in LDS (zero padded to RT*32 columns and to CW rows):
//   MODE 1 (proj [cols, R]):  lds[k][j], row stride RT*32 + 16 halfwords;
//     B fragments come from transposing reads (ds_read_b64_tr_b16).
//   MODE 2 (proj [R, cols]):  lds[j][k], row stride CW + 8 halfwords;
//     B fragments are plain 16-byte reads.
constexpr int QR_XSTRIDE = 64 + 8;  // halfwords per row of a wave's 32x64 tile

template <int RT, int MODE, int WAVES, int CW>
struct QuantLds {
  static constexpr int STRIDE = MODE == 1 ? RT * 32 + 16 : CW + 8;      // halfwords
  static constexpr int ROWS = MODE == 1 ? CW : RT * 32;
  static constexpr int PROJ_HW = MODE == 0 ? 0 : ROWS * STRIDE;
  static constexpr int X_HW = MODE == 0 ? 0 : 32 * QR_XSTRIDE;          // per wave
  static constexpr int SC_ROW = CW / 32;                                 // scale bytes per row of a chunk
  static constexpr int SC_HW = 32 * SC_ROW / 2;                          // per wave: 32 rows of scale bytes
  static constexpr int HALFWORDS = PROJ_HW + WAVES * (X_HW + SC_HW);
};

typedef unsigned short v2u16 __attribute__((ext_vector_type(2)));

// max over the 4 lanes of each aligned quad
__device__ __forceinline__ uint32_t quad_max(uint32_t m) {
  m = max(m, (uint32_t)__builtin_amdgcn_mov_dpp((int)m, 0xB1, 0xF, 0xF, true));  // quad_perm [1,0,3,2]
  m = max(m, (uint32_t)__builtin_amdgcn_mov_dpp((int)m, 0x4E, 0xF, 0xF, true));  // quad_perm [2,3,0,1]
  return m;
}

// One 64-column step of a wave's 8*NQ rows (NQ groups of 8 rows): block
// scales and codes, the scale bytes staged in the wave's LDS rows, and (XT)
// the step's bf16 values in the wave's projection tile.  EDGE: rows past
// the end and blocks past the chunk are zeroed and not stored.
// QM: numerics mode (QM_NOCLIP, QM_SR).  With QM_SR, idx0 is the matrix
// index (row * cols + column) of this lane's first element in group q = 0 and
// rstep8 = 8 * cols (the next group's rows); one Philox call draws the
// uniforms of the lane's 8 elements.
template <bool EDGE, bool XT, int QM = 0, int NQ = 4, class Store>
__device__ __forceinline__ void quant_step(const v4i (&x)[4], int rw0, int rows, bool col_ok, int lr, int lc,
                                           int lane, const Store& store, int st, FT_LDS uint8_t* sc,
                                           int sc_row, FT_LDS uint16_t* xt, const SrKey& key = SrKey{},
                                           uint64_t idx0 = 0, uint64_t rstep8 = 0) {
#pragma unroll
  for (int q = 0; q < NQ; q++) {
    const int row = rw0 + 8 * q + lr;
    const bool ok = !EDGE || (col_ok && row < rows);
    uint32_t w[4];
#pragma unroll
    for (int e = 0; e < 4; e++) w[e] = ok ? (uint32_t)x[q][e] : 0u;
    // largest |bf16| bit pattern: packed 16-bit maxima of the sign-cleared pairs
    v2u16 p[4];
#pragma unroll
    for (int e = 0; e < 4; e++) p[e] = __builtin_bit_cast(v2u16, w[e] & 0x7FFF7FFFu);
    const v2u16 pm = __builtin_elementwise_max(__builtin_elementwise_max(p[0], p[1]),
                                               __builtin_elementwise_max(p[2], p[3]));
    uint32_t m = max((uint32_t)pm[0], (uint32_t)pm[1]);
    m = quad_max(m);
    const uint32_t code = e8m0_of<QM>(m);
    uint32_t o = 0;
    if constexpr ((QM & QM_SR) != 0) {
      const uint64_t blk8 = (idx0 + (uint64_t)q * rstep8) >> 3;
      uint32_t rnd[4];
      philox4x32_10((uint32_t)blk8, (uint32_t)(blk8 >> 32), key.s0, key.s1, key.k0, key.k1, rnd);
      o = sr_fp4x8(w, code, rnd);
    } else {
      const float s = e8m0_to_f32(code);
      o = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(o, __builtin_bit_cast(v2bf, w[0]), s, 0);
      o = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(o, __builtin_bit_cast(v2bf, w[1]), s, 1);
      o = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(o, __builtin_bit_cast(v2bf, w[2]), s, 2);
      o = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(o, __builtin_bit_cast(v2bf, w[3]), s, 3);
    }
    if (ok) store(q, st, o);
    // scale bytes of (row, blocks 2st, 2st+1): the row's first lane takes the
    // second quad's code along (row_shl:4) and writes both
    const uint32_t code2 = (uint32_t)__builtin_amdgcn_mov_dpp((int)code, 0x104, 0xF, 0xF, true);
    if ((lane & 7) == 0) *(FT_LDS uint16_t*)(sc + (8 * q + lr) * sc_row + 2 * st) = (uint16_t)(code | (code2 << 8));
    if constexpr (XT) *(FT_LDS v4i*)(xt + (8 * q + lr) * QR_XSTRIDE + lc) = v4i{(int)w[0], (int)w[1], (int)w[2], (int)w[3]};
  }
}

template <int RT, int MODE, int WAVES, int CW, int QM, bool MC>
__global__ __launch_bounds__(64 * WAVES) void k_quant_rows(const uint16_t* __restrict__ src, int rows,
                                                                     int cols, uint8_t* __restrict__ codes,
                                                                     uint8_t* __restrict__ scales,
                                                                     const uint16_t* __restrict__ proj, int R,
                                                                     float* __restrict__ proj_out, float* __restrict__ parts,
                                                                     SrKey key, int cpw) {
  using L = QuantLds<RT, MODE, WAVES, CW>;
  __shared__ __attribute__((aligned(16))) uint16_t lds[L::HALFWORDS];
  constexpr int NST = CW / 64;     // 64-column steps per chunk
  constexpr int NT = 64 * WAVES;   // threads

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int rw0 = blockIdx.x * 32 * WAVES + wave * 32;  // first row of this wave
  const int nbc = cols >> 5;
  const int lr = lane >> 3, lc = (lane & 7) * 8;     // row within an 8-row group, column within a step
  // This workgroup's chunks: one, or (MC) cpw consecutive ones (the last
  // group may have fewer); the projection accumulates over all of them, so
  // one partial per group leaves the workgroup.
  const int j0 = MC ? blockIdx.y * cpw : blockIdx.y;
  const int j1 = MC ? min(j0 + cpw, (cols + CW - 1) / CW) : j0 + 1;
  v16f acc[RT];
#pragma unroll
  for (int t = 0; t < RT; t++) acc[t] = v16f{};
  FT_LDS uint16_t* xt = (FT_LDS uint16_t*)lds + L::PROJ_HW + wave * L::X_HW;  // this wave's 32x64 tile
  FT_LDS uint8_t* sc = (FT_LDS uint8_t*)((FT_LDS uint16_t*)lds + L::PROJ_HW + WAVES * L::X_HW + wave * L::SC_HW);
  const int r32 = lane & 31, h = lane >> 5;

  for (int jc = j0; jc < j1; jc++) {
    const int c0 = jc * CW;
    const int ncols = min(CW, cols - c0);
    const int nblk = ncols >> 5;
    if (jc > j0) __syncthreads();   // every wave is done with the previous chunk's projection slice

    // The first PF steps' loads go out right after the projection chunk's;
    // each step, once consumed, issues the load PF steps ahead.  Rows past the end and blocks
    // past the chunk read an in-range address; their values become zeros.
    constexpr int PF = NST < (MC ? 4 : 6) ? NST : (MC ? 4 : 6);   // MC: fewer steps in flight (registers)
    v4i xv[NST][4];
    auto issue = [&](int st) {
      const int col = min(64 * st + lc, ncols - 8);
#pragma unroll
      for (int q = 0; q < 4; q++) {
        const int row = min(rw0 + 8 * q + lr, rows - 1);
        xv[st][q] = *(const v4i*)(src + (size_t)row * cols + c0 + col);
      }
    };
    // The projection chunk is loaded first: every step's MFMAs need it, while
    // the steps' own rows arrive one after another behind it.  It is staged
    // in LDS as 16-byte slots, zero outside [R] x [ncols].
    constexpr int SLOTS_PER_ROW = MODE == 1 ? RT * 4 : CW / 8;
    constexpr int NSLOTS = L::ROWS * SLOTS_PER_ROW;
    constexpr int PER_THREAD = MODE == 0 ? 1 : (NSLOTS + NT - 1) / NT;
    [[maybe_unused]] uint4 v[PER_THREAD];
    if constexpr (MODE != 0) {
#pragma unroll
      for (int u = 0; u < PER_THREAD; u++) {
        const int s = tid + NT * u;
        const int rr = s / SLOTS_PER_ROW, cc = (s % SLOTS_PER_ROW) * 8;
        v[u] = make_uint4(0, 0, 0, 0);
        if constexpr (MODE == 1) {  // rr = k within chunk, cc = j
          if (s < NSLOTS && rr < ncols && cc < R) v[u] = *(const uint4*)(proj + (size_t)(c0 + rr) * R + cc);
        } else {                    // rr = j, cc = k within chunk
          if (s < NSLOTS && rr < R && cc < ncols) v[u] = *(const uint4*)(proj + (size_t)rr * cols + c0 + cc);
        }
      }
    }
#pragma unroll
    for (int st = 0; st < PF; st++) issue(st);

    if constexpr (MODE != 0) {
#pragma unroll
      for (int u = 0; u < PER_THREAD; u++) {
        const int s = tid + NT * u;
        if (s < NSLOTS) *(uint4*)(lds + (s / SLOTS_PER_ROW) * L::STRIDE + (s % SLOTS_PER_ROW) * 8) = v[u];
      }
      __syncthreads();
    }

    // code bytes of this lane's rows 8q + lr at the step's first column (steps add 32 bytes)
    uint8_t* cptr[4];
#pragma unroll
    for (int q = 0; q < 4; q++) cptr[q] = codes + (size_t)(rw0 + 8 * q + lr) * (cols >> 1) + ((c0 + lc) >> 1);
    auto store = [&](int q, int st, uint32_t o) { *(uint32_t*)(cptr[q] + 32 * st) = o; };

#pragma unroll
    for (int st = 0; st < NST; st++) {
      if (2 * st >= nblk) break;  // uniform across the workgroup
      if (st + PF < NST) issue(st + PF);
      const int blk = 2 * st + (lane >> 2 & 1);           // this lane's block within the chunk
      const bool col_ok = blk < nblk;
      // interior (every row of the wave and both blocks of the step in range):
      // no masking; the edge path zeroes what lies outside
      const uint64_t idx0 = (uint64_t)(rw0 + lr) * cols + c0 + 64 * st + lc;
      if (rw0 + 32 > rows || 2 * st + 2 > nblk)
        quant_step<true, MODE != 0, QM>(xv[st], rw0, rows, col_ok, lr, lc, lane, store, st, sc, L::SC_ROW, xt, key,
                                        idx0, 8ull * cols);
      else
        quant_step<false, MODE != 0, QM>(xv[st], rw0, rows, col_ok, lr, lc, lane, store, st, sc, L::SC_ROW, xt, key,
                                         idx0, 8ull * cols);

      if constexpr (MODE != 0) {
        const int g16 = lane >> 4, t16 = lane & 15;
#pragma unroll
        for (int kk = 0; kk < 4; kk++) {
          const v8bf a = __builtin_bit_cast(v8bf, *(const FT_LDS v4i*)(xt + r32 * QR_XSTRIDE + 16 * kk + 8 * h));
          const int kloc = 64 * st + 16 * kk + 8 * h;  // chunk position of this lane's 8 elements
#pragma unroll
          for (int t = 0; t < RT; t++) {
            v8bf b;
            if constexpr (MODE == 2) {
              const int j = t * 32 + r32;
              b = __builtin_bit_cast(v8bf, *(const FT_LDS v4i*)((FT_LDS uint16_t*)lds + j * L::STRIDE + kloc));
            } else {
              // group g16 covers columns t*32 + 16*(g16&1) + [0,16), reduction rows kloc..kloc+7
              const int jj = t16 >> 2, qq = t16 & 3;
              const int col = t * 32 + 16 * (g16 & 1) + 4 * qq;
              const FT_LDS uint16_t* base = (FT_LDS uint16_t*)lds + (kloc + jj) * L::STRIDE + col;
              v4s lo = lds_read_tr16(base);
              v4s hi = lds_read_tr16(base + 4 * L::STRIDE);
              b = make_v8bf(lo, hi);
            }
            acc[t] = mfma_bf16_32x32x16(a, b, acc[t]);
          }
        }
      }
    }

    // scales: each row's bytes of this chunk are contiguous; 4-byte stores when
    // rows and the chunk start are 4-byte aligned, else bytes
    {
      constexpr int DW = L::SC_ROW / 4;   // dwords per staged row
      const bool al = (nbc & 3) == 0 && ((c0 >> 5) & 3) == 0;
#pragma unroll
      for (int d0 = 0; d0 < 32 * DW; d0 += 64) {
        const int d = d0 + lane;
        const int rr = d / DW, dw = d % DW;
        const int row = rw0 + rr;
        if (d < 32 * DW && row < rows && 4 * dw < nblk) {
          uint8_t* dst = scales + (size_t)row * nbc + (c0 >> 5) + 4 * dw;
          const FT_LDS uint8_t* srcb = sc + rr * L::SC_ROW + 4 * dw;
          if (al && 4 * dw + 4 <= nblk) {
            *(uint32_t*)dst = *(const FT_LDS uint32_t*)srcb;
          } else {
            for (int b = 0; b < 4 && 4 * dw + b < nblk; b++) dst[b] = srcb[b];
          }
        }
      }
    }
  }

  if constexpr (MODE != 0) {
    // this group's partial (several groups) or the projection itself (one
    // group), one 32-column tile at a time through the wave's own bf16 tile
    // (32 rows x 36 fp32 fit its 32 x 72 halfwords), stored as row-contiguous
    // 16-byte runs: 4 stores per tile instead of 16
    static_assert(32 * 36 * 4 == L::X_HW * 2, "fp32 tile in the bf16 tile's place");
    float* dst = parts ? parts + (size_t)blockIdx.y * rows * R : proj_out;
    FT_LDS float* pst = (FT_LDS float*)xt;
#pragma unroll
    for (int t = 0; t < RT; t++) {
#pragma unroll
      for (int v = 0; v < 16; v++) pst[(8 * (v >> 2) + 4 * h + (v & 3)) * 36 + r32] = acc[t][v];
#pragma unroll
      for (int q = 0; q < 4; q++) {
        const int idx = lane + 64 * q, row = idx >> 3, c4 = idx & 7;
        const v4i val = *(const FT_LDS v4i*)(pst + row * 36 + 4 * c4);   // four fp32, copied as bits
        const int rr = rw0 + row, j = t * 32 + 4 * c4;
        if (rr < rows && j < R) *(v4i*)(dst + (size_t)rr * R + j) = val;
      }
    }
  }
}

// ---------------------------------------------------------------- full rows
// Projection [cols, R] only.  Workgroup = WAVES waves over ROWS = 8*NQ whole
// rows (32, or 24 when that fills more CUs); wave w takes the 64-column
// steps w, w + WAVES, ...  A step is handled as in
// k_quant_rows: row-contiguous loads (every 8 lanes read one 128-byte line),
// block scales and codes from lane quads, the bf16 values through a private
// LDS tile into the MFMA layout.  The step's 64 projection rows come with it,
// also as whole 128-byte lines, into a second private tile that is read back
// transposed.  The waves' partial projections are added in LDS in wave
// order: nothing partial leaves the workgroup and no reduction kernel
// follows.  The price is one read of the projection matrix (from L2) per
// workgroup, on fewer workgroups than the chunked kernel has.  With 24 rows
// the MFMA tile's last 8 rows are zeros and their results are dropped.
constexpr int QF_MAX_BLOCKS = 128;   // scale bytes per row staged in LDS: cols <= 4096
// Waves per whole-row workgroup: 10 (at most 5 of a 48-step row each) where
// the kernel fits 168 VGPRs without spilling, else 8 (stochastic rounding,
// 32-row workgroups).
template <int QM, int NQ>
constexpr int fr_waves() { return ((QM & QM_SR) != 0 || NQ == 4) ? 8 : 10; }

template <int RT, int WAVES>
struct QuantFrLds {
  static constexpr int PSTRIDE = RT * 32 + 16;                        // projection tile [64 k][RT*32] (halfwords)
  static constexpr int PTILE = 64 * PSTRIDE * 2;
  static constexpr int XTILE = 32 * QR_XSTRIDE * 2;
  static constexpr int WAVE_BYTES = PTILE + XTILE;
  static constexpr int RED = WAVES * RT * 16 * 64 * 4;               // the waves' accumulators
  static constexpr int WORK = WAVES * WAVE_BYTES > RED ? WAVES * WAVE_BYTES : RED;
  static constexpr int BYTES = WORK + 32 * QF_MAX_BLOCKS;
};

template <int RT, int WAVES, int QM, int NQ>
__global__ __launch_bounds__(64 * WAVES) void k_quant_rows_fr(const uint16_t* __restrict__ src, int rows, int cols,
                                                              uint8_t* __restrict__ codes,
                                                              uint8_t* __restrict__ scales,
                                                              const uint16_t* __restrict__ proj, int R,
                                                              float* __restrict__ proj_out, SrKey key) {
  using L = QuantFrLds<RT, WAVES>;
  __shared__ __attribute__((aligned(16))) uint8_t lds[L::BYTES];
  constexpr int NT = 64 * WAVES;
  constexpr int NP = 4 * RT;        // 16-byte projection loads per lane and step
  constexpr int NB = WAVES > 8 ? 2 : 3;   // step buffers: NB - 1 steps in flight ahead of the one consumed

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  constexpr int ROWS = 8 * NQ;
  const int row0 = blockIdx.x * ROWS;
  const int lr = lane >> 3, lc = (lane & 7) * 8;     // row within an 8-row group, column within a step
  const int nsteps = (cols + 63) >> 6;
  const int nmine = wave < nsteps ? (nsteps - 1 - wave) / WAVES + 1 : 0;
  const int nbc = cols >> 5;
  FT_LDS uint8_t* sc = (FT_LDS uint8_t*)(lds + L::WORK);             // [32 rows][QF_MAX_BLOCKS] scale bytes
  FT_LDS uint16_t* pt = (FT_LDS uint16_t*)(lds + wave * L::WAVE_BYTES);   // projection tile
  FT_LDS uint16_t* xt = (FT_LDS uint16_t*)(lds + wave * L::WAVE_BYTES + L::PTILE);   // bf16 tile [32][64]
  // Buffer offsets: per lane and constant over the steps (rows past the
  // matrix and projection columns past R get an out-of-range offset and
  // read zeros; projection rows past cols lie past the buffer), plus a
  // uniform offset per step.
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(src, (uint32_t)((size_t)rows * cols * 2));
  const __amdgpu_buffer_rsrc_t rc = make_rsrc(codes, (uint32_t)((size_t)rows * cols / 2));
  const __amdgpu_buffer_rsrc_t rp = make_rsrc(proj, (uint32_t)((size_t)R * cols * 2));
  uint32_t xoff[NQ], coff[NQ], poff[NP];
#pragma unroll
  for (int q = 0; q < NQ; q++) {
    const int r = row0 + 8 * q + lr;
    xoff[q] = r < rows ? (uint32_t)(r * cols + lc) * 2u : kOobOffset;
    coff[q] = r < rows ? (uint32_t)(r * (cols >> 1) + (lc >> 1)) : kOobOffset;
  }
#pragma unroll
  for (int q = 0; q < NP; q++) {   // 16-byte slot lane + 64q of the step's [64 k][RT*32] rows
    const int sl = lane + 64 * q, kr = sl / (RT * 4), c16 = sl % (RT * 4);
    poff[q] = 8 * c16 < R ? (uint32_t)(kr * R + 8 * c16) * 2u : kOobOffset;
  }
  auto store = [&](int q, int st, uint32_t o) {
    __builtin_amdgcn_raw_buffer_store_b32(o, rc, coff[q], 32 * st, 0);
  };

  auto step_of = [&](int k) { return wave + k * WAVES; };

  struct Ops { v4i x[4]; v4i p[NP]; };   // x[q] for q < NQ
  // Loads of local step k.  On the last step of a row whose length is an odd
  // multiple of 32, the upper lanes read past the row; quant_step zeroes those
  // values (the projection rows there lie past the buffer).
  auto issue = [&](int k, Ops& o) {
    const int c = 64 * step_of(k);
#pragma unroll
    for (int q = 0; q < NQ; q++) o.x[q] = __builtin_amdgcn_raw_buffer_load_b128(rx, xoff[q], 2 * c, 0);
#pragma unroll
    for (int q = 0; q < NP; q++)
      o.p[q] = __builtin_amdgcn_raw_buffer_load_b128(rp, poff[q], 2 * c * R, 0);
  };

  v16f acc[RT];
#pragma unroll
  for (int t = 0; t < RT; t++) acc[t] = v16f{};
  const int r32 = lane & 31, h = lane >> 5, g16 = lane >> 4, t16 = lane & 15;
  if constexpr (ROWS < 32) {
    // rows ROWS..31 of the wave's bf16 tile stay zero: the steps write rows < ROWS only
    for (int e = lane; e < (32 - ROWS) * (QR_XSTRIDE / 8); e += 64)
      *(FT_LDS v4i*)(xt + ROWS * QR_XSTRIDE + 8 * e) = v4i{0, 0, 0, 0};
  }

  auto consume = [&](int k, Ops& o) {
    const int st = step_of(k), c = 64 * st;
    const int blk = 2 * st + (lane >> 2 & 1);
    const bool col_ok = blk < nbc;
    const uint64_t idx0 = (uint64_t)(row0 + lr) * cols + c + lc;
    if (row0 + ROWS > rows || c + 64 > cols)
      quant_step<true, true, QM, NQ>(o.x, row0, rows, col_ok, lr, lc, lane, store, st, sc, QF_MAX_BLOCKS, xt, key,
                                     idx0, 8ull * cols);
    else
      quant_step<false, true, QM, NQ>(o.x, row0, rows, col_ok, lr, lc, lane, store, st, sc, QF_MAX_BLOCKS, xt, key,
                                      idx0, 8ull * cols);
    // the step's projection rows
#pragma unroll
    for (int q = 0; q < NP; q++) {
      const int sl = lane + 64 * q, kr = sl / (RT * 4), c16 = sl % (RT * 4);
      *(FT_LDS v4i*)(pt + kr * L::PSTRIDE + 8 * c16) = o.p[q];
    }
#pragma unroll
    for (int kk = 0; kk < 4; kk++) {
      const v8bf a = __builtin_bit_cast(v8bf, *(const FT_LDS v4i*)(xt + r32 * QR_XSTRIDE + 16 * kk + 8 * h));
#pragma unroll
      for (int t = 0; t < RT; t++) {
        // group g16 covers columns t*32 + 16(g16 & 1) + [0,16), reduction rows 16kk + 8h + [0,8)
        const int jj = t16 >> 2, qq = t16 & 3;
        const FT_LDS uint16_t* base = pt + (16 * kk + 8 * h + jj) * L::PSTRIDE + t * 32 + 16 * (g16 & 1) + 4 * qq;
        const v8bf b = make_v8bf(lds_read_tr16((const FT_LDS void*)base),
                                 lds_read_tr16((const FT_LDS void*)(base + 4 * L::PSTRIDE)));
        acc[t] = mfma_bf16_32x32x16(a, b, acc[t]);
      }
    }
  };

  Ops buf[NB];
#pragma unroll
  for (int k = 0; k < NB - 1; k++)
    if (k < nmine) issue(k, buf[k]);
#pragma unroll 1
  for (int k0 = 0; k0 < nmine; k0 += NB) {
#pragma unroll
    for (int u = 0; u < NB; u++) {
      const int k = k0 + u;
      if (k < nmine) {
        if (k + NB - 1 < nmine) issue(k + NB - 1, buf[(u + NB - 1) % NB]);
        consume(k, buf[u]);
      }
    }
  }

  // the waves' partial projections, added in wave order
  __syncthreads();
  float* red = (float*)lds;
#pragma unroll
  for (int t = 0; t < RT; t++)
#pragma unroll
    for (int v = 0; v < 16; v++) red[((wave * RT + t) * 16 + v) * 64 + lane] = acc[t][v];
  __syncthreads();
  constexpr int NOUT = RT * 16 * 64;
  for (int o = tid; o < NOUT; o += NT) {
    float sum = 0.f;
#pragma unroll
    for (int w = 0; w < WAVES; w++) sum += red[w * NOUT + o];
    const int t = o >> 10, v = (o >> 6) & 15, ln = o & 63;
    const int rl = 8 * (v >> 2) + 4 * (ln >> 5) + (v & 3), r = row0 + rl, j = t * 32 + (ln & 31);
    if (rl < ROWS && r < rows && j < R) proj_out[(size_t)r * R + j] = sum;
  }
  // scale bytes of the workgroup's rows
  const int nw = (nbc + 3) >> 2;
  const bool al = (nbc & 3) == 0;
  for (int d = tid; d < ROWS * nw; d += NT) {
    const int rr = d / nw, dw = d % nw, r = row0 + rr;
    if (r >= rows) continue;
    uint8_t* dst = scales + (size_t)r * nbc + 4 * dw;
    const FT_LDS uint8_t* sp = sc + rr * QF_MAX_BLOCKS + 4 * dw;
    if (al) {
      *(uint32_t*)dst = *(const FT_LDS uint32_t*)sp;
    } else {
      for (int b = 0; b < 4 && 4 * dw + b < nbc; b++) dst[b] = sp[b];
    }
  }
}

// ---------------------------------------------------------------- tiles
// One wave per 32x32 tile: lane l takes row l/2, columns 16*(l%2) + [0,16).
// NOCLIP: the no-clip scale rule.  per_row: scales are written as
// [rows, cols/32], every row of a tile carrying the tile's code (2-D blocked
// activations in the layout the GEMM reads), else [rows/32, cols/32].
template <bool NOCLIP>
__global__ __launch_bounds__(256) void k_quant_tiles(const uint16_t* __restrict__ src, int rows, int cols,
                                                     uint8_t* __restrict__ codes, uint8_t* __restrict__ scales,
                                                     int per_row) {
  const int lane = threadIdx.x & 63;
  const int tile = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int nbc = cols >> 5;
  if (tile >= (rows >> 5) * nbc) return;  // whole wave exits together
  const int tr = tile / nbc, tc = tile % nbc;
  const int row = tr * 32 + (lane >> 1);
  const int col = tc * 32 + 16 * (lane & 1);
  const uint4* p = (const uint4*)(src + (size_t)row * cols + col);
  uint4 v0 = p[0], v1 = p[1];
  uint32_t w[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
  uint32_t m = 0;
#pragma unroll
  for (int i = 0; i < 8; i++) {
    uint32_t a = w[i] & 0x7FFF7FFFu;
    m = max(m, max(a & 0xFFFFu, a >> 16));
  }
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off, 64));
  const uint32_t code = NOCLIP ? e8m0_noclip_from_amax_bits(m) : e8m0_from_amax_bits(m);
  const float s = e8m0_to_f32(code);
  uint32_t o0 = 0, o1 = 0;
  o0 = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(o0, __builtin_bit_cast(v2bf, w[0]), s, 0);
  o0 = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(o0, __builtin_bit_cast(v2bf, w[1]), s, 1);
  o0 = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(o0, __builtin_bit_cast(v2bf, w[2]), s, 2);
  o0 = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(o0, __builtin_bit_cast(v2bf, w[3]), s, 3);
  o1 = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(o1, __builtin_bit_cast(v2bf, w[4]), s, 0);
  o1 = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(o1, __builtin_bit_cast(v2bf, w[5]), s, 1);
  o1 = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(o1, __builtin_bit_cast(v2bf, w[6]), s, 2);
  o1 = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(o1, __builtin_bit_cast(v2bf, w[7]), s, 3);
  *(uint2*)(codes + (size_t)row * (cols >> 1) + (col >> 1)) = make_uint2(o0, o1);
  if (per_row) {
    if ((lane & 1) == 0) scales[(size_t)row * nbc + tc] = (uint8_t)code;
  } else if (lane == 0) {
    scales[(size_t)tr * nbc + tc] = (uint8_t)code;
  }
}

// ---------------------------------------------------------------- launchers
// Geometry per mode, from timing at the FLUX shapes: 8 waves (256 rows) per
// workgroup amortize the staged projection chunk.  The [cols, R] projection
// takes 384-column chunks, or 256 when that would leave fewer workgroups
// than CUs (4608 x 3072: 16.5 us against 17.6); more chunks mean more
// partial sums, which dominate for long rows.  The [R, cols] projection
// takes 768-column chunks (fewer partial sums; 384 and 512 are slower)
// while the chunk fits LDS.
// Chunks per workgroup of the chunked kernel (256-row workgroups), so that
// long rows leave fewer partial sums: for [cols, R] as many as 6 while 384
// workgroups remain (18432 x 15360 at 512 columns: 6 partials per row
// instead of 30), for [R, cols] as many as 4 while 512 remain (18432 x 21504:
// 11 instead of 42; 3 or 8 per workgroup measured slower).  Shapes with fewer
// workgroups keep one chunk each.
static int quant_chunks_per_wg(int rows, int cols, int cw, int layout) {
  const size_t rb = (size_t)((rows + 255) / 256), nch = (size_t)((cols + cw - 1) / cw);
  const int cmax = layout == 0 ? 6 : 4;
  const size_t need = layout == 0 ? 384 : 512;
  for (int c = cmax; c > 1; c--)
    if (rb * ((nch + c - 1) / c) >= need) return c;
  return 1;
}

static int quant_chunk_cols(int rows, int cols, int R, int layout) {
  if (R == 0) return 384;
  const int rt = (R + 31) / 32;
  // the widest chunk whose projection slice fits LDS, so fewer partial sums,
  // as long as it still makes a full round of workgroups (4608 x 15360,
  // R = 64: 61-62 us at 384 columns, 58 at 512, 49-51 at 640; 18432 x 15360,
  // R = 96: 300 at 384, 280 at 512; 18432 x 3072: 58-61 -> 50-53 us at
  // R = 96, 49-50 -> 42-43 at R = 64)
  if (layout == 0) {
    const int wide = rt <= 2 ? 640 : rt == 3 ? 512 : 384;
    if ((size_t)((rows + 255) / 256) * ((cols + wide - 1) / wide) >= 256) return wide;
  }
  if (layout == 0) return (size_t)((rows + 255) / 256) * ((cols + 383) / 384) < 256 ? 256 : 384;
  // [R, cols]: the widest chunk whose projection slice fits LDS (18432 x 21504
  // with R = 96: 416-437 us at 384 columns, 385-400 at 512; 4608 x 9216 with
  // R = 64: 28.8 us at 768, 36-37 at 256 or 384), except that 256-column
  // chunks fill the chip when 768-column ones would make fewer than 128
  // workgroups (4608 x 3072: 20.4 -> 16.1 us; 512 x 3072: 17.3 -> 13.8)
  if (rt <= 2 && (size_t)((rows + 255) / 256) * ((cols + 767) / 768) < 128) return 256;
  return rt <= 2 ? 768 : rt == 3 ? 512 : 384;
}

// Whole rows per workgroup (no partial sums) for proj [cols, R] when the
// whole-row workgroups make between 64 and one round of 256, rows are at
// most 4096 long and the projection is at most 64 wide (4608 x 3072: 12.8 to
// 13.5 us, against 13.1 plus a 4.7 us reduction for the chunks).  Longer rows
// make each workgroup read a larger projection matrix (4608 x 15360: 94 us
// against 80).  For proj [R, cols] at 4608 x 9216 the chunked kernel is
// faster (33 against 36 us): the step work of 4608 rows outweighs the
// partial sums.  Rows per whole-row workgroup: 24 when that still makes one
// round (more CUs busy than with 32), else 32.
static int quant_fr_rows(int rows) { return (rows + 23) / 24 <= 256 ? 24 : 32; }

static bool quant_full_rows(int rows, int cols, int R, int layout) {
  const int wg = (rows + quant_fr_rows(rows) - 1) / quant_fr_rows(rows);
  return layout == 0 && R > 0 && R <= 64 && cols <= 32 * QF_MAX_BLOCKS && wg >= 64 && wg <= 256;
}

size_t quant_rows_workspace(int rows, int cols, int R, int layout) {
  if (R == 0 || quant_full_rows(rows, cols, R, layout)) return 0;
  const int cw = quant_chunk_cols(rows, cols, R, layout);
  const int cpw = quant_chunks_per_wg(rows, cols, cw, layout);
  const int groups = ((cols + cw - 1) / cw + cpw - 1) / cpw;
  return groups > 1 ? (size_t)groups * rows * R * sizeof(float) : 0;
}

template <int RT, int MODE, int WAVES, int CW, int QM>
static hipError_t launch_rows_t(const uint16_t* src, int rows, int cols, uint8_t* codes, uint8_t* scales,
                                const uint16_t* proj, int R, float* proj_out, float* ws, const SrKey& key,
                                hipStream_t st) {
  const int cpw = MODE == 0 ? 1 : quant_chunks_per_wg(rows, cols, CW, MODE == 1 ? 0 : 1);
  const int nch = (cols + CW - 1) / CW;
  dim3 grid((rows + 32 * WAVES - 1) / (32 * WAVES), (nch + cpw - 1) / cpw);
  float* parts = MODE != 0 && grid.y > 1 ? ws : nullptr;
  if (cpw > 1)
    k_quant_rows<RT, MODE, WAVES, CW, QM, true><<<grid, 64 * WAVES, 0, st>>>(src, rows, cols, codes, scales, proj, R,
                                                                           proj_out, parts, key, cpw);
  else
    k_quant_rows<RT, MODE, WAVES, CW, QM, false><<<grid, 64 * WAVES, 0, st>>>(src, rows, cols, codes, scales, proj, R,
                                                                            proj_out, parts, key, 1);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !parts) return e;
  return launch_reduce_parts(parts, (int)grid.y, (size_t)rows * R, proj_out, 0, nullptr, false, st);
}

template <int QM>
static hipError_t launch_quant_rows_qm(const uint16_t* src, int rows, int cols, uint8_t* codes, uint8_t* scales,
                                       const uint16_t* proj, int R, int layout, float* proj_out, float* ws,
                                       const SrKey& key, hipStream_t st) {
  if (!proj || R == 0)
    return launch_rows_t<1, 0, 4, 384, QM>(src, rows, cols, codes, scales, nullptr, 0, nullptr, nullptr, key, st);
  const int rt = (R + 31) / 32;
  if (quant_full_rows(rows, cols, R, layout)) {
    const int fr = quant_fr_rows(rows);
    const unsigned grid = (unsigned)((rows + fr - 1) / fr);
#define FT_FR(RT_, NQ_) \
  k_quant_rows_fr<RT_, fr_waves<QM, NQ_>(), QM, NQ_><<<grid, 64 * fr_waves<QM, NQ_>(), 0, st>>>(src, rows, cols, codes, \
                                                                                            scales, proj, R, proj_out, key)
    if (fr == 24) { if (rt == 1) FT_FR(1, 3); else FT_FR(2, 3); }
    else { if (rt == 1) FT_FR(1, 4); else FT_FR(2, 4); }
#undef FT_FR
    return hipGetLastError();
  }
#define FT_ROWS(RT_, MODE_, CW_) \
  launch_rows_t<RT_, MODE_, 8, CW_, QM>(src, rows, cols, codes, scales, proj, R, proj_out, ws, key, st)
  if (layout == 0) {
    const int cw = quant_chunk_cols(rows, cols, R, layout);
    if (cw == 640) return rt == 1 ? FT_ROWS(1, 1, 640) : FT_ROWS(2, 1, 640);
    if (cw == 512) return FT_ROWS(3, 1, 512);
    if (cw == 256) {
      switch (rt) {
        case 1: return FT_ROWS(1, 1, 256);
        case 2: return FT_ROWS(2, 1, 256);
        case 3: return FT_ROWS(3, 1, 256);
        default: return FT_ROWS(4, 1, 256);
      }
    }
    switch (rt) {
      case 1: return FT_ROWS(1, 1, 384);
      case 2: return FT_ROWS(2, 1, 384);
      case 3: return FT_ROWS(3, 1, 384);
      default: return FT_ROWS(4, 1, 384);
    }
  }
  if (quant_chunk_cols(rows, cols, R, layout) == 256) return rt == 1 ? FT_ROWS(1, 2, 256) : FT_ROWS(2, 2, 256);
  switch (rt) {
    case 1: return FT_ROWS(1, 2, 768);
    case 2: return FT_ROWS(2, 2, 768);
    case 3: return FT_ROWS(3, 2, 512);
    default: return FT_ROWS(4, 2, 384);
  }
#undef FT_ROWS
}

hipError_t launch_quant_rows(const uint16_t* src, int rows, int cols, uint8_t* codes, uint8_t* scales,
                             const uint16_t* proj, int R, int layout, float* proj_out, float* ws, hipStream_t st,
                             const QuantMode& mode) {
  const SrKey key{(uint32_t)mode.seed, (uint32_t)(mode.seed >> 32), (uint32_t)mode.stream,
                  (uint32_t)(mode.stream >> 32)};
  switch ((mode.no_clip ? QM_NOCLIP : 0) | (mode.stochastic ? QM_SR : 0)) {
    case 0: return launch_quant_rows_qm<0>(src, rows, cols, codes, scales, proj, R, layout, proj_out, ws, key, st);
    case QM_NOCLIP:
      return launch_quant_rows_qm<QM_NOCLIP>(src, rows, cols, codes, scales, proj, R, layout, proj_out, ws, key, st);
    case QM_SR:
      return launch_quant_rows_qm<QM_SR>(src, rows, cols, codes, scales, proj, R, layout, proj_out, ws, key, st);
    default:
      return launch_quant_rows_qm<QM_NOCLIP | QM_SR>(src, rows, cols, codes, scales, proj, R, layout, proj_out, ws,
                                                     key, st);
  }
}

hipError_t launch_quant_tiles(const uint16_t* src, int rows, int cols, uint8_t* codes, uint8_t* scales,
                              hipStream_t st, const QuantMode& mode) {
  const int tiles = (rows / 32) * (cols / 32);
  if (mode.no_clip)
    k_quant_tiles<true><<<(tiles + 3) / 4, 256, 0, st>>>(src, rows, cols, codes, scales, mode.scales_per_row);
  else
    k_quant_tiles<false><<<(tiles + 3) / 4, 256, 0, st>>>(src, rows, cols, codes, scales, mode.scales_per_row);
  return hipGetLastError();
}

}  // namespace ft
