// Block-wise MXFP4 quantization kernels (gfx950).
//
// k_quant_rows: 1x32 blocks along rows of a bf16 matrix (activations X and
// gradients G, FourTune Sec. 3.1 dynamic quantization), fused with the
// low-rank down-projection of the same rows (Sec. 3.3, LoRA fusion: the
// stabilizer and adapter branches share the input, so one pass reads it once).
// k_quant_tiles: 32x32 tiles of the frozen weight (Sec. 3.2), offline.
#include "ft_device.h"
#include "ft_kernels.h"

namespace ft {

// ---------------------------------------------------------------- rows
// Workgroup = 4 waves; wave w owns 32 rows [row0 + 32w, +32) of one column
// chunk of QR_CW columns.  Lane l holds row l%32 and, for block pair i, the
// 32-element block 2i + l/32 of the chunk: it reads the block's 64 bytes,
// quantizes it alone (no cross-lane reduction), and feeds the same registers
// to the projection MFMAs.  The projection's reduction order is permuted to
// match: MFMA q of pair i takes elements [8q, 8q+8) of each lane's block, and
// the B operand is read from the same chunk positions.
//
// proj chunk staged in LDS (zero padded to RT*32 columns and to QR_CW rows):
//   MODE 1 (proj [cols, R]):  lds[k][j], row stride RT*32 + 16 halfwords;
//     B fragments come from transposing reads (ds_read_b64_tr_b16).
//   MODE 2 (proj [R, cols]):  lds[j][k], row stride QR_CW + 8 halfwords;
//     B fragments are plain 16-byte reads.
template <int RT, int MODE>
struct QuantLds {
  static constexpr int STRIDE = MODE == 1 ? RT * 32 + 16 : QR_CW + 8;   // halfwords
  static constexpr int ROWS = MODE == 1 ? QR_CW : RT * 32;
  static constexpr int HALFWORDS = MODE == 0 ? 8 : ROWS * STRIDE;
};

template <int RT, int MODE>
__global__ __launch_bounds__(256) void k_quant_rows(const uint16_t* __restrict__ src, int rows, int cols,
                                                    uint8_t* __restrict__ codes, uint8_t* __restrict__ scales,
                                                    const uint16_t* __restrict__ proj, int R,
                                                    float* __restrict__ proj_out, int use_atomics) {
  using L = QuantLds<RT, MODE>;
  __shared__ __attribute__((aligned(16))) uint16_t lds[L::HALFWORDS];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int r32 = lane & 31, h = lane >> 5;
  const int row = blockIdx.x * QR_ROWS + wave * 32 + r32;
  const int c0 = blockIdx.y * QR_CW;
  const int ncols = min(QR_CW, cols - c0);
  const int nblk = ncols >> 5;
  const bool row_ok = row < rows;
  const int nbc = cols >> 5;

  if constexpr (MODE != 0) {
    // Stage the projection chunk: 16-byte slots, zero outside [R] x [ncols].
    constexpr int SLOTS_PER_ROW = MODE == 1 ? RT * 4 : QR_CW / 8;
    constexpr int NSLOTS = L::ROWS * SLOTS_PER_ROW;
    for (int s = tid; s < NSLOTS; s += 256) {
      const int rr = s / SLOTS_PER_ROW, cc = (s % SLOTS_PER_ROW) * 8;
      uint4 v = make_uint4(0, 0, 0, 0);
      if constexpr (MODE == 1) {  // rr = k within chunk, cc = j
        if (rr < ncols && cc < R) v = *(const uint4*)(proj + (size_t)(c0 + rr) * R + cc);
      } else {                    // rr = j, cc = k within chunk
        if (rr < R && cc < ncols) v = *(const uint4*)(proj + (size_t)rr * cols + c0 + cc);
      }
      *(uint4*)(lds + rr * L::STRIDE + cc) = v;
    }
    __syncthreads();
  }

  v16f acc[RT];
#pragma unroll
  for (int t = 0; t < RT; t++) acc[t] = v16f{};

#pragma unroll 1
  for (int i = 0; i < QR_CW / 64; i++) {
    if (2 * i >= nblk) break;  // uniform across the workgroup
    const int kb = 2 * i + h;
    const bool ok = row_ok && kb < nblk;
    uint32_t w[16];
    if (ok) {
      const uint4* p = (const uint4*)(src + (size_t)row * cols + c0 + kb * 32);
#pragma unroll
      for (int q = 0; q < 4; q++) {
        uint4 v = load_nt16(p + q);
        w[4 * q + 0] = v.x; w[4 * q + 1] = v.y; w[4 * q + 2] = v.z; w[4 * q + 3] = v.w;
      }
      uint32_t out[4];
      const uint32_t sc = quantize32(w, out);
      *(uint4*)(codes + (size_t)row * (cols >> 1) + ((c0 + kb * 32) >> 1)) = make_uint4(out[0], out[1], out[2], out[3]);
      scales[(size_t)row * nbc + (c0 >> 5) + kb] = (uint8_t)sc;
    } else {
#pragma unroll
      for (int q = 0; q < 16; q++) w[q] = 0;
    }

    if constexpr (MODE != 0) {
      const int g16 = lane >> 4, t16 = lane & 15;
#pragma unroll
      for (int q = 0; q < 4; q++) {
        uint32_t ah[8];
#pragma unroll
        for (int e = 0; e < 4; e++) { ah[2 * e] = w[4 * q + e] & 0xFFFFu; ah[2 * e + 1] = w[4 * q + e] >> 16; }
        const v8bf a = pack_v8bf(ah);
        const int kloc = kb * 32 + 8 * q;  // chunk position of this lane's 8 elements
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

  if constexpr (MODE != 0) {
    const int rbase = blockIdx.x * QR_ROWS + wave * 32;
#pragma unroll
    for (int t = 0; t < RT; t++) {
      const int j = t * 32 + r32;
      if (j >= R) continue;
#pragma unroll
      for (int v = 0; v < 16; v++) {
        const int rr = rbase + 8 * (v >> 2) + 4 * h + (v & 3);
        if (rr < rows) {
          float* dst = proj_out + (size_t)rr * R + j;
          if (use_atomics) atomicAdd(dst, acc[t][v]);
          else *dst = acc[t][v];
        }
      }
    }
  }
}

// ---------------------------------------------------------------- tiles
// One wave per 32x32 tile: lane l takes row l/2, columns 16*(l%2) + [0,16).
__global__ __launch_bounds__(256) void k_quant_tiles(const uint16_t* __restrict__ src, int rows, int cols,
                                                     uint8_t* __restrict__ codes, uint8_t* __restrict__ scales) {
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
  const uint32_t code = e8m0_from_amax_bits(m);
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
  if (lane == 0) scales[(size_t)tr * nbc + tc] = (uint8_t)code;
}

__global__ void k_fill_f32(float* __restrict__ p, size_t n, float v) {
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t st = (size_t)gridDim.x * blockDim.x;
  for (; i < n; i += st) p[i] = v;
}

// ---------------------------------------------------------------- launchers
template <int RT, int MODE>
static hipError_t launch_rows_t(const uint16_t* src, int rows, int cols, uint8_t* codes, uint8_t* scales,
                                const uint16_t* proj, int R, float* proj_out, hipStream_t st) {
  dim3 grid((rows + QR_ROWS - 1) / QR_ROWS, (cols + QR_CW - 1) / QR_CW);
  const int atomics = MODE != 0 && grid.y > 1;
  if (atomics) {
    const size_t n = (size_t)rows * R;
    k_fill_f32<<<(unsigned)std::min<size_t>((n + 255) / 256, 4096), 256, 0, st>>>(proj_out, n, 0.0f);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  k_quant_rows<RT, MODE><<<grid, 256, 0, st>>>(src, rows, cols, codes, scales, proj, R, proj_out, atomics);
  return hipGetLastError();
}

hipError_t launch_quant_rows(const uint16_t* src, int rows, int cols, uint8_t* codes, uint8_t* scales,
                             const uint16_t* proj, int R, int layout, float* proj_out, hipStream_t st) {
  if (!proj || R == 0) return launch_rows_t<1, 0>(src, rows, cols, codes, scales, nullptr, 0, nullptr, st);
  const int rt = (R + 31) / 32;
  if (layout == 0) {
    switch (rt) {
      case 1: return launch_rows_t<1, 1>(src, rows, cols, codes, scales, proj, R, proj_out, st);
      case 2: return launch_rows_t<2, 1>(src, rows, cols, codes, scales, proj, R, proj_out, st);
      case 3: return launch_rows_t<3, 1>(src, rows, cols, codes, scales, proj, R, proj_out, st);
      default: return launch_rows_t<4, 1>(src, rows, cols, codes, scales, proj, R, proj_out, st);
    }
  }
  switch (rt) {
    case 1: return launch_rows_t<1, 2>(src, rows, cols, codes, scales, proj, R, proj_out, st);
    case 2: return launch_rows_t<2, 2>(src, rows, cols, codes, scales, proj, R, proj_out, st);
    case 3: return launch_rows_t<3, 2>(src, rows, cols, codes, scales, proj, R, proj_out, st);
    default: return launch_rows_t<4, 2>(src, rows, cols, codes, scales, proj, R, proj_out, st);
  }
}

hipError_t launch_quant_tiles(const uint16_t* src, int rows, int cols, uint8_t* codes, uint8_t* scales,
                              hipStream_t st) {
  const int tiles = (rows / 32) * (cols / 32);
  k_quant_tiles<<<(tiles + 3) / 4, 256, 0, st>>>(src, rows, cols, codes, scales);
  return hipGetLastError();
}

hipError_t launch_fill_f32(float* p, size_t n, float v, hipStream_t st) {
  if (n == 0) return hipSuccess;
  k_fill_f32<<<(unsigned)std::min<size_t>((n + 255) / 256, 4096), 256, 0, st>>>(p, n, v);
  return hipGetLastError();
}

}  // namespace ft
