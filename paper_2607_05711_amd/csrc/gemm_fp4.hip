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
#include "ft_device.h"
#include "ft_kernels.h"

namespace ft {

constexpr int GB = 256;                 // output tile edge (rows and columns)
constexpr int GK = 256;                 // reduction elements per stage
constexpr int GROW = GK / 2;            // bytes of codes per tile row per stage
constexpr int GSTRIDE = GROW + 16;      // padded LDS row stride (bytes)
constexpr int GTILE = GB * GSTRIDE;     // bytes per operand tile per stage

template <bool BWD, bool OUT_F32>
__global__ __launch_bounds__(256, 1) void k_gemm_fp4(const uint8_t* __restrict__ A, const uint8_t* __restrict__ As,
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

hipError_t launch_gemm_fp4(bool bwd, const uint8_t* a, const uint8_t* as, const uint8_t* wq, const uint8_t* ws,
                           int M, int N, int K, const float* P, int R, const uint16_t* lr,
                           const uint16_t* bias, void* out, bool out_f32, hipStream_t st) {
  const int NO = bwd ? K : N;
  dim3 grid((NO + GB - 1) / GB, (M + GB - 1) / GB);
  if (!bwd) {
    if (out_f32) k_gemm_fp4<false, true><<<grid, 256, 0, st>>>(a, as, wq, ws, M, N, K, P, R, lr, bias, out);
    else k_gemm_fp4<false, false><<<grid, 256, 0, st>>>(a, as, wq, ws, M, N, K, P, R, lr, bias, out);
  } else {
    if (out_f32) k_gemm_fp4<true, true><<<grid, 256, 0, st>>>(a, as, wq, ws, M, N, K, P, R, lr, nullptr, out);
    else k_gemm_fp4<true, false><<<grid, 256, 0, st>>>(a, as, wq, ws, M, N, K, P, R, lr, nullptr, out);
  }
  return hipGetLastError();
}

}  // namespace ft
