// NVFP4 emulation (gfx950): the format FourTune Sec. 3.1 names, as an
// accuracy cross-check of the layer's native MXFP4.  NVFP4 holds E2M1
// elements with one FP8 E4M3 scale per 16 elements (16x16 tiles for the
// weight, Sec. 4.3, so the transposed weight reuses its scales, Sec. 3.2) and
// one FP32 scale per tensor.  gfx950's block-scaled MFMA takes E8M0 scales
// per 32 elements, so NVFP4 has no native rate here: the GEMM dequantizes
// E2M1 x E4M3 (at most 6 significant bits, exact in bf16) into LDS and runs
// bf16 MFMAs with fp32 accumulation; the two tensor scales multiply the
// result.
//
// Quantization, per tensor:
//   st = amax / (6 * 448)                      one correctly rounded fp32 division
//   block scale = E4M3 nearest to amax_b / (6 st)   fp32: 6 st, then the division;
//                                                     ties to the even mantissa, saturating at 448
//   element = E2M1 nearest to |v| / (E4M3 * st)     decided in fp64 (the quotient of a bf16
//                                                     value by a 28-bit product is never within
//                                                     an fp64 rounding of a decision point
//                                                     without lying on it), ties to the even
//                                                     code, saturating at 6, sign copied
// The tensor's amax goes through the caller's 4-byte tensor-scale buffer:
// zeroed, raised with atomic max of the bf16 magnitude bits, read by the
// quantize kernel, and finally overwritten with st.
#include "ft_device.h"
#include "ft_kernels.h"

namespace ft {

__global__ void k_nvfp4_zero(uint32_t* cell) { if (threadIdx.x == 0 && blockIdx.x == 0) cell[0] = 0u; }

// Largest bf16 magnitude bit pattern of src[n] (bf16 magnitudes order like
// their bit patterns).  16-byte loads, then the tail.
__global__ __launch_bounds__(256) void k_nvfp4_amax(const uint16_t* __restrict__ src, size_t n, uint32_t* cell) {
  __shared__ uint32_t wmax[4];
  uint32_t m = 0;
  const size_t n8 = n / 8;
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n8; i += stride) {
    const uint4 v = ((const uint4*)src)[i];
    const uint32_t w[4] = {v.x & 0x7FFF7FFFu, v.y & 0x7FFF7FFFu, v.z & 0x7FFF7FFFu, v.w & 0x7FFF7FFFu};
#pragma unroll
    for (int e = 0; e < 4; e++) m = max(m, max(w[e] & 0xFFFFu, w[e] >> 16));
  }
  for (size_t i = n8 * 8 + (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
    m = max(m, (uint32_t)(src[i] & 0x7FFFu));
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off, 64));
  if ((threadIdx.x & 63) == 0) wmax[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint32_t b = max(max(wmax[0], wmax[1]), max(wmax[2], wmax[3]));
    atomicMax(cell, b);
  }
}

// st from the amax cell: bf16 magnitude bits -> fp32, divided by 6 * 448.
__device__ __forceinline__ float nvfp4_st(const uint32_t* cell) {
  return __fdiv_rn(__uint_as_float(cell[0] << 16), 2688.0f);
}

__global__ void k_nvfp4_finish(uint32_t* cell) {
  if (threadIdx.x == 0 && blockIdx.x == 0) {
    const float st = nvfp4_st(cell);
    cell[0] = __float_as_uint(st);
  }
}

// E4M3 code nearest to d >= 0, ties to the even mantissa, saturating at 448.
__device__ __forceinline__ uint32_t e4m3_nearest(float d) {
  if (!(d < 448.0f)) return 0x7Eu;
  if (d < 0.015625f) return (uint32_t)__builtin_rintf(d * 512.0f);   // subnormals m / 8 * 2^-6 (8 -> 2^-6)
  const uint32_t b = __float_as_uint(d);
  const uint32_t mant = b & 0x7FFFFFu, rem = mant & 0xFFFFFu;
  uint32_t m3 = mant >> 20;
  if (rem > 0x80000u || (rem == 0x80000u && (m3 & 1u))) m3++;
  const uint32_t code = ((((b >> 23) & 0xFFu) - 120u) << 3) + m3;   // exponent field e - 127 + 7
  return code > 0x7Eu ? 0x7Eu : code;
}

__device__ __forceinline__ float e4m3_value(uint32_t code) {
  const uint32_t e = (code >> 3) & 15u, m = code & 7u;
  return e == 0 ? (float)m * 0x1p-9f : __uint_as_float(((e + 120u) << 23) | (m << 20));
}

// E2M1 magnitude code nearest to t >= 0 (ties to the even code, saturating).
__device__ __forceinline__ uint32_t e2m1_nearest(double t) {
  return (uint32_t)(t > 0.25) + (uint32_t)(t >= 0.75) + (uint32_t)(t > 1.25) + (uint32_t)(t >= 1.75) +
         (uint32_t)(t > 2.5) + (uint32_t)(t >= 3.5) + (uint32_t)(t > 5.0);
}

// Codes of n bf16 values (n even) sharing the block scale code sc.
template <int NV>
__device__ __forceinline__ void nvfp4_codes(const uint32_t (&w)[NV / 2], uint32_t sc, float st, uint32_t (&out)[NV / 8]) {
  const double bs = (double)e4m3_value(sc) * (double)st;
#pragma unroll
  for (int i = 0; i < NV / 8; i++) out[i] = 0;
#pragma unroll
  for (int i = 0; i < NV; i++) {
    const uint32_t b = (w[i >> 1] >> (16 * (i & 1))) & 0xFFFFu;
    const double v = (double)__uint_as_float((b & 0x7FFFu) << 16);
    const uint32_t c = bs > 0.0 ? e2m1_nearest(__ddiv_rn(v, bs)) : 0u;
    out[i >> 3] |= (c | ((b >> 12) & 8u)) << (4 * (i & 7));
  }
}

// 1x16 blocks: a lane takes 8 elements, a lane pair one block.
__global__ __launch_bounds__(256) void k_nvfp4_quant_rows(const uint16_t* __restrict__ src, int rows, int cols,
                                                          uint8_t* __restrict__ codes, uint8_t* __restrict__ scales,
                                                          const uint32_t* __restrict__ cell) {
  const size_t per_row = (size_t)cols / 8;
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;   // the grid covers rows * cols / 8 (even)
  const bool live = i < (size_t)rows * per_row;
  const size_t r = live ? i / per_row : 0, c8 = live ? i % per_row : 0;
  uint32_t w[4] = {0, 0, 0, 0};
  if (live) {
    const uint4 v = *(const uint4*)(src + r * cols + 8 * c8);
    w[0] = v.x; w[1] = v.y; w[2] = v.z; w[3] = v.w;
  }
  uint32_t m = 0;
#pragma unroll
  for (int e = 0; e < 4; e++) {
    const uint32_t a = w[e] & 0x7FFF7FFFu;
    m = max(m, max(a & 0xFFFFu, a >> 16));
  }
  m = max(m, (uint32_t)__builtin_amdgcn_mov_dpp((int)m, 0xB1, 0xF, 0xF, true));   // the pair's other lane
  const float st = nvfp4_st(cell);
  const float st6 = 6.0f * st;
  const float amax = __uint_as_float(m << 16);
  const uint32_t sc = st6 > 0.0f ? e4m3_nearest(__fdiv_rn(amax, st6)) : 0u;
  uint32_t o[1];
  nvfp4_codes<8>(w, sc, st, o);
  if (live) {
    *(uint32_t*)(codes + r * (cols / 2) + 4 * c8) = o[0];
    if ((c8 & 1) == 0) scales[r * (cols / 16) + c8 / 2] = (uint8_t)sc;
  }
}

// 16x16 tiles: one wave per tile, lane l takes row l / 4, columns 4 (l % 4) .. + 4.
__global__ __launch_bounds__(256) void k_nvfp4_quant_tiles(const uint16_t* __restrict__ src, int rows, int cols,
                                                           uint8_t* __restrict__ codes, uint8_t* __restrict__ scales,
                                                           const uint32_t* __restrict__ cell) {
  const int lane = threadIdx.x & 63;
  const int tile = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int nbc = cols >> 4;
  if (tile >= (rows >> 4) * nbc) return;   // whole wave
  const int tr = tile / nbc, tc = tile % nbc;
  const int row = tr * 16 + (lane >> 2), col = tc * 16 + 4 * (lane & 3);
  const uint2 v = *(const uint2*)(src + (size_t)row * cols + col);
  const uint32_t w[2] = {v.x, v.y};
  uint32_t m = max(max(w[0] & 0x7FFFu, (w[0] >> 16) & 0x7FFFu), max(w[1] & 0x7FFFu, (w[1] >> 16) & 0x7FFFu));
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off, 64));
  const float st = nvfp4_st(cell);
  const float st6 = 6.0f * st;
  const uint32_t sc = st6 > 0.0f ? e4m3_nearest(__fdiv_rn(__uint_as_float(m << 16), st6)) : 0u;
  const double bs = (double)e4m3_value(sc) * (double)st;
  uint32_t o = 0;
#pragma unroll
  for (int i = 0; i < 4; i++) {
    const uint32_t b = (w[i >> 1] >> (16 * (i & 1))) & 0xFFFFu;
    const double x = (double)__uint_as_float((b & 0x7FFFu) << 16);
    const uint32_t c = bs > 0.0 ? e2m1_nearest(__ddiv_rn(x, bs)) : 0u;
    o |= (c | ((b >> 12) & 8u)) << (4 * i);
  }
  *(uint16_t*)(codes + (size_t)row * (cols >> 1) + (col >> 1)) = (uint16_t)o;
  if (lane == 0) scales[(size_t)tr * nbc + tc] = (uint8_t)sc;
}

hipError_t launch_quant_nvfp4(const uint16_t* src, int rows, int cols, int block_rows, uint8_t* codes,
                              uint8_t* scales, float* tensor_scale, hipStream_t st) {
  uint32_t* cell = (uint32_t*)tensor_scale;
  const size_t n = (size_t)rows * cols;
  k_nvfp4_zero<<<1, 64, 0, st>>>(cell);
  const unsigned g = (unsigned)std::min<size_t>(1024, (n / 8 + 255) / 256 + 1);
  k_nvfp4_amax<<<g, 256, 0, st>>>(src, n, cell);
  if (block_rows == 1) {
    const size_t lanes = n / 8;
    k_nvfp4_quant_rows<<<(unsigned)((lanes + 255) / 256), 256, 0, st>>>(src, rows, cols, codes, scales, cell);
  } else {
    const int tiles = (rows / 16) * (cols / 16);
    k_nvfp4_quant_tiles<<<(unsigned)((tiles + 3) / 4), 256, 0, st>>>(src, rows, cols, codes, scales, cell);
  }
  k_nvfp4_finish<<<1, 64, 0, st>>>(cell);
  return hipGetLastError();
}

// ------------------------------------------------------------------ GEMM
// out[M, NO] fp32 = ta * tw * sum over the reduction of E2M1 x E4M3 products:
//   forward  (BWD = false): out = A[M, K] W[N, K]^T  (A 1x16 blocks along K, W 16x16 tiles)
//   backward (BWD = true):  out = A[M, N] W[N, K]    (A 1x16 blocks along N, W read transposed)
// Workgroup 256 threads (2x2 waves) per 128x128 output tile, each wave 64x64
// as 2x2 bf16 32x32x16 MFMA tiles; 32 reduction elements per step, the
// dequantized operands staged in LDS as [row][reduction] bf16.
constexpr int NV_T = 128, NV_K = 32, NV_S = NV_K + 8;

__device__ __forceinline__ void nvfp4_dequant16(uint2 c, uint32_t sc, uint16_t (&h)[16]) {
  const float s = e4m3_value(sc);
  const float mag[8] = {0.0f, 0.5f, 1.0f, 1.5f, 2.0f, 3.0f, 4.0f, 6.0f};
#pragma unroll
  for (int i = 0; i < 16; i++) {
    const uint32_t nib = ((i < 8 ? c.x : c.y) >> (4 * (i & 7))) & 15u;
    const float v = mag[nib & 7] * s;                        // exact: at most 6 significant bits
    h[i] = (uint16_t)((__float_as_uint(v) >> 16) | ((nib & 8u) << 12));
  }
}

template <bool BWD>
__global__ __launch_bounds__(256) void k_gemm_nvfp4(const uint8_t* __restrict__ A, const uint8_t* __restrict__ As,
                                                    const float* __restrict__ At, const uint8_t* __restrict__ Wq,
                                                    const uint8_t* __restrict__ Ws, const float* __restrict__ Wt,
                                                    int M, int N, int K, float* __restrict__ out) {
  __shared__ __attribute__((aligned(16))) uint16_t la[NV_T * NV_S];
  __shared__ __attribute__((aligned(16))) uint16_t lb[NV_T * NV_S];
  const int NO = BWD ? K : N, KR = BWD ? N : K;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1, r32 = lane & 31, h = lane >> 5;
  const int m0 = blockIdx.y * NV_T, n0 = blockIdx.x * NV_T;
  v16f acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; i++)
#pragma unroll
    for (int j = 0; j < 2; j++) acc[i][j] = v16f{};

  for (int k0 = 0; k0 < KR; k0 += NV_K) {
    {   // A: thread t -> row t/2, reduction elements k0 + 16 (t % 2) .. + 16
      const int r = m0 + (tid >> 1), kk = k0 + 16 * (tid & 1);
      uint16_t v[16] = {};
      if (r < M && kk < KR)
        nvfp4_dequant16(*(const uint2*)(A + (size_t)r * (KR / 2) + kk / 2), As[(size_t)r * (KR / 16) + kk / 16], v);
      uint4* d = (uint4*)(la + (tid >> 1) * NV_S + 16 * (tid & 1));
      d[0] = make_uint4(v[0] | (v[1] << 16), v[2] | (v[3] << 16), v[4] | (v[5] << 16), v[6] | (v[7] << 16));
      d[1] = make_uint4(v[8] | (v[9] << 16), v[10] | (v[11] << 16), v[12] | (v[13] << 16), v[14] | (v[15] << 16));
    }
    if constexpr (!BWD) {   // W rows n, reduction k: as A, scales per 16x16 tile
      const int n = n0 + (tid >> 1), kk = k0 + 16 * (tid & 1);
      uint16_t v[16] = {};
      if (n < N && kk < K)
        nvfp4_dequant16(*(const uint2*)(Wq + (size_t)n * (K / 2) + kk / 2), Ws[(size_t)(n / 16) * (K / 16) + kk / 16], v);
      uint4* d = (uint4*)(lb + (tid >> 1) * NV_S + 16 * (tid & 1));
      d[0] = make_uint4(v[0] | (v[1] << 16), v[2] | (v[3] << 16), v[4] | (v[5] << 16), v[6] | (v[7] << 16));
      d[1] = make_uint4(v[8] | (v[9] << 16), v[10] | (v[11] << 16), v[12] | (v[13] << 16), v[14] | (v[15] << 16));
    } else {   // W rows n (the reduction), output columns k: 16 columns of one row, written transposed
      const int n = k0 + (tid >> 3), kc = n0 + 16 * (tid & 7);
      uint16_t v[16] = {};
      if (n < N && kc < K)
        nvfp4_dequant16(*(const uint2*)(Wq + (size_t)n * (K / 2) + kc / 2), Ws[(size_t)(n / 16) * (K / 16) + kc / 16], v);
#pragma unroll
      for (int i = 0; i < 16; i++) lb[(16 * (tid & 7) + i) * NV_S + (tid >> 3)] = v[i];
    }
    __syncthreads();
#pragma unroll
    for (int ks = 0; ks < 2; ks++) {
      v8bf a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; i++) a[i] = *(const v8bf*)(la + (wm * 64 + 32 * i + r32) * NV_S + 16 * ks + 8 * h);
#pragma unroll
      for (int j = 0; j < 2; j++) b[j] = *(const v8bf*)(lb + (wn * 64 + 32 * j + r32) * NV_S + 16 * ks + 8 * h);
#pragma unroll
      for (int i = 0; i < 2; i++)
#pragma unroll
        for (int j = 0; j < 2; j++) acc[i][j] = mfma_bf16_32x32x16(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
  const float scale = At[0] * Wt[0];
#pragma unroll
  for (int i = 0; i < 2; i++)
#pragma unroll
    for (int j = 0; j < 2; j++)
#pragma unroll
      for (int v = 0; v < 16; v++) {
        const int row = m0 + wm * 64 + 32 * i + 8 * (v >> 2) + 4 * h + (v & 3);
        const int col = n0 + wn * 64 + 32 * j + r32;
        if (row < M && col < NO) out[(size_t)row * NO + col] = acc[i][j][v] * scale;
      }
}

hipError_t launch_gemm_nvfp4(bool bwd, const uint8_t* a, const uint8_t* as, const float* at, const uint8_t* wq,
                             const uint8_t* ws, const float* wt, int M, int N, int K, float* out, hipStream_t st) {
  const int NO = bwd ? K : N;
  dim3 grid((NO + NV_T - 1) / NV_T, (M + NV_T - 1) / NV_T);
  if (bwd) k_gemm_nvfp4<true><<<grid, 256, 0, st>>>(a, as, at, wq, ws, wt, M, N, K, out);
  else k_gemm_nvfp4<false><<<grid, 256, 0, st>>>(a, as, at, wq, ws, wt, M, N, K, out);
  return hipGetLastError();
}

}  // namespace ft
