// Adapter weight gradients (FourTune Sec. 3.2):
//   dB = (X A)^T G      dB[j,n] = sum_m xa[m,j]  G[m,n]
//   dA = X^T (G B^T)    dA[k,j] = sum_m X[m,k]   gbt[m,j]
// Both are out[j, c] = sum_m L[m, j] V[m, c] with a skinny fp32 L (r columns)
// and a wide bf16 V, reduced over the token axis M.  The reduction axis is the
// row axis of both operands in memory, so tiles are staged in LDS as stored
// and the MFMA operands are gathered with transposing 16-bit LDS reads.  L is
// split into two bf16 terms (hi + lo) so its ~16 leading bits take part.
// Workgroups split M into chunks; their partial sums meet in fp32 atomics.
#include "ft_device.h"
#include "ft_kernels.h"

namespace ft {

constexpr int LG_BC = 256;    // output columns per workgroup (4 waves x 2 tiles of 32)
constexpr int LG_BM = 64;     // token rows per LDS stage
constexpr int LG_VSTRIDE = LG_BC + 16;  // halfwords

template <int RTJ>
struct LoraLds {
  static constexpr int LSTRIDE = RTJ * 32 + 16;  // halfwords
  static constexpr int V_HW = LG_BM * LG_VSTRIDE;
  static constexpr int L_HW = LG_BM * LSTRIDE;
};

struct LoraJob {
  const float* L;       // [M, ld], r columns used
  const uint16_t* V;    // [M, C]
  float* out;
  int C;
  int out_rows_are_j;   // 1: out[j * C + c] (dB);  0: out[c * r + j] (dA)
  int ncg;              // column groups
};

template <int RTJ>
__global__ __launch_bounds__(256) void k_lora_grads(LoraJob jb0, LoraJob jb1, int M, int ld, int r, int mchunk,
                                                    int nmch) {
  using Lds = LoraLds<RTJ>;
  __shared__ __attribute__((aligned(16))) uint16_t lv[Lds::V_HW];
  __shared__ __attribute__((aligned(16))) uint16_t lhi[Lds::L_HW];
  __shared__ __attribute__((aligned(16))) uint16_t llo[Lds::L_HW];

  int b = blockIdx.x;
  const int n0blocks = jb0.ncg * nmch;
  const LoraJob job = b < n0blocks ? jb0 : jb1;
  if (b >= n0blocks) b -= n0blocks;
  const int cg = b % job.ncg, mc = b / job.ncg;
  const int c0 = cg * LG_BC;
  const int mbeg = mc * mchunk, mend = min(M, mbeg + mchunk);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r32 = lane & 31, h = lane >> 5, g16 = lane >> 4, t16 = lane & 15;
  const int jj = t16 >> 2, qq = t16 & 3;

  v16f acc[RTJ][2];
#pragma unroll
  for (int t = 0; t < RTJ; t++) { acc[t][0] = v16f{}; acc[t][1] = v16f{}; }

#pragma unroll 1
  for (int m0 = mbeg; m0 < mend; m0 += LG_BM) {
    // stage V[m0 .. m0+64) x [c0 .. c0+256)
#pragma unroll
    for (int i = 0; i < 8; i++) {
      const int s = tid + 256 * i, row = s >> 5, col = (s & 31) * 8;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (m0 + row < mend && c0 + col < job.C)
        v = load_nt16(job.V + (size_t)(m0 + row) * job.C + c0 + col);
      *(uint4*)(lv + row * LG_VSTRIDE + col) = v;
    }
    // stage L[m0 .. m0+64) x [0 .. RTJ*32) as hi/lo bf16
    constexpr int LEL = LG_BM * RTJ * 32;
#pragma unroll
    for (int i = 0; i < LEL / 256; i++) {
      const int s = tid + 256 * i, row = s / (RTJ * 32), j = s % (RTJ * 32);
      float x = 0.0f;
      if (m0 + row < mend && j < r) x = job.L[(size_t)(m0 + row) * ld + j];
      uint32_t hi, lo;
      split_bf16(x, hi, lo);
      lhi[row * Lds::LSTRIDE + j] = (uint16_t)hi;
      llo[row * Lds::LSTRIDE + j] = (uint16_t)lo;
    }
    __syncthreads();
#pragma unroll
    for (int ms = 0; ms < LG_BM / 16; ms++) {
      const int mrow = ms * 16 + 8 * h + jj;   // this lane's source row for the first tr read
      v8bf bv[2];
#pragma unroll
      for (int ct = 0; ct < 2; ct++) {
        const int col = wave * 64 + ct * 32 + 16 * (g16 & 1) + 4 * qq;
        const FT_LDS uint16_t* p = (FT_LDS uint16_t*)lv + mrow * LG_VSTRIDE + col;
        bv[ct] = make_v8bf(lds_read_tr16(p), lds_read_tr16(p + 4 * LG_VSTRIDE));
      }
#pragma unroll
      for (int t = 0; t < RTJ; t++) {
        const int col = t * 32 + 16 * (g16 & 1) + 4 * qq;
        const FT_LDS uint16_t* ph = (FT_LDS uint16_t*)lhi + mrow * Lds::LSTRIDE + col;
        const FT_LDS uint16_t* pl = (FT_LDS uint16_t*)llo + mrow * Lds::LSTRIDE + col;
        const v8bf ah = make_v8bf(lds_read_tr16(ph), lds_read_tr16(ph + 4 * Lds::LSTRIDE));
        const v8bf al = make_v8bf(lds_read_tr16(pl), lds_read_tr16(pl + 4 * Lds::LSTRIDE));
#pragma unroll
        for (int ct = 0; ct < 2; ct++) {
          acc[t][ct] = mfma_bf16_32x32x16(ah, bv[ct], acc[t][ct]);
          acc[t][ct] = mfma_bf16_32x32x16(al, bv[ct], acc[t][ct]);
        }
      }
    }
    __syncthreads();
  }

  // acc[t][ct]: row j = t*32 + 8(v/4) + 4h + v%4, column c = c0 + wave*64 + ct*32 + r32
#pragma unroll
  for (int ct = 0; ct < 2; ct++) {
    const int c = c0 + wave * 64 + ct * 32 + r32;
    if (c >= job.C) continue;
#pragma unroll
    for (int t = 0; t < RTJ; t++)
#pragma unroll
      for (int v = 0; v < 16; v++) {
        const int j = t * 32 + 8 * (v >> 2) + 4 * h + (v & 3);
        if (j < r) {
          float* dst = job.out_rows_are_j ? job.out + (size_t)j * job.C + c : job.out + (size_t)c * r + j;
          atomicAdd(dst, acc[t][ct][v]);
        }
      }
  }
}

hipError_t launch_lora_grads(const uint16_t* x, int M, int K, const uint16_t* dy, int N, const float* xa,
                             const float* dyb, int ld, int r, float* dA, float* dB, bool accumulate,
                             hipStream_t st) {
  if (!accumulate) {
    hipError_t e = launch_fill_f32(dA, (size_t)K * r, 0.0f, st);
    if (e != hipSuccess) return e;
    e = launch_fill_f32(dB, (size_t)r * N, 0.0f, st);
    if (e != hipSuccess) return e;
  }
  if (M == 0) return hipSuccess;
  LoraJob jobB{xa, dy, dB, N, 1, (N + LG_BC - 1) / LG_BC};
  LoraJob jobA{dyb, x, dA, K, 0, (K + LG_BC - 1) / LG_BC};
  const int ncg = jobB.ncg + jobA.ncg;
  const int mblocks = (M + LG_BM - 1) / LG_BM;
  int nmch = std::max(1, std::min(mblocks, (1024 + ncg - 1) / ncg));
  const int mchunk = ((mblocks + nmch - 1) / nmch) * LG_BM;
  nmch = (M + mchunk - 1) / mchunk;
  const unsigned grid = (unsigned)(ncg * nmch);
  switch ((r + 31) / 32) {
    case 1: k_lora_grads<1><<<grid, 256, 0, st>>>(jobB, jobA, M, ld, r, mchunk, nmch); break;
    case 2: k_lora_grads<2><<<grid, 256, 0, st>>>(jobB, jobA, M, ld, r, mchunk, nmch); break;
    case 3: k_lora_grads<3><<<grid, 256, 0, st>>>(jobB, jobA, M, ld, r, mchunk, nmch); break;
    default: k_lora_grads<4><<<grid, 256, 0, st>>>(jobB, jobA, M, ld, r, mchunk, nmch); break;
  }
  return hipGetLastError();
}

}  // namespace ft
