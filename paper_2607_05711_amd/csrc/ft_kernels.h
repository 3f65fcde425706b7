// Internal launch interface between the C ABI (api.hip) and the kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <algorithm>

namespace ft {

// 1x32 row quantization with the fused down-projection.  When the columns
// span several chunks, each chunk's fp32 projection partial goes to `ws`
// (quant_rows_workspace bytes) and a reduction kernel sums them into
// proj_out; otherwise proj_out is written directly and ws is unused.
// Numerics variants of the quantizers: the no-clip scale rule, stochastic
// rounding (Philox4x32-10 bits keyed by seed, counter words 2 and 3 = stream),
// and for 32x32 tiles scales written once per row.
struct QuantMode {
  bool no_clip = false;
  bool stochastic = false;
  uint64_t seed = 0, stream = 0;
  int scales_per_row = 0;
};
size_t quant_rows_workspace(int rows, int cols, int R, int layout);
hipError_t launch_quant_rows(const uint16_t* src, int rows, int cols, uint8_t* codes, uint8_t* scales,
                             const uint16_t* proj, int R, int layout, float* proj_out, float* ws, hipStream_t st,
                             const QuantMode& mode = QuantMode{});
hipError_t launch_quant_tiles(const uint16_t* src, int rows, int cols, uint8_t* codes, uint8_t* scales,
                              hipStream_t st, const QuantMode& mode = QuantMode{});

// out0 (+)= sum of nparts partials [n0 | n1] in ws; likewise out1.  n0, n1 multiples of 4.
hipError_t launch_reduce_parts(const float* ws, int nparts, size_t n0, float* out0, size_t n1, float* out1,
                               bool accumulate, hipStream_t st);

// FP4 GEMM.  bwd = false: out[M, N] = A[M, K] . W[N, K]^T  (+ P . U + bias)
//            bwd = true : out[M, K] = A[M, N] . W[N, K]    (+ P . D^T)
hipError_t launch_gemm_fp4(bool bwd, const uint8_t* a, const uint8_t* as, const uint8_t* wq, const uint8_t* ws,
                           int M, int N, int K, const float* P, int R, const uint16_t* lr,
                           const uint16_t* bias, void* out, bool out_f32, hipStream_t st);

// Epilogues of the MLP pair (the output NO columns feed the next linear).
enum { EPI_PLAIN = 0, EPI_GELU = 1, EPI_DGELU = 2 };
struct GemmEpilogue {
  uint16_t* z_out;        // EPI_GELU: z = bf16(acc) [M, NO]
  const uint16_t* z_in;   // EPI_DGELU: z saved by the forward [M, NO]
  uint16_t* y;            // EPI_GELU: h = bf16(GELU(z));  EPI_DGELU: dz = bf16(acc GELU'(z))  [M, NO]
  uint8_t* q;             // E2M1 codes of y [M, NO/2]
  uint8_t* s;             // E8M0 scales of y [M, NO/32]
  const uint16_t* proj;   // EPI_GELU: D2 [NO, R2];  EPI_DGELU: U1 [R2, NO];  unused when R2 == 0
  int R2;                 // 0, 16, 32, 48 or 64
  float* parts;           // fp32 partials [tiles over NO][M][R2], or the projection when one tile spans NO
};
// Whether the fused epilogues support this shape (the pipelined kernel runs it).
bool gemm_fp4_fused_supported(bool bwd, int M, int N, int K, int R, int R2);
// Number of output column tiles (partials of the fused projection).
int gemm_fp4_col_tiles(int NO);
hipError_t launch_gemm_fp4_fused(bool bwd, const uint8_t* a, const uint8_t* as, const uint8_t* wq, const uint8_t* ws,
                                 int M, int N, int K, const float* P, int R, const uint16_t* lr, const uint16_t* bias,
                                 const GemmEpilogue& ep, float* proj_out, hipStream_t st);

// Adapter gradients; token chunks leave partials in ws (lora_grads_workspace bytes).
size_t lora_grads_workspace(int M, int K, int N, int ld, int r);
hipError_t launch_lora_grads(const uint16_t* x, int M, int K, const uint16_t* dy, int N, const float* xa,
                             const float* dyb, int ld, int r, float* dA, float* dB, bool accumulate, float* ws,
                             hipStream_t st);

// Size of the static device scratch the allocation-free adapter-gradient entry
// point uses in place of a workspace, and its device address on the current
// device (looked up on the first call per device).  Every call on one device
// shares it.
constexpr size_t kLoraScratchBytes = (size_t)32 << 20;
hipError_t lora_grads_scratch(float** ptr);

// NVFP4 emulation: quantization (1x16 or 16x16 blocks, E4M3 scales, the fp32
// tensor scale left in *tensor_scale) and the dequantizing bf16-MFMA GEMM
// (fp32 output, both tensor scales applied).
hipError_t launch_quant_nvfp4(const uint16_t* src, int rows, int cols, int block_rows, uint8_t* codes,
                              uint8_t* scales, float* tensor_scale, hipStream_t st);
hipError_t launch_gemm_nvfp4(bool bwd, const uint8_t* a, const uint8_t* as, const float* at, const uint8_t* wq,
                             const uint8_t* ws, const float* wt, int M, int N, int K, float* out, hipStream_t st);

}  // namespace ft
