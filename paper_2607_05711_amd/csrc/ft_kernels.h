// Internal launch interface between the C ABI (api.hip) and the kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <algorithm>

namespace ft {


hipError_t launch_quant_rows(const uint16_t* src, int rows, int cols, uint8_t* codes, uint8_t* scales,
                             const uint16_t* proj, int R, int layout, float* proj_out, hipStream_t st);
hipError_t launch_quant_tiles(const uint16_t* src, int rows, int cols, uint8_t* codes, uint8_t* scales,
                              hipStream_t st);
hipError_t launch_fill_f32(float* p, size_t n, float v, hipStream_t st);

// FP4 GEMM.  bwd = false: out[M, N] = A[M, K] . W[N, K]^T  (+ P . U + bias)
//            bwd = true : out[M, K] = A[M, N] . W[N, K]    (+ P . D^T)
hipError_t launch_gemm_fp4(bool bwd, const uint8_t* a, const uint8_t* as, const uint8_t* wq, const uint8_t* ws,
                           int M, int N, int K, const float* P, int R, const uint16_t* lr,
                           const uint16_t* bias, void* out, bool out_f32, hipStream_t st);

hipError_t launch_lora_grads(const uint16_t* x, int M, int K, const uint16_t* dy, int N, const float* xa,
                             const float* dyb, int ld, int r, float* dA, float* dB, bool accumulate,
                             hipStream_t st);

}  // namespace ft
