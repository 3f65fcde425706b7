// Sum of fp32 partial results left in a workspace by kernels whose
// workgroups each cover part of a reduction (column chunks of the fused
// down-projection, token chunks of the adapter gradients):
//   out0[i] (+)= sum_p ws[p * (n0 + n1) + i]            i < n0
//   out1[i] (+)= sum_p ws[p * (n0 + n1) + n0 + i]       i < n1
// Plain stores and a fixed summation order: results do not depend on the
// order in which workgroups ran.
#include "ft_device.h"
#include "ft_kernels.h"

namespace ft {

__global__ __launch_bounds__(256) void k_reduce_parts(const float* __restrict__ ws, int nparts, size_t n0,
                                                      float* __restrict__ out0, size_t n1, float* __restrict__ out1,
                                                      int accumulate) {
  const size_t n = n0 + n1;  // floats per part, multiple of 4 (so are n0, n1)
  const size_t i = ((size_t)blockIdx.x * 256 + threadIdx.x) * 4;
  if (i >= n) return;
  float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
  int p = 0;
  for (; p + 4 <= nparts; p += 4) {
    const float4 a = *(const float4*)(ws + (size_t)p * n + i);
    const float4 b = *(const float4*)(ws + (size_t)(p + 1) * n + i);
    const float4 c = *(const float4*)(ws + (size_t)(p + 2) * n + i);
    const float4 d = *(const float4*)(ws + (size_t)(p + 3) * n + i);
    s.x += a.x; s.y += a.y; s.z += a.z; s.w += a.w;
    s.x += b.x; s.y += b.y; s.z += b.z; s.w += b.w;
    s.x += c.x; s.y += c.y; s.z += c.z; s.w += c.w;
    s.x += d.x; s.y += d.y; s.z += d.z; s.w += d.w;
  }
  for (; p < nparts; p++) {
    const float4 a = *(const float4*)(ws + (size_t)p * n + i);
    s.x += a.x; s.y += a.y; s.z += a.z; s.w += a.w;
  }
  float* o = i < n0 ? out0 + i : out1 + (i - n0);
  if (accumulate) {
    const float4 prev = *(const float4*)o;
    s.x += prev.x; s.y += prev.y; s.z += prev.z; s.w += prev.w;
  }
  *(float4*)o = s;
}

hipError_t launch_reduce_parts(const float* ws, int nparts, size_t n0, float* out0, size_t n1, float* out1,
                               bool accumulate, hipStream_t st) {
  const size_t n4 = (n0 + n1) / 4;
  if (n4 == 0) return hipSuccess;
  k_reduce_parts<<<(unsigned)((n4 + 255) / 256), 256, 0, st>>>(ws, nparts, n0, out0, n1, out1, accumulate ? 1 : 0);
  return hipGetLastError();
}

}  // namespace ft
