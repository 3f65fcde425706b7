// C ABI of libfourtune: argument validation, then kernel launches.
// Nothing here allocates, frees or synchronizes.
#include <cstdarg>
#include <cstdio>

#include "../../include/fourtune.h"
#include "ft_kernels.h"

namespace {

thread_local char g_last_error[512] = "";

ft_status fail(ft_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
  va_end(ap);
  return st;
}

ft_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return FT_OK;
  return fail(FT_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

constexpr int64_t kMaxDim = (int64_t)1 << 30;

ft_status check_dim(const char* name, int64_t v, int64_t mult) {
  if (v < 0 || v > kMaxDim) return fail(FT_ERR_SHAPE, "%s = %lld out of range [0, 2^30]", name, (long long)v);
  if (mult > 1 && v % mult != 0)
    return fail(FT_ERR_SHAPE, "%s = %lld is not a multiple of %lld", name, (long long)v, (long long)mult);
  return FT_OK;
}

ft_status check_rank(int32_t R, const void* a, const void* b, const char* an, const char* bn) {
  if (R == 0) {
    if (a || b) return fail(FT_ERR_UNSUPPORTED, "R == 0 but %s/%s given", an, bn);
    return FT_OK;
  }
  if (!a || !b) return fail(FT_ERR_NULL, "R = %d but %s or %s is NULL", R, an, bn);
  if (R < 0 || R > 128 || R % 16 != 0) return fail(FT_ERR_UNSUPPORTED, "R = %d: need 16 <= R <= 128, R %% 16 == 0", R);
  if (!aligned16(a) || !aligned16(b)) return fail(FT_ERR_ALIGN, "%s or %s not 16-byte aligned", an, bn);
  return FT_OK;
}

ft_status check_workspace(const void* ws, size_t bytes, size_t need) {
  if (need == 0) return FT_OK;
  if (!ws) return fail(FT_ERR_NULL, "a workspace of %zu bytes is required", need);
  if (bytes < need) return fail(FT_ERR_SHAPE, "workspace of %zu bytes, %zu required", bytes, need);
  if (!aligned16(ws)) return fail(FT_ERR_ALIGN, "workspace not 16-byte aligned");
  return FT_OK;
}

#define FT_TRY(x)                   \
  do {                              \
    ft_status s_ = (x);             \
    if (s_ != FT_OK) return s_;     \
  } while (0)

}  // namespace

extern "C" {

const char* ft_status_string(ft_status s) {
  switch (s) {
    case FT_OK: return "ok";
    case FT_ERR_NULL: return "null pointer";
    case FT_ERR_SHAPE: return "invalid shape";
    case FT_ERR_ALIGN: return "misaligned pointer";
    case FT_ERR_UNSUPPORTED: return "unsupported argument";
    case FT_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

const char* ft_last_error(void) { return g_last_error; }

size_t ft_quantize_workspace_size(int64_t rows, int64_t cols, int32_t block_rows, int32_t R,
                                  ft_proj_layout proj_layout) {
  if (block_rows != 1 || R <= 0 || R > 128 || rows <= 0 || cols <= 0 || rows > kMaxDim || cols > kMaxDim) return 0;
  return ft::quant_rows_workspace((int)rows, (int)cols, R, (int)proj_layout);
}

static ft_status quantize_impl(const void* src, int64_t rows, int64_t cols, int32_t block_rows, uint8_t* codes,
                               uint8_t* scales, const void* proj, int32_t R, ft_proj_layout proj_layout,
                               float* proj_out, void* workspace, size_t workspace_bytes, const ft::QuantMode& qm,
                               hipStream_t stream) {
  FT_TRY(check_dim("rows", rows, block_rows == 32 ? 32 : 1));
  FT_TRY(check_dim("cols", cols, 32));
  if (block_rows != 1 && block_rows != 32) return fail(FT_ERR_UNSUPPORTED, "block_rows = %d (1 or 32)", block_rows);
  if (rows == 0 || cols == 0) return FT_OK;
  if (!src || !codes || !scales) return fail(FT_ERR_NULL, "src, codes and scales are required");
  if (!aligned16(src) || !aligned16(codes) || !aligned16(scales))
    return fail(FT_ERR_ALIGN, "src, codes and scales must be 16-byte aligned");
  if (proj_layout != FT_PROJ_COLS_BY_R && proj_layout != FT_PROJ_R_BY_COLS)
    return fail(FT_ERR_UNSUPPORTED, "proj_layout = %d", (int)proj_layout);
  FT_TRY(check_rank(R, proj, proj_out, "proj", "proj_out"));
  if (block_rows == 32) {
    if (R != 0) return fail(FT_ERR_UNSUPPORTED, "projection is only fused with 1x32 blocks");
    if (qm.stochastic) return fail(FT_ERR_UNSUPPORTED, "stochastic rounding is only offered for 1x32 blocks");
    return hip_status(ft::launch_quant_tiles((const uint16_t*)src, (int)rows, (int)cols, codes, scales, stream, qm),
                      "quantize 32x32");
  }
  if (qm.scales_per_row) return fail(FT_ERR_UNSUPPORTED, "scales_per_row applies to 32x32 blocks");
  FT_TRY(check_workspace(workspace, workspace_bytes,
                         R ? ft::quant_rows_workspace((int)rows, (int)cols, R, (int)proj_layout) : 0));
  return hip_status(ft::launch_quant_rows((const uint16_t*)src, (int)rows, (int)cols, codes, scales,
                                          (const uint16_t*)proj, R, (int)proj_layout, proj_out, (float*)workspace,
                                          stream, qm),
                    "quantize 1x32");
}

ft_status ft_quantize_blockwise(const void* src, int64_t rows, int64_t cols, int32_t block_rows, uint8_t* codes,
                                uint8_t* scales, const void* proj, int32_t R, ft_proj_layout proj_layout,
                                float* proj_out, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  g_last_error[0] = 0;
  return quantize_impl(src, rows, cols, block_rows, codes, scales, proj, R, proj_layout, proj_out, workspace,
                       workspace_bytes, ft::QuantMode{}, stream);
}

ft_status ft_quantize_blockwise_mode(const void* src, int64_t rows, int64_t cols, int32_t block_rows,
                                     uint8_t* codes, uint8_t* scales, const void* proj, int32_t R,
                                     ft_proj_layout proj_layout, float* proj_out, void* workspace,
                                     size_t workspace_bytes, const ft_quant_mode* mode, hipStream_t stream) {
  g_last_error[0] = 0;
  ft::QuantMode qm;
  if (mode) {
    if (mode->scale_rule != FT_SCALE_FLOOR && mode->scale_rule != FT_SCALE_NO_CLIP)
      return fail(FT_ERR_UNSUPPORTED, "scale_rule = %d", (int)mode->scale_rule);
    if (mode->rounding != FT_ROUND_NEAREST_EVEN && mode->rounding != FT_ROUND_STOCHASTIC)
      return fail(FT_ERR_UNSUPPORTED, "rounding = %d", (int)mode->rounding);
    if (mode->scales_per_row != 0 && mode->scales_per_row != 1)
      return fail(FT_ERR_UNSUPPORTED, "scales_per_row = %d", (int)mode->scales_per_row);
    qm.no_clip = mode->scale_rule == FT_SCALE_NO_CLIP;
    qm.stochastic = mode->rounding == FT_ROUND_STOCHASTIC;
    qm.seed = mode->seed;
    qm.stream = mode->stream;
    qm.scales_per_row = mode->scales_per_row;
  }
  return quantize_impl(src, rows, cols, block_rows, codes, scales, proj, R, proj_layout, proj_out, workspace,
                       workspace_bytes, qm, stream);
}

ft_status ft_linear_fwd(const uint8_t* xq, const uint8_t* xs, int64_t M, int64_t K, const uint8_t* wq,
                        const uint8_t* ws, int64_t N, const float* P, int32_t R, const void* U, const void* bias,
                        void* y, ft_dtype y_dtype, hipStream_t stream) {
  g_last_error[0] = 0;
  FT_TRY(check_dim("M", M, 1));
  FT_TRY(check_dim("K", K, 32));
  FT_TRY(check_dim("N", N, 32));
  if (y_dtype != FT_BF16 && y_dtype != FT_F32) return fail(FT_ERR_UNSUPPORTED, "y_dtype = %d", (int)y_dtype);
  if (M == 0 || N == 0) return FT_OK;
  if (K == 0) return fail(FT_ERR_SHAPE, "K == 0");
  if (!xq || !xs || !wq || !ws || !y) return fail(FT_ERR_NULL, "xq, xs, wq, ws and y are required");
  if (!aligned16(xq) || !aligned16(xs) || !aligned16(wq) || !aligned16(ws) || !aligned16(y) ||
      (bias && !aligned16(bias)))
    return fail(FT_ERR_ALIGN, "xq, xs, wq, ws, y, bias must be 16-byte aligned");
  FT_TRY(check_rank(R, P, U, "P", "U"));
  return hip_status(ft::launch_gemm_fp4(false, xq, xs, wq, ws, (int)M, (int)N, (int)K, P, R, (const uint16_t*)U,
                                        (const uint16_t*)bias, y, y_dtype == FT_F32, stream),
                    "linear fwd");
}

ft_status ft_linear_bwd_input(const uint8_t* gq, const uint8_t* gs, int64_t M, int64_t N, const uint8_t* wq,
                              const uint8_t* ws, int64_t K, const float* Qp, int32_t R, const void* D, void* dx,
                              ft_dtype dx_dtype, hipStream_t stream) {
  g_last_error[0] = 0;
  FT_TRY(check_dim("M", M, 1));
  FT_TRY(check_dim("N", N, 32));
  FT_TRY(check_dim("K", K, 32));
  if (dx_dtype != FT_BF16 && dx_dtype != FT_F32) return fail(FT_ERR_UNSUPPORTED, "dx_dtype = %d", (int)dx_dtype);
  if (M == 0 || K == 0) return FT_OK;
  if (N == 0) return fail(FT_ERR_SHAPE, "N == 0");
  if (!gq || !gs || !wq || !ws || !dx) return fail(FT_ERR_NULL, "gq, gs, wq, ws and dx are required");
  if (!aligned16(gq) || !aligned16(gs) || !aligned16(wq) || !aligned16(ws) || !aligned16(dx))
    return fail(FT_ERR_ALIGN, "gq, gs, wq, ws, dx must be 16-byte aligned");
  FT_TRY(check_rank(R, Qp, D, "Qp", "D"));
  return hip_status(ft::launch_gemm_fp4(true, gq, gs, wq, ws, (int)M, (int)N, (int)K, Qp, R, (const uint16_t*)D,
                                        nullptr, dx, dx_dtype == FT_F32, stream),
                    "linear bwd input");
}

static size_t mlp_workspace(int64_t M, int64_t NO, int32_t R2) {
  if (M <= 0 || NO <= 0 || R2 <= 0 || M > kMaxDim || NO > kMaxDim) return 0;
  const int tiles = ft::gemm_fp4_col_tiles((int)NO);
  return tiles > 1 ? (size_t)tiles * M * R2 * sizeof(float) : 0;
}

size_t ft_linear_fwd_gelu_workspace_size(int64_t M, int64_t N, int32_t R2) { return mlp_workspace(M, N, R2); }

ft_status ft_linear_fwd_gelu(const uint8_t* xq, const uint8_t* xs, int64_t M, int64_t K, const uint8_t* wq,
                             const uint8_t* ws, int64_t N, const float* P, int32_t R, const void* U, const void* bias,
                             void* z, void* h, uint8_t* hq, uint8_t* hs, const void* D2, int32_t R2, float* P2,
                             void* workspace, size_t workspace_bytes, hipStream_t stream) {
  g_last_error[0] = 0;
  FT_TRY(check_dim("M", M, 1));
  FT_TRY(check_dim("K", K, 32));
  FT_TRY(check_dim("N", N, 32));
  if (M == 0 || N == 0) return FT_OK;
  if (K == 0) return fail(FT_ERR_SHAPE, "K == 0");
  if (!xq || !xs || !wq || !ws || !z || !h || !hq || !hs) return fail(FT_ERR_NULL, "xq, xs, wq, ws, z, h, hq, hs are required");
  if (!aligned16(xq) || !aligned16(xs) || !aligned16(wq) || !aligned16(ws) || !aligned16(z) || !aligned16(h) ||
      !aligned16(hq) || !aligned16(hs) || (bias && !aligned16(bias)))
    return fail(FT_ERR_ALIGN, "xq, xs, wq, ws, z, h, hq, hs, bias must be 16-byte aligned");
  FT_TRY(check_rank(R, P, U, "P", "U"));
  if (R2 != 0 && (R2 < 16 || R2 > 64 || R2 % 16 != 0)) return fail(FT_ERR_UNSUPPORTED, "R2 = %d: need 0 or 16..64, R2 %% 16 == 0", R2);
  FT_TRY(check_rank(R2, D2, P2, "D2", "P2"));
  if (!ft::gemm_fp4_fused_supported(false, (int)M, (int)N, (int)K, R, R2))
    return fail(FT_ERR_UNSUPPORTED, "fused GELU epilogue needs K %% 128 == 0 and operands below 2 GiB");
  FT_TRY(check_workspace(workspace, workspace_bytes, mlp_workspace(M, N, R2)));
  const bool parts = mlp_workspace(M, N, R2) > 0;
  ft::GemmEpilogue ep{(uint16_t*)z, nullptr, (uint16_t*)h, hq, hs, (const uint16_t*)D2, R2, parts ? (float*)workspace : P2};
  return hip_status(ft::launch_gemm_fp4_fused(false, xq, xs, wq, ws, (int)M, (int)N, (int)K, P, R, (const uint16_t*)U,
                                              (const uint16_t*)bias, ep, P2, stream),
                    "linear fwd gelu");
}

size_t ft_linear_bwd_input_dgelu_workspace_size(int64_t M, int64_t K, int32_t R1) { return mlp_workspace(M, K, R1); }

ft_status ft_linear_bwd_input_dgelu(const uint8_t* gq, const uint8_t* gs, int64_t M, int64_t N, const uint8_t* wq,
                                    const uint8_t* ws, int64_t K, const float* Qp, int32_t R, const void* D,
                                    const void* z, void* dz, uint8_t* dzq, uint8_t* dzs, const void* U1, int32_t R1,
                                    float* Qp1, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  g_last_error[0] = 0;
  FT_TRY(check_dim("M", M, 1));
  FT_TRY(check_dim("N", N, 32));
  FT_TRY(check_dim("K", K, 32));
  if (M == 0 || K == 0) return FT_OK;
  if (N == 0) return fail(FT_ERR_SHAPE, "N == 0");
  if (!gq || !gs || !wq || !ws || !z || !dz || !dzq || !dzs)
    return fail(FT_ERR_NULL, "gq, gs, wq, ws, z, dz, dzq, dzs are required");
  if (!aligned16(gq) || !aligned16(gs) || !aligned16(wq) || !aligned16(ws) || !aligned16(z) || !aligned16(dz) ||
      !aligned16(dzq) || !aligned16(dzs))
    return fail(FT_ERR_ALIGN, "gq, gs, wq, ws, z, dz, dzq, dzs must be 16-byte aligned");
  FT_TRY(check_rank(R, Qp, D, "Qp", "D"));
  if (R1 != 0 && (R1 < 16 || R1 > 64 || R1 % 16 != 0)) return fail(FT_ERR_UNSUPPORTED, "R1 = %d: need 0 or 16..64, R1 %% 16 == 0", R1);
  FT_TRY(check_rank(R1, U1, Qp1, "U1", "Qp1"));
  if (!ft::gemm_fp4_fused_supported(true, (int)M, (int)N, (int)K, R, R1))
    return fail(FT_ERR_UNSUPPORTED, "fused dGELU epilogue needs N and K multiples of 128 and operands below 2 GiB");
  FT_TRY(check_workspace(workspace, workspace_bytes, mlp_workspace(M, K, R1)));
  const bool parts = mlp_workspace(M, K, R1) > 0;
  ft::GemmEpilogue ep{nullptr, (const uint16_t*)z, (uint16_t*)dz, dzq, dzs, (const uint16_t*)U1, R1,
                      parts ? (float*)workspace : Qp1};
  return hip_status(ft::launch_gemm_fp4_fused(true, gq, gs, wq, ws, (int)M, (int)N, (int)K, Qp, R, (const uint16_t*)D,
                                              nullptr, ep, Qp1, stream),
                    "linear bwd input dgelu");
}

size_t ft_lora_grads_workspace_size(int64_t M, int64_t K, int64_t N, int64_t ld, int32_t r) {
  if (M <= 0 || K <= 0 || N <= 0 || r < 1 || r > 128 || ld < r || M > kMaxDim || K > (1 << 24) || N > (1 << 24) ||
      ld > 4096)
    return 0;
  return ft::lora_grads_workspace((int)M, (int)K, (int)N, (int)ld, r);
}

static ft_status lora_validate(const void* x, int64_t M, int64_t K, const void* dy, int64_t N, const float* xa,
                               const float* dyb, int64_t ld, int32_t r, float* dA, float* dB, int32_t accumulate,
                               bool* nothing) {
  *nothing = false;
  FT_TRY(check_dim("M", M, 1));
  FT_TRY(check_dim("K", K, 32));
  FT_TRY(check_dim("N", N, 32));
  if (r < 1 || r > 128) return fail(FT_ERR_UNSUPPORTED, "r = %d: need 1 <= r <= 128", r);
  if (ld < r || ld % 4 != 0 || ld > 4096) return fail(FT_ERR_SHAPE, "ld = %lld: need r <= ld <= 4096, ld %% 4 == 0", (long long)ld);
  if (accumulate != 0 && accumulate != 1) return fail(FT_ERR_UNSUPPORTED, "accumulate = %d", accumulate);
  if (K == 0 && N == 0) {   // dA [0, r] and dB [r, 0] hold nothing
    *nothing = true;
    return FT_OK;
  }
  if (!dA || !dB) return fail(FT_ERR_NULL, "dA and dB are required");
  if (M > 0 && (!x || !dy || !xa || !dyb)) return fail(FT_ERR_NULL, "x, dy, xa and dyb are required");
  if (K > (1 << 24) || N > (1 << 24)) return fail(FT_ERR_UNSUPPORTED, "K and N above 2^24 are not supported here");
  if ((x && !aligned16(x)) || (dy && !aligned16(dy)) || (xa && !aligned16(xa)) || (dyb && !aligned16(dyb)) ||
      !aligned16(dA) || !aligned16(dB))
    return fail(FT_ERR_ALIGN, "x, dy, xa, dyb, dA, dB must be 16-byte aligned");
  return FT_OK;
}

ft_status ft_lora_grads(const void* x, int64_t M, int64_t K, const void* dy, int64_t N, const float* xa,
                        const float* dyb, int64_t ld, int32_t r, float* dA, float* dB, int32_t accumulate,
                        void* workspace, size_t workspace_bytes, hipStream_t stream) {
  g_last_error[0] = 0;
  bool nothing;
  FT_TRY(lora_validate(x, M, K, dy, N, xa, dyb, ld, r, dA, dB, accumulate, &nothing));
  if (nothing) return FT_OK;
  FT_TRY(check_workspace(workspace, workspace_bytes, ft::lora_grads_workspace((int)M, (int)K, (int)N, (int)ld, r)));
  return hip_status(ft::launch_lora_grads((const uint16_t*)x, (int)M, (int)K, (const uint16_t*)dy, (int)N, xa, dyb,
                                          (int)ld, r, dA, dB, accumulate != 0, (float*)workspace, stream),
                    "lora grads");
}

ft_status ft_lora_grads_noalloc(const void* x, int64_t M, int64_t K, const void* dy, int64_t N, const float* xa,
                                const float* dyb, int64_t ld, int32_t r, float* dA, float* dB, int32_t accumulate,
                                hipStream_t stream) {
  g_last_error[0] = 0;
  bool nothing;
  FT_TRY(lora_validate(x, M, K, dy, N, xa, dyb, ld, r, dA, dB, accumulate, &nothing));
  if (nothing) return FT_OK;
  const size_t need = ft::lora_grads_workspace((int)M, (int)K, (int)N, (int)ld, r);
  if (need > ft::kLoraScratchBytes)
    return fail(FT_ERR_UNSUPPORTED, "these sizes need %zu bytes of scratch, more than the %zu of the allocation-free "
                "entry point; call ft_lora_grads with a workspace", need, ft::kLoraScratchBytes);
  float* scratch = nullptr;
  if (need > 0) FT_TRY(hip_status(ft::lora_grads_scratch(&scratch), "lora grads scratch lookup"));
  return hip_status(ft::launch_lora_grads((const uint16_t*)x, (int)M, (int)K, (const uint16_t*)dy, (int)N, xa, dyb,
                                          (int)ld, r, dA, dB, accumulate != 0, scratch, stream),
                    "lora grads (no allocation)");
}

ft_status ft_quantize_nvfp4(const void* src, int64_t rows, int64_t cols, int32_t block_rows, uint8_t* codes,
                            uint8_t* scales, float* tensor_scale, hipStream_t stream) {
  g_last_error[0] = 0;
  if (block_rows != 1 && block_rows != 16) return fail(FT_ERR_UNSUPPORTED, "block_rows = %d (1 or 16)", block_rows);
  FT_TRY(check_dim("rows", rows, block_rows));
  FT_TRY(check_dim("cols", cols, 16));
  if (rows == 0 || cols == 0) return FT_OK;
  if ((rows / 16 + 1) * (cols / 16) >= ((int64_t)1 << 31)) return fail(FT_ERR_SHAPE, "rows * cols too large");
  if (!src || !codes || !scales || !tensor_scale) return fail(FT_ERR_NULL, "src, codes, scales, tensor_scale are required");
  if (!aligned16(src) || !aligned16(codes) || !aligned16(scales) || ((uintptr_t)tensor_scale & 3u))
    return fail(FT_ERR_ALIGN, "src, codes, scales must be 16-byte aligned and tensor_scale 4-byte aligned");
  return hip_status(ft::launch_quant_nvfp4((const uint16_t*)src, (int)rows, (int)cols, block_rows, codes, scales,
                                           tensor_scale, stream),
                    "quantize nvfp4");
}

static ft_status nvfp4_gemm(bool bwd, const uint8_t* a, const uint8_t* as, const float* at, int64_t M, int64_t KR,
                            const uint8_t* wq, const uint8_t* ws, const float* wt, int64_t NO, float* out,
                            hipStream_t stream) {
  FT_TRY(check_dim("M", M, 1));
  FT_TRY(check_dim(bwd ? "N" : "K", KR, 16));
  FT_TRY(check_dim(bwd ? "K" : "N", NO, 16));
  if (M == 0 || NO == 0) return FT_OK;
  if (KR == 0) return fail(FT_ERR_SHAPE, "empty reduction");
  if (!a || !as || !at || !wq || !ws || !wt || !out) return fail(FT_ERR_NULL, "every operand is required");
  if (!aligned16(a) || !aligned16(as) || !aligned16(wq) || !aligned16(ws) || !aligned16(out) ||
      ((uintptr_t)at & 3u) || ((uintptr_t)wt & 3u))
    return fail(FT_ERR_ALIGN, "codes, scales and out must be 16-byte aligned, tensor scales 4-byte aligned");
  if ((int64_t)M * KR / 2 >= ((int64_t)1 << 31) || (int64_t)M * NO >= ((int64_t)1 << 31))
    return fail(FT_ERR_SHAPE, "operands too large for this path");
  const int N = (int)(bwd ? KR : NO), K = (int)(bwd ? NO : KR);
  return hip_status(ft::launch_gemm_nvfp4(bwd, a, as, at, wq, ws, wt, (int)M, N, K, out, stream), "gemm nvfp4");
}

ft_status ft_linear_fwd_nvfp4(const uint8_t* xq, const uint8_t* xs, const float* xt, int64_t M, int64_t K,
                              const uint8_t* wq, const uint8_t* ws, const float* wt, int64_t N, float* y,
                              hipStream_t stream) {
  g_last_error[0] = 0;
  return nvfp4_gemm(false, xq, xs, xt, M, K, wq, ws, wt, N, y, stream);
}

ft_status ft_linear_bwd_input_nvfp4(const uint8_t* gq, const uint8_t* gs, const float* gt, int64_t M, int64_t N,
                                    const uint8_t* wq, const uint8_t* ws, const float* wt, int64_t K, float* dx,
                                    hipStream_t stream) {
  g_last_error[0] = 0;
  return nvfp4_gemm(true, gq, gs, gt, M, N, wq, ws, wt, K, dx, stream);
}

}  // extern "C"
