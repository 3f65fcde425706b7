/*
 * fourtune.h -- C ABI of the MI355X (gfx950) W4A4G4 triple-branch linear layer.
 *
 * Method: FourTune (arXiv 2607.05711), Section 3.  One linear layer carries
 *   (1) a frozen 4-bit backbone weight W, used through 4-bit GEMMs,
 *   (2) a frozen low-rank "numerical stabilizer" L1 L2 in bf16, and
 *   (3) a trainable low-rank adapter A B in bf16,
 * forward  (Eq. 2):  Y  = Q(X) Q(W)^T + X L1 L2 + X A B (+ bias)
 * backward (Eq. 3):  dX = Q(G) Q(W)   + G (L1 L2)^T + G (A B)^T,   G = dL/dY
 * adapter gradients (Sec. 3.2):  dB = (X A)^T G,  dA = X^T (G B^T).
 * The two low-rank branches share their input, so the library concatenates
 * them: D = [L1 | A] is [K, R] ("down") and U = [L2 ; B] is [R, N] ("up"),
 * R = r_s + r, stabilizer first (Sec. 3.3, LoRA fusion).
 *
 * Number format (paper: NVFP4, Sec. 3.1; read here as the OCP Microscaling
 * MXFP4 format the paper cites in Sec. 2.3, which gfx950's block-scaled MFMA
 * consumes): 4-bit E2M1 codes, two per byte (element 2i in bits 3:0, element
 * 2i+1 in bits 7:4), with one E8M0 power-of-two scale per block.
 *   - X and G: 1x32 blocks along the GEMM reduction axis (K for X, N for G).
 *   - W: 32x32 tiles, scales [N/32, K/32], so the backward GEMM reads the
 *     same codes and scales in transposed order (Sec. 3.2, block-wise
 *     quantization) with no re-quantization.
 * Block rule: e = floor(log2(max|v|)) - 2 clamped to [-127, 127] (a zero block
 * gets e = -127), scale byte = e + 127; each element becomes the nearest
 * E2M1 value of v / 2^e, ties to the even code, saturating at 6, with the
 * input's sign bit (also for -0).
 *
 * Conventions for every call:
 *   - All tensors are dense row-major device buffers owned by the caller.  The
 *     library never allocates, frees or synchronizes; work is enqueued on
 *     `stream` (a hipStream_t; NULL = the default stream) and runs
 *     asynchronously.
 *   - bf16 tensors are passed as `const void*` holding IEEE bfloat16 values.
 *   - Every tensor pointer must be 16-byte aligned, the E8M0 scale arrays
 *     (`scales`, `xs`, `gs`, `ws`, `hs`, `dzs`) included: the kernels move
 *     scales in 4- and 16-byte units.  A misaligned pointer gives
 *     FT_ERR_ALIGN.
 *   - Arguments are validated before anything is enqueued; on error nothing is
 *     launched and the return value says why (ft_last_error() has details).
 *   - FT_ERR_HIP means a launch was rejected by the HIP runtime; earlier
 *     kernels of the same call may already be enqueued.
 *   - Inputs are assumed finite.  Calls on the same stream are ordered; calls
 *     that write the same buffers from different streams race.
 */
#ifndef FOURTUNE_H
#define FOURTUNE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ihipStream_t *hipStream_t;

typedef enum ft_status {
    FT_OK = 0,
    FT_ERR_NULL = 1,         /* a required pointer is NULL */
    FT_ERR_SHAPE = 2,        /* a size is negative, too large, or not a multiple of 32 where required */
    FT_ERR_ALIGN = 3,        /* a tensor pointer is not 16-byte aligned */
    FT_ERR_UNSUPPORTED = 4,  /* valid but unsupported option (e.g. R > 128, R % 16 != 0) */
    FT_ERR_HIP = 5           /* the HIP runtime rejected a launch */
} ft_status;

typedef enum ft_dtype { FT_BF16 = 0, FT_F32 = 1 } ft_dtype;

typedef enum ft_proj_layout {
    FT_PROJ_COLS_BY_R = 0,   /* proj is [cols, R]; proj_out = src . proj   (forward: D) */
    FT_PROJ_R_BY_COLS = 1    /* proj is [R, cols]; proj_out = src . proj^T (backward: U) */
} ft_proj_layout;

/*
 * Block-wise MXFP4 quantization of a bf16 matrix, optionally fused with the
 * low-rank down-projection of the same input (Sec. 3.3: the three branches
 * share their input, so one pass reads it once).
 *
 *   src        bf16 [rows, cols]; cols % 32 == 0.
 *   block_rows 1  -> 1x32 blocks along each row (activations X, gradients G);
 *                    scales is [rows, cols/32].
 *              32 -> 32x32 tiles (the frozen weight, prepared offline);
 *                    rows % 32 == 0; scales is [rows/32, cols/32].
 *   codes      uint8 [rows, cols/2], packed E2M1 (see above).
 *   scales     uint8 E8M0 codes, layout as above.
 *   proj       bf16, NULL for none.  layout FT_PROJ_COLS_BY_R: [cols, R]
 *              (forward, D = [L1|A]); FT_PROJ_R_BY_COLS: [R, cols] (backward,
 *              U = [L2;B]).  Only with block_rows == 1.
 *   R          0 when proj is NULL; else 16 <= R <= 128 and R % 16 == 0.
 *   proj_out   fp32 [rows, R] = src . proj (or src . proj^T), products of the
 *              unquantized bf16 inputs with fp32 accumulation.  Column chunks
 *              of the row leave fp32 partial sums in the workspace, which a
 *              second kernel adds in a fixed order (results are reproducible).
 *   workspace  device memory of at least ft_quantize_workspace_size(...) bytes,
 *              16-byte aligned, owned by the caller; contents on entry are
 *              ignored and on return undefined.  May be NULL when the size is
 *              0 (no projection, or the columns fit one chunk).  Calls that
 *              share a workspace must not overlap.
 * rows == 0 is a no-op.  rows < 2^31, cols < 2^31.
 */
ft_status ft_quantize_blockwise(const void *src, int64_t rows, int64_t cols, int32_t block_rows,
                                uint8_t *codes, uint8_t *scales,
                                const void *proj, int32_t R, ft_proj_layout proj_layout,
                                float *proj_out, void *workspace, size_t workspace_bytes,
                                hipStream_t stream);

/* Workspace bytes ft_quantize_blockwise needs for these arguments (0: none). */
size_t ft_quantize_workspace_size(int64_t rows, int64_t cols, int32_t block_rows, int32_t R,
                                  ft_proj_layout proj_layout);

/*
 * Numerics variants of Q(.).  Sec. 3.1 fixes the 4-bit format but not the
 * quantizer's scale rule or rounding; these options cover the readings the
 * default (floor rule, nearest-even) leaves out.
 *   scale_rule  FT_SCALE_FLOOR (default): e = floor(log2 max|v|) - 2, values
 *               above 6 * 2^e saturate to 6.  FT_SCALE_NO_CLIP: the smallest
 *               e with max|v| <= 6 * 2^e, so nothing saturates (the scale byte
 *               may then change when dequantized values are quantized again;
 *               the values do not).
 *   rounding    FT_ROUND_NEAREST_EVEN (default), or FT_ROUND_STOCHASTIC: an
 *               element between two E2M1 magnitudes lo < t < hi (t = |v| / 2^e)
 *               moves up to hi when (t - lo) / (hi - lo) > (u + 1/2) / 2^16,
 *               u a 16-bit uniform; values on the grid stay.  u comes from the
 *               counter-based generator Philox4x32-10 (Salmon, Moraes, Dror,
 *               Shaw, SC 2011) with key = seed (low word first) and counter =
 *               (i / 8 as two words, stream as two words), i = row * cols +
 *               col; element i takes the 16-bit half i % 2 (low half first) of
 *               output word (i % 8) / 2.  Results depend only on (seed,
 *               stream, i), never on the launch.  1x32 blocks only.
 *   seed, stream  the generator's key and stream (e.g. a run seed and the
 *               training step); ignored with nearest-even rounding.
 *   scales_per_row  block_rows == 32 only (2-D blocked activations): 1 writes
 *               the scales as [rows, cols/32], every row of a 32x32 tile
 *               carrying the tile's code, which is the layout ft_linear_fwd
 *               and ft_linear_bwd_input read for their left operand.
 */
typedef enum ft_scale_rule { FT_SCALE_FLOOR = 0, FT_SCALE_NO_CLIP = 1 } ft_scale_rule;
typedef enum ft_rounding { FT_ROUND_NEAREST_EVEN = 0, FT_ROUND_STOCHASTIC = 1 } ft_rounding;
typedef struct ft_quant_mode {
    int32_t scale_rule;        /* ft_scale_rule */
    int32_t rounding;          /* ft_rounding */
    uint64_t seed;
    uint64_t stream;
    int32_t scales_per_row;    /* 0 or 1 */
} ft_quant_mode;

/*
 * ft_quantize_blockwise with a numerics mode (NULL: the defaults, identical to
 * ft_quantize_blockwise).  Arguments and errors as ft_quantize_blockwise;
 * FT_ERR_UNSUPPORTED for an unknown option, stochastic rounding with 32x32
 * blocks, or scales_per_row with 1x32 blocks.  The fused projection is
 * unaffected by the mode (it uses the unquantized input).
 */
ft_status ft_quantize_blockwise_mode(const void *src, int64_t rows, int64_t cols, int32_t block_rows,
                                     uint8_t *codes, uint8_t *scales,
                                     const void *proj, int32_t R, ft_proj_layout proj_layout,
                                     float *proj_out, void *workspace, size_t workspace_bytes,
                                     const ft_quant_mode *mode, hipStream_t stream);

/*
 * Forward of the triple-branch linear, Eq. (2), in nn.Linear orientation:
 *   y[m,n] = sum_k DQ(xq)[m,k] DQ(wq)[n,k] + sum_j P[m,j] U[j,n] + bias[n]
 * The 4-bit product runs on block-scaled FP4 MFMA with fp32 accumulation; the
 * low-rank up-projection and the bias are added in the same kernel's
 * epilogue (Sec. 3.3).  P is split as P = hi + lo (two bf16 terms) so the
 * up-projection keeps ~16 significant bits of P.
 *
 *   xq, xs   X codes [M, K/2] and 1x32 scales [M, K/32] (ft_quantize_blockwise).
 *   wq, ws   W codes [N, K/2] and 32x32 scales [N/32, K/32].
 *   M >= 0;  K, N multiples of 32.
 *   P        fp32 [M, R] = X . D (from ft_quantize_blockwise); NULL iff R == 0.
 *   U        bf16 [R, N] = [L2 ; B]; NULL iff R == 0.  R % 16 == 0, R <= 128.
 *   bias     bf16 [N] or NULL.
 *   y        [M, N], bf16 (round to nearest even) or fp32.
 */
ft_status ft_linear_fwd(const uint8_t *xq, const uint8_t *xs, int64_t M, int64_t K,
                        const uint8_t *wq, const uint8_t *ws, int64_t N,
                        const float *P, int32_t R, const void *U,
                        const void *bias, void *y, ft_dtype y_dtype, hipStream_t stream);

/*
 * Input gradient of the triple-branch linear, Eq. (3):
 *   dx[m,k] = sum_n DQ(gq)[m,n] DQ(wq)[n,k] + sum_j Qp[m,j] D[k,j]
 * The weight codes and 32x32 scales are the forward's, read in transposed
 * order inside the kernel (Sec. 3.2); nothing is re-quantized.
 *
 *   gq, gs   G codes [M, N/2] and 1x32 scales [M, N/32].
 *   wq, ws   W codes [N, K/2] and 32x32 scales [N/32, K/32].
 *   Qp       fp32 [M, R] = G . U^T (from ft_quantize_blockwise); NULL iff R == 0.
 *   D        bf16 [K, R] = [L1 | A]; NULL iff R == 0.
 *   dx       [M, K], bf16 or fp32.
 */
ft_status ft_linear_bwd_input(const uint8_t *gq, const uint8_t *gs, int64_t M, int64_t N,
                              const uint8_t *wq, const uint8_t *ws, int64_t K,
                              const float *Qp, int32_t R, const void *D,
                              void *dx, ft_dtype dx_dtype, hipStream_t stream);

/*
 * MLP pair, forward of FC1 fused with FC2's input preparation (Sec. 3.3, MLP
 * fusion: the GELU and FC2's quantization and down-projection consume FC1's
 * output tile while it is on chip).  The GEMM is ft_linear_fwd's; then
 *   z[m,n]   = bf16(y[m,n])                         saved for the backward
 *   h[m,n]   = bf16(GELU_tanh(z[m,n]))              FC2's input
 *   hq, hs   = 1x32 MXFP4 codes/scales of h (as ft_quantize_blockwise)
 *   P2[m,j]  = sum_n h[m,n] D2[n,j]                 FC2's P (fp32)
 * GELU_tanh(z) = 0.5 z (1 + tanh(sqrt(2/pi) (z + 0.044715 z^3))), evaluated in
 * fp32.
 *   Arguments up to bias as ft_linear_fwd.  z, h: bf16 [M, N];  hq uint8
 *   [M, N/2]; hs uint8 [M, N/32].  D2: bf16 [N, R2] = FC2's [L1 | A];
 *   R2 in {0, 16, 32, 48, 64} (0: no projection, D2 and P2 NULL);  P2 fp32 [M, R2].
 *   workspace: ft_linear_fwd_gelu_workspace_size(M, N, R2) bytes, 16-byte
 *   aligned (NULL when 0): per-column-tile partials of P2, summed in a fixed
 *   order by a second kernel.
 * Needs K % 128 == 0 (FT_ERR_UNSUPPORTED otherwise).
 */
ft_status ft_linear_fwd_gelu(const uint8_t *xq, const uint8_t *xs, int64_t M, int64_t K,
                             const uint8_t *wq, const uint8_t *ws, int64_t N,
                             const float *P, int32_t R, const void *U, const void *bias,
                             void *z, void *h, uint8_t *hq, uint8_t *hs,
                             const void *D2, int32_t R2, float *P2,
                             void *workspace, size_t workspace_bytes, hipStream_t stream);
size_t ft_linear_fwd_gelu_workspace_size(int64_t M, int64_t N, int32_t R2);

/*
 * MLP pair, backward-input of FC2 fused with FC1's gradient preparation: the
 * GEMM is ft_linear_bwd_input's (its fp32 result dH is not rounded), then
 *   dz[m,k]  = bf16(dH[m,k] * GELU_tanh'(z[m,k]))   FC1's incoming gradient
 *   dzq, dzs = 1x32 MXFP4 codes/scales of dz
 *   Qp1[m,j] = sum_k dz[m,k] U1[j,k]                 FC1's Qp (fp32)
 *   Arguments up to D as ft_linear_bwd_input (N = FC2's output width, K = the
 *   MLP width).  z: bf16 [M, K] from ft_linear_fwd_gelu.  dz bf16 [M, K];  dzq
 *   uint8 [M, K/2];  dzs uint8 [M, K/32].  U1: bf16 [R1, K] = FC1's [L2 ; B];
 *   R1 in {0, 16, 32, 48, 64};  Qp1 fp32 [M, R1].
 *   workspace: ft_linear_bwd_input_dgelu_workspace_size(M, K, R1) bytes.
 * Needs N % 128 == 0 and K % 128 == 0 (FT_ERR_UNSUPPORTED otherwise).
 */
ft_status ft_linear_bwd_input_dgelu(const uint8_t *gq, const uint8_t *gs, int64_t M, int64_t N,
                                    const uint8_t *wq, const uint8_t *ws, int64_t K,
                                    const float *Qp, int32_t R, const void *D,
                                    const void *z, void *dz, uint8_t *dzq, uint8_t *dzs,
                                    const void *U1, int32_t R1, float *Qp1,
                                    void *workspace, size_t workspace_bytes, hipStream_t stream);
size_t ft_linear_bwd_input_dgelu_workspace_size(int64_t M, int64_t K, int32_t R1);

/*
 * Adapter weight gradients (Sec. 3.2):
 *   dA[k,j] = sum_m X[m,k] dyb[m,j]    (dA = X^T (G B^T))
 *   dB[j,n] = sum_m xa[m,j] G[m,n]     (dB = (X A)^T G)
 * X is the unquantized bf16 input saved by the forward pass.
 *
 *   x        bf16 [M, K];  dy: bf16 [M, N] (the incoming gradient G).
 *   xa       fp32, row stride ld: columns [0, r) hold X A (pass P + r_s).
 *   dyb      fp32, row stride ld: columns [0, r) hold G B^T (pass Qp + r_s).
 *   ld       row stride of xa and dyb in elements (R); ld >= r, ld % 4 == 0.
 *            xa and dyb are 16-byte aligned like every tensor (r_s % 4 == 0
 *            when they point into P and Qp).
 *   r        1 <= r <= 128.
 *   dA       fp32 [K, r];  dB: fp32 [r, N].
 *   accumulate  0: overwrite dA and dB;  1: add into them.
 *   workspace  at least ft_lora_grads_workspace_size(M, K, N, ld, r) bytes,
 *            16-byte aligned (NULL when that size is 0): token chunks leave
 *            fp32 partial sums there and a second kernel adds them in a fixed
 *            order (results are reproducible).  Calls sharing a workspace
 *            must not overlap.
 * K, N multiples of 32 and at most 2^24; M >= 0 (M == 0 gives zeros, or
 * leaves dA and dB unchanged when accumulating).  K == N == 0 is a no-op.
 */
ft_status ft_lora_grads(const void *x, int64_t M, int64_t K, const void *dy, int64_t N,
                        const float *xa, const float *dyb, int64_t ld, int32_t r,
                        float *dA, float *dB, int32_t accumulate,
                        void *workspace, size_t workspace_bytes, hipStream_t stream);

/* Workspace bytes ft_lora_grads needs for these arguments (0: none). */
size_t ft_lora_grads_workspace_size(int64_t M, int64_t K, int64_t N, int64_t ld, int32_t r);

/*
 * ft_lora_grads without a workspace, for callers that cannot allocate device
 * memory around the call (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  Arguments, results and errors are those
 * of ft_lora_grads; the results are bit-identical to it (same kernels, same
 * summation order).  The token-chunk partial sums go to a static 32 MiB
 * device array inside the library instead of a workspace: each GPU the
 * library runs on holds one until the process ends, and its address is looked
 * up on the first call on that device (the device current at the call).
 * Every size this layer accepts fits (the partials never exceed 32 MiB);
 * sizes that would need more return FT_ERR_UNSUPPORTED.  Nothing is
 * allocated, freed or synchronized.  All calls on one GPU share the array:
 * calls that overlap in time on the same GPU (different streams, threads or
 * processes' graphs replayed concurrently) race and give undefined results.
 */
ft_status ft_lora_grads_noalloc(const void *x, int64_t M, int64_t K, const void *dy, int64_t N,
                                const float *xa, const float *dyb, int64_t ld, int32_t r,
                                float *dA, float *dB, int32_t accumulate, hipStream_t stream);

/*
 * NVFP4 emulation: the 4-bit format Sec. 3.1 names (E2M1 elements, one FP8
 * E4M3 scale per 16 elements, one FP32 scale per tensor; 16x16 tiles for the
 * weight, Sec. 4.3), as an accuracy cross-check of the layer's native MXFP4.
 * gfx950's block-scaled MFMA takes E8M0 scales per 32 elements, so these
 * calls dequantize to bf16 inside the GEMM (exact: E2M1 x E4M3 has at most 6
 * significant bits) and run bf16 MFMAs; they are not a fast path.
 *
 * ft_quantize_nvfp4:
 *   src          bf16 [rows, cols]; cols % 16 == 0.
 *   block_rows   1 (1x16 blocks along rows; scales [rows, cols/16]) or 16
 *                (16x16 tiles, rows % 16 == 0; scales [rows/16, cols/16]).
 *   codes        uint8 [rows, cols/2], packed E2M1 as ft_quantize_blockwise.
 *   scales       uint8 FP8 E4M3 codes (OCP E4M3: bias 7, no infinities).
 *   tensor_scale one fp32 in device memory, written: st = amax(|src|) / (6 * 448)
 *                rounded once to fp32.  Used as scratch while the call runs.
 * Block scale: the E4M3 value nearest to amax_block / (6 st) (the fp32
 * product 6 st, then the fp32 quotient), ties to the even mantissa,
 * saturating at 448.  Element: the E2M1 value nearest to |v| / (E4M3 * st)
 * (exact), ties to the even code, saturating at 6, sign copied; a zero block
 * scale gives zero codes.
 */
ft_status ft_quantize_nvfp4(const void *src, int64_t rows, int64_t cols, int32_t block_rows,
                            uint8_t *codes, uint8_t *scales, float *tensor_scale, hipStream_t stream);

/*
 * Forward and input-gradient GEMMs on NVFP4 operands (fp32 outputs):
 *   y[m,n]  = xt wt sum_k DQ(xq)[m,k] DQ(wq)[n,k]    x: 1x16 blocks along K; w: 16x16 tiles [N, K]
 *   dx[m,k] = gt wt sum_n DQ(gq)[m,n] DQ(wq)[n,k]    g: 1x16 blocks along N; the same w, read
 *                                                    transposed with its tile scales (Sec. 3.2)
 * DQ = E2M1 x E4M3 without the tensor scale; xt, gt, wt: the tensor scales
 * (device fp32) from ft_quantize_nvfp4.  K and N multiples of 16.
 */
ft_status ft_linear_fwd_nvfp4(const uint8_t *xq, const uint8_t *xs, const float *xt, int64_t M, int64_t K,
                              const uint8_t *wq, const uint8_t *ws, const float *wt, int64_t N,
                              float *y, hipStream_t stream);
ft_status ft_linear_bwd_input_nvfp4(const uint8_t *gq, const uint8_t *gs, const float *gt, int64_t M, int64_t N,
                                    const uint8_t *wq, const uint8_t *ws, const float *wt, int64_t K,
                                    float *dx, hipStream_t stream);

/* Static description of a status code. */
const char *ft_status_string(ft_status status);

/* Detail of the last error returned on the calling thread ("" if none). */
const char *ft_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* FOURTUNE_H */
