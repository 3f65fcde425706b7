// Device-side helpers shared by the gfx950 kernels of libfourtune.
//
// Operand layouts of the CDNA4 matrix instructions used here (lane l of a
// 64-wide wavefront):
//   v_mfma_scale_f32_32x32x64_f8f6f4 (FP4 x FP4, E8M0 block scales):
//     A: row l%32, reduction elements [32*(l/32), +32) as 16 packed bytes
//        (element 2i in the low nibble of byte i), scale byte for that
//        row/32-block chosen from a VGPR by op_sel;
//     B: column l%32, same reduction split;
//     C/D: column l%32, rows 8*(v/4) + 4*(l/32) + v%4 for v = 0..15.
//   v_mfma_f32_32x32x16_bf16: A row l%32 / B column l%32, reduction
//     elements [8*(l/32), +8); C/D as above.
//   ds_read_b64_tr_b4: in each 16-lane group lane s supplies the address of
//     16 nibbles (a row); lane c receives nibble c of rows 0..15, in order.
//   ds_read_b64_tr_b16: in each 16-lane group, output lane i element j is
//     halfword i%4 of source lane 4j + i/4.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ft {

typedef int v2i __attribute__((ext_vector_type(2)));
typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef short v4s __attribute__((ext_vector_type(4)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef __bf16 v2bf __attribute__((ext_vector_type(2)));
typedef float v2f __attribute__((ext_vector_type(2)));
typedef float v4f __attribute__((ext_vector_type(4)));

#define FT_LDS __attribute__((address_space(3)))

// fp32 -> bf16 bits, round to nearest even (finite inputs).
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

__device__ __forceinline__ float bf16_to_f32(uint32_t b) { return __uint_as_float(b << 16); }

// Two-term bf16 split of an fp32 value: x ~= hi + lo with |x - hi - lo| <= 2^-16 |x|.
__device__ __forceinline__ void split_bf16(float x, uint32_t& hi, uint32_t& lo) {
  hi = f32_to_bf16_rne(x);
  lo = f32_to_bf16_rne(x - bf16_to_f32(hi));
}

// The same split for two values at once with the packed round-to-nearest-even
// convert: hi and lo hold bf16 pairs (a in the low half, b in the high half).
// x - hi is exact in fp32, so lo is the rounding of the true remainder.
__device__ __forceinline__ void split_bf16x2(float a, float b, uint32_t& hi, uint32_t& lo) {
  const v2f x = {a, b};
  hi = __builtin_bit_cast(uint32_t, __builtin_convertvector(x, v2bf));
  const v2f hf = {__uint_as_float(hi << 16), __uint_as_float(hi & 0xFFFF0000u)};
  lo = __builtin_bit_cast(uint32_t, __builtin_convertvector(x - hf, v2bf));
}

// E8M0 block scale from the largest |bf16| bit pattern of a block (sign
// cleared): floor(log2 amax) - 2 + 127, clamped at 0.  A zero or subnormal
// amax gives 0 (e = -127).
__device__ __forceinline__ uint32_t e8m0_from_amax_bits(uint32_t amax_bits) {
  int e = (int)((amax_bits >> 7) & 0xFF) - 2;
  return e > 0 ? (uint32_t)e : 0u;
}

// The no-clip variant: the smallest e with amax / 2^e <= 6 (nothing
// saturates).  With amax = m 2^E, m in [1, 2): e = E - 2 when m <= 1.5
// (mantissa bits <= 0x40), else E - 1; clamped at code 0.
__device__ __forceinline__ uint32_t e8m0_noclip_from_amax_bits(uint32_t amax_bits) {
  int e = (int)((amax_bits >> 7) & 0xFF) - 2 + ((amax_bits & 0x7F) > 0x40 ? 1 : 0);
  return e > 0 ? (uint32_t)e : 0u;
}

// Numerics mode of the 1x32 quantizers (a template argument): bit 0 selects
// the no-clip scale rule, bit 1 stochastic rounding.
enum { QM_NOCLIP = 1, QM_SR = 2 };

template <int QM>
__device__ __forceinline__ uint32_t e8m0_of(uint32_t amax_bits) {
  if constexpr ((QM & QM_NOCLIP) != 0) return e8m0_noclip_from_amax_bits(amax_bits);
  else return e8m0_from_amax_bits(amax_bits);
}

// Philox4x32-10 (Salmon, Moraes, Dror and Shaw, SC 2011): ten rounds of two
// 32x32->64-bit products of counter words 0 and 2 with fixed odd constants;
// the high halves xor the other counter words and the round key, the key
// grows by two Weyl constants per round.
__device__ __forceinline__ void philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3, uint32_t k0,
                                              uint32_t k1, uint32_t (&out)[4]) {
#pragma unroll
  for (int round = 0; round < 10; round++) {
    const uint32_t lo0 = 0xD2511F53u * c0, hi0 = __umulhi(0xD2511F53u, c0);
    const uint32_t lo1 = 0xCD9E8D57u * c2, hi1 = __umulhi(0xCD9E8D57u, c2);
    c0 = hi1 ^ c1 ^ k0;
    c1 = lo1;
    c2 = hi0 ^ c3 ^ k1;
    c3 = lo0;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

// Random stream of stochastic rounding: key = seed, counter words 2 and 3 =
// stream; counter words 0 and 1 = (element index) / 8.
struct SrKey { uint32_t k0, k1, s0, s1; };

// Stochastic rounding of 8 consecutive bf16 (packed in w, element 2e in the
// low half of w[e]) to E2M1 with the block's E8M0 code.  rnd[e] holds the
// 16-bit uniforms of elements 2e (low half) and 2e + 1.  With t = |v| / 2^e
// between grid values lo <= t < hi, the element moves up to hi when
// (t - lo) / (hi - lo) > (u + 1/2) / 2^16; every step is exact in fp32
// (t has 8 significant bits, the grid spacings are powers of two).  t >= 6
// saturates.  The sign bit is copied.  Returns 8 codes, element 0 in the low
// nibble.
__device__ __forceinline__ uint32_t sr_fp4x8(const uint32_t (&w)[4], uint32_t scale_code, const uint32_t (&rnd)[4]) {
  const float inv = __uint_as_float((254u - scale_code) << 23);   // 2^-e, a normal fp32 for every code <= 253
  uint32_t o = 0;
#pragma unroll
  for (int i = 0; i < 8; i++) {
    const uint32_t b = (w[i >> 1] >> (16 * (i & 1))) & 0xFFFFu;
    const uint32_t u = (rnd[i >> 1] >> (16 * (i & 1))) & 0xFFFFu;
    const float t = __uint_as_float((b & 0x7FFFu) << 16) * inv;
    const float t2 = 2.0f * t;
    const float f2 = floorf(t2), f1 = floorf(t);
    uint32_t code;
    float x;
    if (t < 2.0f) { code = (uint32_t)f2; x = t2 - f2; }
    else if (t < 4.0f) { code = (uint32_t)f1 + 2u; x = t - f1; }
    else if (t < 6.0f) { code = 6u; x = (t - 4.0f) * 0.5f; }
    else { code = 7u; x = 0.0f; }
    code += x * 65536.0f > (float)u + 0.5f ? 1u : 0u;
    o |= (code | ((b >> 12) & 8u)) << (4 * i);
  }
  return o;
}

// 2^(code-127) as an fp32 (2^-127 is the subnormal 0x00400000).
__device__ __forceinline__ float e8m0_to_f32(uint32_t code) {
  return __uint_as_float(code ? (code << 23) : 0x00400000u);
}

// tanh-approximated GELU, 0.5 z (1 + tanh(u)) with u = c0 (z + c1 z^3), and
// its derivative, in fp32.  With e = exp(-2u) = 2^(z (a + b z^2)),
// a = -2 c0 log2(e), b = a c1, and r = 1 / (1 + e) = 0.5 (1 + tanh u):
//   GELU(z)  = z r,
//   GELU'(z) = r + z r (1 - r) (2 c0 + 6 c0 c1 z^2)      (1 - tanh(u)^2 = 4 r (1 - r)).
// For very negative z, e overflows to +inf and r is 0: GELU(z) = -0 and
// GELU'(z) = 0, where the exact values are below 2^-120 in magnitude.
constexpr float kGeluA = -2.302208198e+00f;   // -2 sqrt(2/pi) log2(e)
constexpr float kGeluB = -1.029432396e-01f;   // kGeluA * 0.044715
constexpr float kGeluG1 = 1.595769122e+00f;  // 2 sqrt(2/pi)
constexpr float kGeluG3 = 2.140644488e-01f;  // 6 sqrt(2/pi) 0.044715
__device__ __forceinline__ float gelu_tanh(float z) {
  const float e = __builtin_amdgcn_exp2f(z * fmaf(kGeluB, z * z, kGeluA));
  return z * __builtin_amdgcn_rcpf(1.0f + e);   // hardware reciprocal (1 ulp)
}
__device__ __forceinline__ float gelu_tanh_grad(float z) {
  const float t = z * z;
  const float e = __builtin_amdgcn_exp2f(z * fmaf(kGeluB, t, kGeluA));
  const float r = __builtin_amdgcn_rcpf(1.0f + e);
  return fmaf(z * fmaf(kGeluG3, t, kGeluG1) * (1.0f - r), r, r);
}

// Quantize 8 consecutive bf16 (packed in w) of a 32-element block held by a
// lane quad: the block absmax is reduced across the quad with DPP.  Returns
// the 8 E2M1 codes (element 0 in the low nibble) and the block's E8M0 code.
__device__ __forceinline__ uint32_t quad_quantize8(const uint32_t (&w)[4], uint32_t& scale_code) {
  uint32_t m = 0;
#pragma unroll
  for (int e = 0; e < 4; e++) {
    const uint32_t a = w[e] & 0x7FFF7FFFu;
    m = max(m, max(a & 0xFFFFu, a >> 16));
  }
  m = max(m, (uint32_t)__builtin_amdgcn_mov_dpp((int)m, 0xB1, 0xF, 0xF, true));  // quad_perm [1,0,3,2]
  m = max(m, (uint32_t)__builtin_amdgcn_mov_dpp((int)m, 0x4E, 0xF, 0xF, true));  // quad_perm [2,3,0,1]
  scale_code = e8m0_from_amax_bits(m);
  const float s = e8m0_to_f32(scale_code);
  uint32_t o = 0;
  o = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(o, __builtin_bit_cast(v2bf, w[0]), s, 0);
  o = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(o, __builtin_bit_cast(v2bf, w[1]), s, 1);
  o = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(o, __builtin_bit_cast(v2bf, w[2]), s, 2);
  o = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(o, __builtin_bit_cast(v2bf, w[3]), s, 3);
  return o;
}


__device__ __forceinline__ v4s lds_read_tr16(const FT_LDS void* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((FT_LDS v4s*)p);
}

__device__ __forceinline__ v2i lds_read_tr4(const FT_LDS void* p) {
  return __builtin_amdgcn_ds_read_tr4_b64_v2i32((FT_LDS v2i*)p);
}

__device__ __forceinline__ v8bf make_v8bf(v4s a, v4s b) {
  struct { v4s x, y; } t = {a, b};
  return __builtin_bit_cast(v8bf, t);
}

__device__ __forceinline__ v8bf pack_v8bf(const uint32_t (&h)[8]) {
  v4i t;
  t[0] = (int)(h[0] | (h[1] << 16));
  t[1] = (int)(h[2] | (h[3] << 16));
  t[2] = (int)(h[4] | (h[5] << 16));
  t[3] = (int)(h[6] | (h[7] << 16));
  return __builtin_bit_cast(v8bf, t);
}

__device__ __forceinline__ v16f mfma_bf16_32x32x16(v8bf a, v8bf b, v16f c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// FP4 x FP4 block-scaled MFMA.  a, b: 16 packed bytes each (upper half of the
// 8-dword operand unused for FP4).  sa, sb: E8M0 bytes, byte SEL of the word.
template <int SEL>
__device__ __forceinline__ v16f mfma_fp4_32x32x64(v4i a, v4i b, v16f c, int sa, int sb) {
  v8i a8 = {a[0], a[1], a[2], a[3], 0, 0, 0, 0};
  v8i b8 = {b[0], b[1], b[2], b[3], 0, 0, 0, 0};
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a8, b8, c, 4, 4, SEL, sa, SEL, sb);
}

// Raw buffer resource over [base, base + bytes): loads at offsets >= bytes
// return zeros, which handles ragged tiles without branches.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

// An offset no buffer here reaches: a load from it returns zeros.
constexpr uint32_t kOobOffset = 0x80000000u;

// Cache policy of buffer stores whose data no kernel reads soon (GEMM outputs,
// the MLP epilogues' activations and codes): non-temporal, so they stream to
// HBM without displacing operand lines from L2.
constexpr int kStoreNT = 2;

// Buffer resource words for the asm loads below (same layout as make_rsrc).
__device__ __forceinline__ v4i rsrc_words(const void* base, uint32_t bytes) {
  const uint64_t a = (uint64_t)base;
  return v4i{(int)(uint32_t)a, (int)(uint32_t)(a >> 32) & 0xFFFF, (int)bytes, 0x00020000};
}

// LDS byte address of a pointer into a __shared__ array.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const FT_LDS void*)p;
}

// Wait until at most N_ vector memory operations of this wave are outstanding.
template <int N_>
__device__ __forceinline__ void wait_vm() {
  // vmcnt(N_) with expcnt/lgkmcnt left unconstrained (gfx9 encoding)
  __builtin_amdgcn_s_waitcnt((N_ & 15) | ((N_ >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Buffer -> LDS loads issued as inline asm: lane L writes lds_base + 16L (or
// + 4L).  The compiler does not see these as LDS writes, so it never adds
// waits for them; callers publish the data with an explicit vmcnt wait and a
// barrier.  lds_base must be wave-uniform.
// The byte offset is voff (per lane) + soff (uniform); a voff at or beyond the
// buffer size reads zeros whatever soff is.
// The uniform operands pass through readfirstlane: the compiler may hold a
// uniform value in a VGPR, which an "s" asm operand would not convert.
// The LDS destination travels in M0, which the compiler reserves: the asm
// saves M0 in a scratch SGPR and restores it after the load has issued (the
// load reads M0 at issue), so M0 holds the same value before and after the
// statement whatever the compiler keeps there.  An LDS DMA needs one wait
// state after a scalar write of M0.
__device__ __forceinline__ void dma16(v4i rsrc, uint32_t lds_base, uint32_t voff, uint32_t soff) {
  uint32_t keep;
  asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\ts_nop 0\n\t"
               "buffer_load_dwordx4 %2, %3, %4 offen lds\n\ts_mov_b32 m0, %0"
               : "=&s"(keep)
               : "s"(__builtin_amdgcn_readfirstlane(lds_base)), "v"(voff), "s"(rsrc),
                 "s"(__builtin_amdgcn_readfirstlane(soff))
               : "memory");
}
__device__ __forceinline__ void dma4(v4i rsrc, uint32_t lds_base, uint32_t voff, uint32_t soff) {
  uint32_t keep;
  asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\ts_nop 0\n\t"
               "buffer_load_dword %2, %3, %4 offen lds\n\ts_mov_b32 m0, %0"
               : "=&s"(keep)
               : "s"(__builtin_amdgcn_readfirstlane(lds_base)), "v"(voff), "s"(rsrc),
                 "s"(__builtin_amdgcn_readfirstlane(soff))
               : "memory");
}

}  // namespace ft
