// Device-side format codecs shared by the quantizer kernels (qf_quant.hip, qf_lora.hip):
// bit-pattern encoders / decoders of bf16, E2M1, E4M3, E8M0 and FP16, the 16-byte chunk
// (8 bf16 along K) helpers, and the per-chunk quantize-dequantize of each format.  A lane
// owns one chunk; a format block spans B/8 adjacent lanes (NVFP4: 2, MXFP4: 4, Q4_K
// sub-block: 4, Q4_K super-block: 32) whose extremes are reduced with DPP quad permutes and
// ds_swizzle inside the wavefront, so all lanes of a block must call the chunk function
// together.  Arithmetic is integer on the bit patterns wherever a format is defined on bits,
// plus single IEEE FP32 operations for the scale products and quotients (the library is
// built with -ffp-contract=off).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace qf {
namespace codec {

__device__ __forceinline__ float as_f32(uint32_t u) { return __uint_as_float(u); }
__device__ __forceinline__ uint32_t as_u32(float f) { return __float_as_uint(f); }

// ---- cross-lane helpers --------------------------------------------------------------------
// DPP quad permutes: lane ^ 1 and lane ^ 2 inside each group of four lanes.
__device__ __forceinline__ uint32_t xor1_u32(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false);
}
__device__ __forceinline__ uint32_t xor2_u32(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false);
}
// ds_swizzle bit-mask mode inside groups of 32 lanes: lane ^ MASK.
template <int MASK>
__device__ __forceinline__ uint32_t xor_swz_u32(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_ds_swizzle((int)v, (MASK << 10) | 0x1F);
}
__device__ __forceinline__ float xor1_f(float v) { return as_f32(xor1_u32(as_u32(v))); }
__device__ __forceinline__ float xor2_f(float v) { return as_f32(xor2_u32(as_u32(v))); }
template <int MASK>
__device__ __forceinline__ float xor_swz_f(float v) { return as_f32(xor_swz_u32<MASK>(as_u32(v))); }

// ---- format codecs on bit patterns ---------------------------------------------------------
// binary32 -> bfloat16, round to nearest even; NaN -> 0x7FC0.
__device__ __forceinline__ uint32_t bf16_rne(float f) {
  uint32_t u = as_u32(f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0u;
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

// Two binary32 values -> bfloat16 pair (lo in bits 0-15), round to nearest even, with the
// hardware conversion: equal to bf16_rne for every input except NaN (whose sign and payload
// it keeps), so callers use it only on values that cannot be NaN.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t bf16x2_rne_nonnan(float lo, float hi) {
  const f32x2_t v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

// The two E2M1 codes in byte P of w (low nibble first) as signed binary32 values +-V, exact.
template <int P>
__device__ __forceinline__ f32x2_t e2m1_pair(uint32_t w) {
  return __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w, 1.0f, P);
}

// E2M1 magnitude as binary32 (code 0..7).
__device__ __forceinline__ float e2m1_value(uint32_t m) {
  uint32_t b = m >= 2u ? (m + 252u) << 22 : (m == 1u ? 0x3F000000u : 0u);
  return as_f32(b);
}

// OCP E4M3 ("FN", bias 7, max 448) code of t >= 0: round to nearest even, saturating at
// 448 (code 0x7E); NaN -> 0x7F.
// Both candidate codes are formed and one is selected (no branch).
__device__ __forceinline__ uint32_t e4m3_code(float t) {
  const uint32_t sub = (uint32_t)__builtin_rintf(t * 512.0f);     // subnormals m * 2^-9
  const uint32_t u = as_u32(t);
  const uint32_t r = u + 0x7FFFFu + ((u >> 20) & 1u);
  uint32_t c = (r >> 20) - (120u << 3);                              // normals
  c = c < 0x7Eu ? c : 0x7Eu;
  c = t < 0x1p-6f ? sub : c;
  return t < 448.0f ? c : (t != t ? 0x7Fu : 0x7Eu);
}

__device__ __forceinline__ float e4m3_value(uint32_t c) {
  uint32_t e = (c >> 3) & 15u, m = c & 7u;
  if (e == 0u) return (float)m * 0x1p-9f;
  return as_f32(((e + 120u) << 23) | (m << 20));
}

// binary32 -> binary16, round to nearest even, subnormals kept, finite overflow saturating to
// 65504; NaN -> 0x7E00.  The hardware conversion (round to nearest even in the default mode,
// binary16 subnormals kept) on the value clamped to +-65504: every binary32 above 65504 in
// magnitude would round to 65504 or to infinity, and the clamp makes it 65504.  Equal to the
// bit-level rounding for all 2^32 inputs (checked on the GPU).
__device__ __forceinline__ uint32_t f16_rne_sat(float f) {
  const float c = __builtin_fminf(__builtin_fmaxf(f, -65504.0f), 65504.0f);
  const uint32_t h = __builtin_bit_cast(uint16_t, (_Float16)c);
  return f != f ? 0x7E00u : h;
}

// binary16 bits -> binary32 (hardware conversion: exact, subnormals kept, infinity and NaN
// as infinity and NaN).
__device__ __forceinline__ float f16_value(uint32_t h) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)h);
}

// fl(x / C) for x >= 0 (zero, subnormal, normal, infinity or NaN) and C = 15 or 63: the product
// with the rounded reciprocal, its exact residual by FMA and one correcting FMA (the
// Markstein correction, which is correctly rounded here).  Equal to the IEEE quotient for
// every non-negative binary32 input, checked exhaustively for both constants; an infinite
// product is returned as is (the residual would be NaN).
template <int C>
__device__ __forceinline__ float div_nonneg_by(float x) {
  static_assert(C == 15 || C == 63, "checked for 15 and 63 only");
  constexpr float c = (float)C, rc = 1.0f / (float)C;
  const float q0 = x * rc;
  const float r = __builtin_fmaf(-q0, c, x);
  const float q1 = __builtin_fmaf(r, rc, q0);
  return __builtin_isinf(q0) ? q0 : q1;
}

__device__ __forceinline__ uint32_t lo16(uint32_t w) { return w & 0xFFFFu; }
__device__ __forceinline__ uint32_t hi16(uint32_t w) { return w >> 16; }

__device__ __forceinline__ void unpack8(const uint4& v, uint32_t h[8]) {
  h[0] = lo16(v.x); h[1] = hi16(v.x); h[2] = lo16(v.y); h[3] = hi16(v.y);
  h[4] = lo16(v.z); h[5] = hi16(v.z); h[6] = lo16(v.w); h[7] = hi16(v.w);
}
__device__ __forceinline__ uint4 pack8(const uint32_t h[8]) {
  return make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16),
                    h[6] | (h[7] << 16));
}

__device__ __forceinline__ uint32_t max_abs_bits8(const uint32_t h[8]) {
  uint32_t m = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    uint32_t a = h[i] & 0x7FFFu;
    m = a > m ? a : m;
  }
  return m;
}

// ======================================================================= per-chunk codecs
// Each function quantizes and dequantizes this lane's 8 elements h[] (bf16 bits); the lanes
// of one format block must run it together (cross-lane reductions).

// ---- gfx950 FP4 conversions ----------------------------------------------------------------
// v_cvt_scalef32_pk_fp4_{bf16,f32} encode two values as E2M1 codes of x / 2^s (nearest, ties to
// the even code, saturating at 6, sign copied including -0; NaN encodes as magnitude 7), and
// v_cvt_scalef32_pk_bf16_fp4 decodes two codes to bf16(+-V * 2^s); both use only the exponent
// field of the FP32 scale (2^s; field 0 means 2^-127).  These equalities were checked on the
// GPU for every bf16 input and scale exponents -127..127, and the quantizer parity tests pin
// them against the oracle.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float e8m0_scale(uint32_t e) {     // 2^(e - 127), e in 0..254
  return as_f32((e << 23) | 0x00400000u);
}

// Four E2M1 bytes (8 codes, element k in nibble k) of the bf16 words w[0..3] divided by 2^s.
__device__ __forceinline__ uint32_t fp4_encode8(const uint32_t w[4], float scale) {
  uint32_t cw = 0;
  cw = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(cw, __builtin_bit_cast(bf16x2_t, w[0]), scale, 0);
  cw = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(cw, __builtin_bit_cast(bf16x2_t, w[1]), scale, 1);
  cw = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(cw, __builtin_bit_cast(bf16x2_t, w[2]), scale, 2);
  cw = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(cw, __builtin_bit_cast(bf16x2_t, w[3]), scale, 3);
  return cw;
}

// bf16 words (two elements each) of the 8 codes in cw times 2^s.
__device__ __forceinline__ void fp4_decode8(uint32_t cw, float scale, uint32_t w[4]) {
  w[0] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(cw, scale, 0));
  w[1] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(cw, scale, 1));
  w[2] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(cw, scale, 2));
  w[3] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(cw, scale, 3));
}

// ---- decoders of packed codes (Eqs. nvfp4-dequant, mxfp4-dequant, q4k-dequant) ------------
// Each returns the bf16 x_hat of 8 consecutive elements as 4 words (element 2q in the low half
// of word q).  The quantizers below produce their x_hat through the same functions, and the
// packed-operand GEMM prologue and the transposing dequantizer decode with them too, so x_hat
// is bit-identical wherever it is formed.

// NVFP4: 8 codes cw (element k in nibble k: bit 3 sign, bits 0-2 magnitude) of blocks whose
// decode scale is D = fl(S * s_E4M3): x_hat = bf16(fl(+-V * D)).
// For a finite D: V from the hardware E2M1 decode (exact), one FP32 product, the hardware
// round-to-nearest-even pack (|V D| <= 6 D is finite, so the pack rounds as bf16_rne would).
__device__ __forceinline__ void nvfp4_decode8_finite(uint32_t cw, float D, uint32_t w[4]) {
  const f32x2_t v0 = e2m1_pair<0>(cw), v1 = e2m1_pair<1>(cw);
  const f32x2_t v2 = e2m1_pair<2>(cw), v3 = e2m1_pair<3>(cw);
  w[0] = bf16x2_rne_nonnan(v0.x * D, v0.y * D);
  w[1] = bf16x2_rne_nonnan(v1.x * D, v1.y * D);
  w[2] = bf16x2_rne_nonnan(v2.x * D, v2.y * D);
  w[3] = bf16x2_rne_nonnan(v3.x * D, v3.y * D);
}
// D = fl(S * s_E4M3) is finite exactly when the tensor scale S is (s_E4M3 <= 480), so a caller
// holding one S for many blocks may test S once and call nvfp4_decode8_finite.
__device__ __forceinline__ void nvfp4_decode8(uint32_t cw, float D, uint32_t w[4]) {
  if (__builtin_isfinite(D)) {
    nvfp4_decode8_finite(cw, D, w);
  } else {                                  // tensor scale from a non-finite amax
    uint32_t xh[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const float mag = e2m1_value((cw >> (4 * k)) & 7u) * D;
      xh[k] = bf16_rne((cw >> (4 * k + 3)) & 1u ? -mag : mag);
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) w[q] = xh[2 * q] | (xh[2 * q + 1] << 16);
  }
}

// The NVFP4 block decode scale D = fl(S * s_E4M3) of E4M3 code sc under tensor scale S.
__device__ __forceinline__ float nvfp4_block_scale(float S, uint32_t sc) {
  return S * e4m3_value(sc);
}

// MXFP4: 8 codes of a block with E8M0 scale code e: x_hat = +-V * 2^(e - 127); a block whose
// scale code is 0xFF (it held Inf / NaN) decodes to NaN (0x7FC0).
__device__ __forceinline__ void mxfp4_decode8(uint32_t cw, uint32_t e, uint32_t w[4]) {
  fp4_decode8(cw, e8m0_scale(e), w);
  const bool nan = e == 0xFFu;
#pragma unroll
  for (int q = 0; q < 4; ++q) w[q] = nan ? 0x7FC07FC0u : w[q];
}

// Q4_K: 8 unsigned codes q of a sub-block with step t1 = fl(d s6) and offset t2 = fl(dmin m6):
// x_hat = bf16(fl(t1 q - t2)).  t1 q is exact (at most 21 significant bits, far from the FP32
// range limits), so a fused multiply-add rounds t1 q - t2 exactly once, as the separate product
// and difference do.  The codes as FP32 integers 0..15 (qf[k] for element k):
__device__ __forceinline__ void q4k_decode8f(const float qf[8], float t1, float t2,
                                            uint32_t w[4]) {
#pragma unroll
  for (int q = 0; q < 4; ++q)
    w[q] = bf16x2_rne_nonnan(__builtin_fmaf(t1, qf[2 * q], -t2),
                             __builtin_fmaf(t1, qf[2 * q + 1], -t2));
}
// ... and as bytes (element k in byte k % 4 of qw[k / 4]).
__device__ __forceinline__ void q4k_decode8(const uint32_t qw[2], float t1, float t2,
                                           uint32_t w[4]) {
  float qf[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) qf[k] = (float)((qw[k >> 2] >> (8 * (k & 3))) & 0xFFu);
  q4k_decode8f(qf, t1, t2, w);
}

// The block decode scale D = fl(S * s_E4M3) of every E4M3 code under one tensor scale S, with
// its reciprocal fl(1 / D) (0 where D = 0), as the NVFP4 encoder uses them: computed per call
// (Nvfp4Direct), or read from a 128-entry table of all codes (Nvfp4Table) that a workgroup
// fills once with nvfp4_fill_table (same operations, so the same values).
__device__ __forceinline__ f32x2_t nvfp4_scale_pair(float S, uint32_t sc) {
  const float D = nvfp4_block_scale(S, sc);
  return f32x2_t{D, D != 0.0f ? 1.0f / D : 0.0f};
}
struct Nvfp4Direct {
  float S;
  __device__ __forceinline__ f32x2_t operator()(uint32_t sc) const { return nvfp4_scale_pair(S, sc); }
};
struct Nvfp4Table {
  const f32x2_t* tab;                       // 128 entries (codes 0x00..0x7F), LDS
  __device__ __forceinline__ f32x2_t operator()(uint32_t sc) const { return tab[sc]; }
};
// Threads 0..127 of a workgroup each write one entry; the caller synchronizes before use.
__device__ __forceinline__ void nvfp4_fill_table(float S, f32x2_t* tab, int t) {
  if (t < 128) tab[t] = nvfp4_scale_pair(S, (uint32_t)t);
}

// NVFP4 steps for a 16-block held by this lane and lane ^ 1 (both lanes call each step):
// the block's max |x| as bf16 magnitude bits ...
__device__ __forceinline__ uint32_t nvfp4_block_max(const uint32_t h[8]) {
  const uint32_t ab = max_abs_bits8(h);
  const uint32_t o = xor1_u32(ab);         // partner lane holds the other 8 of the 16-block
  return o > ab ? o : ab;
}
// ... its E4M3 scale code from t_b = a_b / (6 S) (S is the FP32 tensor scale g / (6 * 448),
// six_s = 6 S; S = 0 gives code 0) ...
__device__ __forceinline__ uint32_t nvfp4_scale_code(uint32_t ab, float S, float six_s) {
  return S != 0.0f ? e4m3_code(as_f32(ab << 16) / six_s) : 0u;
}
// ... and the 4-bit codes cw (element k in nibble k) and x_hat bits xh of this lane's 8
// elements h under scale code sc, with bs(sc) giving the block's (D, 1 / D).
template <class BlockScale>
__device__ __forceinline__ void nvfp4_encode(const uint32_t h[8], uint32_t ab, uint32_t sc,
                                             const BlockScale& bs, uint32_t& cw, uint32_t xh[8]) {
  const f32x2_t dr = bs(sc);
  const float D = dr.x, rcp = dr.y;         // block decode scale s_FP32 * s_E4M3,b, 1 / D
  const uint32_t w[4] = {h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16),
                         h[6] | (h[7] << 16)};
  uint32_t p[4];
  if (ab < 0x7F80u && __builtin_isfinite(rcp) && __builtin_isfinite(D)) {
    // A finite block under a finite reciprocal (0 when D = 0): fl(x * rcp) is the signed
    // fl(|x| * rcp) (-0 for x = -0), and the conversion copies the sign bit, so each code is
    // the sign of x over the magnitude code of fl(|x| * rcp), as defined.
    uint32_t c = 0;
    c = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c, as_f32(w[0] << 16) * rcp,
                                                 as_f32(w[0] & 0xFFFF0000u) * rcp, 1.0f, 0);
    c = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c, as_f32(w[1] << 16) * rcp,
                                                 as_f32(w[1] & 0xFFFF0000u) * rcp, 1.0f, 1);
    c = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c, as_f32(w[2] << 16) * rcp,
                                                 as_f32(w[2] & 0xFFFF0000u) * rcp, 1.0f, 2);
    c = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c, as_f32(w[3] << 16) * rcp,
                                                 as_f32(w[3] & 0xFFFF0000u) * rcp, 1.0f, 3);
    cw = c;
    nvfp4_decode8_finite(cw, D, p);
  } else {
    // magnitude codes of fl(|x| * rcp) (scale 2^0), then the sign bit of each input; D = 0
    // gives magnitude 0 for every element (also for Inf / NaN inputs under a caller's g = 0).
    // A NaN product (a NaN input, or 0 * Inf where fl(1 / D) overflows for a D below 2^-128)
    // encodes magnitude 0: no E2M1 value is nearest to it (the conversion would give 7).
    uint32_t mc = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      float v0 = as_f32((h[2 * q] & 0x7FFFu) << 16) * rcp;
      float v1 = as_f32((h[2 * q + 1] & 0x7FFFu) << 16) * rcp;
      v0 = v0 != v0 ? 0.0f : v0;
      v1 = v1 != v1 ? 0.0f : v1;
      const uint32_t c2 = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(0u, v0, v1, 1.0f, 0);
      mc |= (c2 & 0xFFu) << (8 * q);
    }
    if (D == 0.0f) mc = 0;
    cw = mc;                                // magnitudes leave bit 3 of each nibble clear
#pragma unroll
    for (int k = 0; k < 8; ++k) cw |= (h[k] >> 15) << (4 * k + 3);
    nvfp4_decode8(cw, D, p);
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    xh[2 * q] = p[q] & 0xFFFFu;
    xh[2 * q + 1] = p[q] >> 16;
  }
}

// NVFP4 of one chunk: codes cw, E4M3 block scale sc, x_hat bits xh.
template <class BlockScale>
__device__ __forceinline__ void nvfp4_chunk(const uint32_t h[8], float S, float six_s,
                                            const BlockScale& bs, uint32_t& cw, uint32_t& sc,
                                            uint32_t xh[8]) {
  const uint32_t ab = nvfp4_block_max(h);
  sc = nvfp4_scale_code(ab, S, six_s);
  nvfp4_encode(h, ab, sc, bs, cw, xh);
}
__device__ __forceinline__ void nvfp4_chunk(const uint32_t h[8], float S, float six_s,
                                            uint32_t& cw, uint32_t& sc, uint32_t xh[8]) {
  nvfp4_chunk(h, S, six_s, Nvfp4Direct{S}, cw, sc, xh);
}

// MXFP4 (32-block = the 4 lanes of a quad): codes cw, E8M0 scale code e (0xFF for a block
// holding Inf / NaN, whose x_hat is NaN and codes 0), x_hat bits xh.
__device__ __forceinline__ void mxfp4_chunk(const uint32_t h[8], uint32_t& cw, uint32_t& scale,
                                            uint32_t xh[8]) {
  uint32_t ab = max_abs_bits8(h);
  uint32_t o = xor1_u32(ab);
  ab = o > ab ? o : ab;
  o = xor2_u32(ab);
  ab = o > ab ? o : ab;                     // max |x| of the 32-block (4 lanes)
  const bool nonfinite = ab >= 0x7F80u;     // Inf or NaN somewhere in the block
  const uint32_t E = ab >> 7;               // biased exponent of the block max
  const uint32_t e = E >= 2u ? E - 2u : 0u; // scale code: floor(log2 a) - 2, clamped
  const float sc = e8m0_scale(e);
  const uint32_t w[4] = {h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16),
                         h[6] | (h[7] << 16)};
  cw = fp4_encode8(w, sc);                  // nearest E2M1 of x / 2^(e - 127)
  scale = e;
  if (nonfinite) {
    cw = 0;
    scale = 0xFFu;
  }
  uint32_t d[4];
  mxfp4_decode8(cw, scale, d);              // x_hat = +-V * 2^(e - 127), or NaN
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    xh[2 * p] = d[p] & 0xFFFFu;
    xh[2 * p + 1] = d[p] >> 16;
  }
}

// Q4_K (32 lanes per 256-element super-block; lane L holds elements 8L..8L+7, sub-block L/4):
// FP16 bits of d and dmin, this sub-block's 6-bit scale / min, the 4-bit codes of this
// lane (qlo: elements 0-3, qhi: 4-7, one per byte) and x_hat bits xh.
struct Q4kChunk {
  uint32_t dh, mh, ls, lm, qlo, qhi;
};

// Q4_K element codes q[k] = min(max(rint(fl(a[k] / t)), 0), 15) for a normal t > 0, as FP32
// integers.  With rt = 1 / t from v_rcp_f32 (within 1 ulp), y = fl(a rt) is within
// 2.4e-7 |a / t| of fl(a / t): within 4e-6 for |a / t| <= 16, and further out both clamp
// alike, so whenever y lies more than 1e-5 from a half-integer both round to the same integer.
// A chunk with any element closer than that takes the exact quotients for all eight (y - rint y
// is exact, so |y - rint y| >= 0.49999 is the test; a NaN or infinite y fails it and clamps as
// the exact quotient does).
__device__ __forceinline__ void q4_codes8(const float a[8], float t, float q[8]) {
  const float rt = __builtin_amdgcn_rcpf(t);
  float dm = 0.0f;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const float y = a[k] * rt;
    const float n = __builtin_rintf(y);
    dm = fmaxf(dm, __builtin_fabsf(y - n));     // a NaN distance is dropped
    q[k] = fminf(fmaxf(n, 0.0f), 15.0f);
  }
  if (dm >= 0.49999f) {
#pragma unroll
    for (int k = 0; k < 8; ++k) q[k] = fminf(fmaxf(__builtin_rintf(a[k] / t), 0.0f), 15.0f);
  }
}

// Four codes held as FP32 integers 0..15 -> one byte each (element k in byte k).
__device__ __forceinline__ uint32_t q4_bytes4(const float q[4]) {
  uint32_t w = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) w = __builtin_amdgcn_cvt_pk_u8_f32(q[k], k, w);
  return w;
}

// Q4_K 6-bit sub-block code min(max(rint(fl(a / t)), 0), 63) for a normal t > 0: as above,
// y = fl(a * v_rcp(t)) is within 1.6e-5 of fl(a / t) for |a / t| <= 64, so a margin of 1e-4
// around half-integers decides; closer, the exact quotient.  The exact quotient sits behind a
// wavefront-uniform test, so it costs nothing unless some lane needs it.
__device__ __forceinline__ uint32_t q6_code(float a, float t) {
  float y = a * __builtin_amdgcn_rcpf(t);
  const bool near = !(__builtin_fabsf(__builtin_amdgcn_fractf(y) - 0.5f) > 1e-4f);
  if (__builtin_amdgcn_ballot_w64(near) != 0) {
    const float e = a / t;
    y = near ? e : y;
  }
  return (uint32_t)fminf(fmaxf(__builtin_rintf(y), 0.0f), 63.0f);
}

__device__ __forceinline__ void q4k_chunk(const uint32_t h[8], Q4kChunk& r, uint32_t xh[8]) {
  float xv[8];
  float lo = 0.0f, hi = -__builtin_huge_valf();
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    xv[k] = as_f32(h[k] << 16);
    lo = fminf(lo, xv[k]);
    hi = fmaxf(hi, xv[k]);
  }
  lo = fminf(lo, xor1_f(lo)); hi = fmaxf(hi, xor1_f(hi));
  lo = fminf(lo, xor2_f(lo)); hi = fmaxf(hi, xor2_f(hi));
  lo = lo + 0.0f;                           // signed zeros count as +0 (the extremes only:
  hi = hi + 0.0f;                           // x + t2 below treats -0 as +0 by itself)
  const float a = div_nonneg_by<15>(hi - lo);   // step of the sub-block, fl((hi - lo) / 15)
  const float mu = 0.0f - lo;               // offset (subtracted), never negative
  float A = a, Mx = mu;
  A = fmaxf(A, xor_swz_f<4>(A)); Mx = fmaxf(Mx, xor_swz_f<4>(Mx));
  A = fmaxf(A, xor_swz_f<8>(A)); Mx = fmaxf(Mx, xor_swz_f<8>(Mx));
  A = fmaxf(A, xor_swz_f<16>(A)); Mx = fmaxf(Mx, xor_swz_f<16>(Mx));
  r.dh = f16_rne_sat(div_nonneg_by<63>(A));
  r.mh = f16_rne_sat(div_nonneg_by<63>(Mx));
  const float d = f16_value(r.dh), dmin = f16_value(r.mh);
  r.ls = 0;
  r.lm = 0;
  if (d != 0.0f) r.ls = q6_code(a, d);
  if (dmin != 0.0f) r.lm = q6_code(mu, dmin);
  const float t1 = d * (float)r.ls;
  const float t2 = dmin * (float)r.lm;  // >= +0, so x + t2 is +0 for x = -0 and t2 = 0
  float qv[8] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
  if (t1 != 0.0f) {
    float av[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) av[k] = xv[k] + t2;
    q4_codes8(av, t1, qv);
  }
  r.qlo = q4_bytes4(qv);
  r.qhi = q4_bytes4(qv + 4);
  // t1 q - t2 is finite for every input (t1, t2 come from FP16 scales), so the hardware pack
  // rounds it exactly as bf16_rne would
  uint32_t p[4];
  q4k_decode8f(qv, t1, t2, p);
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    xh[2 * k] = p[k] & 0xFFFFu;
    xh[2 * k + 1] = p[k] >> 16;
  }
}


// ---- Q4_K, sixteen elements per lane ---------------------------------------------------------
// The row quantizer's form: lane L of a group of 16 holds elements 16 L .. 16 L + 15 of a
// super-block (sub-block L / 2, its half L % 2), so a sub-block's extremes take one lane
// exchange and the per-sub-block work (step, offset, 6-bit codes, FP16 scales, block header) is
// shared by twice as many elements as in q4k_chunk.  Every value comes from the same operations
// as there (minima and maxima do not depend on the order of their reductions), so the codes,
// scales and x_hat are the same bits.
// DPP row mirrors: lane i <-> 7 - i inside each 8 lanes, 15 - i inside each 16.
__device__ __forceinline__ uint32_t half_mirror_u32(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xF, 0xF, false);
}
__device__ __forceinline__ uint32_t mirror_u32(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x140, 0xF, 0xF, false);
}
// Maximum over a group of 16 lanes of a value that lanes 2j and 2j + 1 hold alike: quads by
// lane ^ 2, then the two quads of each 8 by the half mirror, then the two 8s by the mirror.
__device__ __forceinline__ float max16_pairs(float v) {
  v = fmaxf(v, as_f32(xor2_u32(as_u32(v))));
  v = fmaxf(v, as_f32(half_mirror_u32(as_u32(v))));
  return fmaxf(v, as_f32(mirror_u32(as_u32(v))));
}

struct Q4kChunk16 {
  uint32_t dh, mh, ls, lm, q[4];            // q: the 16 codes, element k in byte k % 4 of q[k / 4]
};

// h: the lane's 16 bf16 inputs; xw: x_hat as 8 words of bf16 pairs (element 2i in the low half).
__device__ __forceinline__ void q4k_chunk16(const uint32_t h[16], Q4kChunk16& r, uint32_t xw[8]) {
  float xv[16];
  float lo = 0.0f, hi = -__builtin_huge_valf();
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    xv[k] = as_f32(h[k] << 16);
    lo = fminf(lo, xv[k]);
    hi = fmaxf(hi, xv[k]);
  }
  lo = fminf(lo, xor1_f(lo)); hi = fmaxf(hi, xor1_f(hi));
  lo = lo + 0.0f;                           // signed zeros count as +0 (as in q4k_chunk)
  hi = hi + 0.0f;
  const float a = div_nonneg_by<15>(hi - lo);   // step of the sub-block, fl((hi - lo) / 15)
  const float mu = 0.0f - lo;               // offset (subtracted), never negative
  const float A = max16_pairs(a), Mx = max16_pairs(mu);
  r.dh = f16_rne_sat(div_nonneg_by<63>(A));
  r.mh = f16_rne_sat(div_nonneg_by<63>(Mx));
  const float d = f16_value(r.dh), dmin = f16_value(r.mh);
  r.ls = 0;
  r.lm = 0;
  if (d != 0.0f) r.ls = q6_code(a, d);
  if (dmin != 0.0f) r.lm = q6_code(mu, dmin);
  const float t1 = d * (float)r.ls;
  const float t2 = dmin * (float)r.lm;
  float qv[16];
#pragma unroll
  for (int k = 0; k < 16; ++k) qv[k] = 0.0f;
  if (t1 != 0.0f) {
    float av[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) av[k] = xv[k] + t2;
    q4_codes8(av, t1, qv);
    q4_codes8(av + 8, t1, qv + 8);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) r.q[i] = q4_bytes4(qv + 4 * i);
  q4k_decode8f(qv, t1, t2, xw);
  q4k_decode8f(qv + 8, t1, t2, xw + 4);
}

// Packs the super-block held by 16 lanes (lane L: sub-block L / 2, half L % 2) into its 144-byte
// block at blk, in the layout q4k_store writes.  Every lane of the group must call it
// (cross-lane moves); `store` predicates the writes.
__device__ __forceinline__ void q4k_store16(const Q4kChunk16& q, int L, bool store, uint8_t* blk) {
  // Lane 2j holds sub-block j's scale and min.  Bytes j and 4 + j come together at lane 2j,
  // pairs of them at lanes 0 and 4 (lane ^ 2), all eight at lane 0 (lane ^ 4); bytes 8 + j
  // start at lane 8 + 2j and meet at lane 8, then lane 0.
  const uint32_t own = q.ls | (q.lm << 16);
  const uint32_t up = xor_swz_u32<8>(own);                   // scale, min of sub-block j + 4
  const uint32_t v = (own & 0x003F003Fu) | (((up >> 4) & 0x00030003u) << 6);  // bytes j, 4+j
  const uint32_t v2 = xor2_u32(v);
  const uint32_t pv = (v & 0x00FF00FFu) | ((v2 & 0x00FF00FFu) << 8);  // lane 0: b0 b1 b4 b5
  const uint32_t pv4 = xor_swz_u32<4>(pv);                   // lane 0: b2 b3 b6 b7
  const uint32_t w0 = (q.ls & 15u) | ((q.lm & 15u) << 4);    // lane 8 + 2j: byte 8 + j
  const uint32_t pw = w0 | (xor2_u32(w0) << 8);              // lane 8: b8 b9, lane 12: b10 b11
  const uint32_t pw4 = xor_swz_u32<4>(pw);
  const uint32_t sw = xor_swz_u32<8>(pw | (pw4 << 16));      // lane 0: b8 b9 b10 b11
  // codes of the odd sub-block (lane L ^ 2) go to the high nibbles of the even one's bytes
  uint32_t pq[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) pq[i] = xor2_u32(q.q[i]);
  if (!store) return;
  if (L == 0)
    *reinterpret_cast<uint4*>(blk) =
        make_uint4(q.dh | (q.mh << 16), (pv & 0xFFFFu) | (pv4 << 16),
                   (pv >> 16) | (pv4 & 0xFFFF0000u), sw);
  if ((L & 2) == 0)
    *reinterpret_cast<uint4*>(blk + 16 + 32 * (L >> 2) + 16 * (L & 1)) =
        make_uint4(q.q[0] | (pq[0] << 4), q.q[1] | (pq[1] << 4), q.q[2] | (pq[2] << 4),
                   q.q[3] | (pq[3] << 4));
}

// ---- Q4_K with searched sub-block steps ------------------------------------------------------
// Sums over a 32-element sub-block in one fixed order: this lane's 8 elements from +0 in
// index order, then the quad tree (g0 + g1) + (g2 + g3) (lane ^ 1, then lane ^ 2; the same
// value lands on all four lanes since each step adds a commutative pair).
__device__ __forceinline__ float sub_sum(const float f[8]) {
  float s = 0.0f;
#pragma unroll
  for (int k = 0; k < 8; ++k) s += f[k];
  s = s + xor1_f(s);
  return s + xor2_f(s);
}
// Super-block total of per-sub-block sums (lane L holds sub-block L / 4):
// ((s0 + s1) + (s2 + s3)) + ((s4 + s5) + (s6 + s7)).
__device__ __forceinline__ float super_sum(float s) {
  s = s + xor_swz_f<4>(s);
  s = s + xor_swz_f<8>(s);
  return s + xor_swz_f<16>(s);
}

// The final stage shared by both candidates of a super-block: 6-bit scale / min quantization
// of (a, mu), codes of the min-max reading's last step, FP32 decode t1 C - t2 and the
// super-block's squared-error sum.
__device__ __forceinline__ float q4k_finish(const float xv[8], float a, float mu, Q4kChunk& r,
                                            float xf[8]) {
  float A = a, Mx = mu;
  A = fmaxf(A, xor_swz_f<4>(A)); Mx = fmaxf(Mx, xor_swz_f<4>(Mx));
  A = fmaxf(A, xor_swz_f<8>(A)); Mx = fmaxf(Mx, xor_swz_f<8>(Mx));
  A = fmaxf(A, xor_swz_f<16>(A)); Mx = fmaxf(Mx, xor_swz_f<16>(Mx));
  r.dh = f16_rne_sat(div_nonneg_by<63>(A));
  r.mh = f16_rne_sat(div_nonneg_by<63>(Mx));
  const float d = f16_value(r.dh), dmin = f16_value(r.mh);
  r.ls = 0;
  r.lm = 0;
  if (d != 0.0f) r.ls = q6_code(a, d);
  if (dmin != 0.0f) r.lm = q6_code(mu, dmin);
  const float t1 = d * (float)r.ls;
  const float t2 = dmin * (float)r.lm;
  float e2[8];
  float qv[8] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
  if (t1 != 0.0f) {
    float av[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) av[k] = xv[k] + t2;
    q4_codes8(av, t1, qv);
  }
  r.qlo = q4_bytes4(qv);
  r.qhi = q4_bytes4(qv + 4);
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    xf[k] = t1 * qv[k] - t2;
    const float e = xv[k] - xf[k];
    e2[k] = e * e;
  }
  return super_sum(sub_sum(e2));
}

// Q4_K whose sub-block (step, offset) come from a search of ||x - x_hat||^2: anchors lo =
// min(0, min x), hi = max x, mu0 = -lo; candidate k = 0..16 quantizes with the step
// (hi - lo) / (14 + k/4), refits step and offset to those codes by least squares (offset
// constrained to >= 0; a degenerate or non-positive refit keeps the candidate), and the
// candidate with the smallest error sum wins (the first on ties).  The super-block then keeps
// the searched steps or the min-max ones (q4k_chunk), whichever gives the smaller final error.
__device__ __forceinline__ void q4k_mse_chunk(const uint32_t h[8], Q4kChunk& r, uint32_t xh[8]) {
  float xv[8];
  float lo = 0.0f, hi = -__builtin_huge_valf();
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    xv[k] = as_f32(h[k] << 16) + 0.0f;      // signed zeros count as +0
    lo = fminf(lo, xv[k]);
    hi = fmaxf(hi, xv[k]);
  }
  lo = fminf(lo, xor1_f(lo)); hi = fmaxf(hi, xor1_f(hi));
  lo = fminf(lo, xor2_f(lo)); hi = fmaxf(hi, xor2_f(hi));
  const float range = hi - lo, mu0 = 0.0f - lo;
  const float sx = sub_sum(xv);
  float best_e = __builtin_huge_valf(), best_a = div_nonneg_by<15>(range), best_mu = mu0;
#pragma unroll 1
  for (int k = 0; k <= 16; ++k) {
    const float Dk = 14.0f + 0.25f * (float)k;
    const float ak = range / Dk;
    float q[8], ac = ak, mc = mu0;
    if (ak == 0.0f) {
#pragma unroll
      for (int i = 0; i < 8; ++i) q[i] = 0.0f;
    } else {
      const float rc = 1.0f / ak;
      float qq[8], qx[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        q[i] = fminf(fmaxf(__builtin_rintf((xv[i] + mu0) * rc), 0.0f), 15.0f);
        qq[i] = q[i] * q[i];
        qx[i] = q[i] * xv[i];
      }
      const float sq = sub_sum(q), sqq = sub_sum(qq), sqx = sub_sum(qx);
      const float den = 32.0f * sqq - sq * sq;
      if (den > 0.0f) {
        ac = (32.0f * sqx - sq * sx) / den;
        mc = (ac * sq - sx) / 32.0f;
        if (mc < 0.0f) {
          mc = 0.0f;
          ac = sqx / sqq;
        }
        if (!(ac > 0.0f)) {
          ac = ak;
          mc = mu0;
        }
      }
    }
    float e2[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float e = xv[i] - (ac * q[i] - mc);
      e2[i] = e * e;
    }
    const float err = sub_sum(e2);
    if (err < best_e) {
      best_e = err;
      best_a = ac;
      best_mu = mc;
    }
  }
  Q4kChunk rs, rm;
  float xs[8], xm[8];
  const float es = q4k_finish(xv, best_a, best_mu, rs, xs);
  const float em = q4k_finish(xv, div_nonneg_by<15>(range), mu0, rm, xm);
  const bool use_s = es < em;
  r = use_s ? rs : rm;
#pragma unroll
  for (int k = 0; k < 8; ++k) xh[k] = bf16_rne(use_s ? xs[k] : xm[k]);
}

// Packs one Q4_K super-block held by the 32 lanes of a half-wave (lane L = this lane's index
// inside the super-block, elements 8L..8L+7) into the 144-byte llama.cpp block at blk: FP16 d
// and dmin, twelve bytes of 6-bit scales / mins, then 128 bytes of codes (sub-block 2p in the
// low nibbles of bytes 16 + 32p.., sub-block 2p+1 in the high nibbles).  Every lane of the
// half-wave must call it (cross-lane moves); `store` predicates the writes.
__device__ __forceinline__ void q4k_store(const Q4kChunk& q, int L, bool store, uint8_t* blk) {
  // The twelve scale bytes: byte j (j < 4) = low 6 bits of scale j | top 2 bits of scale j + 4
  // << 6, byte 4 + j the same for the mins, byte 8 + j = low nibble of scale j + 4 | low
  // nibble of min j + 4 << 4.  Lane 4j of the half-wave holds sub-block j's scale and min.
  // Every lane computes both forms; swizzles inside the half-wave bring lanes 0, 4, 8, 12
  // (bytes j, 4 + j) and 16, 20, 24, 28 (bytes 8 + j) together at lane 0.
  const uint32_t own = q.ls | (q.lm << 16);
  const uint32_t up = xor_swz_u32<16>(own);                  // scale, min of sub-block j + 4
  const uint32_t v = (own & 0x003F003Fu) | (((up >> 4) & 0x00030003u) << 6);  // bytes j, 4+j
  const uint32_t v4 = xor_swz_u32<4>(v);
  const uint32_t pv = (v & 0x00FF00FFu) | ((v4 & 0x00FF00FFu) << 8);  // lane 0: b0 b1 b4 b5
  const uint32_t pv8 = xor_swz_u32<8>(pv);                   // lane 0: b2 b3 b6 b7
  const uint32_t w0 = (q.ls & 15u) | ((q.lm & 15u) << 4);    // lane 16 + 4j: byte 8 + j
  const uint32_t w4 = xor_swz_u32<4>(w0);
  const uint32_t pw = w0 | (w4 << 8);
  const uint32_t pw8 = xor_swz_u32<8>(pw);
  const uint32_t sw = xor_swz_u32<16>(pw | (pw8 << 16));     // lane 0: b8 b9 b10 b11
  // codes of sub-block j+1 (odd) go to the high nibbles of sub-block j's bytes
  const uint32_t plo = xor_swz_u32<4>(q.qlo);
  const uint32_t phi = xor_swz_u32<4>(q.qhi);
  if (!store) return;
  if (L == 0)
    *reinterpret_cast<uint4*>(blk) =
        make_uint4(q.dh | (q.mh << 16), (pv & 0xFFFFu) | (pv8 << 16),
                   (pv >> 16) | (pv8 & 0xFFFF0000u), sw);
  const int sub = L >> 2;
  if ((sub & 1) == 0) {
    const int off = 16 + 32 * (sub >> 1) + 8 * (L & 3);
    *reinterpret_cast<uint2*>(blk + off) = make_uint2(q.qlo | (plo << 4), q.qhi | (phi << 4));
  }
}

// ---- 64 x 256 tiles with transposed output ---------------------------------------------------
// A workgroup of 256 lanes quantizes a 64-row x 256-column tile: lane t owns chunk t % 32 of
// rows 8 i + t / 32 (i = 0..7), so each half-wave holds one 256-element row segment and every
// format block (the Q4_K super-block included) stays inside one half-wave.  For transposed
// output the lanes park x_hat chunks in LDS (chunk c of row r at slot c ^ (((r >> 3) & 7) << 1),
// which spreads both the row writes and the 8 x 8 block reads over the banks), then each lane
// transposes an 8 x 8 block in registers and writes 8 output rows of 16 bytes.
constexpr int kTR = 64, kTC = 256;

__device__ __forceinline__ int tslot(int r, int c) { return c ^ (((r >> 3) & 7) << 1); }

// Output row j (0..7) of the transposed 8 x 8 block of 16-bit values whose input row i is
// w[i] (element 2q + h in half h of word q): word d holds input rows 2d and 2d + 1.
__device__ __forceinline__ uint4 block_row_transposed(const uint32_t w[8][4], int j) {
  uint32_t o[4];
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    const uint32_t lo = w[2 * d][j >> 1], hi = w[2 * d + 1][j >> 1];
    o[d] = __builtin_amdgcn_perm(hi, lo, (j & 1) ? 0x07060302u : 0x05040100u);
  }
  return make_uint4(o[0], o[1], o[2], o[3]);
}

// out[c0 + k][oc0 + r] = tile(r, k) for the 64 x 256 tile in LDS (after a barrier); output rows
// at or past K and output columns at or past col_end are skipped (both multiples of 8).
__device__ __forceinline__ void store_tile_transposed(const uint4* tile, int t, uint16_t* out,
                                                      int64_t ldo, int64_t c0, int64_t oc0,
                                                      int64_t K, int64_t col_end) {
  const int rb = t & 7, cb = t >> 3;
  uint32_t w[8][4];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int row = rb * 8 + i;
    const uint4 v = tile[row * 32 + tslot(row, cb)];
    w[i][0] = v.x; w[i][1] = v.y; w[i][2] = v.z; w[i][3] = v.w;
  }
  const int64_t orow0 = c0 + cb * 8, ocol = oc0 + rb * 8;
  if (ocol >= col_end) return;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    if (orow0 + j >= K) break;
    *reinterpret_cast<uint4*>(out + (orow0 + j) * ldo + ocol) = block_row_transposed(w, j);
  }
}

// Tile origin of the grouped transposes (64-row tiles, grid.y = y): expert e's rows
// [off[e], off[e+1]) go to the 64-aligned output columns starting at 64 kstart[e], so tile y
// reads input rows [r0, r_end) and writes output columns from oc0 (the columns past the
// expert's last row as zeros).  False for the tiles past the last expert's (uniform per block).
__device__ __forceinline__ bool grouped_tile(int y, const int64_t* off, const int* kstart, int E,
                                             int64_t& r0, int64_t& r_end, int64_t& oc0) {
  if (y >= kstart[E]) return false;
  int lo = 0, hi = E;                            // kstart[e] <= y < kstart[e+1]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (kstart[mid] <= y) lo = mid; else hi = mid;
  }
  r0 = off[lo] + (int64_t)(y - kstart[lo]) * kTR;
  r_end = off[lo + 1];
  oc0 = (int64_t)y * kTR;
  return true;
}

}  // namespace codec
}  // namespace qf
