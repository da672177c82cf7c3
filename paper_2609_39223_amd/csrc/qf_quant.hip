// Fake-quantization kernels for gfx950: tensor amax, NVFP4, MXFP4 and Q4_K.
//
// Work layout shared by the quantizers: one lane owns one 16-byte chunk (8 bf16 along K),
// loaded with a single 128-bit load.  A format block of B elements spans B/8 adjacent
// lanes (NVFP4: 2, MXFP4: 4, Q4_K sub-block: 4, Q4_K super-block: 32), so block extremes
// are reduced with DPP quad permutes / ds_swizzle inside the wavefront, never through LDS.
// A workgroup of 256 lanes covers 256 consecutive chunks of one row; blockIdx.y walks
// groups of rows.  Every lane stays active through the cross-lane steps (loads and stores
// are predicated), so partial tiles never read a disabled lane.
//
// Arithmetic is integer on the bit patterns wherever the formats are defined on bits
// (exponent extraction, E4M3 / E2M1 / FP16 / BF16 round-to-nearest-even), plus single IEEE
// FP32 operations where the scale arithmetic is a product or quotient.  The library is
// compiled with -ffp-contract=off, so no step is fused into an FMA.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "qf.h"
#include "qf_internal.h"

namespace qf {
namespace {

constexpr int kThreads = 256;

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

// E2M1 magnitude code of v >= 0 (finite or +inf): nearest of {0,.5,1,1.5,2,3,4,6}, ties to
// the even code, saturating at 6.  Below 1 the spacing is 0.5 (round 2v); from 1 up the
// value has one fraction bit, so round the binary32 fraction to 1 bit on the bit pattern.
__device__ __forceinline__ uint32_t e2m1_code(float v) {
  if (v < 1.0f) return (uint32_t)__builtin_rintf(v * 2.0f);
  uint32_t u = as_u32(v);
  uint32_t r = u + 0x1FFFFFu + ((u >> 22) & 1u);
  uint32_t m = (r >> 22) - 252u;          // (biased exp 127,128,129) x 2 + fraction bit - 252
  return m < 7u ? m : 7u;
}

// E2M1 magnitude as binary32 (code 0..7).
__device__ __forceinline__ float e2m1_value(uint32_t m) {
  uint32_t b = m >= 2u ? (m + 252u) << 22 : (m == 1u ? 0x3F000000u : 0u);
  return as_f32(b);
}

// OCP E4M3 ("FN", bias 7, max 448) code of t >= 0: round to nearest even, saturating at
// 448 (code 0x7E); NaN -> 0x7F.
__device__ __forceinline__ uint32_t e4m3_code(float t) {
  if (!(t < 448.0f)) return t != t ? 0x7Fu : 0x7Eu;
  if (t < 0x1p-6f) return (uint32_t)__builtin_rintf(t * 512.0f);   // subnormals m * 2^-9
  uint32_t u = as_u32(t);
  uint32_t r = u + 0x7FFFFu + ((u >> 20) & 1u);
  uint32_t c = (r >> 20) - (120u << 3);
  return c < 0x7Eu ? c : 0x7Eu;
}

__device__ __forceinline__ float e4m3_value(uint32_t c) {
  uint32_t e = (c >> 3) & 15u, m = c & 7u;
  if (e == 0u) return (float)m * 0x1p-9f;
  return as_f32(((e + 120u) << 23) | (m << 20));
}

// binary32 -> binary16, round to nearest even, subnormals kept, finite overflow saturating to
// 65504; NaN -> 0x7E00.
__device__ __forceinline__ uint32_t f16_rne_sat(float f) {
  uint32_t u = as_u32(f);
  uint32_t s = (u >> 16) & 0x8000u;
  uint32_t a = u & 0x7FFFFFFFu;
  if (a > 0x7F800000u) return 0x7E00u;
  float af = as_f32(a);
  if (af >= 65504.0f) return s | 0x7BFFu;
  if (af < 0x1p-14f) return s | (uint32_t)__builtin_rintf(af * 16777216.0f);
  uint32_t r = a + 0xFFFu + ((a >> 13) & 1u);
  uint32_t h = (r >> 13) - (112u << 10);
  return s | (h < 0x7BFFu ? h : 0x7BFFu);
}

__device__ __forceinline__ float f16_value(uint32_t h) {
  uint32_t e = (h >> 10) & 31u, f = h & 1023u;
  float v = e == 0u ? (float)f * 0x1p-24f : as_f32(((e + 112u) << 23) | (f << 13));
  return (h & 0x8000u) ? -v : v;
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

// ============================================================================= fill / amax
__global__ void fill_f32_kernel(float* p, int64_t n, float v) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

// max |x| as bf16 magnitude bits (NaN bit patterns sort above +inf), folded into *amax as the
// binary32 pattern with an integer atomic max (order independent, so the result is exact and
// deterministic).  grid.z indexes equally shaped tensors when batched (stride R*K elements).
__global__ __launch_bounds__(kThreads) void amax_kernel(const uint16_t* __restrict__ x, int64_t R,
                                                        int64_t K, int64_t ldx, int64_t tstride,
                                                        float* __restrict__ amax) {
  constexpr int RPT = 8;                      // rows per pass: 8 independent 16-byte loads
  const int64_t chunks = K >> 3;
  const uint16_t* xt = x + (int64_t)blockIdx.z * tstride;
  uint32_t m = 0;
  for (int64_t c = (int64_t)blockIdx.x * kThreads + threadIdx.x; c < chunks;
       c += (int64_t)gridDim.x * kThreads) {
    for (int64_t r0 = (int64_t)blockIdx.y * RPT; r0 < R; r0 += (int64_t)gridDim.y * RPT) {
      uint4 v[RPT];
#pragma unroll
      for (int i = 0; i < RPT; ++i) {
        v[i] = make_uint4(0, 0, 0, 0);
        if (r0 + i < R) v[i] = *reinterpret_cast<const uint4*>(xt + (r0 + i) * ldx + c * 8);
      }
#pragma unroll
      for (int i = 0; i < RPT; ++i) {
        uint32_t h[8];
        unpack8(v[i], h);
        const uint32_t a = max_abs_bits8(h);
        m = a > m ? a : m;
      }
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    uint32_t o = (uint32_t)__shfl_xor((int)m, off, 64);
    m = o > m ? o : m;
  }
  __shared__ uint32_t wmax[kThreads / 64];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  if (lane == 0) wmax[wid] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t b = wmax[0];
    for (int i = 1; i < kThreads / 64; ++i) b = wmax[i] > b ? wmax[i] : b;
    if (b != 0u) atomicMax(reinterpret_cast<unsigned int*>(amax + blockIdx.z), b << 16);
  }
}

// ======================================================================= per-chunk codecs
// Each function quantizes and dequantizes this lane's 8 elements h[] (bf16 bits); the lanes
// of one format block must run it together (cross-lane reductions).

// NVFP4 (16-block = this lane and lane ^ 1): 4-bit codes cw (element k in nibble k), E4M3
// block scale sc, x_hat bits xh.  S is the FP32 tensor scale g / (6 * 448), six_s = 6 S.
__device__ __forceinline__ void nvfp4_chunk(const uint32_t h[8], float S, float six_s,
                                            uint32_t& cw, uint32_t& sc, uint32_t xh[8]) {
  uint32_t ab = max_abs_bits8(h);
  const uint32_t o = xor1_u32(ab);         // partner lane holds the other 8 of the 16-block
  ab = o > ab ? o : ab;
  sc = 0;
  if (S != 0.0f) {
    const float t = as_f32(ab << 16) / six_s;   // t_b = a_b / (6 S)
    sc = e4m3_code(t);
  }
  const float D = S * e4m3_value(sc);       // block decode scale s_FP32 * s_E4M3,b
  const float rcp = D != 0.0f ? 1.0f / D : 0.0f;
  cw = 0;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const uint32_t sign = h[k] >> 15;
    uint32_t m = 0;
    if (D != 0.0f) m = e2m1_code(as_f32((h[k] & 0x7FFFu) << 16) * rcp);
    cw |= ((sign << 3) | m) << (4 * k);
    const float mag = e2m1_value(m) * D;
    xh[k] = bf16_rne(sign ? -mag : mag);
  }
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
  const float up = as_f32((254u - e) << 23);  // 2^(127 - e): divides by the scale exactly
  cw = 0;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const uint32_t sign = h[k] >> 15;
    const uint32_t m = e2m1_code(as_f32((h[k] & 0x7FFFu) << 16) * up);
    // x_hat = +-V(m) * 2^(e-127) written directly as bf16 bits
    uint32_t b;
    if (m == 0u) b = 0u;
    else if (e < 2u && m < 4u) b = m << (e + 5u);             // bf16 subnormal range
    else b = (e << 7) - 128u + (m >= 2u ? 64u * m : 0u);
    cw |= ((sign << 3) | m) << (4 * k);
    xh[k] = b | (sign << 15);
  }
  scale = e;
  if (nonfinite) {
    cw = 0;
    scale = 0xFFu;
#pragma unroll
    for (int k = 0; k < 8; ++k) xh[k] = 0x7FC0u;
  }
}

// Q4_K (32 lanes per 256-element super-block; lane L holds elements 8L..8L+7, sub-block L/4):
// FP16 bits of d and dmin, this sub-block's 6-bit scale / min, the 4-bit codes of this
// lane (qlo: elements 0-3, qhi: 4-7, one per byte) and x_hat bits xh.
struct Q4kChunk {
  uint32_t dh, mh, ls, lm, qlo, qhi;
};
__device__ __forceinline__ void q4k_chunk(const uint32_t h[8], Q4kChunk& r, uint32_t xh[8]) {
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
  const float a = (hi - lo) / 15.0f;        // step of the sub-block
  const float mu = 0.0f - lo;               // offset (subtracted), never negative
  float A = a, Mx = mu;
  A = fmaxf(A, xor_swz_f<4>(A)); Mx = fmaxf(Mx, xor_swz_f<4>(Mx));
  A = fmaxf(A, xor_swz_f<8>(A)); Mx = fmaxf(Mx, xor_swz_f<8>(Mx));
  A = fmaxf(A, xor_swz_f<16>(A)); Mx = fmaxf(Mx, xor_swz_f<16>(Mx));
  r.dh = f16_rne_sat(A / 63.0f);
  r.mh = f16_rne_sat(Mx / 63.0f);
  const float d = f16_value(r.dh), dmin = f16_value(r.mh);
  r.ls = 0;
  r.lm = 0;
  if (d != 0.0f) r.ls = (uint32_t)fminf(fmaxf(__builtin_rintf(a / d), 0.0f), 63.0f);
  if (dmin != 0.0f) r.lm = (uint32_t)fminf(fmaxf(__builtin_rintf(mu / dmin), 0.0f), 63.0f);
  const float t1 = d * (float)r.ls;
  const float t2 = dmin * (float)r.lm;
  r.qlo = 0;
  r.qhi = 0;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    uint32_t q = 0;
    if (t1 != 0.0f) q = (uint32_t)fminf(fmaxf(__builtin_rintf((xv[k] + t2) / t1), 0.0f), 15.0f);
    if (k < 4) r.qlo |= q << (8 * k);
    else r.qhi |= q << (8 * (k - 4));
    const float prod = t1 * (float)q;
    xh[k] = bf16_rne(prod - t2);
  }
}

// ============================================================================= NVFP4
// grid.z indexes batched tensors (expert weights): tensor z uses g[z] and element offset
// z * tstride (input) / z * R * K (outputs).
template <int RPT>
__global__ __launch_bounds__(kThreads) void nvfp4_kernel(
    const uint16_t* __restrict__ x, int64_t R, int64_t K, int64_t ldx, int64_t tstride,
    const float* __restrict__ gptr, float* __restrict__ s_out, uint8_t* __restrict__ codes,
    uint8_t* __restrict__ scales, uint16_t* __restrict__ xhat) {
  const int64_t chunks = K >> 3;
  const int64_t c = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  const bool col_ok = c < chunks;
  const int64_t z = blockIdx.z;
  const float g = gptr[z];
  const float S = g / 2688.0f;             // decode tensor scale s_FP32: g maps to 6 * 448
  const float six_s = 6.0f * S;
  if (s_out && blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) s_out[z] = S;
  const uint16_t* xt = x + z * tstride;
  const int64_t obase = z * R * K;
  uint4 vin[RPT];
#pragma unroll
  for (int i = 0; i < RPT; ++i) {           // all loads first: RPT requests in flight
    const int64_t r = (int64_t)blockIdx.y * RPT + i;
    vin[i] = make_uint4(0, 0, 0, 0);
    if (col_ok && r < R) vin[i] = *reinterpret_cast<const uint4*>(xt + r * ldx + c * 8);
  }
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    const int64_t r = (int64_t)blockIdx.y * RPT + i;
    const bool ok = col_ok && r < R;
    uint32_t h[8], cw, sc, xh[8];
    unpack8(vin[i], h);
    nvfp4_chunk(h, S, six_s, cw, sc, xh);
    if (ok) {
      if (codes) *reinterpret_cast<uint32_t*>(codes + obase / 2 + r * (K / 2) + c * 4) = cw;
      if (scales && (c & 1) == 0) scales[obase / 16 + r * (K / 16) + c / 2] = (uint8_t)sc;
      if (xhat) *reinterpret_cast<uint4*>(xhat + obase + r * K + c * 8) = pack8(xh);
    }
  }
}

// ============================================================================= MXFP4
template <int RPT>
__global__ __launch_bounds__(kThreads) void mxfp4_kernel(
    const uint16_t* __restrict__ x, int64_t R, int64_t K, int64_t ldx, uint8_t* __restrict__ codes,
    uint8_t* __restrict__ scales, uint16_t* __restrict__ xhat) {
  const int64_t chunks = K >> 3;
  const int64_t c = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  const bool col_ok = c < chunks;
  uint4 vin[RPT];
#pragma unroll
  for (int i = 0; i < RPT; ++i) {           // all loads first: RPT requests in flight
    const int64_t r = (int64_t)blockIdx.y * RPT + i;
    vin[i] = make_uint4(0, 0, 0, 0);
    if (col_ok && r < R) vin[i] = *reinterpret_cast<const uint4*>(x + r * ldx + c * 8);
  }
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    const int64_t r = (int64_t)blockIdx.y * RPT + i;
    const bool ok = col_ok && r < R;
    uint32_t h[8], cw, e, xh[8];
    unpack8(vin[i], h);
    mxfp4_chunk(h, cw, e, xh);
    if (ok) {
      if (codes) *reinterpret_cast<uint32_t*>(codes + r * (K / 2) + c * 4) = cw;
      if (scales && (c & 3) == 0) scales[r * (K / 32) + c / 4] = (uint8_t)e;
      if (xhat) *reinterpret_cast<uint4*>(xhat + r * K + c * 8) = pack8(xh);
    }
  }
}

// ============================================================================= Q4_K
// 32 lanes per 256-element super-block; lane L of the super-block holds elements 8L..8L+7,
// i.e. sub-block j = L / 4.
template <int RPT>
__global__ __launch_bounds__(kThreads) void q4k_kernel(const uint16_t* __restrict__ x, int64_t R,
                                                       int64_t K, int64_t ldx,
                                                       uint8_t* __restrict__ packed,
                                                       uint16_t* __restrict__ xhat) {
  const int64_t chunks = K >> 3;
  const int64_t c = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  const bool col_ok = c < chunks;
  const int L = threadIdx.x & 31;           // lane within the super-block
  const int64_t sb = c >> 5;
  const int sub = L >> 2;
#pragma unroll 1
  for (int i = 0; i < RPT; ++i) {
    const int64_t r = (int64_t)blockIdx.y * RPT + i;
    const bool ok = col_ok && r < R;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (ok) v = *reinterpret_cast<const uint4*>(x + r * ldx + c * 8);
    uint32_t h[8], xh[8];
    unpack8(v, h);
    Q4kChunk q;
    q4k_chunk(h, q, xh);
    const uint32_t ls = q.ls, lm = q.lm, qlo = q.qlo, qhi = q.qhi, dh = q.dh, mh = q.mh;
    // gather the eight 6-bit scales / mins at lane 0 of the super-block
    uint32_t LS[8], LM[8];
    const int base = (threadIdx.x & 63) & ~31;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      LS[j] = (uint32_t)__shfl((int)ls, base + 4 * j, 64);
      LM[j] = (uint32_t)__shfl((int)lm, base + 4 * j, 64);
    }
    // codes of sub-block j+1 (odd) go to the high nibbles of sub-block j's bytes
    const uint32_t plo = xor_swz_u32<4>(qlo);
    const uint32_t phi = xor_swz_u32<4>(qhi);
    if (ok && packed) {
      uint8_t* blk = packed + (r * (K / 256) + sb) * 144;
      if (L == 0) {
        uint32_t w[4];
        w[0] = dh | (mh << 16);
        uint32_t sc[12];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          sc[j] = (LS[j] & 63u) | ((LS[j + 4] >> 4) << 6);
          sc[j + 4] = (LM[j] & 63u) | ((LM[j + 4] >> 4) << 6);
          sc[j + 8] = (LS[j + 4] & 15u) | ((LM[j + 4] & 15u) << 4);
        }
        w[1] = sc[0] | (sc[1] << 8) | (sc[2] << 16) | (sc[3] << 24);
        w[2] = sc[4] | (sc[5] << 8) | (sc[6] << 16) | (sc[7] << 24);
        w[3] = sc[8] | (sc[9] << 8) | (sc[10] << 16) | (sc[11] << 24);
        *reinterpret_cast<uint4*>(blk) = make_uint4(w[0], w[1], w[2], w[3]);
      }
      if ((sub & 1) == 0) {
        const int off = 16 + 32 * (sub >> 1) + 8 * (L & 3);
        *reinterpret_cast<uint2*>(blk + off) = make_uint2(qlo | (plo << 4), qhi | (phi << 4));
      }
    }
    if (ok && xhat) *reinterpret_cast<uint4*>(xhat + r * K + c * 8) = pack8(xh);
  }
}

// ===================================================== quantize-dequantize, transposed output
// out[k][r] = x_hat[r][k]: the backward's NT GEMMs take W_hat^T and A_hat^T, which this
// writes in one pass instead of x_hat followed by a transpose.  A block quantizes a 64 x 256
// tile (thread t: row 8 i + t / 32, chunk t % 32, so each 32-lane half-wave holds one full
// 256-element row -- every format block, the Q4_K super-block included, stays inside one
// half-wave), parks x_hat in LDS (chunk c of row r at slot c ^ (((r >> 3) & 7) << 1)), then
// every lane transposes an 8 x 8 block in registers and writes 8 output rows of 16 bytes.
// grid.z indexes batched tensors; NVFP4 tensor z uses the tensor amax g[z].  R and K are
// multiples of 8; K a multiple of the format block.
constexpr int kTR = 64, kTC = 256;

__device__ __forceinline__ int tslot(int r, int c) { return c ^ (((r >> 3) & 7) << 1); }

template <int FMT, bool GROUPED>
__global__ __launch_bounds__(kThreads) void quant_t_kernel(const uint16_t* __restrict__ x,
                                                           int64_t R, int64_t K, int64_t ldx,
                                                           int64_t xbs, const float* __restrict__ g,
                                                           uint16_t* __restrict__ out,
                                                           int64_t ldo, int64_t obs,
                                                           const int64_t* __restrict__ off,
                                                           const int* __restrict__ kstart, int E) {
  __shared__ uint4 tile[kTR * (kTC / 8)];
  const int t = threadIdx.x;
  const int64_t c0 = (int64_t)blockIdx.x * kTC;
  // Input rows [r0, r_end) of this tile; output columns start at oc0.
  int64_t r0 = (int64_t)blockIdx.y * kTR, r_end = R, oc0 = r0;
  if (GROUPED) {
    // Expert e's rows [off[e], off[e+1]) go to the 64-aligned output columns starting at
    // 64 kstart[e]; the columns past its last row are written as zeros.
    const int y = blockIdx.y;
    if (y >= kstart[E]) return;                  // uniform over the block
    int lo = 0, hi = E;                          // kstart[e] <= y < kstart[e+1]
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (kstart[mid] <= y) lo = mid; else hi = mid;
    }
    r0 = off[lo] + (int64_t)(y - kstart[lo]) * kTR;
    r_end = off[lo + 1];
    oc0 = (int64_t)y * kTR;
  }
  x += (int64_t)blockIdx.z * xbs;
  out += (int64_t)blockIdx.z * obs;
  float S = 0.0f, six_s = 0.0f;
  if (FMT == QF_FMT_NVFP4) {
    S = g[blockIdx.z] / 2688.0f;            // g maps to 6 * 448
    six_s = 6.0f * S;
  }
  uint4 vin[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {             // all eight loads first
    const int64_t gr = r0 + i * 8 + (t >> 5), gc = c0 + (t & 31) * 8;
    vin[i] = make_uint4(0, 0, 0, 0);
    if (gr < r_end && gc < K) vin[i] = *reinterpret_cast<const uint4*>(x + gr * ldx + gc);
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int row = i * 8 + (t >> 5), cc = t & 31;
    uint32_t h[8], xh[8];
    unpack8(vin[i], h);
    if (FMT == QF_FMT_NVFP4) {
      uint32_t cw, sc;
      nvfp4_chunk(h, S, six_s, cw, sc, xh);
    } else if (FMT == QF_FMT_MXFP4) {
      uint32_t cw, e;
      mxfp4_chunk(h, cw, e, xh);
    } else if (FMT == QF_FMT_Q4K) {
      Q4kChunk q;
      q4k_chunk(h, q, xh);
    } else {
#pragma unroll
      for (int k = 0; k < 8; ++k) xh[k] = h[k];
    }
    tile[row * 32 + tslot(row, cc)] = pack8(xh);
  }
  __syncthreads();
  const int rb = t & 7, cb = t >> 3;
  uint32_t w[8][4];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int row = rb * 8 + i;
    const uint4 v = tile[row * 32 + tslot(row, cb)];
    w[i][0] = v.x; w[i][1] = v.y; w[i][2] = v.z; w[i][3] = v.w;
  }
  const int64_t orow0 = c0 + cb * 8, ocol = oc0 + rb * 8;
  if (!GROUPED && ocol >= R) return;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    if (orow0 + j >= K) break;
    uint32_t o[4];
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      const uint32_t lo = w[2 * d][j >> 1], hi = w[2 * d + 1][j >> 1];
      o[d] = (j & 1) ? ((lo >> 16) | (hi & 0xFFFF0000u)) : ((lo & 0xFFFFu) | (hi << 16));
    }
    *reinterpret_cast<uint4*>(out + (orow0 + j) * ldo + ocol) = make_uint4(o[0], o[1], o[2], o[3]);
  }
}

inline dim3 row_grid(int64_t R, int64_t K, int rpt) {
  const int64_t chunks = K >> 3;
  return dim3((unsigned)((chunks + kThreads - 1) / kThreads), (unsigned)((R + rpt - 1) / rpt), 1);
}

}  // namespace

// ================================================================================ launchers
hipError_t launch_fill_f32(float* p, int64_t n, float v, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_f32_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, p, n, v);
  return hipGetLastError();
}

// At most ~1000 blocks (one atomic each) for one tensor: 8 rows per pass, grid-strided.
static dim3 amax_grid(int64_t R, int64_t K, int64_t E) {
  const int64_t chunks = K >> 3;
  int64_t gx = (chunks + kThreads - 1) / kThreads;
  if (gx > 64) gx = 64;
  int64_t gy = (R + 7) / 8;
  const int64_t cap = (1024 + gx - 1) / gx;
  if (gy > cap) gy = cap;
  if (gy < 1) gy = 1;
  return dim3((unsigned)gx, (unsigned)gy, (unsigned)E);
}

hipError_t launch_amax(const uint16_t* x, int64_t R, int64_t K, int64_t ldx, float* amax,
                       hipStream_t s) {
  if (R == 0 || K == 0) return hipSuccess;
  hipLaunchKernelGGL(amax_kernel, amax_grid(R, K, 1), dim3(kThreads), 0, s, x, R, K, ldx,
                     (int64_t)0, amax);
  return hipGetLastError();
}

hipError_t launch_amax_batched(const uint16_t* x, int64_t E, int64_t R, int64_t K, float* amax,
                               hipStream_t s) {
  if (E == 0 || R == 0 || K == 0) return hipSuccess;
  dim3 grid = amax_grid(R, K, E);
  const int64_t gy = (R + 7) / 8 < 16 ? (R + 7) / 8 : 16;
  grid.y = (unsigned)(gy < 1 ? 1 : gy);
  hipLaunchKernelGGL(amax_kernel, grid, dim3(kThreads), 0, s, x, R, K, K, R * K, amax);
  return hipGetLastError();
}

constexpr int kRowsPerThread = 4;

hipError_t launch_nvfp4(const uint16_t* x, int64_t R, int64_t K, int64_t ldx, const float* g,
                        float* s_out, uint8_t* codes, uint8_t* scales, uint16_t* xhat,
                        hipStream_t s) {
  if (R == 0 || K == 0) {
    if (s_out) return hipSuccess;  // nothing to quantize; S is left to the caller
    return hipSuccess;
  }
  hipLaunchKernelGGL(nvfp4_kernel<kRowsPerThread>, row_grid(R, K, kRowsPerThread),
                     dim3(kThreads), 0, s, x, R, K, ldx, (int64_t)0, g, s_out, codes, scales,
                     xhat);
  return hipGetLastError();
}

hipError_t launch_nvfp4_batched(const uint16_t* x, int64_t E, int64_t R, int64_t K,
                                const float* g, uint16_t* xhat, hipStream_t s) {
  if (E == 0 || R == 0 || K == 0) return hipSuccess;
  dim3 grid = row_grid(R, K, kRowsPerThread);
  grid.z = (unsigned)E;
  hipLaunchKernelGGL(nvfp4_kernel<kRowsPerThread>, grid, dim3(kThreads), 0, s, x, R, K, K,
                     R * K, g, (float*)nullptr, (uint8_t*)nullptr, (uint8_t*)nullptr, xhat);
  return hipGetLastError();
}

hipError_t launch_mxfp4(const uint16_t* x, int64_t R, int64_t K, int64_t ldx, uint8_t* codes,
                        uint8_t* scales, uint16_t* xhat, hipStream_t s) {
  if (R == 0 || K == 0) return hipSuccess;
  hipLaunchKernelGGL(mxfp4_kernel<kRowsPerThread>, row_grid(R, K, kRowsPerThread),
                     dim3(kThreads), 0, s, x, R, K, ldx, codes, scales, xhat);
  return hipGetLastError();
}

hipError_t launch_q4k(const uint16_t* x, int64_t R, int64_t K, int64_t ldx, uint8_t* packed,
                      uint16_t* xhat, hipStream_t s) {
  if (R == 0 || K == 0) return hipSuccess;
  hipLaunchKernelGGL(q4k_kernel<2>, row_grid(R, K, 2), dim3(kThreads), 0, s, x, R, K, ldx,
                     packed, xhat);
  return hipGetLastError();
}

template <bool GROUPED>
hipError_t launch_quant_t_impl(int fmt, const uint16_t* x, int64_t R, int64_t K, int64_t ldx,
                               int64_t batch, int64_t xbs, const float* g, uint16_t* out,
                               int64_t ldo, int64_t obs, const int64_t* off, const int* kstart,
                               int E, int64_t ytiles, hipStream_t s) {
  const dim3 grid((unsigned)((K + kTC - 1) / kTC), (unsigned)ytiles, (unsigned)batch);
  switch (fmt) {
#define QF_QT(F)                                                                            \
  hipLaunchKernelGGL((quant_t_kernel<F, GROUPED>), grid, dim3(kThreads), 0, s, x, R, K, ldx, \
                     xbs, g, out, ldo, obs, off, kstart, E);                                 \
  break;
    case QF_FMT_NONE: QF_QT(QF_FMT_NONE)
    case QF_FMT_NVFP4: QF_QT(QF_FMT_NVFP4)
    case QF_FMT_MXFP4: QF_QT(QF_FMT_MXFP4)
    case QF_FMT_Q4K: QF_QT(QF_FMT_Q4K)
#undef QF_QT
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_quant_t(int fmt, const uint16_t* x, int64_t R, int64_t K, int64_t ldx,
                          int64_t batch, int64_t xbs, const float* g, uint16_t* out, int64_t ldo,
                          int64_t obs, hipStream_t s) {
  if (R == 0 || K == 0 || batch == 0) return hipSuccess;
  return launch_quant_t_impl<false>(fmt, x, R, K, ldx, batch, xbs, g, out, ldo, obs, nullptr,
                                    nullptr, 0, (R + kTR - 1) / kTR, s);
}

hipError_t launch_quant_t_grouped(int fmt, const uint16_t* x, int64_t T, int64_t K,
                                  const int64_t* off, const int* kstart, int64_t E,
                                  uint16_t* out, int64_t ldo, hipStream_t s) {
  if (T == 0 || K == 0 || E == 0) return hipSuccess;
  // 64-row tiles: at most sum_e ceil(T_e / 64) <= T / 64 + E
  return launch_quant_t_impl<true>(fmt, x, T, K, K, 1, 0, nullptr, out, ldo, 0, off, kstart,
                                   (int)E, (T + kTR - 1) / kTR + E, s);
}

}  // namespace qf
