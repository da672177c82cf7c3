// QAD distillation loss for gfx950 (QATFactory Sec. 3.3, Eq. qad-objective): per token row of
// teacher and student logits (bf16 [L, V]), the forward KL of the two softmax distributions,
// its gradient with respect to the student's logits, and the teacher-student top-1 agreement.
//
// One workgroup per row, two passes over the row:
//   pass 1  online base-2 statistics of both rows, with a = z log2(e):
//             m = max a,  S = sum 2^(a - m)                         (teacher and student)
//             Q = sum 2^(a_T - m_T) (z_T - z_S)                      (teacher-weighted gap)
//           and the first index of each row's maximum logit.  Each 8-logit chunk updates the
//           maxima from its raw maximum (z -> z log2(e) is monotone), each exponent is one
//           FMA (z log2(e) - m), and the index search runs only when a chunk's maximum beats
//           the lane's running one.  Then, in natural units,
//             lse = ln2 (m + log2 S),   KL = Q / S_T + lse_S - lse_T
//           (sum_v p_T (log p_T - log p_S) with log p = z - lse).
//   pass 2  grad[v] = scale (2^(a_S - c_S) - 2^(a_T - c_T)), c = m + log2 S, i.e.
//           scale (p_S - p_T), written as bf16.
// Each lane folds its 16-byte chunks in a fixed order and the workgroup merges the lanes'
// statistics in a fixed tree, so the results are deterministic.  One 1024-lane workgroup
// fits a CU (68 VGPRs: 7 waves per SIMD), so 256 rows (~155 MB of logits at a 152K
// vocabulary) are in flight, and part of the second read hits the 256 MB last-level cache;
// the gradient goes out with non-temporal stores so it does not evict the logits (512-lane
// workgroups, two per CU, read faster in the first pass but lose that reuse: slower overall).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "qf.h"
#include "qf_codecs.h"
#include "qf_internal.h"

namespace qf {
namespace {

using namespace codec;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int kUnroll = 2;                            // chunks per lane in flight per operand
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

struct Stat {   // online softmax statistics in base 2
  float m, S, Q;
};

__device__ __forceinline__ float exp2_safe(float d) {   // 2^d with 2^(-inf) = 0
  return __builtin_amdgcn_exp2f(d);
}

// (m1, S1, Q1) + (m2, S2, Q2) -> common maximum; an empty side (m = -inf) contributes nothing.
__device__ __forceinline__ Stat merge(Stat x, Stat y) {
  const float m = fmaxf(x.m, y.m);
  const float fx = x.m == m ? 1.0f : exp2_safe(x.m - m);
  const float fy = y.m == m ? 1.0f : exp2_safe(y.m - m);
  return Stat{m, x.S * fx + y.S * fy, x.Q * fx + y.Q * fy};
}

struct ArgMax {  // value and first index of a maximum
  float v;
  int64_t i;
};

__device__ __forceinline__ ArgMax amax_merge(ArgMax x, ArgMax y) {
  if (y.v > x.v || (y.v == x.v && y.i < x.i)) return y;
  return x;
}

// The 8 bf16 logits of a 16-byte chunk as FP32 (element k in half k % 2 of dword k / 2).
__device__ __forceinline__ void unpack8_f32(uint4 v, float x[8]) {
  const uint32_t d[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    x[2 * q] = as_f32(d[q] << 16);
    x[2 * q + 1] = as_f32(d[q] & 0xFFFF0000u);
  }
}

__device__ __forceinline__ float max8(const float x[8]) {
  return fmaxf(fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])),
               fmaxf(fmaxf(x[4], x[5]), fmaxf(x[6], x[7])));
}

// First k with x[k] == m (m is the maximum of x, so one exists).
__device__ __forceinline__ int first_eq8(const float x[8], float m) {
  int k0 = 7;
#pragma unroll
  for (int k = 6; k >= 0; --k) k0 = x[k] == m ? k : k0;
  return k0;
}

template <int NT>
__global__ __launch_bounds__(NT) void qad_kl_kernel(const uint16_t* __restrict__ zt, int64_t ldt,
                                                    const uint16_t* __restrict__ zs, int64_t lds_,
                                                    int64_t V, float gscale,
                                                    float* __restrict__ row_kl,
                                                    uint16_t* __restrict__ grad, int64_t ldg,
                                                    int32_t* __restrict__ agree) {
  constexpr int NW = NT / 64;
  __shared__ float sm_t[NW], sS_t[NW], sQ[NW], sm_s[NW], sS_s[NW];
  __shared__ float sva[NW], svb[NW];
  __shared__ int64_t sia[NW], sib[NW];
  __shared__ float row_c[2];
  const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
  const int64_t row = blockIdx.x;
  const uint16_t* pt = zt + row * ldt;
  const uint16_t* ps = zs + row * lds_;
  const int64_t chunks = V >> 3;

  Stat st{-__builtin_huge_valf(), 0.0f, 0.0f};
  Stat ss{-__builtin_huge_valf(), 0.0f, 0.0f};
  ArgMax at{-__builtin_huge_valf(), INT64_MAX}, as{-__builtin_huge_valf(), INT64_MAX};

  for (int64_t c0 = t; c0 < chunks; c0 += (int64_t)NT * kUnroll) {
    uint4 vt[kUnroll], vs[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {               // all loads first
      const int64_t c = c0 + (int64_t)u * NT;
      vt[u] = make_uint4(0, 0, 0, 0);
      vs[u] = make_uint4(0, 0, 0, 0);
      if (c < chunks) {
        vt[u] = *reinterpret_cast<const uint4*>(pt + c * 8);
        vs[u] = *reinterpret_cast<const uint4*>(ps + c * 8);
      }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t c = c0 + (int64_t)u * NT;
      if (c >= chunks) break;
      float xt[8], xs[8];
      unpack8_f32(vt[u], xt);
      unpack8_f32(vs[u], xs);
      const float mt = max8(xt), ms = max8(xs);
      if (mt > at.v) at = ArgMax{mt, c * 8 + first_eq8(xt, mt)};
      if (ms > as.v) as = ArgMax{ms, c * 8 + first_eq8(xs, ms)};
      // rescale the running sums to the new maxima, then add the chunk
      const float nmt = fmaxf(st.m, mt * kLog2e), nms = fmaxf(ss.m, ms * kLog2e);
      const float ft = st.m == nmt ? 1.0f : exp2_safe(st.m - nmt);
      const float fs = ss.m == nms ? 1.0f : exp2_safe(ss.m - nms);
      float S_t = st.S * ft, Q_t = st.Q * ft, S_s = ss.S * fs;
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const float et = exp2_safe(__builtin_fmaf(xt[k], kLog2e, -nmt));
        S_t += et;
        Q_t = __builtin_fmaf(et, xt[k] - xs[k], Q_t);
        S_s += exp2_safe(__builtin_fmaf(xs[k], kLog2e, -nms));
      }
      st = Stat{nmt, S_t, Q_t};
      ss = Stat{nms, S_s, 0.0f};
    }
  }

  // workgroup merge in a fixed tree: within each wave by halving offsets, then waves in order
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    Stat ot{__shfl_down(st.m, off, 64), __shfl_down(st.S, off, 64), __shfl_down(st.Q, off, 64)};
    Stat os{__shfl_down(ss.m, off, 64), __shfl_down(ss.S, off, 64), 0.0f};
    ArgMax oa{__shfl_down(at.v, off, 64), (int64_t)__shfl_down((long long)at.i, off, 64)};
    ArgMax ob{__shfl_down(as.v, off, 64), (int64_t)__shfl_down((long long)as.i, off, 64)};
    if (lane + off < 64) {
      st = merge(st, ot);
      ss = merge(ss, os);
      at = amax_merge(at, oa);
      as = amax_merge(as, ob);
    }
  }
  if (lane == 0) {
    sm_t[wv] = st.m; sS_t[wv] = st.S; sQ[wv] = st.Q; sm_s[wv] = ss.m; sS_s[wv] = ss.S;
    sva[wv] = at.v; sia[wv] = at.i; svb[wv] = as.v; sib[wv] = as.i;
  }
  __syncthreads();
  if (t == 0) {
    Stat T{sm_t[0], sS_t[0], sQ[0]}, Sx{sm_s[0], sS_s[0], 0.0f};
    ArgMax A{sva[0], sia[0]}, B{svb[0], sib[0]};
    for (int w = 1; w < NW; ++w) {
      T = merge(T, Stat{sm_t[w], sS_t[w], sQ[w]});
      Sx = merge(Sx, Stat{sm_s[w], sS_s[w], 0.0f});
      A = amax_merge(A, ArgMax{sva[w], sia[w]});
      B = amax_merge(B, ArgMax{svb[w], sib[w]});
    }
    const float ct = T.m + __builtin_amdgcn_logf(T.S);     // base-2 log-sum-exp
    const float cs = Sx.m + __builtin_amdgcn_logf(Sx.S);
    row_kl[row] = T.Q / T.S + (cs - ct) * kLn2;
    if (agree) agree[row] = A.i == B.i ? 1 : 0;
    row_c[0] = ct;
    row_c[1] = cs;
  }
  if (!grad) return;
  __syncthreads();
  const float ct = row_c[0], cs = row_c[1];
  uint16_t* pg = grad + row * ldg;
  // Finite row statistics make every probability finite, so the hardware bf16 pack rounds
  // exactly as bf16_rne; rows with non-finite logits keep the bit-level rounding (uniform per
  // workgroup).
  const bool finite = __builtin_isfinite(ct) && __builtin_isfinite(cs);
  for (int64_t c0 = t; c0 < chunks; c0 += (int64_t)NT * kUnroll) {
    uint4 vt[kUnroll], vs[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t c = c0 + (int64_t)u * NT;
      vt[u] = make_uint4(0, 0, 0, 0);
      vs[u] = make_uint4(0, 0, 0, 0);
      if (c < chunks) {
        vt[u] = *reinterpret_cast<const uint4*>(pt + c * 8);
        vs[u] = *reinterpret_cast<const uint4*>(ps + c * 8);
      }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t c = c0 + (int64_t)u * NT;
      if (c >= chunks) break;
      float xt[8], xs[8], g[8];
      unpack8_f32(vt[u], xt);
      unpack8_f32(vs[u], xs);
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const float p_t = exp2_safe(__builtin_fmaf(xt[k], kLog2e, -ct));
        const float p_s = exp2_safe(__builtin_fmaf(xs[k], kLog2e, -cs));
        g[k] = gscale * (p_s - p_t);
      }
      uint32_t o[4];
      if (finite) {
#pragma unroll
        for (int q = 0; q < 4; ++q) o[q] = bf16x2_rne_nonnan(g[2 * q], g[2 * q + 1]);
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q) o[q] = bf16_rne(g[2 * q]) | (bf16_rne(g[2 * q + 1]) << 16);
      }
      const u32x4 ov = {o[0], o[1], o[2], o[3]};
      __builtin_nontemporal_store(ov, reinterpret_cast<u32x4*>(pg + c * 8));
    }
  }
}

// loss = (1 / L) sum_t row_kl[t] in a fixed order (one workgroup).
__global__ __launch_bounds__(256) void mean_kernel(const float* __restrict__ x, int64_t n,
                                                   float* __restrict__ out) {
  __shared__ float part[256];
  float acc = 0.0f;                                   // x[t], x[t + 256], ... in order,
  int64_t i = threadIdx.x;                            // eight loads in flight per batch
  for (; i + 7 * 256 < n; i += 8 * 256) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = x[i + u * 256];
#pragma unroll
    for (int u = 0; u < 8; ++u) acc += v[u];
  }
  for (; i < n; i += 256) acc += x[i];
  part[threadIdx.x] = acc;
  __syncthreads();
  for (int s = 128; s >= 1; s >>= 1) {
    if ((int)threadIdx.x < s) part[threadIdx.x] += part[threadIdx.x + s];
    __syncthreads();
  }
  if (threadIdx.x == 0) *out = n > 0 ? part[0] / (float)n : 0.0f;
}

}  // namespace

hipError_t launch_qad_kl(const uint16_t* zt, int64_t ldt, const uint16_t* zs, int64_t lds_,
                         int64_t L, int64_t V, float gscale, float* row_kl, float* loss,
                         uint16_t* grad, int64_t ldg, int32_t* agree, hipStream_t s) {
  if (L > 0) {
    hipLaunchKernelGGL(qad_kl_kernel<1024>, dim3((unsigned)L), dim3(1024), 0, s, zt, ldt, zs, lds_,
                       V, gscale, row_kl, grad, ldg, agree);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (loss) {
    hipLaunchKernelGGL(mean_kernel, dim3(1), dim3(256), 0, s, row_kl, L, loss);
    return hipGetLastError();
  }
  return hipSuccess;
}

}  // namespace qf
