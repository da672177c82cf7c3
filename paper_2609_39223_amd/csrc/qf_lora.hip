// LoRA-QAD kernels for gfx950 (QATFactory Sec. 3.3, Eqs. qad-lora and export-lora).
//
// Forward / export: W_hat = Q^-1(Q(W + s B A)) with the rank-r update merged inside the
// quantizer's tile load, so the merged weight never goes to HBM.  W is bf16 [N, K], A FP32
// [r, K], B FP32 [N, r].  Each merged element is
//     acc = sum_j B[n][j] A[j][k]   (binary32, one fused multiply-add per rank term, j rising)
//     m   = bf16(W[n][k] + fl(s * acc))
// and then goes through the same per-chunk codec as an unmerged tensor.
//
// Backward (straight-through, Eq. ste): the merged weight's gradient G = dY^T A_hat is never
// formed; the factor gradients are regrouped around the rank-r products
//     dB = s G A^T = s dY^T (A_hat A^T),      dA = s B^T G = s (dY B)^T A_hat,
// i.e. two row-dot products (U = A_hat A^T, V = dY B: [M, r], contraction over the
// contiguous axis) and two column sums (dY^T U: [N, r], V^T A_hat: [r, K], contraction over
// the M rows).  All four stream a bf16 matrix once from HBM against a small FP32 factor
// held on chip; the column sums split M into row ranges whose FP32 partials are added in a
// fixed order (deterministic results).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "qf.h"
#include "qf_codecs.h"
#include "qf_internal.h"

namespace qf {
namespace {

using namespace codec;

constexpr int kThreads = 256;
constexpr int kRC = 16;   // rank terms staged per pass (B rows in LDS; row-dot outputs)
constexpr int64_t kGroupChunk = 1024;   // rows per column-sum chunk in grouped mode

// ====================================================================== merged quantizer
enum { kOutRows = 0, kOutTransposed = 1, kOutAmax = 2 };

struct MergeArgs {
  const uint16_t* w;      // [N, K] row stride ldw; tensor z at w + z * wbs
  int64_t N, K, ldw, wbs;
  const float* A;         // [r, K] (row stride K); tensor z at A + z * abs (0: shared)
  int64_t abs;
  const float* B;         // [N, r] (row stride r); tensor z at B + z * bbs (0: shared)
  int64_t bbs;
  int r;
  float scale;
  const float* g;         // NVFP4 tensor amax per tensor (read)
  float* amax;            // kOutAmax: running max per tensor (bit-pattern atomic max)
  float* s_out;           // NVFP4 decode scale per tensor, or null
  uint8_t* codes;         // [N, K/2] per tensor, or null
  uint8_t* scales;        // [N, K/16] E4M3 or [N, K/32] E8M0 per tensor, or null
  uint8_t* packed;        // Q4_K [N, K/256, 144] per tensor, or null
  uint16_t* xhat;         // [N, K] per tensor, or null
  uint16_t* out;          // kOutTransposed: [K, N] row stride ldo, tensor z at out + z * obs
  int64_t ldo, obs;
};

// One 64 x 256 tile of tensor blockIdx.z (the tile layout of store_tile_transposed: lane t
// owns chunk t % 32 of rows 8 i + t / 32).
template <int FMT, int OUT>
__global__ __launch_bounds__(kThreads) void lora_quant_kernel(MergeArgs p) {
  __shared__ float bs[kTR * kRC];                     // B rows of the tile, one rank pass
  __shared__ uint4 tile[OUT == kOutTransposed ? kTR * (kTC / 8) : 1];
  const int t = threadIdx.x, cc = t & 31, rs = t >> 5;
  const int64_t z = blockIdx.z;
  const int64_t c0 = (int64_t)blockIdx.x * kTC, r0 = (int64_t)blockIdx.y * kTR;
  const int64_t col = c0 + cc * 8;
  const int64_t N = p.N, K = p.K;
  const bool col_ok = col < K;
  const uint16_t* w = p.w + z * p.wbs;
  const float* A = p.A + z * p.abs;
  const float* B = p.B + z * p.bbs;

  uint4 vin[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {                       // the W tile's loads go out first
    const int64_t row = r0 + 8 * i + rs;
    vin[i] = make_uint4(0, 0, 0, 0);
    if (row < N && col_ok) vin[i] = *reinterpret_cast<const uint4*>(w + row * p.ldw + col);
  }

  float acc[8][8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int k = 0; k < 8; ++k) acc[i][k] = 0.0f;

  for (int j0 = 0; j0 < p.r; j0 += kRC) {
    const int nj = p.r - j0 < kRC ? p.r - j0 : kRC;
    __syncthreads();                                  // previous pass's reads of bs are done
    for (int idx = t; idx < kTR * kRC; idx += kThreads) {
      const int rr = idx / kRC, jj = idx % kRC;
      const int64_t row = r0 + rr;
      bs[idx] = (row < N && jj < nj) ? B[row * p.r + j0 + jj] : 0.0f;
    }
    __syncthreads();
#pragma unroll 2
    for (int jj = 0; jj < nj; ++jj) {
      float a[8];
      if (col_ok) {
        const float4 lo = *reinterpret_cast<const float4*>(A + (int64_t)(j0 + jj) * K + col);
        const float4 hi = *reinterpret_cast<const float4*>(A + (int64_t)(j0 + jj) * K + col + 4);
        a[0] = lo.x; a[1] = lo.y; a[2] = lo.z; a[3] = lo.w;
        a[4] = hi.x; a[5] = hi.y; a[6] = hi.z; a[7] = hi.w;
      } else {
#pragma unroll
        for (int k = 0; k < 8; ++k) a[k] = 0.0f;
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float b = bs[(8 * i + rs) * kRC + jj];
#pragma unroll
        for (int k = 0; k < 8; ++k) acc[i][k] = __builtin_fmaf(b, a[k], acc[i][k]);
      }
    }
  }

  float S = 0.0f, six_s = 0.0f;
  if (FMT == QF_FMT_NVFP4 && OUT != kOutAmax) {
    S = p.g[z] / 2688.0f;                             // g maps to 6 * 448
    six_s = 6.0f * S;
    if (OUT == kOutRows && p.s_out && blockIdx.x == 0 && blockIdx.y == 0 && t == 0) p.s_out[z] = S;
  }
  uint32_t mx = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int64_t row = r0 + 8 * i + rs;
    const bool ok = row < N && col_ok;
    uint32_t h[8], xh[8];
    unpack8(vin[i], h);
#pragma unroll
    for (int k = 0; k < 8; ++k) {                     // m = bf16(W + fl(s * acc))
      const float upd = p.scale * acc[i][k];
      h[k] = bf16_rne(as_f32(h[k] << 16) + upd);
    }
    if (OUT == kOutAmax) {
      const uint32_t a = ok ? max_abs_bits8(h) : 0u;
      mx = a > mx ? a : mx;
      continue;
    }
    uint32_t cw = 0, sc = 0;
    if (FMT == QF_FMT_NVFP4) {
      nvfp4_chunk(h, S, six_s, cw, sc, xh);
    } else if (FMT == QF_FMT_MXFP4) {
      mxfp4_chunk(h, cw, sc, xh);
    } else if (FMT == QF_FMT_Q4K) {
      Q4kChunk q;
      q4k_chunk(h, q, xh);
      if (OUT == kOutRows && p.packed) {
        const int64_t kb = K / 256;
        q4k_store(q, cc, ok, p.packed + ((z * N + row) * kb + col / 256) * 144);
      }
    } else {
#pragma unroll
      for (int k = 0; k < 8; ++k) xh[k] = h[k];
    }
    if (OUT == kOutTransposed) {
      const int lr = 8 * i + rs;
      tile[lr * 32 + tslot(lr, cc)] = pack8(xh);
    } else if (ok) {
      const int64_t e = (z * N + row) * K + col;      // element index of this chunk
      if (FMT == QF_FMT_NVFP4 || FMT == QF_FMT_MXFP4) {
        if (p.codes) *reinterpret_cast<uint32_t*>(p.codes + e / 2) = cw;
        constexpr int kBlk = FMT == QF_FMT_NVFP4 ? 16 : 32;
        if (p.scales && (cc & (kBlk / 8 - 1)) == 0) p.scales[e / kBlk] = (uint8_t)sc;
      }
      if (p.xhat) *reinterpret_cast<uint4*>(p.xhat + e) = pack8(xh);
    }
  }
  if (OUT == kOutAmax) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      const uint32_t o = (uint32_t)__shfl_xor((int)mx, off, 64);
      mx = o > mx ? o : mx;
    }
    __shared__ uint32_t wmax[kThreads / 64];
    if ((t & 63) == 0) wmax[t >> 6] = mx;
    __syncthreads();
    if (t == 0) {
      uint32_t b = wmax[0];
      for (int i = 1; i < kThreads / 64; ++i) b = wmax[i] > b ? wmax[i] : b;
      if (b != 0u) atomicMax(reinterpret_cast<unsigned int*>(p.amax + z), b << 16);
    }
  }
  if (OUT == kOutTransposed) {
    __syncthreads();
    store_tile_transposed(tile, t, p.out + z * p.obs, p.ldo, c0, r0, K, N);
  }
}

// ======================================================================== expert groups
// Grouped (mixture-of-experts) mode of the row-dot and column-sum kernels: rows
// [off[e], off[e+1]) belong to expert e, and blocks are dealt expert-aligned row chunks:
// block y covers chunk y - pre[e] of expert e, where pre[e] <= y < pre[e+1] and pre is the
// prefix of ceil(rows_e / chunk) (group_prefix_kernel).  The host never reads off or pre, so
// grids are sized for the worst case (T / chunk + E) and blocks past pre[E] exit.
struct Groups {
  const int64_t* off;   // null: one group of M rows (dense)
  const int* pre;
  int E;
};

__device__ __forceinline__ int find_group(const int* pre, int E, int y) {
  int lo = 0, hi = E;                                 // pre[lo] <= y < pre[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (pre[mid] <= y) lo = mid; else hi = mid;
  }
  return lo;
}

// pre[e] = sum over experts before e of ceil(rows / q); one thread (E <= 1024).
__global__ void group_prefix_kernel(const int64_t* __restrict__ off, int E, int q,
                                    int* __restrict__ pre) {
  if (threadIdx.x != 0) return;
  int acc = 0;
  pre[0] = 0;
  for (int e = 0; e < E; ++e) {
    acc += (int)((off[e + 1] - off[e] + q - 1) / q);
    pre[e + 1] = acc;
  }
}

// ============================================================================ row-dot
// P[m][j0 + j] = sum_k X[m][k] F[j0 + j][k] for j < 16: X bf16 [M, K] (row stride ldx),
// F FP32 [r, K] (row stride ldf), P FP32 [M, ldp] with ldp >= r rounded up to 16 (the ranks
// past r get zeros).  On v_mfma_f32_16x16x32_bf16: each FP32 factor value f is split into
// bf16 hi = rn(f) and lo = rn(f - hi) (|f - hi - lo| <= 2^-18 |f|; f - hi is exact), and the
// row block accumulates X hi + X lo in FP32 (X is bf16, exact as an MFMA operand).  A block of
// 4 waves covers 16 rows x 16 ranks; wave w takes the 32-deep k steps w, w + 4, ..., each lane
// loading its 8 consecutive k of one X row (A operand: row lane % 16, k 8 (lane / 16) + 0..7)
// and of one F row (B operand: rank lane % 16).  The waves' 16 x 16 partials are added in wave
// order through LDS, so the sums are deterministic.  Grouped: a block's 16 rows come from one
// expert's chunk and use F + e * fstride.
constexpr int kRowBlock = 16;
constexpr int kDotUnroll = 4;                         // k steps in flight per wave

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

// hi / lo bf16 halves of 8 FP32 values (round to nearest even; the inputs are finite factors).
__device__ __forceinline__ void split_bf16x8(const float f[8], bf16x8_t& hi, bf16x8_t& lo) {
  uint32_t h[4], l[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    h[q] = bf16x2_rne_nonnan(f[2 * q], f[2 * q + 1]);
    const float r0 = f[2 * q] - as_f32(h[q] << 16);
    const float r1 = f[2 * q + 1] - as_f32(h[q] & 0xFFFF0000u);
    l[q] = bf16x2_rne_nonnan(r0, r1);
  }
  hi = __builtin_bit_cast(bf16x8_t, make_uint4(h[0], h[1], h[2], h[3]));
  lo = __builtin_bit_cast(bf16x8_t, make_uint4(l[0], l[1], l[2], l[3]));
}

__global__ __launch_bounds__(kThreads) void lora_rowdot_kernel(const uint16_t* __restrict__ X,
                                                               int64_t M, int64_t K, int64_t ldx,
                                                               const float* F,
                                                               int64_t ldf, int r,
                                                               float* __restrict__ P,
                                                               int64_t ldp, Groups g,
                                                               int64_t fstride) {
  __shared__ f32x4_t red[4][64];
  const int t = threadIdx.x, lane = t & 63;
  const int wv = __builtin_amdgcn_readfirstlane(t >> 6);
  const int j0 = blockIdx.y * kRowBlock;
  int64_t m0 = (int64_t)blockIdx.x * kRowBlock;
  if (g.off) {                                        // uniform over the block
    const int y = blockIdx.x;
    if (y >= g.pre[g.E]) return;
    const int e = find_group(g.pre, g.E, y);
    m0 = g.off[e] + (int64_t)(y - g.pre[e]) * kRowBlock;
    M = g.off[e + 1];
    F += e * fstride;
  }
  const int row = lane & 15, kq = (lane >> 4) * 8;
  const bool rok = m0 + row < M, jok = j0 + row < r;  // A row / B rank of this lane
  const uint16_t* xp = X + (rok ? m0 + row : m0) * ldx + kq;
  const float* fp = F + (int64_t)(jok ? j0 + row : 0) * ldf + kq;
  f32x4_t acc = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int64_t k0 = (int64_t)wv * 32; k0 < K; k0 += 4 * 32 * kDotUnroll) {
    uint4 xa[kDotUnroll];
    float4 fa[kDotUnroll][2];
#pragma unroll
    for (int u = 0; u < kDotUnroll; ++u) {            // all loads first
      const int64_t k = k0 + u * 4 * 32;
      const bool kin = k + kq < K;                    // K % 8 == 0: a lane's 8 are all in or out
      xa[u] = make_uint4(0, 0, 0, 0);
      fa[u][0] = fa[u][1] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
      if (kin && rok) xa[u] = *reinterpret_cast<const uint4*>(xp + k);
      if (kin && jok) {
        fa[u][0] = *reinterpret_cast<const float4*>(fp + k);
        fa[u][1] = *reinterpret_cast<const float4*>(fp + k + 4);
      }
    }
#pragma unroll
    for (int u = 0; u < kDotUnroll; ++u) {
      const float f[8] = {fa[u][0].x, fa[u][0].y, fa[u][0].z, fa[u][0].w,
                          fa[u][1].x, fa[u][1].y, fa[u][1].z, fa[u][1].w};
      bf16x8_t hi, lo;
      split_bf16x8(f, hi, lo);
      const bf16x8_t a = __builtin_bit_cast(bf16x8_t, xa[u]);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, hi, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, lo, acc, 0, 0, 0);
    }
  }
  red[wv][lane] = acc;
  __syncthreads();
  if (wv != 0) return;
  const f32x4_t s = ((red[0][lane] + red[1][lane]) + red[2][lane]) + red[3][lane];
  // D[i][j]: lane holds rows 4 (lane / 16) + v, rank lane % 16
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int64_t m = m0 + 4 * (lane >> 4) + v;
    if (m < M) P[m * ldp + j0 + (lane & 15)] = s[v];   // ranks past r: zeros (F rows read as 0)
  }
}

// ======================================================================== column sums
// part[s][j0 + j][c] = sum over rows m of split s of Big[m][c] Sm[m][j0 + j], j < 16:
// Big bf16 [M, C] (row stride ldb), Sm FP32 [M, lds_] (row stride a multiple of 16, zeros
// past rank r, as the row-dot writes it).  On v_mfma_f32_16x16x32_bf16 as D[j][c] =
// sum_m Sm^T[j][m] Big[m][c], with Sm split into bf16 hi + lo like the row-dot's factor.  A
// block covers 256 columns of one row split and one 16-rank block; per 32-row step it stages
// the Big tile [32][256] (row pitch 544 bytes) and Sm^T [16][32] in LDS (double-buffered, the
// next step's global loads in flight while the current one computes).  Wave w owns columns
// 64 w .. 64 w + 63 as four 16-column MFMA blocks: the A operand (rank lane % 16, rows
// 8 (lane / 16) + 0..7) is read from Sm^T, the B operand (column lane % 16, the same rows)
// with two ds_read_b64_tr_b16 per block.  Waves own disjoint columns, so no cross-wave sum.
// part is [splits][r][C] FP32.  Grouped: split y is chunk y - pre[e] (rows_per_split rows)
// of expert e.
constexpr int kColTile = 256;                         // columns per block
constexpr int kColStep = 32;                          // rows per step
constexpr int kColPitch = kColTile * 2 + 32;          // Big tile row pitch in LDS (bytes)

typedef short v4i16_t __attribute__((ext_vector_type(4)));
typedef short v8i16_t __attribute__((ext_vector_type(8)));

// ds_read_b64_tr_b16: within each group of 16 lanes, source lane 4 j + a gives the address of
// row kb + j, columns c0 + 4 a .. + 3; output lane L receives rows kb .. kb + 3 of column c0 + L.
__device__ __forceinline__ v4i16_t lds_tr16(const char* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) v4i16_t*)(__attribute__((address_space(3))) char*)(p));
}

__global__ __launch_bounds__(kThreads) void lora_colsum_kernel(const uint16_t* __restrict__ Big,
                                                               int64_t M, int64_t C, int64_t ldb,
                                                               const float* __restrict__ Sm,
                                                               int64_t lds_, int r,
                                                               int64_t rows_per_split,
                                                               float* __restrict__ part,
                                                               Groups g) {
  __shared__ __attribute__((aligned(16))) char tile[2][kColStep * kColPitch];
  __shared__ __attribute__((aligned(16))) float smt[2][kRC * kColStep];   // [j][m]
  const int t = threadIdx.x, lane = t & 63;
  const int wv = __builtin_amdgcn_readfirstlane(t >> 6);
  const int j0 = blockIdx.z * kRC;
  const int nj = r - j0 < kRC ? r - j0 : kRC;
  const int64_t s = blockIdx.y;
  const int64_t cb = (int64_t)blockIdx.x * kColTile;
  int64_t mb = s * rows_per_split, end = M;
  if (g.off) {                                        // uniform over the block
    if (s >= g.pre[g.E]) return;
    const int e = find_group(g.pre, g.E, (int)s);
    mb = g.off[e] + (s - g.pre[e]) * rows_per_split;
    end = g.off[e + 1];
  }
  const int64_t me = mb + rows_per_split < end ? mb + rows_per_split : end;
  // staging: thread t loads Big rows t / 32 + 8 q (q < 4), 16-byte chunk t % 32, and Sm row
  // t / 8, ranks 2 (t % 8) + {0, 1}
  const int srow = t >> 5, schunk = t & 31;
  const int64_t scol = cb + schunk * 8;
  const bool scol_ok = scol < C;                      // C % 4 == 0, chunks of 8 may be partial
  const int mrow = t >> 3, mj = 2 * (t & 7);
  uint4 bv[4];
  float2 sv;
  auto load = [&](int64_t m0) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int64_t m = m0 + srow + 8 * q;
      bv[q] = make_uint4(0, 0, 0, 0);
      if (m < me) {
        if (scol + 8 <= C) {
          bv[q] = *reinterpret_cast<const uint4*>(Big + m * ldb + scol);
        } else if (scol_ok) {                         // 4 valid columns
          const uint2 h = *reinterpret_cast<const uint2*>(Big + m * ldb + scol);
          bv[q] = make_uint4(h.x, h.y, 0, 0);
        }
      }
    }
    sv = make_float2(0.0f, 0.0f);
    if (m0 + mrow < me) sv = *reinterpret_cast<const float2*>(Sm + (m0 + mrow) * lds_ + j0 + mj);
  };
  auto store = [&](int b) {
#pragma unroll
    for (int q = 0; q < 4; ++q)
      *reinterpret_cast<uint4*>(tile[b] + (srow + 8 * q) * kColPitch + schunk * 16) = bv[q];
    smt[b][mj * kColStep + mrow] = sv.x;
    smt[b][(mj + 1) * kColStep + mrow] = sv.y;
  };
  // fragment addresses: A from Sm^T row lane % 16, columns 8 (lane / 16) + 0..7; B per
  // column block cb4: rows 8 (lane / 16) + 4 h + (lane % 16) / 4, columns 16 cb4 + 4 (lane % 4)
  const int grp = lane >> 4, lj = (lane & 15) >> 2, la = lane & 3;
  const int a_off = (lane & 15) * kColStep + 8 * grp;
  const int b_off = (8 * grp + lj) * kColPitch + (wv * 64 + 4 * la) * 2;
  f32x4_t acc[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) acc[i] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
  if (mb < me) {
    load(mb);
    store(0);
    __syncthreads();
    int b = 0;
    for (int64_t m0 = mb; m0 < me; m0 += kColStep) {
      const bool more = m0 + kColStep < me;           // uniform
      if (more) load(m0 + kColStep);
      const float4 a0 = *reinterpret_cast<const float4*>(&smt[b][a_off]);
      const float4 a1 = *reinterpret_cast<const float4*>(&smt[b][a_off + 4]);
      const float f[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
      bf16x8_t hi, lo;
      split_bf16x8(f, hi, lo);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const char* p = tile[b] + b_off + i * 32;
        const v4i16_t r0 = lds_tr16(p);
        const v4i16_t r1 = lds_tr16(p + 4 * kColPitch);
        const v8i16_t v = __builtin_shufflevector(r0, r1, 0, 1, 2, 3, 4, 5, 6, 7);
        const bf16x8_t bb = __builtin_bit_cast(bf16x8_t, v);
        acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(hi, bb, acc[i], 0, 0, 0);
        acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lo, bb, acc[i], 0, 0, 0);
      }
      if (more) {
        store(b ^ 1);
        __syncthreads();                              // next tile published
        b ^= 1;
      }
    }
  }
  // D[j][c]: lane holds ranks 4 (lane / 16) + v of column lane % 16 of each block
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t c = cb + wv * 64 + i * 16 + (lane & 15);
    if (c >= C) continue;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int jj = 4 * grp + v;
      if (jj < nj) part[(s * r + j0 + jj) * C + c] = acc[i][v];
    }
  }
}

// out = scale * sum_s part[s] in split order (part [splits][r][C]); out[c][j] (row stride r)
// or, transposed, out[j][c] (row stride C).  Grouped with per_group: output e = blockIdx.y
// (at out + e * C * r) sums splits [pre[e], pre[e+1]); grouped without: all pre[E] splits.
__global__ void lora_finish_kernel(const float* __restrict__ part, int64_t splits, int64_t C,
                                   int r, float scale, int transposed, float* __restrict__ out,
                                   Groups g, int per_group) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;   // j * C + c
  if (idx >= C * r) return;
  int64_t s0 = 0, s1 = splits;
  if (g.off) {
    const int e = blockIdx.y;
    s0 = per_group ? g.pre[e] : 0;
    s1 = per_group ? g.pre[e + 1] : g.pre[g.E];
    out += (int64_t)e * C * r;
  }
  // splits added in order; eight loads in flight per batch
  const int64_t stride = C * r;
  float acc = 0.0f;
  int64_t s = s0;
  for (; s + 8 <= s1; s += 8) {
    float v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = part[(s + i) * stride + idx];
#pragma unroll
    for (int i = 0; i < 8; ++i) acc += v[i];
  }
  for (; s < s1; ++s) acc += part[s * stride + idx];
  const float v = scale * acc;
  const int64_t j = idx / C, c = idx % C;
  if (transposed) out[idx] = v;
  else out[c * r + j] = v;
}

// Ft[z][j][n] = F[z][n][j] for small FP32 [N, r] matrices (batch z = blockIdx.y).
__global__ void transpose_f32_kernel(const float* __restrict__ F, int64_t N, int r,
                                     float* __restrict__ Ft) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= N * r) return;
  const int64_t z = blockIdx.y;
  const int64_t n = idx / r, j = idx % r;
  Ft[z * N * r + j * N + n] = F[z * N * r + idx];
}

inline dim3 tile_grid(int64_t N, int64_t K, int64_t batch) {
  return dim3((unsigned)((K + kTC - 1) / kTC), (unsigned)((N + kTR - 1) / kTR), (unsigned)batch);
}

template <int OUT>
hipError_t launch_merge(int fmt, const MergeArgs& a, int64_t batch, hipStream_t s) {
  const dim3 grid = tile_grid(a.N, a.K, batch);
  switch (fmt) {
#define QF_LQ(F)                                                                      \
  hipLaunchKernelGGL((lora_quant_kernel<F, OUT>), grid, dim3(kThreads), 0, s, a); \
  break;
    case QF_FMT_NONE: QF_LQ(QF_FMT_NONE)
    case QF_FMT_NVFP4: QF_LQ(QF_FMT_NVFP4)
    case QF_FMT_MXFP4: QF_LQ(QF_FMT_MXFP4)
    case QF_FMT_Q4K: QF_LQ(QF_FMT_Q4K)
#undef QF_LQ
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

MergeArgs merge_args(const LoraOperand& L, const uint16_t* w, int64_t N, int64_t K, int64_t ldw,
                     int64_t wbs) {
  MergeArgs a{};
  a.w = w; a.N = N; a.K = K; a.ldw = ldw; a.wbs = wbs;
  a.A = L.A; a.abs = L.a_stride;
  a.B = L.B; a.bbs = L.b_stride;
  a.r = (int)L.r; a.scale = L.scale;
  return a;
}

}  // namespace

// ================================================================================ launchers
hipError_t launch_lora_amax(const LoraOperand& L, const uint16_t* w, int64_t N, int64_t K,
                            int64_t ldw, int64_t batch, int64_t wbs, float* amax, hipStream_t s) {
  if (N == 0 || K == 0 || batch == 0) return hipSuccess;
  MergeArgs a = merge_args(L, w, N, K, ldw, wbs);
  a.amax = amax;
  return launch_merge<kOutAmax>(QF_FMT_NONE, a, batch, s);
}

hipError_t launch_lora_quant(int fmt, const LoraOperand& L, const uint16_t* w, int64_t N,
                             int64_t K, int64_t ldw, int64_t batch, int64_t wbs, const float* g,
                             float* s_out, uint8_t* codes, uint8_t* scales, uint8_t* packed,
                             uint16_t* xhat, hipStream_t s) {
  if (N == 0 || K == 0 || batch == 0) return hipSuccess;
  MergeArgs a = merge_args(L, w, N, K, ldw, wbs);
  a.g = g; a.s_out = s_out; a.codes = codes; a.scales = scales; a.packed = packed; a.xhat = xhat;
  return launch_merge<kOutRows>(fmt, a, batch, s);
}

hipError_t launch_lora_quant_t(int fmt, const LoraOperand& L, const uint16_t* w, int64_t N,
                               int64_t K, int64_t ldw, int64_t batch, int64_t wbs, const float* g,
                               uint16_t* out, int64_t ldo, int64_t obs, hipStream_t s) {
  if (N == 0 || K == 0 || batch == 0) return hipSuccess;
  MergeArgs a = merge_args(L, w, N, K, ldw, wbs);
  a.g = g; a.out = out; a.ldo = ldo; a.obs = obs;
  return launch_merge<kOutTransposed>(fmt, a, batch, s);
}

hipError_t launch_group_prefix(const int64_t* off, int64_t E, int q, int* pre, hipStream_t s) {
  hipLaunchKernelGGL(group_prefix_kernel, dim3(1), dim3(64), 0, s, off, (int)E, q, pre);
  return hipGetLastError();
}

hipError_t launch_lora_rowdot(const uint16_t* X, int64_t M, int64_t K, int64_t ldx, const float* F,
                              int64_t ldf, int64_t r, float* P, int64_t ldp, const int64_t* off,
                              const int* pre, int64_t E, int64_t fstride, hipStream_t s) {
  if (M == 0 || r == 0) return hipSuccess;
  constexpr int64_t rows = kRowBlock;
  const int64_t blocks = off ? M / rows + E : (M + rows - 1) / rows;
  const dim3 grid((unsigned)blocks, (unsigned)((r + kRowBlock - 1) / kRowBlock));
  hipLaunchKernelGGL(lora_rowdot_kernel, grid, dim3(kThreads), 0, s, X, M, K, ldx, F, ldf, (int)r,
                     P, ldp, Groups{off, pre, (int)E}, fstride);
  return hipGetLastError();
}

int64_t lora_colsum_splits(int64_t M, int64_t C) {
  const int64_t cblocks = (C + 255) / 256;
  int64_t sp = (1024 + cblocks - 1) / cblocks;       // ~1024 workgroups
  const int64_t by_rows = (M + 127) / 128;           // at least 128 rows per split
  if (sp > by_rows) sp = by_rows;
  return sp < 1 ? 1 : sp;
}

size_t lora_colsum_part_bytes(int64_t M, int64_t C, int64_t r) {
  return (size_t)lora_colsum_splits(M, C) * (size_t)C * (size_t)r * 4;
}

size_t lora_colsum_grouped_part_bytes(int64_t T, int64_t E, int64_t C, int64_t r) {
  return (size_t)(T / kGroupChunk + E) * (size_t)C * (size_t)r * 4;
}

hipError_t launch_lora_colsum(const uint16_t* Big, int64_t M, int64_t C, int64_t ldb,
                              const float* Sm, int64_t lds_, int64_t r, float scale,
                              float* part, int transposed, float* out, const int64_t* off,
                              const int* pre, int64_t E, int per_group, hipStream_t s) {
  if (C == 0 || r == 0) return hipSuccess;
  const Groups g{off, pre, (int)E};
  int64_t splits = 0, rps = 0;
  if (off) {
    splits = M / kGroupChunk + E;
    rps = kGroupChunk;
  } else if (M > 0) {
    splits = lora_colsum_splits(M, C);
    rps = (M + splits - 1) / splits;
  }
  if (splits > 0 && M > 0) {
    const dim3 grid((unsigned)((C + 255) / 256), (unsigned)splits, (unsigned)((r + kRC - 1) / kRC));
    hipLaunchKernelGGL(lora_colsum_kernel, grid, dim3(kThreads), 0, s, Big, M, C, ldb, Sm, lds_,
                       (int)r, rps, part, g);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const int64_t n = C * r;
  const unsigned outs = off && per_group ? (unsigned)E : 1u;
  hipLaunchKernelGGL(lora_finish_kernel, dim3((unsigned)((n + 255) / 256), outs), dim3(256), 0, s,
                     part, M > 0 ? splits : 0, C, (int)r, scale, transposed, out, g, per_group);
  return hipGetLastError();
}

hipError_t launch_transpose_f32(const float* F, int64_t N, int64_t r, int64_t batch, float* Ft,
                                hipStream_t s) {
  const int64_t n = N * r;
  if (n == 0 || batch == 0) return hipSuccess;
  hipLaunchKernelGGL(transpose_f32_kernel, dim3((unsigned)((n + 255) / 256), (unsigned)batch),
                     dim3(256), 0, s, F, N, (int)r, Ft);
  return hipGetLastError();
}

}  // namespace qf
