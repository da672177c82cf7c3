// BF16 MFMA GEMMs for the quantization-aware linear layer on gfx950 (CDNA4).
//
//   C[m, n] = sum_k A(m, k) * B(n, k)        FP32 accumulation, bf16 or FP32 output
//
// Each operand is either k-major (stored [MN][K], contraction contiguous: X, W, dY in the
// forward and dX GEMMs) or mn-major (stored [K][MN]: W_hat as the right operand of
// dX = dY W_hat, and both operands of dW = dY^T A_hat).  The three products of the layer
// (Eqs. fakequant, ste, activation-ste) are the three layout combinations (k,k), (k,mn),
// (mn,mn) of one kernel template.
//
// Block tile 256 x 256 x 64, 256 lanes = 4 wavefronts in a 2 x 2 grid, each wavefront
// owning a 128 x 128 sub-tile as 4 x 4 v_mfma_f32_32x32x16_bf16 accumulators (256 AGPRs).
// Operand tiles are staged global -> VGPR -> LDS with 128-bit accesses and double buffered
// in LDS (2 x 64 KB of the 160 KB per CU), so the next tile's global loads overlap the
// current tile's MFMAs and one barrier per 64-deep step suffices.
//
// LDS holds both operands k-contiguous: row r (an m or n index) of 64 bf16 = 8 chunks of
// 16 bytes; chunk c of row r sits at chunk slot c ^ (r & 7) ^ ((r >> 3) & 7).  The swizzle
// keeps the 8 lanes served per LDS cycle on distinct banks for all three access streams:
// MFMA fragment reads (8 consecutive rows, same chunk), k-major stores (one row, 8
// chunks) and mn-major stores (rows 8 apart after the in-register 8x8 transpose).
//
// Block order: workgroups are dispatched round-robin over the 8 XCDs, each with its own L2.
// The linear block id is remapped so each XCD receives a contiguous range of tiles, and
// tiles are walked in groups of 8 tile-rows so concurrently running blocks share operand
// tiles in that XCD's L2.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "qf_internal.h"

namespace qf {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int BM = 256, BN = 256, BK = 64, NTHR = 256;
constexpr int kTileBytes = BM * BK * 2;   // one operand stage: 32 KB
constexpr int kGroupM = 8;
constexpr int kXcds = 8;

enum Mode { kDense = 0, kGroupRows = 1, kGroupWgrad = 2 };

struct GemmArgs {
  const uint16_t* A;
  const uint16_t* B;
  void* C;
  int64_t lda, ldb, ldc;
  int64_t bstride;   // grouped: elements between consecutive experts' B
  int64_t cstride;   // grouped wgrad: elements between consecutive experts' C
  int64_t M, N, K;
  int tiles_m, tiles_n;
  const int64_t* off;      // grouped: device [E+1] row offsets
  const int* tile_start;   // grouped rows: [E+1] prefix of per-expert m-tile counts
  const int* order;        // grouped wgrad: experts by decreasing row count
  int E;
};

__device__ __forceinline__ int lds_off(int r, int c) {
  return r * 128 + ((c ^ (r & 7) ^ ((r >> 3) & 7)) << 4);
}

__device__ __forceinline__ uint32_t bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0u;
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

// Operand tile [256 mn][64 k] read from global into registers.
// k-major: element (mn, k) at P[mn * ld + k]; lane t reads chunks (r = 32 i + t / 8, c = t % 8).
// mn-major: element (mn, k) at P[k * ld + mn]; lane t reads rows k = 8 (t / 32) + i of the
//   8 mn values starting at 8 (t % 32), to be transposed in registers before the LDS store.
template <bool KMAJOR>
struct Stage {
  uint4 v[8];

  __device__ __forceinline__ void load(const uint16_t* __restrict__ P, int64_t ld, int64_t mn0,
                                       int64_t mn_end, int64_t k0, int64_t k_end, int tid) {
    if (KMAJOR) {
      const int c = tid & 7;
      const int64_t k = k0 + c * 8;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int64_t mn = mn0 + i * 32 + (tid >> 3);
        v[i] = make_uint4(0, 0, 0, 0);
        if (mn < mn_end && k < k_end) v[i] = *reinterpret_cast<const uint4*>(P + mn * ld + k);
      }
    } else {
      const int64_t mn = mn0 + (tid & 31) * 8;
      const int64_t kb = k0 + (tid >> 5) * 8;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        v[i] = make_uint4(0, 0, 0, 0);
        if (mn < mn_end && kb + i < k_end)
          v[i] = *reinterpret_cast<const uint4*>(P + (kb + i) * ld + mn);
      }
    }
  }

  __device__ __forceinline__ void store(char* __restrict__ lds, int tid) const {
    if (KMAJOR) {
      const int c = tid & 7;
#pragma unroll
      for (int i = 0; i < 8; ++i)
        *reinterpret_cast<uint4*>(lds + lds_off(i * 32 + (tid >> 3), c)) = v[i];
    } else {
      const int mg = tid & 31, kg = tid >> 5;
      uint32_t w[8][4];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        w[i][0] = v[i].x; w[i][1] = v[i].y; w[i][2] = v[i].z; w[i][3] = v[i].w;
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        uint32_t o[4];
#pragma unroll
        for (int d = 0; d < 4; ++d) {
          const uint32_t lo = w[2 * d][j >> 1], hi = w[2 * d + 1][j >> 1];
          o[d] = (j & 1) ? ((lo >> 16) | (hi & 0xFFFF0000u)) : ((lo & 0xFFFFu) | (hi << 16));
        }
        *reinterpret_cast<uint4*>(lds + lds_off(mg * 8 + j, kg)) = make_uint4(o[0], o[1], o[2], o[3]);
      }
    }
  }
};

__device__ __forceinline__ int remap_xcd(int bid, int nb) {
  const int full = nb - nb % kXcds;
  if (bid >= full) return bid;
  return (bid % kXcds) * (full / kXcds) + bid / kXcds;
}

template <bool A_KM, bool B_KM, bool C_F32, int MODE>
__global__ __launch_bounds__(NTHR, 1) void gemm_kernel(GemmArgs p) {
  __shared__ __attribute__((aligned(16))) char smem[4 * kTileBytes];
  const int tid = threadIdx.x;
  const int lane = tid & 63, w = tid >> 6, wm = w >> 1, wn = w & 1;
  const int bid = remap_xcd(blockIdx.x, gridDim.x);

  // ---- resolve this block's problem -------------------------------------------------------
  const uint16_t* Ap = p.A;
  const uint16_t* Bp = p.B;
  char* Cp = reinterpret_cast<char*>(p.C);
  int64_t m0, m_end, n0, n_end = p.N, kb = 0, ke = p.K;
  if (MODE == kDense) {
    const int per_group = kGroupM * p.tiles_n;
    const int g = bid / per_group;
    const int first = g * kGroupM;
    const int gs = min(p.tiles_m - first, kGroupM);
    const int tm = first + (bid % per_group) % gs;
    const int tn = (bid % per_group) / gs;
    m0 = (int64_t)tm * BM; m_end = p.M;
    n0 = (int64_t)tn * BN;
  } else if (MODE == kGroupRows) {
    const int mt = bid / p.tiles_n, tn = bid % p.tiles_n;
    if (mt >= p.tile_start[p.E]) return;        // uniform over the block
    int lo = 0, hi = p.E;                       // find e: tile_start[e] <= mt < tile_start[e+1]
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (p.tile_start[mid] <= mt) lo = mid; else hi = mid;
    }
    const int e = lo;
    m0 = p.off[e] + (int64_t)(mt - p.tile_start[e]) * BM;
    m_end = p.off[e + 1];
    n0 = (int64_t)tn * BN;
    Bp += (int64_t)e * p.bstride;
  } else {
    const int tpe = p.tiles_m * p.tiles_n;
    const int e = p.order[bid / tpe];
    const int t = bid % tpe;
    m0 = (int64_t)(t / p.tiles_n) * BM; m_end = p.M;
    n0 = (int64_t)(t % p.tiles_n) * BN;
    kb = p.off[e]; ke = p.off[e + 1];
    Cp += (int64_t)e * p.cstride * (C_F32 ? 4 : 2);
  }

  f32x16_t acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x16_t{};

  const int64_t nk = ke > kb ? (ke - kb + BK - 1) / BK : 0;
  Stage<A_KM> sa;
  Stage<B_KM> sb;
  if (nk > 0) {
    sa.load(Ap, p.lda, m0, m_end, kb, ke, tid);
    sb.load(Bp, p.ldb, n0, n_end, kb, ke, tid);
    sa.store(smem, tid);
    sb.store(smem + kTileBytes, tid);
  }
  __syncthreads();

  for (int64_t kt = 0; kt < nk; ++kt) {
    char* cur = smem + (kt & 1) * 2 * kTileBytes;
    char* nxt = smem + ((kt + 1) & 1) * 2 * kTileBytes;
    const bool more = kt + 1 < nk;
    if (more) {
      const int64_t k0 = kb + (kt + 1) * BK;
      sa.load(Ap, p.lda, m0, m_end, k0, ke, tid);
      sb.load(Bp, p.ldb, n0, n_end, k0, ke, tid);
    }
    const char* As = cur;
    const char* Bs = cur + kTileBytes;
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      const int c = kk * 2 + (lane >> 5);
      bf16x8_t af[4], bfr[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        af[i] = *reinterpret_cast<const bf16x8_t*>(As + lds_off(wm * 128 + i * 32 + (lane & 31), c));
#pragma unroll
      for (int j = 0; j < 4; ++j)
        bfr[j] = *reinterpret_cast<const bf16x8_t*>(Bs + lds_off(wn * 128 + j * 32 + (lane & 31), c));
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (more) {
      sa.store(nxt, tid);
      sb.store(nxt + kTileBytes, tid);
    }
    __syncthreads();
  }

  // ---- epilogue: accumulator (row 8(v/4) + 4(lane/32) + v%4, col lane%32) -> C -------------
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t col = n0 + wn * 128 + j * 32 + (lane & 31);
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int64_t row = m0 + wm * 128 + i * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
        if (row < m_end && col < n_end) {
          if (C_F32)
            reinterpret_cast<float*>(Cp)[row * p.ldc + col] = acc[i][j][v];
          else
            reinterpret_cast<uint16_t*>(Cp)[row * p.ldc + col] = (uint16_t)bf16_rne(acc[i][j][v]);
        }
      }
    }
  }
}

// Per-expert tile prefix (grouped rows) and experts ordered by decreasing row count (grouped
// wgrad, so the longest contractions start first).  One block, E <= 1024 lanes.
__global__ void grouped_prep_kernel(const int64_t* __restrict__ off, int E, int* tile_start,
                                    int* order) {
  __shared__ int cnt[1024];
  const int e = threadIdx.x;
  int64_t rows = 0;
  if (e < E) rows = off[e + 1] - off[e];
  if (e < E) cnt[e] = (int)((rows + BM - 1) / BM);
  __syncthreads();
  if (e == 0) {
    int s = 0;
    for (int i = 0; i < E; ++i) { tile_start[i] = s; s += cnt[i]; }
    tile_start[E] = s;
  }
  if (e < E && order) {
    int rank = 0;
    for (int i = 0; i < E; ++i) {
      const int64_t ri = off[i + 1] - off[i];
      rank += (ri > rows) || (ri == rows && i < e);
    }
    order[rank] = e;
  }
}

template <bool A_KM, bool B_KM, bool C_F32, int MODE>
hipError_t launch(const GemmArgs& a, int blocks, hipStream_t s) {
  hipLaunchKernelGGL((gemm_kernel<A_KM, B_KM, C_F32, MODE>), dim3(blocks), dim3(NTHR), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm(int64_t M, int64_t N, int64_t K, const uint16_t* A, int64_t lda,
                       int a_kmajor, const uint16_t* B, int64_t ldb, int b_kmajor, void* C,
                       int64_t ldc, int c_f32, hipStream_t s) {
  if (M == 0 || N == 0) return hipSuccess;
  GemmArgs a{};
  a.A = A; a.B = B; a.C = C; a.lda = lda; a.ldb = ldb; a.ldc = ldc;
  a.M = M; a.N = N; a.K = K;
  a.tiles_m = (int)((M + BM - 1) / BM);
  a.tiles_n = (int)((N + BN - 1) / BN);
  const int blocks = a.tiles_m * a.tiles_n;
  const int key = (a_kmajor ? 4 : 0) | (b_kmajor ? 2 : 0) | (c_f32 ? 1 : 0);
  switch (key) {
    case 7: return launch<true, true, true, kDense>(a, blocks, s);
    case 6: return launch<true, true, false, kDense>(a, blocks, s);
    case 5: return launch<true, false, true, kDense>(a, blocks, s);
    case 4: return launch<true, false, false, kDense>(a, blocks, s);
    case 3: return launch<false, true, true, kDense>(a, blocks, s);
    case 2: return launch<false, true, false, kDense>(a, blocks, s);
    case 1: return launch<false, false, true, kDense>(a, blocks, s);
    default: return launch<false, false, false, kDense>(a, blocks, s);
  }
}

hipError_t launch_grouped_prep(const int64_t* off, int64_t E, int* tile_start, int* order,
                               hipStream_t s) {
  hipLaunchKernelGGL(grouped_prep_kernel, dim3(1), dim3(1024), 0, s, off, (int)E, tile_start,
                     order);
  return hipGetLastError();
}

hipError_t launch_grouped_rows_ws(int64_t E, int64_t T, int64_t N, int64_t K, const int64_t* off,
                                  const int* tile_start, const uint16_t* A, int64_t lda,
                                  const uint16_t* B, int64_t ldb, int64_t bstride, int b_kmajor,
                                  uint16_t* C, int64_t ldc, hipStream_t s) {
  if (T == 0 || N == 0 || E == 0) return hipSuccess;
  GemmArgs a{};
  a.A = A; a.B = B; a.C = C; a.lda = lda; a.ldb = ldb; a.ldc = ldc; a.bstride = bstride;
  a.M = T; a.N = N; a.K = K; a.off = off; a.tile_start = tile_start; a.E = (int)E;
  a.tiles_n = (int)((N + BN - 1) / BN);
  a.tiles_m = (int)((T + BM - 1) / BM + E);   // upper bound on sum_e ceil(M_e / BM)
  const int blocks = a.tiles_m * a.tiles_n;
  if (b_kmajor) return launch<true, true, false, kGroupRows>(a, blocks, s);
  return launch<true, false, false, kGroupRows>(a, blocks, s);
}

hipError_t launch_grouped_wgrad_ws(int64_t E, int64_t T, int64_t N, int64_t K, const int64_t* off,
                                   const int* order, const uint16_t* dY, int64_t ldy,
                                   const uint16_t* X, int64_t ldx, float* C, hipStream_t s) {
  if (E == 0 || N == 0 || K == 0) return hipSuccess;
  GemmArgs a{};
  a.A = dY; a.B = X; a.C = C; a.lda = ldy; a.ldb = ldx; a.ldc = K; a.cstride = N * K;
  a.M = N; a.N = K; a.K = T; a.off = off; a.order = order; a.E = (int)E;
  a.tiles_m = (int)((N + BM - 1) / BM);
  a.tiles_n = (int)((K + BN - 1) / BN);
  const int blocks = a.tiles_m * a.tiles_n * (int)E;
  return launch<false, false, true, kGroupWgrad>(a, blocks, s);
}

}  // namespace qf
