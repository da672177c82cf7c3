// NT BF16 MFMA GEMM for gfx950: C[m, n] = sum_k A[m, k] * B[n, k], both operands k-contiguous.
//
// Every product of the quantization-aware layer is issued in this form (the backward's
// transposed operands come from the transposing quantizer / transpose kernels), so this is
// the one kernel that carries the layer's FLOPs:
//   forward  Y  = A_hat W_hat^T        A = A_hat [M, K],   B = W_hat [N, K]
//   dX          = dY W_hat             A = dY [M, N],      B = W_hat^T [K, N]
//   dW          = dY^T A_hat           A = dY^T [N, M],    B = A_hat^T [K, M]
//
// Design (256 x 256 block tile, 512 lanes = 8 wavefronts, two per SIMD):
//  - Each wavefront owns a 128 x 64 sub-tile as 4 x 2 v_mfma_f32_32x32x16_bf16 accumulators
//    (128 AGPRs); the second wavefront on a SIMD issues MFMAs while the first waits.
//  - Operands move global -> LDS with direct-to-LDS loads (global_load_lds_dwordx4): no
//    staging registers and no ds_write instructions.  Wavefronts 0-3 load A, 4-7 load B.
//  - The k loop runs in 32-deep stages through a 5-stage ring (5 x 32 KB = the whole 160 KB
//    LDS).  Loads for stage s+4 are issued at step s, three steps before they are needed, so
//    L2-miss latency is hidden; before the one barrier per step each wavefront waits only for
//    its own loads of stage s+2 (s_waitcnt vmcnt(8)).
//  - After the barrier every wavefront prefetches the first fragments of the next stage
//    while the current stage's MFMAs run, so no fragment read waits behind the barrier.
//  - LDS rows hold 32 bf16 (4 chunks of 16 bytes); chunk c of row r is stored at slot
//    c ^ ((r >> 2) & 3), which keeps 16 consecutive fragment rows on 16 distinct bank groups.
//  - Rows past the matrix edge load the last valid row (their outputs are never stored); a
//    partial last k stage goes through a masked register path after the ring drains.
//  - Block ids are remapped so each XCD (own L2) works on a contiguous group of tiles.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "qf_internal.h"

namespace qf {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int BM = 256, BN = 256, BK = 32, NSTAGE = 5;
constexpr int kOpStage = BM * BK * 2;            // 16 KB: one operand, one stage
constexpr int kStage = 2 * kOpStage;             // 32 KB: A then B
constexpr int kGroupM = 8;
constexpr int kXcds = 8;

enum Mode { kDense = 0, kGroupRows = 1 };
constexpr int kNtWaves = 8;   // wavefronts per block (the 4-wavefront form is kept compilable)

struct NtArgs {
  const uint16_t* A;
  const uint16_t* B;
  void* C;
  int64_t lda, ldb, ldc;
  int64_t bstride;        // grouped rows: elements between experts' B
  int64_t M, N, K;
  int tiles_m, tiles_n;
  const int64_t* off;     // grouped rows: [E+1] row offsets
  const int* tile_start;  // grouped rows: [E+1] per-expert tile prefix
  int E;
};

#define QF_LDS(p) ((__attribute__((address_space(3))) void*)(p))

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding).
#define QF_WAIT_VMCNT(n) \
  __builtin_amdgcn_s_waitcnt(((n) & 15) | (7 << 4) | (15 << 8) | ((((n) >> 4) & 3) << 14))

// 16-byte direct-to-LDS load: lane l's 16 bytes land at lds + 16 l (lds wave-uniform).
// (A plain function: device builtins with template-dependent operands keep the host pass
// from emitting the kernel's launch stub.)
__device__ __forceinline__ void dma16(const void* g, void* lds) {
  __builtin_amdgcn_global_load_lds(g, QF_LDS(lds), 16, 0, 0);
}

__device__ __forceinline__ uint32_t bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0u;
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ int remap_xcd(int bid, int nb) {
  const int full = nb - nb % kXcds;
  if (bid >= full) return bid;
  return (bid % kXcds) * (full / kXcds) + bid / kXcds;
}

// NW = 8: two wavefronts per SIMD, 128 x 64 each, wavefronts 0-3 load A and 4-7 load B.
// NW = 4: one wavefront per SIMD, 128 x 128 each, every wavefront loads both operands.
template <bool C_F32, int MODE, int NW>
__global__ __launch_bounds__(NW * 64, 1) void gemm_nt_kernel(NtArgs p) {
  constexpr int NJ = NW == 8 ? 2 : 4;            // 32-column accumulator blocks per wave
  constexpr int WN = NJ * 32;                    // columns per wavefront
  constexpr int NLD = NW == 8 ? 4 : 8;           // direct-to-LDS loads per wave per stage
  __shared__ __attribute__((aligned(16))) char smem[NSTAGE * kStage];
  const int tid = threadIdx.x;
  const int lane = tid & 63, w = tid >> 6;
  const int wm = NW == 8 ? w >> 2 : w >> 1, wn = NW == 8 ? w & 3 : w & 1;
  const int bid = remap_xcd(blockIdx.x, gridDim.x);

  const uint16_t* Bp = p.B;
  int64_t m0, m_end, n0;
  if (MODE == kDense) {
    const int per_group = kGroupM * p.tiles_n;
    const int g = bid / per_group;
    const int first = g * kGroupM;
    const int gs = min(p.tiles_m - first, kGroupM);
    m0 = (int64_t)(first + (bid % per_group) % gs) * BM;
    m_end = p.M;
    n0 = (int64_t)((bid % per_group) / gs) * BN;
  } else {
    const int mt = bid / p.tiles_n, tn = bid % p.tiles_n;
    if (mt >= p.tile_start[p.E]) return;         // uniform over the block
    int lo = 0, hi = p.E;                        // tile_start[e] <= mt < tile_start[e+1]
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (p.tile_start[mid] <= mt) lo = mid; else hi = mid;
    }
    m0 = p.off[lo] + (int64_t)(mt - p.tile_start[lo]) * BM;
    m_end = p.off[lo + 1];
    n0 = (int64_t)tn * BN;
    Bp += (int64_t)lo * p.bstride;
  }
  const int64_t n_end = p.N, K = p.K;

  // ---- this lane's loads: direct-to-LDS instructions of 16 rows each ------------------------
  // Load q of wavefront w fills LDS rows R0 = (4 (w & 3) + (q & 3)) * 16 .. R0 + 15 of operand
  // (NW == 8 ? w >> 2 : q >> 2); lane l lands at row R0 + l / 4, slot l % 4, which holds
  // logical chunk (l % 4) ^ ((l / 16) % 4).
  const int lw = w & 3;
  const int chunk = (lane & 3) ^ ((lane >> 4) & 3);
  const char* gbase[2];
  uint32_t goff[NLD];
  int lofs[NLD];
#pragma unroll
  for (int op = 0; op < 2; ++op) {
    const uint16_t* P = op ? Bp : p.A;
    const int64_t r0 = op ? n0 : m0;
    gbase[op] = reinterpret_cast<const char*>(P + r0 * (op ? p.ldb : p.lda));
  }
#pragma unroll
  for (int q = 0; q < NLD; ++q) {
    const int op = NW == 8 ? (w >> 2) : (q >> 2);
    const int64_t ld = op ? p.ldb : p.lda;
    const int64_t rlim = (op ? n_end : m_end) - (op ? n0 : m0) - 1;
    const int64_t row = (lw * 4 + (q & 3)) * 16 + (lane >> 2);
    const int64_t rc = row < rlim ? row : rlim;
    goff[q] = (uint32_t)((rc * ld + chunk * 8) * 2);
    lofs[q] = op * kOpStage + (lw * 4 + (q & 3)) * 1024;
  }
  const int gsel = NW == 8 ? (w >> 2) : 0;

  // ---- fragment offsets: slice kk, fragment i at fo[kk] + i * 2048 (32 rows of 64 bytes) -----
  int foa[2], fob[2];
  {
    const int ra = wm * 128 + (lane & 31), rb = wn * WN + (lane & 31);
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const int c = 2 * kk + (lane >> 5);
      foa[kk] = ra * 64 + ((c ^ ((ra >> 2) & 3)) << 4);
      fob[kk] = kOpStage + rb * 64 + ((c ^ ((rb >> 2) & 3)) << 4);
    }
  }

  f32x16_t acc[4][NJ];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j) acc[i][j] = f32x16_t{};
  bf16x8_t a0[4], b0[NJ], a1[4], b1[NJ];

  auto issue = [&](int64_t s, int buf) {
    char* l = smem + buf * kStage;
#pragma unroll
    for (int q = 0; q < NLD; ++q) {
      const char* g = gbase[NW == 8 ? gsel : (q >> 2)] + s * (BK * 2);
      dma16(g + goff[q], l + lofs[q]);
    }
  };
  auto frags = [&](const char* st, int kk, bf16x8_t* a, bf16x8_t* b) {
#pragma unroll
    for (int i = 0; i < 4; ++i) a[i] = *reinterpret_cast<const bf16x8_t*>(st + foa[kk] + i * 2048);
#pragma unroll
    for (int j = 0; j < NJ; ++j) b[j] = *reinterpret_cast<const bf16x8_t*>(st + fob[kk] + j * 2048);
  };
  auto mfma = [&](const bf16x8_t* a, const bf16x8_t* b) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < NJ; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
  };

  const int64_t nfull = K / BK;
  const int64_t krem = K % BK;
  if (nfull > 0) {
    const int64_t last = nfull - 1;
    // Ring slot of stage s is s % NSTAGE.  Stage s+4 is issued at the top of step s into the
    // slot stage s-1 used; the barrier that ends step s-1 guarantees every wavefront has
    // consumed that slot.  The barrier that ends step s guarantees stage s+2 has landed, so
    // step s+1 may prefetch its fragments.  Each wavefront issues exactly 4 loads per step
    // (stages past the end re-load the last stage into a slot nobody reads again), so
    // "stages up to t landed" is always "at most 8 loads outstanding" at the barrier.
#pragma unroll
    for (int s = 0; s < NSTAGE - 1; ++s) issue(s < last ? s : last, s);
    QF_WAIT_VMCNT(2 * NLD);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    frags(smem, 0, a0, b0);
    int buf = 0;
    for (int64_t s = 0; s < nfull; ++s) {
      const int64_t s4 = s + NSTAGE - 1;
      const int bufp = buf == 0 ? NSTAGE - 1 : buf - 1;
      const int bufn = buf == NSTAGE - 1 ? 0 : buf + 1;
      issue(s4 < last ? s4 : last, bufp);
      frags(smem + buf * kStage, 1, a1, b1);
      mfma(a0, b0);
      frags(smem + bufn * kStage, 0, a0, b0);      // next stage, slice 0
      mfma(a1, b1);
      QF_WAIT_VMCNT(2 * NLD);                            // own loads of stage s+2 landed
      __builtin_amdgcn_s_barrier();
      __builtin_amdgcn_sched_barrier(0);
      buf = bufn;
    }
    QF_WAIT_VMCNT(0);                              // drain the ring before LDS is reused
  }
  if (krem > 0) {
    // Partial last stage: masked loads through registers into ring slot 0.
    QF_WAIT_VMCNT(0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    const int64_t k0 = nfull * BK + chunk * 8;
#pragma unroll
    for (int q = 0; q < NLD; ++q) {
      uint4 v = make_uint4(0, 0, 0, 0);
      const char* g = gbase[NW == 8 ? gsel : (q >> 2)] + nfull * (BK * 2);
      if (k0 < K) v = *reinterpret_cast<const uint4*>(g + goff[q]);
      *reinterpret_cast<uint4*>(smem + lofs[q] + lane * 16) = v;
    }
    __syncthreads();
    frags(smem, 0, a0, b0);
    frags(smem, 1, a1, b1);
    mfma(a0, b0);
    mfma(a1, b1);
  }

  // ---- epilogue: accumulator element v sits at row 8(v/4) + 4(lane/32) + v%4, col lane%32 ----
  char* Cp = reinterpret_cast<char*>(p.C);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int64_t col = n0 + wn * WN + j * 32 + (lane & 31);
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

}  // namespace

hipError_t launch_gemm_nt(int64_t M, int64_t N, int64_t K, const uint16_t* A, int64_t lda,
                          const uint16_t* B, int64_t ldb, void* C, int64_t ldc, int c_f32,
                          hipStream_t s) {
  if (M == 0 || N == 0) return hipSuccess;
  NtArgs a{};
  a.A = A; a.B = B; a.C = C; a.lda = lda; a.ldb = ldb; a.ldc = ldc;
  a.M = M; a.N = N; a.K = K;
  a.tiles_m = (int)((M + BM - 1) / BM);
  a.tiles_n = (int)((N + BN - 1) / BN);
  const dim3 grid((unsigned)(a.tiles_m * a.tiles_n));
  if (c_f32) hipLaunchKernelGGL((gemm_nt_kernel<true, kDense, kNtWaves>), grid, dim3(kNtWaves * 64), 0, s, a);
  else hipLaunchKernelGGL((gemm_nt_kernel<false, kDense, kNtWaves>), grid, dim3(kNtWaves * 64), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_grouped_nt_rows(int64_t E, int64_t T, int64_t N, int64_t K, const int64_t* off,
                                  const int* tile_start, const uint16_t* A, int64_t lda,
                                  const uint16_t* B, int64_t ldb, int64_t bstride, uint16_t* C,
                                  int64_t ldc, hipStream_t s) {
  if (T == 0 || N == 0 || E == 0) return hipSuccess;
  NtArgs a{};
  a.A = A; a.B = B; a.C = C; a.lda = lda; a.ldb = ldb; a.ldc = ldc; a.bstride = bstride;
  a.M = T; a.N = N; a.K = K; a.off = off; a.tile_start = tile_start; a.E = (int)E;
  a.tiles_n = (int)((N + BN - 1) / BN);
  a.tiles_m = (int)((T + BM - 1) / BM + E);
  const dim3 grid((unsigned)(a.tiles_m * a.tiles_n));
  hipLaunchKernelGGL((gemm_nt_kernel<false, kGroupRows, kNtWaves>), grid, dim3(kNtWaves * 64), 0, s, a);
  return hipGetLastError();
}

}  // namespace qf
