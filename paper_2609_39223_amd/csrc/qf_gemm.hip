// BF16 MFMA GEMMs for the quantization-aware linear layer on gfx950 (CDNA4).
//
//   C[m, n] = sum_k A(m, k) * B(n, k)        FP32 accumulation, bf16 or FP32 output
//
// Each operand is either k-major (stored [MN][K], contraction contiguous) or mn-major
// (stored [K][MN]).  The layer's products run on the NT kernel (qf_gemm_nt.hip) with both
// operands k-major; this template covers the other layouts of the plain GEMM entry point and
// the layer backward when the token count is not a multiple of 8 (dX = dY W_hat as (k,mn),
// dW = dY^T A_hat as (mn,mn)), reading mn-major operands in place.
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

enum Mode { kDense = 0 };

struct GemmArgs {
  const uint16_t* A;
  const uint16_t* B;
  void* C;
  int64_t lda, ldb, ldc;
  int64_t M, N, K;
  int tiles_m, tiles_n;
};

__device__ __forceinline__ int lds_off(int r, int c) {
  return r * 128 + ((c ^ (r & 7) ^ ((r >> 3) & 7)) << 4);
}

__device__ __forceinline__ uint32_t bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0u;
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

// LDS layout (128 KB): [A stage buffer 0 | A buffer 1 | B buffer 0 | B buffer 1], 32 KB each.
constexpr int kLdsB = 2 * kTileBytes;

// One operand's staging state for the block.
// k-major: element (mn, k) at P[mn * ld + k]; lane t owns chunks (row 32 i + t / 8, chunk t % 8).
// mn-major: element (mn, k) at P[k * ld + mn]; lane t owns the 8 x 8 block of rows
//   k = 8 (t / 32) + i and columns mn = 8 (t % 32) + j, transposed in registers so that LDS
//   holds it k-contiguous like the k-major operand.
// `base` (uniform) is the tile origin at the block's first k; a 64-deep step advances it by
// `step` bytes; `off` are per-lane byte offsets (rows past the matrix end are clamped to the
// last row: they only feed outputs that are never stored).  `wr` are per-lane LDS offsets.
template <bool KMAJOR>
struct Operand {
  const char* base;
  int64_t step;
  uint32_t off[8];
  int wr[8];
  uint4 v[8];

  __device__ __forceinline__ void init(const uint16_t* P, int64_t ld, int64_t mn0,
                                       int64_t mn_end, int64_t kb, int tid) {
    if (KMAJOR) {
      base = reinterpret_cast<const char*>(P + mn0 * ld + kb);
      step = (int64_t)BK * 2;
      const int c = tid & 7;
      const int64_t lim = mn_end - mn0 - 1;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int rel = i * 32 + (tid >> 3);
        const int64_t rc = rel < lim ? rel : lim;
        off[i] = (uint32_t)((rc * ld + c * 8) * 2);
        wr[i] = lds_off(rel, c);
      }
    } else {
      base = reinterpret_cast<const char*>(P + kb * ld + mn0);
      step = (int64_t)BK * ld * 2;
      const int mg = tid & 31, kg = tid >> 5;
      const int64_t lim = mn_end - mn0 - 8;
      const int64_t cc = mg * 8 < lim ? mg * 8 : lim;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        off[i] = (uint32_t)(((int64_t)(kg * 8 + i) * ld + cc) * 2);
        wr[i] = lds_off(mg * 8 + i, kg);
      }
    }
  }

  __device__ __forceinline__ void load(int i, int64_t s) {
    v[i] = *reinterpret_cast<const uint4*>(base + s * step + off[i]);
  }
  __device__ __forceinline__ void load_all(int64_t s) {
#pragma unroll
    for (int i = 0; i < 8; ++i) load(i, s);
  }
  // Partial last step: contraction indices >= krem (relative to the step) read as zero.
  __device__ __forceinline__ void load_tail(int64_t s, int64_t krem, int tid) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int64_t k = KMAJOR ? (tid & 7) * 8 : (tid >> 5) * 8 + i;
      v[i] = make_uint4(0, 0, 0, 0);
      if (k < krem) load(i, s);
    }
  }
  // k-major: chunk i -> its LDS slot.
  __device__ __forceinline__ void write(int i, char* lds) const {
    *reinterpret_cast<uint4*>(lds + wr[i]) = v[i];
  }
  // mn-major: transpose the 8 x 8 bf16 block and store the 8 k-contiguous chunks.
  __device__ __forceinline__ void write_transposed(char* lds) const {
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
      *reinterpret_cast<uint4*>(lds + wr[j]) = make_uint4(o[0], o[1], o[2], o[3]);
    }
  }
  __device__ __forceinline__ void write_all(char* lds) const {
    if (KMAJOR) {
#pragma unroll
      for (int i = 0; i < 8; ++i) write(i, lds);
    } else {
      write_transposed(lds);
    }
  }
};

// Which chunks of an operand are written to LDS in which k-slice of a step (see the pipeline
// below).  k-major operands spread their 8 chunks as pairs over slices 3, 0, 1, 2; mn-major
// operands write all 8 at once (the transpose needs all eight rows): A in slice 3, B in 0.
template <bool KMAJOR, bool IS_A>
__device__ __forceinline__ constexpr bool writes_in(int slice, int i) {
  return KMAJOR ? ((i >> 1) == ((slice + 1) & 3)) : (slice == (IS_A ? 3 : 0));
}

template <bool KMAJOR, bool IS_A>
__device__ __forceinline__ void stage_slice(Operand<KMAJOR>& op, int slice, char* wbuf,
                                            int64_t load_stage) {
  if (KMAJOR) {
#pragma unroll
    for (int i = 0; i < 8; ++i)
      if (writes_in<KMAJOR, IS_A>(slice, i)) { op.write(i, wbuf); op.load(i, load_stage); }
  } else if (writes_in<KMAJOR, IS_A>(slice, 0)) {
    op.write_transposed(wbuf);
    op.load_all(load_stage);
  }
}

// Per-lane LDS byte offsets of this wave's MFMA fragments: fragment i of k-slice kk sits at
// frag_off[kk][i & 1] + i * 4096 (row 32 i further; the swizzle term (row >> 3) & 7 flips by
// 4 for odd i).
__device__ __forceinline__ void frag_offsets(int rbase, int lane, int fo[4][2]) {
  const int r = rbase + (lane & 31);
  const int g = (lane >> 5) ^ (r & 7) ^ ((r >> 3) & 7);
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) {
    fo[kk][0] = r * 128 + ((g ^ (2 * kk)) << 4);
    fo[kk][1] = r * 128 + ((g ^ (2 * kk) ^ 4) << 4);
  }
}

__device__ __forceinline__ void read_frags(const char* __restrict__ a, const char* __restrict__ b,
                                           const int fa[2], const int fb[2], bf16x8_t af[4],
                                           bf16x8_t bfr[4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
    af[i] = *reinterpret_cast<const bf16x8_t*>(a + fa[i & 1] + i * 4096);
#pragma unroll
  for (int j = 0; j < 4; ++j)
    bfr[j] = *reinterpret_cast<const bf16x8_t*>(b + fb[j & 1] + j * 4096);
}

__device__ __forceinline__ void mfma16(f32x16_t acc[4][4], const bf16x8_t af[4],
                                       const bf16x8_t bfr[4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
      acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
}

// Scheduling-group masks (AMDGPU backend): MFMA, DS read, DS write, VMEM read.
#define QF_SG(mask, n) __builtin_amdgcn_sched_group_barrier(mask, n, 0)
constexpr int kSgMfma = 0x008, kSgDsRead = 0x100, kSgDsWrite = 0x200, kSgVmemRead = 0x020;

// Interleave one k-slice: 16 MFMAs with 8 fragment reads and this slice's LDS writes and
// global loads.
__device__ __forceinline__ void sched_slice(int nw) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    QF_SG(kSgMfma, 1);
    QF_SG(kSgDsRead, 1);
    if (i < nw) { QF_SG(kSgDsWrite, 1); QF_SG(kSgVmemRead, 1); }
    QF_SG(kSgMfma, 1);
    if (i + 8 < nw) { QF_SG(kSgDsWrite, 1); QF_SG(kSgVmemRead, 1); }
  }
}

template <bool KM>
__device__ __forceinline__ constexpr int nwrites(int slice, bool is_a) {
  return KM ? 2 : ((slice == (is_a ? 3 : 0)) ? 8 : 0);
}

__device__ __forceinline__ int remap_xcd(int bid, int nb) {
  const int full = nb - nb % kXcds;
  if (bid >= full) return bid;
  return (bid % kXcds) * (full / kXcds) + bid / kXcds;
}

// Software pipeline over 64-deep k steps, one barrier per step, LDS double buffer.
// During step kt (reading stage kt from buffer kt&1):
//   slices 0-2: MFMAs on slices 0-2 of stage kt; fragment reads of slices 1-3; LDS writes of
//               the slice-0..2 chunks of stage kt+1 into buffer (kt+1)&1, each followed by the
//               global load of the same chunk of stage kt+2 into the freed registers
//   barrier   : stage kt+1 is complete in LDS; every wave is done reading buffer kt&1
//   slice 3   : MFMAs on slice 3; fragment reads of slice 0 of stage kt+1; LDS writes of the
//               slice-3 chunks of stage kt+2 into buffer kt&1, then loads of stage kt+3
// Every chunk is therefore loaded one full step before it is written to LDS.  Loads past the
// last full stage re-read the last stage (uniform clamp) and are never used.
template <bool A_KM, bool B_KM, int CUR>
__device__ __forceinline__ void pipeline_step(int64_t kt, int64_t last, Operand<A_KM>& A,
                                              Operand<B_KM>& B, char* smem, const int fa[4][2],
                                              const int fb[4][2], bf16x8_t af0[4],
                                              bf16x8_t bf0[4], bf16x8_t af1[4], bf16x8_t bf1[4],
                                              f32x16_t acc[4][4]) {
  char* aCur = smem + CUR * kTileBytes;
  char* aNxt = smem + (1 - CUR) * kTileBytes;
  char* bCur = smem + kLdsB + CUR * kTileBytes;
  char* bNxt = smem + kLdsB + (1 - CUR) * kTileBytes;
  const int64_t s2 = kt + 2 <= last ? kt + 2 : last;
  const int64_t s3 = kt + 3 <= last ? kt + 3 : last;
  // slice 0
  read_frags(aCur, bCur, fa[1], fb[1], af1, bf1);
  stage_slice<A_KM, true>(A, 0, aNxt, s2);
  stage_slice<B_KM, false>(B, 0, bNxt, s2);
  mfma16(acc, af0, bf0);
  sched_slice(nwrites<A_KM>(0, true) + nwrites<B_KM>(0, false));
  // slice 1
  read_frags(aCur, bCur, fa[2], fb[2], af0, bf0);
  stage_slice<A_KM, true>(A, 1, aNxt, s2);
  stage_slice<B_KM, false>(B, 1, bNxt, s2);
  mfma16(acc, af1, bf1);
  sched_slice(nwrites<A_KM>(1, true) + nwrites<B_KM>(1, false));
  // slice 2
  read_frags(aCur, bCur, fa[3], fb[3], af1, bf1);
  stage_slice<A_KM, true>(A, 2, aNxt, s2);
  stage_slice<B_KM, false>(B, 2, bNxt, s2);
  mfma16(acc, af0, bf0);
  sched_slice(nwrites<A_KM>(2, true) + nwrites<B_KM>(2, false));
  __syncthreads();
  // slice 3
  read_frags(aNxt, bNxt, fa[0], fb[0], af0, bf0);
  stage_slice<A_KM, true>(A, 3, aCur, s3);
  stage_slice<B_KM, false>(B, 3, bCur, s3);
  mfma16(acc, af1, bf1);
  sched_slice(nwrites<A_KM>(3, true) + nwrites<B_KM>(3, false));
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
  }

  f32x16_t acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x16_t{};

  Operand<A_KM> A;
  Operand<B_KM> B;
  A.init(Ap, p.lda, m0, m_end, kb, tid);
  B.init(Bp, p.ldb, n0, n_end, kb, tid);
  int fa[4][2], fb[4][2];
  frag_offsets(wm * 128, lane, fa);
  frag_offsets(wn * 128, lane, fb);
  bf16x8_t af0[4], bf0[4], af1[4], bf1[4];
  const int64_t depth = ke > kb ? ke - kb : 0;
  const int64_t nfull = depth / BK;
  const int64_t krem = depth % BK;

  if (nfull > 0) {
    const int64_t last = nfull - 1;
    // prologue: stage 0 -> buffer 0; stage 1's slice-3 chunks -> buffer 1; registers hold
    // stage 1 for slices 0-2 and stage 2 for slice 3.
    A.load_all(0);
    B.load_all(0);
    A.write_all(smem);
    B.write_all(smem + kLdsB);
    A.load_all(last < 1 ? last : 1);
    B.load_all(last < 1 ? last : 1);
    stage_slice<A_KM, true>(A, 3, smem + kTileBytes, last < 2 ? last : 2);
    stage_slice<B_KM, false>(B, 3, smem + kLdsB + kTileBytes, last < 2 ? last : 2);
    __syncthreads();
    read_frags(smem, smem + kLdsB, fa[0], fb[0], af0, bf0);
    int64_t kt = 0;
    for (; kt + 1 < nfull; kt += 2) {
      pipeline_step<A_KM, B_KM, 0>(kt, last, A, B, smem, fa, fb, af0, bf0, af1, bf1, acc);
      pipeline_step<A_KM, B_KM, 1>(kt + 1, last, A, B, smem, fa, fb, af0, bf0, af1, bf1, acc);
    }
    if (kt < nfull)
      pipeline_step<A_KM, B_KM, 0>(kt, last, A, B, smem, fa, fb, af0, bf0, af1, bf1, acc);
  }
  if (krem > 0) {
    // partial last step, outside the pipeline: masked loads straight into buffer 0
    __syncthreads();
    A.load_tail(nfull, krem, tid);
    B.load_tail(nfull, krem, tid);
    A.write_all(smem);
    B.write_all(smem + kLdsB);
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      read_frags(smem, smem + kLdsB, fa[kk], fb[kk], af0, bf0);
      mfma16(acc, af0, bf0);
    }
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
                                    int* order, int* kstart, int* korder) {
  __shared__ int cnt[1024], cnt64[1024];
  const int e = threadIdx.x;
  int64_t rows = 0;
  if (e < E) rows = off[e + 1] - off[e];
  if (e < E) cnt[e] = (int)((rows + BM - 1) / BM);
  if (e < E) cnt64[e] = (int)((rows + 63) / 64);
  __syncthreads();
  if (e == 0) {
    int s = 0;
    for (int i = 0; i < E; ++i) { tile_start[i] = s; s += cnt[i]; }
    tile_start[E] = s;
  }
  if (e == 0 && kstart) {                        // 64-row units: padded k ranges of dW
    int s = 0;
    for (int i = 0; i < E; ++i) { kstart[i] = s; s += cnt64[i]; }
    kstart[E] = s;
  }
  if (e < E && order) {
    int rank = 0;
    for (int i = 0; i < E; ++i) {
      const int64_t ri = off[i + 1] - off[i];
      rank += (ri > rows) || (ri == rows && i < e);
    }
    order[rank] = e;
    if (korder) {
      // Balanced over the 8 XCDs for launches whose items run as 8 contiguous ranges (one per
      // XCD): ranks are dealt in a snake (0..7 to XCDs 0..7, 8..15 to XCDs 7..0, ...), and
      // each XCD's experts stay in decreasing order.  Needs E % 8 == 0 (else the plain order).
      int pos = rank;
      if (E % 8 == 0) {
        const int k = rank / 8, i = rank % 8;
        const int x = (k & 1) ? 7 - i : i;
        pos = x * (E / 8) + k;
      }
      korder[pos] = e;
    }
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
                               int* kstart, int* korder, hipStream_t s) {
  hipLaunchKernelGGL(grouped_prep_kernel, dim3(1), dim3(1024), 0, s, off, (int)E, tile_start,
                     order, kstart, korder);
  return hipGetLastError();
}

}  // namespace qf
