// NT BF16 MFMA GEMM for gfx950: C[m, n] = sum_k A[m, k] * B[n, k], both operands k-contiguous.
//
// Every product of the quantization-aware layer is issued in this form (the backward's
// transposed operands come from the transpose kernel), so this is the one kernel that carries
// the layer's FLOPs:
//   forward  Y  = A_hat W_hat^T        A = A_hat [M, K],   B = W_hat [N, K]
//   dX          = dY W_hat             A = dY [M, N],      B = W_hat^T [K, N]
//   dW          = dY^T A_hat           A = dY^T [N, M],    B = A_hat^T [K, M]
//
// Design (256 x 256 block tile):
//  - k-contiguous operands (every layer product): 4 wavefronts, one per SIMD, each owning a
//    128 x 128 sub-tile as 4 x 4 v_mfma_f32_32x32x16_bf16 accumulators (256 AGPRs).  Operands
//    stored with K as rows: 8 wavefronts, two per SIMD, 128 x 64 each (4 x 2 accumulators).
//    The bullets below describe the eight-wavefront load split; the four-wavefront form loads
//    64 rows of both operands per wavefront (see the kernel).
//  - K advances in 64-deep stages, double-buffered in LDS (2 x 64 KB).  A stage row is 128
//    bytes, so every global request is a whole 128-byte cache line (32-deep stages fetch half
//    lines and double the L2 request count).
//  - Operands move global -> LDS with direct-to-LDS loads (no staging registers, no ds_write):
//    wavefronts 0-3 load A, 4-7 load B, 8 loads of 8 rows each per wavefront and stage.  The
//    loads of stage s+1 are spread over four slices (the last of step s-1, right after the
//    barrier that frees its buffer, and the first two of step s), so the memory pipe sees a
//    steady stream rather than a burst, and the last of them has a full slice to land.
//  - Each MFMA is followed by one fragment read for the next slice (and, in three slices of
//    four, up to one direct-to-LDS load), so the LDS and memory pipes work while the MFMA pipe
//    is busy.
//    One barrier per step, before the last slice: it publishes stage s+1 (all loads waited)
//    and retires every read of stage s (so step s+1 may overwrite that buffer).
//  - LDS rows hold 64 bf16 (8 chunks of 16 bytes); chunk c of row r sits at slot
//    c ^ ((r >> 1) & 7), so the 16 rows a fragment read serves in one pass fall on 16
//    distinct 16-byte bank groups.
//  - Rows past the matrix edge load the last valid row (their outputs are never stored); a
//    partial last k stage goes through a masked register path.
//  - The epilogue stages the tile through LDS (rows padded so both half-waves of a write hit
//    different banks) and writes whole rows with 16-byte stores; FP32 tiles go in two halves.
//  - Block ids are remapped so each XCD (own L2) works on a contiguous group of tiles, and
//    each XCD walks K from its own rotated start (HBM channel spread).
//  - Optionally (kDenseAT / kGroupRowsAT, the backward's dX = dY W_hat, dense or per expert)
//    the launch also writes A^T: each staged k stage of A is split into 16 pieces of 4 k-rows,
//    each owned by one tile of the row panel, which gathers its piece from LDS before the
//    step's barrier and stores it as whole 128-byte rows after it.  That replaces a separate
//    transpose pass over dY (grouped: into the padded per-expert columns of the weight
//    gradient, zeros included).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <type_traits>

#include "qf.h"
#include "qf_codecs.h"
#include "qf_internal.h"

namespace qf {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef short v8i16 __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned u32x2_t __attribute__((ext_vector_type(2)));

constexpr int BM = 256, BN = 256, BK = 64;
constexpr int kRow = BK * 2;                     // 128 bytes per LDS row
constexpr int kOpStage = BM * kRow;              // 32 KB: one operand, one stage
constexpr int kStage = 2 * kOpStage;             // 64 KB: A then B
// Dense tile order: groups of kGroupM row tiles, walked column by column (the 9B layer step
// measured 31.2 / 30.2 / 29.5 / 29.9 / 32.0 / 36.4 ms for groups of 1 / 2 / 4 / 8 / 16 / 32).
constexpr int kGroupM = 4;
constexpr int kXcds = 8;
constexpr int64_t kMaxSplitTiles = 128;          // split tiles of the last round, at most
constexpr int kPitch16 = BN * 2 + 16;            // epilogue LDS row pitch, bf16 tile (528 B)
constexpr int kPitch32 = BN * 4 + 32;            // epilogue LDS row pitch, FP32 half tile
constexpr int kSmemEpi = (BM * kPitch16 > 128 * kPitch32) ? BM * kPitch16 : 128 * kPitch32;
constexpr int kSmem = (2 * kStage > kSmemEpi) ? 2 * kStage : kSmemEpi;

// Fragment-major layout of a B operand [N, K] (K a multiple of 16): block (nb, kb) holds rows
// 32 nb .. 32 nb + 31 and columns 16 kb .. 16 kb + 15 as the 64 lanes' MFMA operands of
// v_mfma_f32_32x32x16_bf16 (lane L: row 32 nb + L % 32, columns 16 kb + 8 (L / 32) .. +7, 16
// bytes), blocks ordered nb-major: element (n, k) at
//   ((n / 32) (K / 16) + k / 16) kBfBlock + ((n % 32) + 32 ((k / 8) % 2)) 8 + k % 8,
// rows past N zero.  A wavefront's operand of one slice and block is one contiguous 1 KB load.
constexpr int kBfBlock = 512;                    // elements per block (64 lanes x 8)
// kDenseAT / kGroupRowsAT: dense / grouped rows, and the launch also writes A^T (NtArgs::at).
enum Mode { kDense = 0, kGroupRows = 1, kGroupK = 2, kDenseAT = 3, kGroupRowsAT = 4 };

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
  // grouped K (per-expert weight gradient): expert e contracts over k in
  // [BK kstart[e], BK kstart[e+1]) and writes C + e cstride; order[] lists experts by
  // decreasing work.  Every XCD owns the same contiguous eighth of each expert's tile grid
  // and runs its share of the experts in that order (see the item mapping in the kernel).
  const int* kstart;
  const int* order;
  int64_t cstride;
  int vec_store;          // C and ldc allow 16-byte stores
  // FP32 split of the last partial round.  Tiles [split_from, tiles) are computed as two
  // K-halves (stages [0, split_stage) and the rest); half h of tile split_from + i writes its
  // 256 x 256 FP32 partial to part[2 i + h].  Work items are laid out per XCD (each XCD runs
  // a contiguous range, see remap_xcd): full_per_xcd whole tiles, then split_per_xcd tiles as
  // 2 halves each, so every XCD ends with a full round of half-length items.
  float* part;
  int split_from, full_per_xcd, split_per_xcd;
  int64_t split_stage;
  // kDenseAT / kGroupRowsAT: A^T (row stride ldat) is written as a by-product of the main
  // loop, from the A tiles in LDS (see the kernel).  Dense: A^T [K][M].  Grouped rows: the
  // padded layout of the grouped weight gradient, expert e's rows at columns 64 kstart[e] + i
  // and zeros up to 64 kstart[e+1].
  uint16_t* at;
  int64_t ldat;
  // Packed B (the forward's weight, gemm_nt_kernel's BQ != 0): NVFP4 / MXFP4 codes [N][K/2]
  // (element 2i in the low nibble) and block scales [N][K/16 | K/32], NVFP4's tensor decode
  // scale S at bq_S; or Q4_K blocks [N][K/256][144] at bq_codes.  Each stage's B tile is
  // decoded from these in the main loop (K a multiple of 64).
  const uint8_t* bq_codes;
  const uint8_t* bq_scales;
  const float* bq_S;
};

#define QF_LDS(p) ((__attribute__((address_space(3))) void*)(p))

// 16-byte direct-to-LDS loads: lane l's 16 bytes land at lds + 16 l (lds wave-uniform).
// The buffer form (buffer_load_dwordx4 ... lds) reads at voff + soff from a resource whose
// range ends at the operand's last valid byte (reads past it return zeros).  The global form
// is plain pointer arithmetic, but the compiler counts it as an LDS access of unknown order,
// which turns the fine-grained lgkmcnt waits of the fragment reads that follow into full
// waits.  (Plain functions: device builtins with template-dependent operands keep the host
// pass from emitting the kernel's launch stub.)
#ifndef QF_NT_GLOBAL_LDS
#define QF_NT_GLOBAL_LDS 0
#endif
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int64_t bytes) {
  const int64_t n = bytes < 0xFFFFFFFFll ? bytes : 0xFFFFFFFFll;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)(uint32_t)n,
                                           0x00020000);
}
__device__ __forceinline__ void dma16_buf(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff,
                                          void* lds) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, QF_LDS(lds), 16, (int)voff, (int)soff, 0, 0);
}
__device__ __forceinline__ void dma16_global(const void* g, void* lds) {
  __builtin_amdgcn_global_load_lds(g, QF_LDS(lds), 16, 0, 0);
}

// ds_read_b64_tr_b16 (gfx950): transposing 4 x 16-bit LDS read, see the fragment offsets.
__device__ __forceinline__ v4i16 lds_tr16(const char* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) v4i16*)(__attribute__((address_space(3))) char*)(p));
}

// Workgroup barrier that orders LDS accesses only: outstanding global stores are not waited
// for (a plain __syncthreads() would drain them).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// 16-byte store of an output row segment.  Output tiles go out non-temporally: they are not
// read again by this launch, and as ordinary stores their lines displace operand panels in L2
// (measured 2-5 % slower on whole launches); split partials, read back right away, stay cached.
__device__ __forceinline__ void store_c16(void* dst, uint4 v, bool nt) {
  if (nt) __builtin_nontemporal_store(u32x4_t{v.x, v.y, v.z, v.w}, reinterpret_cast<u32x4_t*>(dst));
  else *reinterpret_cast<uint4*>(dst) = v;
}

// Two FP32 values -> packed bf16 pair (lo in bits 0-15), round to nearest even.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const f32x2_t v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

__device__ __forceinline__ int remap_xcd(int bid, int nb) {
  const int full = nb - nb % kXcds;
  if (bid >= full) return bid;
  return (bid % kXcds) * (full / kXcds) + bid / kXcds;
}

// WAVES = 8: each wavefront owns a 128 x 64 sub-tile (4 x 2 accumulator blocks) and loads
// one operand (8 loads per stage); operands stored [K][rows] (A_MN / B_MN) need this form.
// WAVES = 4: each wavefront owns a 128 x 128 sub-tile (4 x 4 blocks, 256 accumulators in
// AGPRs) and loads 64 rows of both operands (16 loads per stage); one wavefront per SIMD and a
// third less LDS fragment traffic per MFMA (0.5 KB instead of 0.75 KB).  Both visit every
// output element's k slices in the same order, so their results are bit-identical.
//
// BQ != 0 (QF_FMT_NVFP4 / MXFP4 / Q4K; four wavefronts, dense, k-contiguous, bf16 C): B is the
// packed quantized weight instead of a bf16 matrix.  Each lane owns one B row of its
// wavefront's 64 (row 64 w + lane) and, one step ahead, loads that row's codes and scales for
// a stage into registers (32 bytes of codes plus 4 / 2 scale bytes, or the Q4_K block's 16-byte
// header and 32 code bytes); in the next step it decodes them with the quantizers' own decode
// functions (so the B tile holds x_hat bit for bit) and writes the 8 chunks into the stage's
// LDS buffer with 16-byte writes, interleaved with that step's MFMAs, before the barrier that
// publishes the stage.  A keeps its direct-to-LDS loads.
//
// BF (four wavefronts, k-contiguous A, dense modes, K a multiple of 64): B comes in the
// fragment-major layout (see kBfBlock) straight from memory into the MFMA operand registers,
// one fully coalesced 1 KB load per 32-row block and 16-deep slice, and never enters LDS: LDS
// then carries only A (its direct-to-LDS copies and fragment reads), half of the traffic of
// the form above, which is the budget the MFMAs wait on.  Each B fragment of stage s+1 is
// loaded right after the last MFMA that uses the same register for stage s, so it has a whole
// step to arrive; A's copies of stage s+1 all go out at the start of step s, ahead of every B
// load of the step, and the barrier waits for them while leaving that step's B loads in flight.
//
// AT2 (A^T modes): a tile may own two A^T pieces per stage (fewer than 16 tile columns); without
// it the launch has at least 16 and a tile owns at most one.
template <bool C_F32, int MODE, bool A_MN, bool B_MN, int WAVES, int BQ = 0, bool BF = false,
          bool AT2 = false>
__global__ __launch_bounds__(WAVES * 64, 1) void gemm_nt_kernel(NtArgs p) {
  static_assert(WAVES == 8 || (!A_MN && !B_MN), "operands stored [K][rows] need 8 wavefronts");
  static_assert(BQ == 0 || (WAVES == 4 && MODE == kDense && !C_F32),
                "packed B: the four-wavefront dense bf16 form");
  static_assert(!BF || (WAVES == 4 && BQ == 0 && (MODE == kDense || MODE == kDenseAT)),
                "fragment-major B: the four-wavefront dense forms");
  constexpr int NJ = WAVES == 8 ? 2 : 4;         // 32-column accumulator blocks per wavefront
  // direct-to-LDS loads per wavefront per stage (packed or fragment-major B: A's only)
  constexpr int NLD = (WAVES == 8 || BQ != 0 || BF) ? 8 : 16;
  // stage s+1's loads: L0 in the last slice of step s-1, L1 in slice 0 and L2 in slice 1
  // (fragment-major B: all of A's in slice 0)
  constexpr int L0 = BF ? 0 : NLD == 8 ? 3 : 6, L1 = BF ? 8 : NLD == 8 ? 3 : 5;
  constexpr int L2 = NLD - L0 - L1;
  __shared__ __attribute__((aligned(16))) char smem[kSmem];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform (scalar) index
  const int wm = WAVES == 8 ? w >> 2 : w >> 1, wn = WAVES == 8 ? w & 3 : w & 1;
  constexpr bool DENSE = MODE == kDense || MODE == kDenseAT;
  constexpr bool AT = MODE == kDenseAT || MODE == kGroupRowsAT;
  static_assert(!AT || (!C_F32 && WAVES == 4 && !A_MN && !B_MN), "A^T output: bf16 4-wave form");
  const int item = remap_xcd(blockIdx.x, gridDim.x);
  int bid = item, half = -1, pidx = 0;
  if (DENSE && C_F32 && p.part != nullptr) {
    const int per_xcd = p.full_per_xcd + 2 * p.split_per_xcd;
    const int x = item / per_xcd, j = item % per_xcd;
    if (j < p.full_per_xcd) {
      bid = x * p.full_per_xcd + j;
    } else {
      const int i = x * p.split_per_xcd + ((j - p.full_per_xcd) >> 1);
      bid = p.split_from + i;
      half = (j - p.full_per_xcd) & 1;
      pidx = 2 * i + half;
    }
  }

  const uint16_t* Bp = p.B;
  int64_t m0, m_end, n0;
  int ks0 = 0, ks1 = (int)(p.K / BK);            // stage range of this item
  int64_t cofs = 0;                              // element offset of this item's C
  // A^T columns of this tile's first row and the end of its A^T range: rows whose column is
  // below at_end but lie past the operand get zeros (grouped padding)
  int64_t at_col0 = 0, at_end = 0;
  if (DENSE || MODE == kGroupK) {
    int t = bid;
    if (MODE == kGroupK) {
      // Block b runs on XCD x = b % 8 as that XCD's item j = b / 8.  XCD x owns tiles
      // [x tpe / 8, (x + 1) tpe / 8) of every expert; its items walk the experts in order[]
      // (decreasing work), cmax = ceil(tpe / 8) items per expert, the surplus ones empty.  So
      // the 8 XCDs carry equal work however skewed the routing is, and each XCD's CUs take
      // the largest tiles first.
      const int tpe = p.tiles_m * p.tiles_n;
      const int cmax = (tpe + kXcds - 1) / kXcds;
      const int x = blockIdx.x % kXcds, j = blockIdx.x / kXcds;
      const int lo = x * tpe / kXcds, hi = (x + 1) * tpe / kXcds;
      t = lo + j % cmax;
      if (t >= hi) return;                         // uniform over the block
      const int e = p.order[j / cmax];
      ks0 = p.kstart[e];
      ks1 = p.kstart[e + 1];
      cofs = (int64_t)e * p.cstride;
    }
    const int per_group = kGroupM * p.tiles_n;
    const int g = t / per_group;
    const int first = g * kGroupM;
    const int gs = min(p.tiles_m - first, kGroupM);
    m0 = (int64_t)(first + (t % per_group) % gs) * BM;
    m_end = p.M;
    n0 = (int64_t)((t % per_group) / gs) * BN;
    at_col0 = m0;
    at_end = m_end;
  } else {
    // The grid is sized for the most row tiles any routing can need; the real count is
    // tile_start[E].  Block b runs on XCD x = b % 8 as its item j = b / 8, and XCD x takes the
    // contiguous range [x per, (x + 1) per) of the real items (per = ceil(items / 8)), so the
    // XCDs get equal shares and their 32 CUs share the expert weight panels in their L2.
    const int items = p.tile_start[p.E] * p.tiles_n;
    const int per = (items + kXcds - 1) / kXcds;
    const int j = blockIdx.x / kXcds, it = (blockIdx.x % kXcds) * per + j;
    if (j >= per || it >= items) return;         // uniform over the block
    const int mt = it / p.tiles_n, tn = it % p.tiles_n;
    int lo = 0, hi = p.E;                        // tile_start[e] <= mt < tile_start[e+1]
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (p.tile_start[mid] <= mt) lo = mid; else hi = mid;
    }
    m0 = p.off[lo] + (int64_t)(mt - p.tile_start[lo]) * BM;
    m_end = p.off[lo + 1];
    n0 = (int64_t)tn * BN;
    if (AT) {
      at_col0 = 64 * (int64_t)p.kstart[lo] + (m0 - p.off[lo]);
      at_end = 64 * (int64_t)p.kstart[lo + 1];
    }
    Bp += (int64_t)lo * p.bstride;
  }
  const int64_t n_end = p.N, K = p.K;

  // ---- this lane's loads ----------------------------------------------------------------------
  // WAVES = 8: wavefront w loads operand w >> 2, rows (or k-rows) of quarter w & 3, 8 loads of
  // 1 KB per stage.  WAVES = 4: wavefront w loads quarter w of both operands, loads 0-7 for A
  // and 8-15 for B.  Load q of quarter lw at LDS offset op * 32 KB + 8 KB lw + 1 KB (q % 8).
  // k-major operand ([rows][K], a stage is 256 rows x 128 B): load q covers tile rows
  // R = 64 lw + 8 (q % 8) .. R + 7, lane l lands at row R + l / 8, slot l % 8 and so fetches
  // logical chunk (l % 8) ^ ((row >> 1) % 8) = (l % 8) ^ ((4 (q % 2) + l / 16) % 8).
  // mn-major operand ([K][rows], a stage is 64 k-rows x 512 B): load q covers k-rows
  // 16 lw + 2 q + {0, 1}; lane l lands at k-row 16 lw + 2 q + l / 32, 16-byte slot l % 32,
  // and fetches logical chunk (l % 32) ^ (4 (k-row % 4)) (chunk c = columns 8c..8c+7).
  const int lw = WAVES == 8 ? w & 3 : w;
  const int wop = WAVES == 8 ? w >> 2 : 0;       // WAVES = 8: this wavefront's operand
  auto op_of = [&](int q) { return WAVES == 8 ? wop : q >> 3; };
  const char* gb[2];
  __amdgpu_buffer_rsrc_t rs[2];
  int64_t sstride = kRow;                        // bytes from one stage to the next
  uint32_t goff[NLD];
  bool mn = false;
#pragma unroll
  for (int op = 0; op < 2; ++op) {
    if (WAVES == 8 && op != wop) continue;       // uniform
    if ((BQ != 0 || BF) && op == 1) continue;    // packed / fragment-major B: registers
    const bool omn = op ? B_MN : A_MN;
    const int64_t ld = op ? p.ldb : p.lda;
    const int64_t r0 = op ? n0 : m0;
    const int64_t rlim = (op ? n_end : m_end) - r0 - 1;   // last valid row (k-major) / column
    if (!omn) {
      gb[op] = reinterpret_cast<const char*>((op ? Bp : p.A) + r0 * ld);
      rs[op] = make_rsrc(gb[op], (rlim * ld + K) * 2);
#pragma unroll
      for (int q = 0; q < NLD; ++q) {
        if (WAVES == 4 && (q >> 3) != op) continue;
        const int qq = q & 7;
        const int64_t row = lw * 64 + qq * 8 + (lane >> 3);
        const int64_t rc = row < rlim ? row : rlim;
        const int c = (lane & 7) ^ ((4 * (qq & 1) + (lane >> 4)) & 7);
        goff[q] = (uint32_t)((rc * ld + c * 8) * 2);
      }
    } else {
      mn = true;
      gb[op] = reinterpret_cast<const char*>((op ? Bp : p.A) + r0);
      rs[op] = make_rsrc(gb[op], ((K - 1) * ld + rlim + 1) * 2);
      sstride = (int64_t)BK * ld * 2;
      const int clim = (int)(rlim / 8);          // last chunk holding valid columns
#pragma unroll
      for (int q = 0; q < NLD; ++q) {
        const int kr = lw * 16 + q * 2 + (lane >> 5);
        int c = (lane & 31) ^ (4 * (kr & 3));
        c = c < clim ? c : clim;
        goff[q] = (uint32_t)(((int64_t)kr * ld + c * 8) * 2);
      }
    }
  }
  auto lds_of = [&](int q) { return op_of(q) * kOpStage + lw * 8192 + (q & 7) * 1024; };

  // ---- packed B (BQ != 0): this lane's row and its per-stage loads -------------------------
  // Row brow = 64 w + lane of the tile (rows past N decode the last valid row; their outputs
  // are never stored).  Registers of one stage: c0, c1 = the 32 code bytes (element 2i in the
  // low nibble; Q4_K: byte l holds sub-block 2g's element l low and 2g+1's high), sc = the
  // block scales (NVFP4 4 bytes, MXFP4 2) or hd = the Q4_K block header (d, dmin, 12 scale bytes).
  struct BqRegs {
    uint4 c0, c1, hd;
    uint32_t sc;
  };
  const int brow = lw * 64 + lane;
  const uint8_t* bq_row = nullptr;
  const uint8_t* bq_srow = nullptr;
  float bq_S = 0.0f;
  if (BQ != 0) {
    const int64_t gr = n0 + brow < n_end ? n0 + brow : n_end - 1;
    if (BQ == QF_FMT_Q4K) {
      bq_row = p.bq_codes + gr * (K / 256) * 144;
    } else {
      bq_row = p.bq_codes + gr * (K / 2);
      bq_srow = p.bq_scales + gr * (K / (BQ == QF_FMT_NVFP4 ? 16 : 32));
    }
    if (BQ == QF_FMT_NVFP4) bq_S = p.bq_S[0];    // the quantizer's S = fl(g / 2688)
  }
  auto bq_load = [&](int64_t se, BqRegs& r) __attribute__((always_inline)) {
    if (BQ == QF_FMT_Q4K) {
      const uint8_t* blk = bq_row + (se >> 2) * 144;
      r.hd = *reinterpret_cast<const uint4*>(blk);
      r.c0 = *reinterpret_cast<const uint4*>(blk + 16 + 32 * (se & 3));
      r.c1 = *reinterpret_cast<const uint4*>(blk + 32 + 32 * (se & 3));
    } else {
      r.c0 = *reinterpret_cast<const uint4*>(bq_row + se * 32);
      r.c1 = *reinterpret_cast<const uint4*>(bq_row + se * 32 + 16);
      if (BQ == QF_FMT_NVFP4) r.sc = *reinterpret_cast<const uint32_t*>(bq_srow + se * 4);
      else r.sc = *reinterpret_cast<const uint16_t*>(bq_srow + se * 2);
    }
  };
  // x_hat of logical chunk c (elements 8c .. 8c+7 of the stage) into LDS buffer buf.
  auto bq_decode = [&](const BqRegs& r, int64_t se, int c, int buf) __attribute__((always_inline)) {
    const uint32_t cw[8] = {r.c0.x, r.c0.y, r.c0.z, r.c0.w, r.c1.x, r.c1.y, r.c1.z, r.c1.w};
    uint32_t o[4];
    if (BQ == QF_FMT_NVFP4) {
      // (with a non-finite tensor scale the decoded NaN operands may differ from the
      // quantizer's x_hat in NaN sign and payload only, which the NaN sums do not show)
      codec::nvfp4_decode8_finite(
          cw[c], codec::nvfp4_block_scale(bq_S, (r.sc >> (8 * (c >> 1))) & 0xFFu), o);
    } else if (BQ == QF_FMT_MXFP4) {
      codec::mxfp4_decode8(cw[c], (r.sc >> (8 * (c >> 2))) & 0xFFu, o);
    } else {
      // sub-block j = 2 (se % 4) + (c >= 4): its 6-bit scale and min from the header
      const int j = 2 * (int)(se & 3) + (c >> 2);
      const int jj = j & 3, sh = 8 * jj;
      uint32_t ls, lm;
      if (j < 4) {
        ls = (r.hd.y >> sh) & 63u;
        lm = (r.hd.z >> sh) & 63u;
      } else {
        ls = ((r.hd.w >> sh) & 15u) | (((r.hd.y >> (sh + 6)) & 3u) << 4);
        lm = ((r.hd.w >> (sh + 4)) & 15u) | (((r.hd.z >> (sh + 6)) & 3u) << 4);
      }
      const float t1 = codec::f16_value(r.hd.x & 0xFFFFu) * (float)ls;
      const float t2 = codec::f16_value(r.hd.x >> 16) * (float)lm;
      const int b = (c & 3) * 2;                  // code bytes 8 (c % 4) .. +7
      const uint32_t sh4 = c >= 4 ? 4u : 0u;      // sub-block 2g + 1 in the high nibbles
      const uint32_t qw[2] = {(cw[b] >> sh4) & 0x0F0F0F0Fu, (cw[b + 1] >> sh4) & 0x0F0F0F0Fu};
      codec::q4k_decode8(qw, t1, t2, o);
    }
    *reinterpret_cast<uint4*>(smem + buf * kStage + kOpStage + brow * kRow +
                              ((c ^ ((brow >> 1) & 7)) << 4)) = make_uint4(o[0], o[1], o[2], o[3]);
  };
  BqRegs bq_cur{}, bq_nxt{};
  // The main loop decodes a stage as a chain of small operations, one after each MFMA of the
  // step's first three slices, so that no gap between two MFMAs holds more than a few VALU
  // instructions (one wavefront per SIMD: nothing else issues while this one decodes).
  //   NVFP4, 48 operations: per chunk c, the block decode scale D (even c), the four element
  //          pairs (E2M1 -> FP32, x D, bf16 pack), the 16-byte LDS write.
  //   MXFP4, 24 (every other MFMA): per chunk, pairs 0-1 with the E8M0 scale, pairs 2-3, the
  //          NaN-block select and the write.
  //   Q4_K, 43: the super-block's d and dmin, the two sub-blocks' step t1 and offset t2, then
  //          per chunk four element pairs (the first also extracts the chunk's nibbles) and
  //          the write.
  // The arithmetic is the decode functions' (codec::*_decode8), split up.
  float bq_D = 0.0f, bq_d = 0.0f, bq_dmin = 0.0f, bq_t1[2] = {0.0f, 0.0f}, bq_t2[2] = {0.0f, 0.0f};
  uint32_t bq_o[4] = {0, 0, 0, 0}, bq_qw[2] = {0, 0}, bq_e = 0;
  auto bq_word = [&](const BqRegs& r, int c) __attribute__((always_inline)) -> uint32_t {
    switch (c) {
      case 0: return r.c0.x; case 1: return r.c0.y; case 2: return r.c0.z; case 3: return r.c0.w;
      case 4: return r.c1.x; case 5: return r.c1.y; case 6: return r.c1.z; default: return r.c1.w;
    }
  };
  auto bq_store = [&](int c, int buf) __attribute__((always_inline)) {
    *reinterpret_cast<uint4*>(smem + buf * kStage + kOpStage + brow * kRow +
                              ((c ^ ((brow >> 1) & 7)) << 4)) =
        make_uint4(bq_o[0], bq_o[1], bq_o[2], bq_o[3]);
  };
  constexpr int kBqOps = BQ == QF_FMT_NVFP4 ? 48 : BQ == QF_FMT_MXFP4 ? 24 : 43;
  auto bq_op = [&](const BqRegs& r, int64_t se, int u, int buf) __attribute__((always_inline)) {
    if (BQ == QF_FMT_NVFP4) {
      const int c = u / 6, k = u % 6;
      const uint32_t cw = bq_word(r, c);
      if (k == 0) {
        if ((c & 1) == 0) bq_D = codec::nvfp4_block_scale(bq_S, (r.sc >> (8 * (c >> 1))) & 0xFFu);
      } else if (k <= 4) {
        // (with a non-finite tensor scale the decoded NaN operands may differ from the
        // quantizer's x_hat in NaN sign and payload only, which the NaN sums do not show)
        codec::f32x2_t v;
        switch (k) {
          case 1: v = codec::e2m1_pair<0>(cw); break;
          case 2: v = codec::e2m1_pair<1>(cw); break;
          case 3: v = codec::e2m1_pair<2>(cw); break;
          default: v = codec::e2m1_pair<3>(cw); break;
        }
        bq_o[k - 1] = codec::bf16x2_rne_nonnan(v.x * bq_D, v.y * bq_D);
      } else {
        bq_store(c, buf);
      }
    } else if (BQ == QF_FMT_MXFP4) {
      const int c = u / 3, k = u % 3;
      const uint32_t cw = bq_word(r, c);
      if (k == 0) bq_e = (r.sc >> (8 * (c >> 2))) & 0xFFu;
      const float sc = codec::e8m0_scale(bq_e);
      if (k == 0) {
        bq_o[0] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(cw, sc, 0));
        bq_o[1] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(cw, sc, 1));
      } else if (k == 1) {
        bq_o[2] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(cw, sc, 2));
        bq_o[3] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(cw, sc, 3));
      } else {
        const bool nan = bq_e == 0xFFu;                // (codec::mxfp4_decode8's NaN block)
#pragma unroll
        for (int q = 0; q < 4; ++q) bq_o[q] = nan ? 0x7FC07FC0u : bq_o[q];
        bq_store(c, buf);
      }
    } else {
      if (u == 0) {
        bq_d = codec::f16_value(r.hd.x & 0xFFFFu);        // d and dmin of the super-block
        bq_dmin = codec::f16_value(r.hd.x >> 16);
      } else if (u < 3) {
        // sub-block j = 2 (se % 4) + u - 1: its 6-bit scale and min from the header
        const int j = 2 * (int)(se & 3) + u - 1;
        const int sh = 8 * (j & 3);
        uint32_t ls, lm;
        if (j < 4) {
          ls = (r.hd.y >> sh) & 63u;
          lm = (r.hd.z >> sh) & 63u;
        } else {
          ls = ((r.hd.w >> sh) & 15u) | (((r.hd.y >> (sh + 6)) & 3u) << 4);
          lm = ((r.hd.w >> (sh + 4)) & 15u) | (((r.hd.z >> (sh + 6)) & 3u) << 4);
        }
        bq_t1[u - 1] = bq_d * (float)ls;
        bq_t2[u - 1] = bq_dmin * (float)lm;
      } else {
        const int c = (u - 3) / 5, k = (u - 3) % 5, h = c >> 2;
        if (k == 0) {
          const int b = (c & 3) * 2;                // code bytes 8 (c % 4) .. +7
          const uint32_t sh4 = h ? 4u : 0u;         // sub-block 2g + 1 in the high nibbles
          bq_qw[0] = (bq_word(r, b) >> sh4) & 0x0F0F0F0Fu;
          bq_qw[1] = (bq_word(r, b + 1) >> sh4) & 0x0F0F0F0Fu;
        }
        if (k < 4) {
          // elements 2k, 2k + 1: bf16(fl(t1 q - t2)) as in codec::q4k_decode8
          const uint32_t q = bq_qw[k >> 1] >> (16 * (k & 1));
          const float a0 = __builtin_fmaf(bq_t1[h], (float)(q & 0xFFu), -bq_t2[h]);
          const float a1 = __builtin_fmaf(bq_t1[h], (float)((q >> 8) & 0xFFu), -bq_t2[h]);
          bq_o[k] = codec::bf16x2_rne_nonnan(a0, a1);
        } else {
          bq_store(c, buf);
        }
      }
    }
  };

  // ---- fragment offsets ----------------------------------------------------------------------
  // k-major: slice kk, fragment i at fo[kk] + i * 4096 (32 rows of 128 bytes); fragment rows
  // start 32-aligned, so the swizzle term (row >> 1) & 7 is (lane >> 1) & 7.
  // mn-major: two ds_read_b64_tr_b16 per fragment (k 0-3 and 4-7 of the lane's 8).  Within
  // each group of 16 lanes that instruction hands output lane L element j of source lane
  // 4 j + L / 4 (element L % 4), so source lane 4 j + a points at k-row kb + j, columns
  // c0 + 4 a .. +3: output lane L then holds k-rows kb .. kb+3 of column c0 + L.  Lane l
  // (group g = l / 16) serves MFMA lane rows 16 (g % 2) + L and k-half g / 2; fragment f's base
  // is fo[f], plus (16 kk + 4 h) * 512 bytes for slice kk, half h.
  int foa[4], fob[4];
  {
    const int ra = wm * 128 + (lane & 31), rb = wn * (NJ * 32) + (lane & 31);
    const int sw = (lane >> 1) & 7;
    const int g = lane >> 4, j = (lane >> 2) & 3, a = lane & 3;
#pragma unroll
    for (int x = 0; x < 4; ++x) {
      const int c = 2 * x + (lane >> 5);
      // mn-major fragment x: columns start at (wm * 128 or wn * 64) + 32 x
      const int rowj = 8 * (g >> 1) + j;
      if (A_MN) foa[x] = rowj * 512 + ((4 * ((wm * 4 + x) ^ j) + 2 * (g & 1) + (a >> 1)) << 4) + 8 * (a & 1);
      else foa[x] = ra * kRow + ((c ^ sw) << 4);
      if (B_MN) fob[x] = kOpStage + rowj * 512 + ((4 * ((wn * NJ + x) ^ j) + 2 * (g & 1) + (a >> 1)) << 4) + 8 * (a & 1);
      else fob[x] = kOpStage + rb * kRow + ((c ^ sw) << 4);
    }
  }

  f32x16_t acc[4][NJ];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j) acc[i][j] = f32x16_t{};
  bf16x8_t fa[2][4], fb[2][NJ];
  // Fragment-major B (BF): fbr[kk][j] holds the B fragment of 16-deep slice kk and 32-row
  // block j of this wavefront's 128 columns for the stage in use.  Block j's fragments start at
  // bf_base[j]; slice kk of global stage se is kBfBlock elements further per (4 se + kk).
  bf16x8_t fbr[BF ? 4 : 1][BF ? 4 : 1];
  const uint16_t* bf_base[BF ? 4 : 1];
  if (BF) {
    const int64_t nblocks = (p.N + 31) / 32, kblocks = p.K / 16;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      int64_t nb = (n0 + wn * 128) / 32 + j;
      nb = nb < nblocks ? nb : nblocks - 1;      // blocks past N: outputs never stored
      bf_base[j] = p.B + (nb * kblocks) * kBfBlock + lane * 8;
    }
  }
  auto bf_load = [&](int64_t se, int kk, int j) __attribute__((always_inline)) {
    if (BF) fbr[kk][j] = *reinterpret_cast<const bf16x8_t*>(bf_base[j] + (se * 4 + kk) * kBfBlock);
  };

  // K order: the stages of this item's range [ks0, ks1) are visited rotated by an offset that
  // depends on the XCD (blockIdx.x % 8).  The 32 CUs of an XCD stay in step, so the panels
  // they share still meet in its L2, but the eight XCDs stream from eight different k offsets:
  // with row strides that are large powers of two, k-aligned requests from all CUs otherwise
  // pile onto the same HBM channels.  Each tile's sum order is fixed, so results are
  // deterministic.
  // (Stage indices are 32-bit: fewer scalar instructions in the main loop's issue slots.)
  if (half == 1) ks0 = (int)p.split_stage;
  if (half == 0) ks1 = (int)p.split_stage;
  const int klen = ks1 > ks0 ? ks1 - ks0 : 1;
  const int krot = (int)(blockIdx.x % kXcds) * (klen / kXcds);
  // global stage of loop stage s
  auto gstage = [&](int s) __attribute__((always_inline)) -> int {
    const int se = s + krot;
    return se >= ks1 ? se - klen : se;
  };
  const uint32_t sstride32 = (uint32_t)sstride;
  // load q of global stage se into buffer buf
  auto dma = [&](int se, int buf, int q) __attribute__((always_inline)) {
    char* l = smem + buf * kStage + lds_of(q);
    const int op = op_of(q);
    if (QF_NT_GLOBAL_LDS) dma16_global(gb[op] + (int64_t)se * sstride + goff[q], l);
    else dma16_buf(rs[op], goff[q], (uint32_t)se * sstride32, l);
  };
  // Fragment read r of a slice, in the order the slice's MFMAs consume them: A0, B0, B1, A1..A3.
  auto frag = [&](const char* st, int kk, int f, bool is_b) __attribute__((always_inline)) -> bf16x8_t {
    const bool mnf = is_b ? B_MN : A_MN;
    if (!mnf) {
      const int* fo = is_b ? fob : foa;
      return *reinterpret_cast<const bf16x8_t*>(st + fo[kk] + f * 4096);
    }
    const char* base = st + (is_b ? fob[f] : foa[f]) + kk * 16 * 512;
    const v4i16 lo = lds_tr16(base);
    const v4i16 hi = lds_tr16(base + 4 * 512);
    const v8i16 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    return __builtin_bit_cast(bf16x8_t, v);
  };
  auto read_one = [&](const char* st, int kk, int r, bf16x8_t* a, bf16x8_t* b) __attribute__((always_inline)) {
    if (r == 0) a[0] = frag(st, kk, 0, false);
    else if (r <= NJ) { if (!BF) b[r - 1] = frag(st, kk, r - 1, true); }
    else a[r - NJ] = frag(st, kk, r - NJ, false);
  };
  auto read_all = [&](const char* st, int kk, bf16x8_t* a, bf16x8_t* b) __attribute__((always_inline)) {
#pragma unroll
    for (int r = 0; r < 4 + NJ; ++r) read_one(st, kk, r, a, b);
  };
  // ---- A^T output (kDenseAT, kGroupRowsAT) ---------------------------------------------------
  // A stage's A^T is 16 pieces: piece u is k columns 4 u .. 4 u + 3 over the tile's 256 rows, so
  // each of its rows of A^T is written as whole 128-byte lines, each line by one store.  Piece
  // u of global stage se belongs to tile column (16 se + u) mod tiles_n, so with tiles_n >= 8 a
  // tile has at most two pieces per stage.  at_read gathers this lane's part of piece u from
  // the stage in LDS (rows r0 .. r0 + 3, r0 = 64 w + 4 (l % 16), of k column kc = 4 u + l / 16;
  // four 2-byte reads through the row swizzle) before the step's barrier; at_store writes
  // those 8 bytes to A^T row se * 64 + kc, columns at_col0 + r0 .. +3 (at_col0 = m0 dense, the
  // padded column of the tile's first row grouped), after it, so the store has a whole step to
  // complete before the next barrier's wait.  Rows past the operand store zeros while their
  // column is below at_end (an expert's padding) and nothing beyond it.  Stores go through a
  // buffer resource over the stage's rows of A^T: lanes with nothing to store (or columns at
  // or past kvalid) get an offset beyond its range, which the hardware drops.  (Plain LDS reads:
  // the transposing read builtin makes the compiler wait for every direct-to-LDS load in
  // flight first.)
  const int64_t at_tn = n0 / BN;                 // this tile's column
  const int at_r = w * 64 + 4 * (lane & 15), at_c = lane >> 4;
  // (the four values stay unpacked until the store: packing them at the read would make the
  // wavefront wait for the reads there)
  auto at_read = [&](const char* st, int u) __attribute__((always_inline)) -> u32x4_t {
    const int kc = 4 * u + at_c;
    u32x4_t h;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int row = at_r + e;
      h[e] = *reinterpret_cast<const uint16_t*>(
          st + row * kRow + ((((kc >> 3) ^ (row >> 1)) & 7) << 4) + (kc & 7) * 2);
    }
    return h;
  };
  // byte offset of this lane's 8 bytes of piece 0 within a stage's rows of A^T (below 2^31)
  const int at_off = (int)(((int64_t)at_c * p.ldat + at_col0 + at_r) * 2);
  const int at_ld8 = (int)(p.ldat * 8);          // bytes of 4 rows of A^T
  const bool at_rok = m0 + at_r < m_end;          // data rows
  const bool at_zok = at_col0 + at_r < at_end;     // data or zero-padding columns
  auto at_store = [&](int64_t se, int kvalid, int u, u32x4_t h) __attribute__((always_inline)) {
    const u32x2_t v = at_rok ? u32x2_t{h[0] | (h[1] << 16), h[2] | (h[3] << 16)} : u32x2_t{0, 0};
    const bool ok = at_zok && 4 * u + at_c < kvalid;
    const int off = ok ? at_off + u * at_ld8 : 0x7FFFFFF8;
    __builtin_amdgcn_raw_buffer_store_b64(
        v, make_rsrc(p.at + se * BK * p.ldat, (int64_t)kvalid * p.ldat * 2), off, 0, 0);
  };
  // first piece of stage se owned by this tile, (tn - 16 se) mod tiles_n (>= 16: none); the
  // second is at + tiles_n.  In the loop it is stepped, not divided: stage se + 1's is
  // this one minus 16 mod tiles_n.
  auto at_first = [&](int64_t se) -> int {
    const int64_t t = p.tiles_n;
    return (int)((at_tn - (se * 16) % t + t) % t);
  };
  int at_u = 0;
  int at_u_wrap = 0, at_d = 0;
  if (AT) {
    at_u_wrap = at_first(ks0);                   // the stage after the wrap to ks0
    at_d = (int)(16 % p.tiles_n);
  }
  // The main loop's form of at_read / at_store, split into small pieces that go into the
  // issue slots between MFMAs (with one wavefront per SIMD a slot has room for a few
  // instructions only; more stall the MFMA stream).  With kc = 4 u + at_c (at_c < 4),
  // kc >> 3 = u >> 1 and kc & 7 = 4 (u & 1) + at_c, so element e of piece u sits at
  // at_lb[e] + ((u >> 1) << 4 ^ at_sw[e >> 1]) + 8 (u & 1) in the stage (rows at_r + e share
  // (row >> 1) & 7 in pairs).  at_read2 reads elements e0, e0 + 1 of piece u (u < 16) from
  // buffer buf.
  int at_lb[4], at_sw[2];
#pragma unroll
  for (int e = 0; e < 4; ++e) at_lb[e] = (at_r + e) * kRow + at_c * 2;
#pragma unroll
  for (int e = 0; e < 2; ++e) at_sw[e] = (((at_r + 2 * e) >> 1) & 7) << 4;
  auto at_read2 = [&](int buf, int u, int e0, u32x4_t& h) __attribute__((always_inline)) {
    const int xs = (u >> 1) << 4, ad = buf * kStage + ((u & 1) << 3);
    const int x = xs ^ at_sw[e0 >> 1];
    h[e0] = *reinterpret_cast<const uint16_t*>(smem + at_lb[e0] + x + ad);
    h[e0 + 1] = *reinterpret_cast<const uint16_t*>(smem + at_lb[e0 + 1] + x + ad);
  };
  // bytes of a stage's rows of A^T (below 2^31: ldat < 2^24)
  const uint32_t at_sbytes = (uint32_t)(BK * p.ldat * 2);
  auto at_pack = [&](const u32x4_t& h) __attribute__((always_inline)) -> u32x2_t {
    return at_rok ? u32x2_t{h[0] | (h[1] << 16), h[2] | (h[3] << 16)} : u32x2_t{0, 0};
  };
  auto at_put = [&](__amdgpu_buffer_rsrc_t r, int u, u32x2_t v) __attribute__((always_inline)) {
    const int off = at_zok && u < 16 ? at_off + u * at_ld8 : 0x7FFFFFF8;
    __builtin_amdgcn_raw_buffer_store_b64(v, r, off, 0, 2);   // non-temporal
  };
  constexpr bool at_two = AT && AT2;             // a second piece per stage is possible
  // One 16-deep slice of MFMAs from (a, b), with the fragment reads of the next slice (from
  // rst / rkk into ra, rb) and, if LOADS, the direct-to-LDS loads of global stage ls into
  // buffer lbuf, issued one per MFMA.  The scheduling fences keep that interleave.
  // extra(t) runs after MFMA t (the A^T reads and stores, the packed-B decode, index updates).
  auto slice = [&](auto reads, auto loads, const bf16x8_t* a, const bf16x8_t* b,
                   const char* rst, int rkk, bf16x8_t* ra, bf16x8_t* rb, int ls, int lbuf,
                   int qa, int nq, auto extra) __attribute__((always_inline)) {
    constexpr bool READS = decltype(reads)::value, LOADS = decltype(loads)::value;
    constexpr int NM = 4 * NJ, NR = 4 + NJ;
#pragma unroll
    for (int t = 0; t < NM; ++t) {
      acc[t / NJ][t % NJ] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b[t % NJ], a[t / NJ],
                                                                    acc[t / NJ][t % NJ], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
      if (READS && t < NR) read_one(rst, rkk, t, ra, rb);
      if (LOADS) {
        // loads [qa, qa + nq) of stage ls, one per MFMA from the first
        if (t < nq) dma(ls, lbuf, qa + t);
      }
      extra(t);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  // Loads are spread over the step: stage s+1's loads go out L0 in the last slice of step s-1
  // (right after its barrier freed stage s-1's buffer), L1 in slice 0 and L2 in slice 1 of
  // step s; the barrier before slice 3 waits for them.  A step knows the global stages of
  // loop stages s and s+1 (e_cur, e_nx1, handed on by the step before) and works out that of
  // s+2 (e_nx2) in a free slot of slice 2.  LD1 / LD2: loop stages s+1 / s+2 exist (no copies
  // are issued for stages past the end, so the epilogue does not wait for any).  cur: the
  // buffer holding stage s.
  int e_cur = 0, e_nx1 = 0;
  auto step = [&](int s, int s_end, auto last, auto ld1, auto ld2, int cur)
      __attribute__((always_inline)) {
    constexpr bool LAST = decltype(last)::value, LD1 = decltype(ld1)::value;
    constexpr bool LD2 = decltype(ld2)::value;
    const int nxt = cur ^ 1;
    const char* cs = smem + cur * kStage;
    // packed or fragment-major B use stage s+2's index from slice 0 on
    constexpr bool EARLY = BQ != 0 || BF;
    int e_nx2 = 0;
    auto calc_nx2 = [&]() __attribute__((always_inline)) {
      e_nx2 = gstage(s + 2 < s_end ? s + 2 : s_end - 1);
    };
    if (EARLY) calc_nx2();
    // A^T modes: this tile's A^T pieces of the stage (u0 and, with fewer than 16 tile columns,
    // u0 + tiles_n; >= 16: none) are read in slice 1, while the stage is resident, and stored
    // in slice 3, after the barrier; at_u then moves on to stage s+1's piece.
    const int u0 = at_u, u1 = at_u + p.tiles_n;
    u32x4_t v0 = {0, 0, 0, 0}, v1 = {0, 0, 0, 0};
    u32x2_t w0 = {0, 0}, w1 = {0, 0};
    // the main loop's stores cover a full stage (kvalid = BK) of A^T rows
    __amdgpu_buffer_rsrc_t at_rs;
    const char* at_base = nullptr;
    auto at_hook1 = [&](int t) __attribute__((always_inline)) {
      if (!AT) return;
      if (t == 8) at_read2(cur, u0 & 15, 0, v0);
      if (t == 9) at_read2(cur, u0 & 15, 2, v0);
      if (at_two && t == 10) at_read2(cur, u1 & 15, 0, v1);
      if (at_two && t == 11) at_read2(cur, u1 & 15, 2, v1);
    };
    auto at_hook2 = [&](int t) __attribute__((always_inline)) {
      if (AT && t == 12)
        at_base = reinterpret_cast<const char*>(p.at) + (uint64_t)(uint32_t)e_cur * at_sbytes;
      if (AT && t == 13) at_rs = make_rsrc(at_base, (int64_t)at_sbytes);
    };
    auto at_hook3 = [&](int t) __attribute__((always_inline)) {
      if (!AT) return;
      if (t == 8) w0 = at_pack(v0);
      if (t == 9) at_put(at_rs, u0, w0);
      if (at_two && t == 10) w1 = at_pack(v1);
      if (at_two && t == 11) at_put(at_rs, u1, w1);
      if (!LAST && t == 13) {
        int u = e_nx1 == ks0 ? at_u_wrap : at_u - at_d;
        at_u = u < 0 ? u + p.tiles_n : u;
      }
    };
    // Packed B: stage s+2's registers are loaded in slice 0 (they have the rest of the step,
    // up to the barrier's wait), and stage s+1's (loaded one step earlier) are decoded into
    // buffer nxt in small operations spread over slices 0-2.
    // slot g (0..47) = the MFMA of slices 0-2 that the operation follows
    auto bq_slot = [&](int g) __attribute__((always_inline)) {
      if (BQ != 0) {
        if (g == 1) bq_load(e_nx2, bq_nxt);
        if (BQ == QF_FMT_MXFP4) {
          if ((g & 1) == 0 && g / 2 < kBqOps) bq_op(bq_cur, e_nx1, g / 2, nxt);
        } else if (g < kBqOps) {
          bq_op(bq_cur, e_nx1, g, nxt);
        }
      }
    };
    // Fragment-major B: after MFMA t = 12 + j of slice kk (the last one using fbr[kk][j]), that
    // register is loaded with stage s+1's fragment (not in the last step).
    auto bf_hook = [&](int kk, int t) __attribute__((always_inline)) {
      if (BF && !LAST && t >= 12) bf_load(e_nx1, kk, t - 12);
    };
    auto hook0 = [&](int t) __attribute__((always_inline)) {
      bq_slot(t);
      bf_hook(0, t);
    };
    auto hook1 = [&](int t) __attribute__((always_inline)) {
      bq_slot(16 + t);
      at_hook1(t);
      bf_hook(1, t);
    };
    auto hook2 = [&](int t) __attribute__((always_inline)) {
      bq_slot(32 + t);
      at_hook2(t);
      if (!EARLY && t == 2 * NJ + 1) calc_nx2();   // a free slot (slices hold 4 NJ MFMAs)
      bf_hook(2, t);
    };
    auto hook3 = [&](int t) __attribute__((always_inline)) {
      at_hook3(t);
      bf_hook(3, t);
    };
    slice(std::true_type{}, std::integral_constant<bool, LD1>{}, fa[0], BF ? fbr[0] : fb[0], cs,
          1, fa[1], fb[1], e_nx1, nxt, L0, L1, hook0);
    slice(std::true_type{}, std::integral_constant<bool, LD1>{}, fa[1],
          BF ? fbr[1 % (BF ? 4 : 1)] : fb[1], cs, 2, fa[0], fb[0], e_nx1, nxt, L0 + L1, L2, hook1);
    slice(std::true_type{}, std::false_type{}, fa[0], BF ? fbr[2 % (BF ? 4 : 1)] : fb[0], cs, 3,
          fa[1], fb[1], 0, 0, 0, 0, hook2);
    if (BF && !LAST) {
      // A's copies of stage s+1 and everything before them; the 12 B loads issued after them in
      // slices 0-2 stay in flight (vmcnt(12); expcnt not waited; lgkmcnt(0): this wavefront's
      // reads of stage s are done before the barrier lets stage s+2's copies overwrite it)
      __builtin_amdgcn_s_waitcnt(12 | (7 << 4) | (0 << 8));
    } else {
      __builtin_amdgcn_s_waitcnt(0);
    }
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    if (BQ != 0) bq_cur = bq_nxt;               // complete: the wait above covered its loads
    slice(std::integral_constant<bool, !LAST>{}, std::integral_constant<bool, LD2>{}, fa[1],
          BF ? fbr[3 % (BF ? 4 : 1)] : fb[1], smem + nxt * kStage, 0, fa[0], fb[0], e_nx2, cur, 0,
          L0, hook3);
    e_cur = e_nx1;
    e_nx1 = e_nx2;
  };

  const int64_t nfull = K / BK;                 // the K tail (dense, second half) follows it
  // (packed or fragment-major B: K is a multiple of BK, checked on the host)
  const int64_t krem = (half == 0 || MODE == kGroupK || BQ != 0 || BF) ? 0 : K % BK;
  const int s0 = ks0, s1 = ks1;
  if (s1 > s0) {
    e_cur = gstage(s0);
    e_nx1 = gstage(s0 + 1 < s1 ? s0 + 1 : s1 - 1);
#pragma unroll
    for (int q = 0; q < NLD; ++q) dma(e_cur, 0, q);
    if (BF) {
#pragma unroll
      for (int kk = 0; kk < 4; ++kk)
#pragma unroll
        for (int j = 0; j < 4; ++j) bf_load(e_cur, kk, j);
    }
    if (BQ != 0) {
      // stage s0's B decoded now; stage s0+1's registers for the first step
      BqRegs first;
      bq_load(e_cur, first);
      bq_load(e_nx1, bq_cur);
#pragma unroll
      for (int c = 0; c < 8; ++c) bq_decode(first, e_cur, c, 0);
    }
    if (s0 + 1 < s1) {
#pragma unroll
      for (int q = 0; q < L0; ++q) dma(e_nx1, 1, q);
    }
    __builtin_amdgcn_s_waitcnt(0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    read_all(smem, 0, fa[0], fb[0]);
    int s = s0;
    if (AT) at_u = at_first(e_cur);
    const std::true_type T{};
    const std::false_type F{};
    if (WAVES == 4) {
      // two steps per iteration: with one loop-carried copy of the 256 accumulators the
      // register allocator keeps them in place (a one-step loop body rotates them through
      // other AGPRs at every back edge)
      for (; s + 3 < s1; s += 2) {
        step(s, s1, F, T, T, 0);
        step(s + 1, s1, F, T, T, 1);
      }
    }
    for (; s + 2 < s1; ++s) step(s, s1, F, T, T, (s - s0) & 1);
    if (s + 1 < s1) {
      step(s, s1, F, T, F, (s - s0) & 1);
      ++s;
    }
    step(s, s1, T, F, F, (s - s0) & 1);
  }
  if (krem > 0) {
    // Partial last stage: masked loads through registers into buffer 0.  The wait + barrier
    // retires every earlier read of that buffer.
    __builtin_amdgcn_s_waitcnt(0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int q = 0; q < NLD; ++q) {
      bool valid;
      if (!mn) {
        const int c = (lane & 7) ^ ((4 * (q & 1) + (lane >> 4)) & 7);
        valid = nfull * BK + c * 8 < K;
      } else {
        valid = nfull * BK + lw * 16 + q * 2 + (lane >> 5) < K;
      }
      uint4 v = make_uint4(0, 0, 0, 0);
      if (valid) v = *reinterpret_cast<const uint4*>(gb[op_of(q)] + nfull * sstride + goff[q]);
      *reinterpret_cast<uint4*>(smem + lds_of(q) + lane * 16) = v;
    }
    __syncthreads();
    if (AT) {                      // the tail stage, same ownership
      for (int u = at_first(nfull); u < 16; u += p.tiles_n)
        at_store(nfull, (int)krem, u, at_read(smem, u));
    }
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      if (kk * 16 >= krem) break;                // uniform: the rest of the stage is zeros
      read_all(smem, kk, fa[0], fb[0]);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[0][j], fa[0][i], acc[i][j], 0, 0, 0);
    }
  }

  // ---- epilogue: the tile goes through LDS and leaves as whole-row 16-byte stores ----------
  // Each MFMA takes the B fragment as its first operand, so accumulator block (i, j) holds the
  // transposed product: element v sits at row lane % 32 of the block and column
  // 8 (v / 4) + 4 (lane / 32) + v % 4, i.e. a lane owns four consecutive columns of one row per
  // group v / 4, written to LDS with one 8-byte (bf16) or 16-byte (FP32) store.
  __syncthreads();                               // every wavefront is done with the operands
  // Destination: the output tile, or (split halves) a dense 256 x 256 FP32 partial.
  char* Cp = reinterpret_cast<char*>(p.C) + cofs * (C_F32 ? 4 : 2);
  int64_t ldc = p.ldc, em0 = m0, em_end = m_end, en0 = n0, en_end = n_end;
  int vec = p.vec_store;
  if (half >= 0) {
    Cp = reinterpret_cast<char*>(p.part + (int64_t)pidx * BM * BN);
    ldc = BN; em0 = 0; em_end = BM; en0 = 0; en_end = BN; vec = 1;
  }
  const int er = wm * 128 + (lane & 31);          // this lane's row in block (0, *)
  const int ec = wn * (NJ * 32) + 4 * (lane >> 5);  // its first column in block (*, 0), group 0
  if (!C_F32) {
    // bf16 pairs by the hardware pack (round to nearest even; a NaN result stays a quiet NaN)
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < NJ; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const f32x16_t& a = acc[i][j];
          const uint2 w = make_uint2(pack_bf16x2(a[4 * g], a[4 * g + 1]),
                                     pack_bf16x2(a[4 * g + 2], a[4 * g + 3]));
          *reinterpret_cast<uint2*>(smem + (er + 32 * i) * kPitch16 + (ec + 32 * j + 8 * g) * 2) = w;
        }
    lds_barrier();
    const int c8 = (tid & 31) * 8;
    const int64_t gcol = en0 + c8;
    constexpr int kRowsPerPass = WAVES * 64 / 32;  // 32 lanes cover a row
#pragma unroll 4
    for (int it = 0; it < BM / kRowsPerPass; ++it) {
      const int r = it * kRowsPerPass + (tid >> 5);
      const int64_t grow = em0 + r;
      if (grow >= em_end || gcol >= en_end) continue;
      const uint4 v = *reinterpret_cast<const uint4*>(smem + r * kPitch16 + c8 * 2);
      uint16_t* dst = reinterpret_cast<uint16_t*>(Cp) + grow * ldc + gcol;
      if (vec && gcol + 8 <= en_end) {
        store_c16(dst, v, half < 0);
      } else {
        const uint32_t wv[4] = {v.x, v.y, v.z, v.w};
        for (int e = 0; e < 8 && gcol + e < en_end; ++e)
          dst[e] = (uint16_t)(wv[e >> 1] >> (16 * (e & 1)));
      }
    }
  } else {
    // FP32 tile (256 KB) in two halves: in half h every wavefront writes its row blocks 2h and
    // 2h + 1, so LDS row q (0..127) holds tile row (q / 64) * 128 + 64 h + q % 64.
    const int c4 = (tid & 63) * 4;
    const int64_t gcol = en0 + c4;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      if (h) lds_barrier();                      // half 0 has been read out of LDS
#pragma unroll
      for (int ii = 0; ii < 2; ++ii)
#pragma unroll
        for (int j = 0; j < NJ; ++j)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const f32x16_t& a = acc[2 * h + ii][j];
            const int q = wm * 64 + ii * 32 + (lane & 31);
            *reinterpret_cast<float4*>(smem + q * kPitch32 + (ec + 32 * j + 8 * g) * 4) =
                make_float4(a[4 * g], a[4 * g + 1], a[4 * g + 2], a[4 * g + 3]);
          }
      lds_barrier();
      constexpr int kRowsPerPass32 = WAVES;       // 64 lanes cover a row
#pragma unroll 4
      for (int it = 0; it < 128 / kRowsPerPass32; ++it) {
        const int q = it * kRowsPerPass32 + (tid >> 6);
        const int64_t grow = em0 + (q >> 6) * 128 + 64 * h + (q & 63);
        if (grow >= em_end || gcol >= en_end) continue;
        const uint4 v = *reinterpret_cast<const uint4*>(smem + q * kPitch32 + c4 * 4);
        float* dst = reinterpret_cast<float*>(Cp) + grow * ldc + gcol;
        if (vec && gcol + 4 <= en_end) {
          store_c16(dst, v, half < 0);
        } else {
          const uint32_t wv[4] = {v.x, v.y, v.z, v.w};
          for (int e = 0; e < 4 && gcol + e < en_end; ++e) dst[e] = __uint_as_float(wv[e]);
        }
      }
    }
  }
}

// C[tile] = part[2 i] + part[2 i + 1] for the split tiles split_from + i (dense mode, FP32):
// four consecutive columns per lane.  The two halves are added in a fixed order, so the
// result does not depend on which half finished first.
__global__ __launch_bounds__(256) void split_reduce_kernel(NtArgs p) {
  const int i = blockIdx.y;
  const int t = p.split_from + i;
  const int per_group = kGroupM * p.tiles_n;
  const int g = t / per_group;
  const int first = g * kGroupM;
  const int gs = min(p.tiles_m - first, kGroupM);
  const int64_t m0 = (int64_t)(first + (t % per_group) % gs) * BM;
  const int64_t n0 = (int64_t)((t % per_group) / gs) * BN;
  const int e = (blockIdx.x * 256 + threadIdx.x) * 4;      // element of the 256 x 256 tile
  const int r = e / BN, c = e % BN;
  const int64_t grow = m0 + r, gcol = n0 + c;
  if (grow >= p.M || gcol >= p.N) return;
  const float4 a = *reinterpret_cast<const float4*>(p.part + (int64_t)(2 * i) * BM * BN + e);
  const float4 b = *reinterpret_cast<const float4*>(p.part + (int64_t)(2 * i + 1) * BM * BN + e);
  const float sum[4] = {a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w};
  float* dst = reinterpret_cast<float*>(p.C) + grow * p.ldc + gcol;
  if (p.vec_store && gcol + 4 <= p.N) {
    *reinterpret_cast<float4*>(dst) = make_float4(sum[0], sum[1], sum[2], sum[3]);
  } else {
    for (int k = 0; k < 4 && gcol + k < p.N; ++k) dst[k] = sum[k];
  }
}

// Blocks resident at once: one block per CU (its LDS).
int64_t resident_blocks() {
  int dev = 0, ncu = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      ncu <= 0)
    return 256;
  return ncu;
}

// The loads address a tile with 32-bit byte offsets from its first element: a k-major operand
// spans 256 rows, an mn-major one all K rows.
bool nt_offsets_fit(int64_t K, int64_t lda, int64_t ldb, bool a_mn = false, bool b_mn = false) {
  const int64_t lim = (int64_t)1 << 31;
  const int64_t ra = a_mn ? K + BK : BM, rb = b_mn ? K + BK : BN;
  return K * 2 < lim && ra * lda * 2 < lim && rb * ldb * 2 < lim;
}

int vec_store_ok(const void* C, int64_t ldc, int esize) {
  return (reinterpret_cast<uintptr_t>(C) % 16 == 0) && ((ldc * esize) % 16 == 0);
}

}  // namespace

size_t gemm_nt_split_bytes(int64_t M, int64_t N) {
  const int64_t tiles = ((M + BM - 1) / BM) * ((N + BN - 1) / BN);
  return (size_t)(2 * std::min<int64_t>(tiles, kMaxSplitTiles)) * BM * BN * sizeof(float);
}

namespace {

// Shared launch of the dense NT GEMM: bf = B in the fragment-major layout (a_mn = b_mn = 0,
// K a multiple of 64).
hipError_t launch_dense(int64_t M, int64_t N, int64_t K, const uint16_t* A, int64_t lda, int a_mn,
                        const uint16_t* B, int64_t ldb, int b_mn, bool bf, void* C, int64_t ldc,
                        int c_f32, float* part, hipStream_t s, uint16_t* at, int64_t ldat) {
  // (a stage's 64 rows of A^T, 128 ldat bytes, stay below 2^31: 32-bit store offsets)
  if (at != nullptr && (c_f32 || a_mn || b_mn || M % 8 != 0 || ldat < M || ldat % 4 != 0 ||
                        ldat >= kGemmAtMaxLd || reinterpret_cast<uintptr_t>(at) % 8 != 0))
    return hipErrorInvalidValue;
  if (bf && (a_mn || b_mn || K % BK != 0 || reinterpret_cast<uintptr_t>(B) % 16 != 0))
    return hipErrorInvalidValue;
  if (at != nullptr && (N == 0 || (N + BN - 1) / BN < 8)) {
    // no tiles, or fewer than 8 tile columns (a tile would own more than two A^T pieces per
    // stage): the transpose kernel writes A^T instead
    if (M > 0 && K > 0) {
      const hipError_t e = launch_transpose_bf16(A, M, K, lda, at, ldat, 1, 0, 0, s);
      if (e != hipSuccess) return e;
    }
    at = nullptr;
  }
  if (M == 0 || N == 0) return hipSuccess;
  if (!nt_offsets_fit(K, lda, bf ? K : ldb, a_mn, b_mn)) return hipErrorInvalidValue;
  NtArgs a{};
  a.A = A; a.B = B; a.C = C; a.lda = lda; a.ldb = ldb; a.ldc = ldc;
  a.M = M; a.N = N; a.K = K;
  a.at = at; a.ldat = ldat;
  a.vec_store = vec_store_ok(C, ldc, c_f32 ? 4 : 2);
  a.tiles_m = (int)((M + BM - 1) / BM);
  a.tiles_n = (int)((N + BN - 1) / BN);
  const int64_t tiles = (int64_t)a.tiles_m * a.tiles_n;
  int64_t items = tiles;
  // A last round that would leave at least half the CUs idle runs as K-halves instead (FP32
  // output only; needs a partial buffer and at least two full stages).
  // The split is decided per XCD: each runs tiles / 8 tiles on cus / 8 CUs.
  const int64_t cus = resident_blocks();
  const int64_t rem = tiles % cus;
  if (c_f32 && part != nullptr && tiles % kXcds == 0 && cus % kXcds == 0 && rem > 0 &&
      2 * rem <= cus && rem <= kMaxSplitTiles && K / BK >= 2) {
    a.part = part;
    a.split_from = (int)(tiles - rem);
    a.full_per_xcd = (int)((tiles - rem) / kXcds);
    a.split_per_xcd = (int)(rem / kXcds);
    a.split_stage = (K / BK) / 2;
    items = tiles + rem;
  }
  const dim3 grid((unsigned)items);
  const dim3 b8(8 * 64), b4(4 * 64);
  if (bf) {
    if (c_f32) hipLaunchKernelGGL((gemm_nt_kernel<true, kDense, false, false, 4, 0, true>), grid, b4, 0, s, a);
    else if (at != nullptr) hipLaunchKernelGGL((gemm_nt_kernel<false, kDenseAT, false, false, 4, 0, true, true>), grid, b4, 0, s, a);
    else hipLaunchKernelGGL((gemm_nt_kernel<false, kDense, false, false, 4, 0, true>), grid, b4, 0, s, a);
  } else if (c_f32) {
    if (a_mn && b_mn) hipLaunchKernelGGL((gemm_nt_kernel<true, kDense, true, true, 8>), grid, b8, 0, s, a);
    else if (b_mn) hipLaunchKernelGGL((gemm_nt_kernel<true, kDense, false, true, 8>), grid, b8, 0, s, a);
    else if (a_mn) hipLaunchKernelGGL((gemm_nt_kernel<true, kDense, true, false, 8>), grid, b8, 0, s, a);
    else hipLaunchKernelGGL((gemm_nt_kernel<true, kDense, false, false, 4>), grid, b4, 0, s, a);
  } else {
    if (a_mn && b_mn) hipLaunchKernelGGL((gemm_nt_kernel<false, kDense, true, true, 8>), grid, b8, 0, s, a);
    else if (b_mn) hipLaunchKernelGGL((gemm_nt_kernel<false, kDense, false, true, 8>), grid, b8, 0, s, a);
    else if (a_mn) hipLaunchKernelGGL((gemm_nt_kernel<false, kDense, true, false, 8>), grid, b8, 0, s, a);
    else if (at != nullptr && a.tiles_n < 16) hipLaunchKernelGGL((gemm_nt_kernel<false, kDenseAT, false, false, 4, 0, false, true>), grid, b4, 0, s, a);
    else if (at != nullptr) hipLaunchKernelGGL((gemm_nt_kernel<false, kDenseAT, false, false, 4>), grid, b4, 0, s, a);
    else hipLaunchKernelGGL((gemm_nt_kernel<false, kDense, false, false, 4>), grid, b4, 0, s, a);
  }
  if (a.part != nullptr)
    hipLaunchKernelGGL(split_reduce_kernel, dim3(BM * BN / (256 * 4), (unsigned)rem), dim3(256),
                       0, s, a);
  return hipGetLastError();
}

// Row-major bf16 B [N, K] (row stride ld) -> fragment-major (kBfBlock): one lane per 16-byte
// operand; rows past N (to the next multiple of 32) are zeros.
__global__ __launch_bounds__(256) void frag_pack_kernel(const uint16_t* __restrict__ B, int64_t N,
                                                        int64_t K, int64_t ld,
                                                        uint16_t* __restrict__ out,
                                                        int64_t total) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;   // 16-byte operand index
  if (i >= total) return;
  const int64_t blk = i / 64, L = i % 64;
  const int64_t kblocks = K / 16;
  const int64_t nb = blk / kblocks, kb = blk % kblocks;
  const int64_t n = nb * 32 + L % 32, k = kb * 16 + 8 * (L / 32);
  uint4 v = make_uint4(0, 0, 0, 0);
  if (n < N) v = *reinterpret_cast<const uint4*>(B + n * ld + k);
  *reinterpret_cast<uint4*>(out + i * 8) = v;
}

}  // namespace

size_t gemm_frag_bytes(int64_t N, int64_t K) { return (size_t)((N + 31) / 32) * 32 * K * 2; }

hipError_t launch_frag_pack(const uint16_t* B, int64_t N, int64_t K, int64_t ld, uint16_t* out,
                            hipStream_t s) {
  if (N == 0 || K == 0) return hipSuccess;
  if (K % 16 || ld % 8 || reinterpret_cast<uintptr_t>(B) % 16 || reinterpret_cast<uintptr_t>(out) % 16)
    return hipErrorInvalidValue;
  const int64_t total = (N + 31) / 32 * (K / 16) * 64;
  hipLaunchKernelGGL(frag_pack_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, B,
                     N, K, ld, out, total);
  return hipGetLastError();
}

hipError_t launch_gemm_nt(int64_t M, int64_t N, int64_t K, const uint16_t* A, int64_t lda,
                          int a_mn, const uint16_t* B, int64_t ldb, int b_mn, void* C,
                          int64_t ldc, int c_f32, float* part, hipStream_t s, uint16_t* at,
                          int64_t ldat) {
  return launch_dense(M, N, K, A, lda, a_mn, B, ldb, b_mn, false, C, ldc, c_f32, part, s, at,
                      ldat);
}

hipError_t launch_gemm_nt_bf(int64_t M, int64_t N, int64_t K, const uint16_t* A, int64_t lda,
                             const uint16_t* Bf, void* C, int64_t ldc, int c_f32, float* part,
                             hipStream_t s, uint16_t* at, int64_t ldat) {
  return launch_dense(M, N, K, A, lda, 0, Bf, K, 0, true, C, ldc, c_f32, part, s, at, ldat);
}

hipError_t launch_gemm_nt_packed_b(int64_t M, int64_t N, int64_t K, const uint16_t* A,
                                   int64_t lda, int bfmt, const uint8_t* codes,
                                   const uint8_t* scales, const float* S, uint16_t* C,
                                   int64_t ldc, hipStream_t s) {
  if (K % BK != 0 || (bfmt == QF_FMT_Q4K && K % 256 != 0) || codes == nullptr ||
      (bfmt != QF_FMT_Q4K && scales == nullptr) || (bfmt == QF_FMT_NVFP4 && S == nullptr))
    return hipErrorInvalidValue;
  if (M == 0 || N == 0) return hipSuccess;
  if (!nt_offsets_fit(K, lda, K)) return hipErrorInvalidValue;
  NtArgs a{};
  a.A = A; a.B = nullptr; a.C = C; a.lda = lda; a.ldb = K; a.ldc = ldc;
  a.M = M; a.N = N; a.K = K;
  a.bq_codes = codes; a.bq_scales = scales; a.bq_S = S;
  a.vec_store = vec_store_ok(C, ldc, 2);
  a.tiles_m = (int)((M + BM - 1) / BM);
  a.tiles_n = (int)((N + BN - 1) / BN);
  const dim3 grid((unsigned)((int64_t)a.tiles_m * a.tiles_n)), b4(4 * 64);
  switch (bfmt) {
    case QF_FMT_NVFP4:
      hipLaunchKernelGGL((gemm_nt_kernel<false, kDense, false, false, 4, QF_FMT_NVFP4>), grid, b4, 0, s, a);
      break;
    case QF_FMT_MXFP4:
      hipLaunchKernelGGL((gemm_nt_kernel<false, kDense, false, false, 4, QF_FMT_MXFP4>), grid, b4, 0, s, a);
      break;
    case QF_FMT_Q4K:
      hipLaunchKernelGGL((gemm_nt_kernel<false, kDense, false, false, 4, QF_FMT_Q4K>), grid, b4, 0, s, a);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_grouped_nt_rows(int64_t E, int64_t T, int64_t N, int64_t K, const int64_t* off,
                                  const int* tile_start, const uint16_t* A, int64_t lda,
                                  const uint16_t* B, int64_t ldb, int b_mn, int64_t bstride,
                                  uint16_t* C, int64_t ldc, hipStream_t s, uint16_t* at,
                                  int64_t ldat, const int* kstart) {
  if (at != nullptr && (b_mn || (N + BN - 1) / BN < 8 || kstart == nullptr || ldat % 4 != 0 ||
                        ldat >= kGemmAtMaxLd || reinterpret_cast<uintptr_t>(at) % 8 != 0))
    return hipErrorInvalidValue;
  if (T == 0 || N == 0 || E == 0) return hipSuccess;
  if (!nt_offsets_fit(K, lda, ldb, false, b_mn)) return hipErrorInvalidValue;
  NtArgs a{};
  a.A = A; a.B = B; a.C = C; a.lda = lda; a.ldb = ldb; a.ldc = ldc; a.bstride = bstride;
  a.M = T; a.N = N; a.K = K; a.off = off; a.tile_start = tile_start; a.E = (int)E;
  a.at = at; a.ldat = ldat; a.kstart = kstart;
  a.vec_store = vec_store_ok(C, ldc, 2);
  a.tiles_n = (int)((N + BN - 1) / BN);
  a.tiles_m = (int)((T + BM - 1) / BM + E);
  const int64_t per = ((int64_t)a.tiles_m * a.tiles_n + kXcds - 1) / kXcds;
  const dim3 grid((unsigned)(kXcds * per));
  if (b_mn) hipLaunchKernelGGL((gemm_nt_kernel<false, kGroupRows, false, true, 8>), grid, dim3(8 * 64), 0, s, a);
  else if (at != nullptr && a.tiles_n < 16) hipLaunchKernelGGL((gemm_nt_kernel<false, kGroupRowsAT, false, false, 4, 0, false, true>), grid, dim3(4 * 64), 0, s, a);
  else if (at != nullptr) hipLaunchKernelGGL((gemm_nt_kernel<false, kGroupRowsAT, false, false, 4>), grid, dim3(4 * 64), 0, s, a);
  else hipLaunchKernelGGL((gemm_nt_kernel<false, kGroupRows, false, false, 4>), grid, dim3(4 * 64), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_grouped_nt_k(int64_t E, int64_t M, int64_t N, int64_t Kpad, const int* kstart,
                                const int* order, const uint16_t* A, int64_t lda,
                                const uint16_t* B, int64_t ldb, float* C, int64_t ldc,
                                int64_t cstride, hipStream_t s) {
  if (E == 0 || M == 0 || N == 0) return hipSuccess;
  if (!nt_offsets_fit(Kpad, lda, ldb)) return hipErrorInvalidValue;
  NtArgs a{};
  a.A = A; a.B = B; a.C = C; a.lda = lda; a.ldb = ldb; a.ldc = ldc; a.cstride = cstride;
  a.M = M; a.N = N; a.K = Kpad; a.kstart = kstart; a.order = order; a.E = (int)E;
  a.vec_store = vec_store_ok(C, ldc, 4) && (cstride * 4) % 16 == 0;
  a.tiles_m = (int)((M + BM - 1) / BM);
  a.tiles_n = (int)((N + BN - 1) / BN);
  const int64_t cmax = ((int64_t)a.tiles_m * a.tiles_n + kXcds - 1) / kXcds;
  const dim3 grid((unsigned)(kXcds * E * cmax));
  hipLaunchKernelGGL((gemm_nt_kernel<true, kGroupK, false, false, 4>), grid, dim3(4 * 64), 0, s, a);
  return hipGetLastError();
}

}  // namespace qf
