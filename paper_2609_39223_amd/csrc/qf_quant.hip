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

#include <atomic>

#include "qf.h"
#include "qf_codecs.h"
#include "qf_internal.h"

namespace qf {
namespace {

using namespace codec;

constexpr int kThreads = 256;

// ============================================================================= fill / amax
__global__ void fill_f32_kernel(float* p, int64_t n, float v) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

// ---- tensor amax --------------------------------------------------------------------------
// max |x| as bf16 magnitude bits (NaN bit patterns sort above +inf), reduced per workgroup and
// folded with integer atomic maxima (order independent, so the result is exact and
// deterministic).  A fold word is 64 bits: the running maximum (binary32 bits) in the low word
// and a ticket count of the contributors that have folded theirs in in the high word; the
// contributor that takes the last ticket holds the maximum of all of them and returns the word
// to zero.  Words start at zero when the library loads, so no pass needs a clearing dispatch.
// A pass folds in two levels: workgroup i into first-level word i mod kAmaxSub, the last
// workgroup of each of those into the top word, whose last contributor writes the result
// (*amax = m, or max(*amax, m) when accumulating, compared as bits).  Every word sits on a
// 256-byte line of its own: device-scope atomics on one line are performed one after another,
// and a single word per pass cost ~2 us more at the end of a 14336 x 4096 pass.  The host hands
// each pass its own slot (one per tensor of a batch) from a ring of kAmaxSlots, so passes
// running concurrently on different streams do not share one unless kAmaxSlots slots are taken
// in between.
constexpr uint32_t kAmaxSlots = 1024;
constexpr uint32_t kAmaxSub = 8;                     // first-level words per slot
constexpr uint32_t kAmaxLine = 32;                   // 64-bit words per 256-byte line
// slot s: first-level words at lines 9s .. 9s+7, the top word at line 9s+8
__device__ uint64_t g_amax_slot[kAmaxSlots * (kAmaxSub + 1) * kAmaxLine];

// Folds v into word w as one of n contributors.  Returns true for the last one, with the
// maximum of all n in m, after clearing the word.  Device-scope atomics are performed at the
// device's coherence point.  The fold is acknowledged before the ticket is taken (the wait), so
// every fold precedes the last ticket, and the ticket's returned word carries the maximum of all
// of them; no cache write-back is needed for that (a release ordering would write back this
// XCD's L2 in every workgroup).
__device__ __forceinline__ bool fold_word(uint64_t* w, uint32_t v, uint32_t n, uint32_t& m) {
  if (v != 0u)
    __hip_atomic_fetch_max(reinterpret_cast<uint32_t*>(w), v, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
  __builtin_amdgcn_s_waitcnt(0x0F70);            // vmcnt(0): the fold is acknowledged
  const uint64_t old =
      __hip_atomic_fetch_add(w, 1ull << 32, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if ((uint32_t)(old >> 32) != n - 1u) return false;
  m = (uint32_t)old;
  __hip_atomic_store(w, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return true;
}

// Called by thread 0 of every workgroup of a pass with the workgroup's maximum b.  The pass's
// nblocks workgroups are those of one grid z plane, numbered x + y * gridDim.x.
__device__ __forceinline__ void amax_fold(uint32_t b, uint32_t slot, uint32_t nblocks,
                                          float* amax, int accumulate) {
  uint64_t* rec = &g_amax_slot[(slot % kAmaxSlots) * (kAmaxSub + 1) * kAmaxLine];
  const uint32_t i = blockIdx.x + blockIdx.y * gridDim.x;
  const uint32_t sub = i % kAmaxSub;
  uint32_t m;
  if (!fold_word(rec + sub * kAmaxLine, b << 16, (nblocks - sub + kAmaxSub - 1u) / kAmaxSub, m))
    return;
  if (!fold_word(rec + kAmaxSub * kAmaxLine, m, nblocks < kAmaxSub ? nblocks : kAmaxSub, m))
    return;
  uint32_t* out = reinterpret_cast<uint32_t*>(amax);
  const uint32_t prev = accumulate ? *out : 0u;
  *out = prev > m ? prev : m;
}

// Block-wide maximum of m, then the fold by thread 0.
__device__ __forceinline__ void amax_block_fold(uint32_t m, uint32_t slot, uint32_t nblocks,
                                                float* amax, int accumulate) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const uint32_t o = (uint32_t)__shfl_xor((int)m, off, 64);
    m = o > m ? o : m;
  }
  __shared__ uint32_t wmax[kThreads / 64];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  if (lane == 0) wmax[wid] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t b = wmax[0];
    for (int i = 1; i < kThreads / 64; ++i) b = wmax[i] > b ? wmax[i] : b;
    amax_fold(b, slot, nblocks, amax, accumulate);
  }
}

// max |x| over the eight bf16 of a 16-byte chunk, as magnitude bits
__device__ __forceinline__ uint32_t max_abs_chunk(const uint4& v) {
  const uint32_t w[4] = {v.x & 0x7FFF7FFFu, v.y & 0x7FFF7FFFu, v.z & 0x7FFF7FFFu,
                         v.w & 0x7FFF7FFFu};
  uint32_t m = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const uint32_t a = w[q] & 0xFFFFu, b = w[q] >> 16;
    m = a > m ? a : m;
    m = b > m ? b : m;
  }
  return m;
}

// Contiguous tensors (n 16-byte chunks each, tensor z at chunk z * n): a grid-stride loop with
// kAmaxFlatLoads loads in flight per lane; about one workgroup per CU over all tensors.
constexpr int kAmaxFlatLoads = 8;
__global__ __launch_bounds__(kThreads) void amax_flat_kernel(const uint4* __restrict__ x,
                                                             int64_t n, uint32_t slot0,
                                                             float* __restrict__ amax,
                                                             int accumulate) {
  const uint4* xt = x + (int64_t)blockIdx.z * n;
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  uint32_t m = 0;
  for (int64_t base = (int64_t)blockIdx.x * kThreads + threadIdx.x; base < n;
       base += stride * kAmaxFlatLoads) {
    uint4 v[kAmaxFlatLoads];
#pragma unroll
    for (int j = 0; j < kAmaxFlatLoads; ++j) {
      const int64_t i = base + j * stride;
      v[j] = i < n ? xt[i] : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < kAmaxFlatLoads; ++j) {
      const uint32_t a = max_abs_chunk(v[j]);
      m = a > m ? a : m;
    }
  }
  amax_block_fold(m, slot0 + blockIdx.z, gridDim.x, amax + blockIdx.z, accumulate);
}

// Strided rows or a row length that is not a multiple of 8: chunks along K (a last partial
// chunk holds K % 8 elements), kAmaxRows rows per lane pass (all loads issued before the
// reduction); the grid is sized for about one pass per lane.
constexpr int kAmaxRows = 16;
__global__ __launch_bounds__(kThreads) void amax_rows_kernel(const uint16_t* __restrict__ x,
                                                             int64_t R, int64_t K, int64_t ldx,
                                                             uint32_t slot, float* __restrict__ amax,
                                                             int accumulate) {
  const int64_t chunks = (K + 7) >> 3;
  uint32_t m = 0;
  for (int64_t c = (int64_t)blockIdx.x * kThreads + threadIdx.x; c < chunks;
       c += (int64_t)gridDim.x * kThreads) {
    const bool whole = c * 8 + 8 <= K;
    for (int64_t r0 = (int64_t)blockIdx.y * kAmaxRows; r0 < R;
         r0 += (int64_t)gridDim.y * kAmaxRows) {
      uint4 v[kAmaxRows];
#pragma unroll
      for (int i = 0; i < kAmaxRows; ++i) {
        v[i] = make_uint4(0, 0, 0, 0);
        if (r0 + i < R) {
          const uint16_t* src = x + (r0 + i) * ldx + c * 8;
          if (whole) {
            v[i] = *reinterpret_cast<const uint4*>(src);
          } else {                                  // the row's last K % 8 elements only
            uint32_t h[8] = {0, 0, 0, 0, 0, 0, 0, 0};
            for (int e = 0; e < (int)(K - c * 8); ++e) h[e] = src[e];
            v[i] = pack8(h);
          }
        }
      }
#pragma unroll
      for (int i = 0; i < kAmaxRows; ++i) {
        const uint32_t a = max_abs_chunk(v[i]);
        m = a > m ? a : m;
      }
    }
  }
  amax_block_fold(m, slot, gridDim.x * gridDim.y, amax, accumulate);
}

// Plain or non-temporal stores of 4 and 16 bytes (aligned).
template <bool NT>
__device__ __forceinline__ void store_u32(void* p, uint32_t v) {
  if (NT) __builtin_nontemporal_store(v, reinterpret_cast<uint32_t*>(p));
  else *reinterpret_cast<uint32_t*>(p) = v;
}
template <bool NT>
__device__ __forceinline__ void store_u128(void* p, uint4 v) {
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  if (NT) __builtin_nontemporal_store(u32x4{v.x, v.y, v.z, v.w}, reinterpret_cast<u32x4*>(p));
  else *reinterpret_cast<uint4*>(p) = v;
}

// ============================================================================= NVFP4
// grid.z indexes batched tensors (expert weights): tensor z uses g[z] and element offset
// z * tstride (input) / z * R * K (outputs).
// STREAM: the outputs are written with non-temporal stores, which do not allocate in the
// last-level cache, so an input read just before (by the amax pass) stays there for this
// kernel's read.
template <int RPT, bool STREAM>
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
  __shared__ f32x2_t tab[128];              // (D, 1 / D) of every E4M3 code under this S
  nvfp4_fill_table(S, tab, threadIdx.x);
  __syncthreads();
  const Nvfp4Table bs{tab};
  // The two lanes of a block pair split the scale codes: the even lane encodes rows 0, 2, ..
  // and the odd lane rows 1, 3, .. of this thread's RPT, and each takes the other's over DPP.
  static_assert(RPT % 2 == 0, "rows are taken in pairs");
  // With K a multiple of 64 each group of 8 lanes (4 blocks) lies wholly inside or outside a
  // row and its 4 scale bytes start at a multiple of 4 (for an aligned scales pointer): one
  // word store per group; otherwise one byte per block.
  const bool wide_scales = scales && (K & 63) == 0 && (reinterpret_cast<uintptr_t>(scales) & 3) == 0;
  const bool odd = (threadIdx.x & 1) != 0;
  const uint32_t odd_mask = 0u - (threadIdx.x & 1u);
  uint32_t ab[RPT], scs[RPT];
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    uint32_t h[8];
    unpack8(vin[i], h);
    ab[i] = nvfp4_block_max(h);
  }
#pragma unroll
  for (int i = 0; i < RPT; i += 2) {
    // (a mask select: a conditional on the array index would put ab[] in memory)
    const uint32_t a = ab[i] ^ ((ab[i] ^ ab[i + 1]) & odd_mask);
    const uint32_t mine = nvfp4_scale_code(a, S, six_s);
    const uint32_t theirs = xor1_u32(mine);
    scs[i] = odd ? theirs : mine;
    scs[i + 1] = odd ? mine : theirs;
  }
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    const int64_t r = (int64_t)blockIdx.y * RPT + i;
    const bool ok = col_ok && r < R;
    uint32_t h[8], cw, xh[8];
    const uint32_t sc = scs[i];
    unpack8(vin[i], h);
    nvfp4_encode(h, ab[i], sc, bs, cw, xh);
    // lane 8j gathers the scale bytes of its 4 blocks (lanes 8j, +2, +4, +6) into one word
    uint32_t s4 = sc | (xor2_u32(sc) << 8);
    s4 |= xor_swz_u32<4>(s4) << 16;
    if (ok) {
      if (codes) store_u32<STREAM>(codes + obase / 2 + r * (K / 2) + c * 4, cw);
      uint8_t* srow = scales + obase / 16 + r * (K / 16);
      if (wide_scales) {
        if ((c & 7) == 0) store_u32<STREAM>(srow + c / 2, s4);
      } else if (scales && (c & 1) == 0) {
        srow[c / 2] = (uint8_t)sc;
      }
      if (xhat) store_u128<STREAM>(xhat + obase + r * K + c * 8, pack8(xh));
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
template <int RPT, bool MSE>
__global__ __launch_bounds__(kThreads) void q4k_kernel(const uint16_t* __restrict__ x, int64_t R,
                                                       int64_t K, int64_t ldx,
                                                       uint8_t* __restrict__ packed,
                                                       uint16_t* __restrict__ xhat) {
  const int64_t chunks = K >> 3;
  const int64_t c = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  const bool col_ok = c < chunks;
  const int L = threadIdx.x & 31;           // lane within the super-block
  const int64_t sb = c >> 5;
#pragma unroll 1
  for (int i = 0; i < RPT; ++i) {
    const int64_t r = (int64_t)blockIdx.y * RPT + i;
    const bool ok = col_ok && r < R;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (ok) v = *reinterpret_cast<const uint4*>(x + r * ldx + c * 8);
    uint32_t h[8], xh[8];
    unpack8(v, h);
    Q4kChunk q;
    if (MSE) q4k_mse_chunk(h, q, xh);
    else q4k_chunk(h, q, xh);
    q4k_store(q, L, ok && packed, packed ? packed + (r * (K / 256) + sb) * 144 : nullptr);
    if (ok && xhat) *reinterpret_cast<uint4*>(xhat + r * K + c * 8) = pack8(xh);
  }
}

// Q4_K rows with sixteen elements per lane (q4k_chunk16): a group of 16 lanes holds one
// 256-element super-block, so the per-sub-block work of the min-max encoder (VALU-bound at
// eight elements per lane) is shared by twice the elements.  A wavefront covers 1024
// consecutive elements of a row (K a multiple of 1024).  Its loads and x_hat stores stay fully
// coalesced 1 KB accesses: lane l < 32 moves 16-byte chunks 2l and 64 + 2l of the wavefront's
// 128, lane l + 32 chunks 2l + 1 and 65 + 2l, and one exchange between the wavefront's halves
// (v_permlane32_swap: the first chunk of the high lanes for the second of the low ones) turns
// that into chunks 2l, 2l + 1 for every lane l, i.e. elements 16 l .. 16 l + 15 (the same
// exchange undoes it before the stores).  Reading 32 contiguous bytes per lane instead (two
// loads at a 32-byte stride) measured 46.8-47.2 us against 41.8-42.6 us at 14336 x 4096.
__device__ __forceinline__ void swap_halves(uint4& a, uint4& b) {
  // a in the high 32 lanes <-> b in the low 32 lanes
  auto x = __builtin_amdgcn_permlane32_swap(a.x, b.x, false, false);
  auto y = __builtin_amdgcn_permlane32_swap(a.y, b.y, false, false);
  auto z = __builtin_amdgcn_permlane32_swap(a.z, b.z, false, false);
  auto w = __builtin_amdgcn_permlane32_swap(a.w, b.w, false, false);
  a = make_uint4(x[0], y[0], z[0], w[0]);
  b = make_uint4(x[1], y[1], z[1], w[1]);
}

template <int RPT>
__global__ __launch_bounds__(kThreads) void q4k16_kernel(const uint16_t* __restrict__ x, int64_t R,
                                                         int64_t K, int64_t ldx,
                                                         uint8_t* __restrict__ packed,
                                                         uint16_t* __restrict__ xhat) {
  const int64_t c = (int64_t)blockIdx.x * kThreads + threadIdx.x;   // 16-element chunk
  // K is a multiple of 1024, so a wavefront lies wholly inside the row or wholly past it
  const bool col_ok = c < (K >> 4);
  const int L = threadIdx.x & 15;           // lane within the super-block
  const int64_t sb = c >> 4;
  const int lw = threadIdx.x & 63;          // lane within the wavefront
  const int64_t wbase = (c - lw) * 16;      // the wavefront's first element in the row
  const int q0 = lw < 32 ? 2 * lw : 2 * lw - 63;   // 16-byte chunk moved first (second: + 64)
#pragma unroll 1
  for (int i = 0; i < RPT; ++i) {
    const int64_t r = (int64_t)blockIdx.y * RPT + i;
    const bool ok = col_ok && r < R;        // uniform over the wavefront
    uint4 v0 = make_uint4(0, 0, 0, 0), v1 = make_uint4(0, 0, 0, 0);
    if (ok) {
      const uint16_t* xr = x + r * ldx + wbase + 8 * q0;
      v0 = *reinterpret_cast<const uint4*>(xr);
      v1 = *reinterpret_cast<const uint4*>(xr + 512);
    }
    swap_halves(v0, v1);
    uint32_t h[16], xw[8];
    unpack8(v0, h);
    unpack8(v1, h + 8);
    Q4kChunk16 q;
    q4k_chunk16(h, q, xw);
    q4k_store16(q, L, ok && packed, packed ? packed + (r * (K / 256) + sb) * 144 : nullptr);
    uint4 o0 = make_uint4(xw[0], xw[1], xw[2], xw[3]), o1 = make_uint4(xw[4], xw[5], xw[6], xw[7]);
    swap_halves(o0, o1);
    if (ok && xhat) {
      uint16_t* xo = xhat + r * K + wbase + 8 * q0;
      *reinterpret_cast<uint4*>(xo) = o0;
      *reinterpret_cast<uint4*>(xo + 512) = o1;
    }
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
  if (GROUPED && !grouped_tile(blockIdx.y, off, kstart, E, r0, r_end, oc0)) return;
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
  store_tile_transposed(tile, t, out, ldo, c0, oc0, K, GROUPED ? INT64_MAX : R);
}

// ============================================ dequantize from packed codes, transposed output
// out[k][r] = x_hat[r][k] of a tensor stored as packed codes (the layer's saved operands): the
// tile and store of quant_t_kernel, with each lane's chunk decoded from its 4 code bytes and
// block scale (Q4_K: 8 code bytes of its super-block plus the block header) by the quantizers'
// own decode functions, so the output equals quant_t_kernel's for the tensor the codes came
// from, bit for bit.  NVFP4 takes the stored tensor decode scale S.  R and K multiples of 8.
template <int FMT>
__global__ __launch_bounds__(kThreads) void dequant_t_kernel(const uint8_t* __restrict__ codes,
                                                             const uint8_t* __restrict__ scales,
                                                             const float* __restrict__ Sp,
                                                             int64_t R, int64_t K,
                                                             uint16_t* __restrict__ out,
                                                             int64_t ldo, int64_t obs) {
  __shared__ uint4 tile[kTR * (kTC / 8)];
  const int t = threadIdx.x;
  const int64_t c0 = (int64_t)blockIdx.x * kTC, r0 = (int64_t)blockIdx.y * kTR;
  // grid.z indexes equally shaped tensors stored back to back (expert weights): tensor z's
  // codes / scales / blocks follow the z before it, its decode scale is Sp[z], and its output
  // starts obs elements after tensor z - 1's
  const int64_t z = blockIdx.z;
  if (FMT == QF_FMT_Q4K) {
    codes += z * R * (K / 256) * 144;
  } else {
    codes += z * R * (K / 2);
    scales += z * R * (K / (FMT == QF_FMT_NVFP4 ? 16 : 32));
  }
  out += z * obs;
  const float S = FMT == QF_FMT_NVFP4 ? Sp[z] : 0.0f;
  uint32_t cw[8], sc[8];
  uint4 hd[8];
  const int cc = t & 31;
  const int64_t gc = c0 + cc * 8;                 // first element of this lane's chunk
#pragma unroll
  for (int i = 0; i < 8; ++i) {                   // all loads first
    const int64_t gr = r0 + i * 8 + (t >> 5);
    cw[i] = 0; sc[i] = 0; hd[i] = make_uint4(0, 0, 0, 0);
    if (gr < R && gc < K) {
      if (FMT == QF_FMT_Q4K) {
        // element e = 8 cc of super-block gc / 256: code bytes 32 (e / 64) + e % 32 .. +7,
        // low nibbles for e % 64 < 32, high nibbles otherwise
        const uint8_t* blk = codes + (gr * (K / 256) + gc / 256) * 144;
        hd[i] = *reinterpret_cast<const uint4*>(blk);
        const int e = (int)(gc % 256);
        const uint2 q = *reinterpret_cast<const uint2*>(blk + 16 + 32 * (e / 64) + e % 32);
        const uint32_t sh = (e % 64) >= 32 ? 4u : 0u;
        cw[i] = (q.x >> sh) & 0x0F0F0F0Fu;
        sc[i] = (q.y >> sh) & 0x0F0F0F0Fu;        // (the second 4 codes)
      } else {
        cw[i] = *reinterpret_cast<const uint32_t*>(codes + gr * (K / 2) + gc / 2);
        sc[i] = scales[gr * (K / (FMT == QF_FMT_NVFP4 ? 16 : 32)) + gc / (FMT == QF_FMT_NVFP4 ? 16 : 32)];
      }
    }
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int row = i * 8 + (t >> 5);
    uint32_t w[4];
    if (FMT == QF_FMT_NVFP4) {
      nvfp4_decode8(cw[i], nvfp4_block_scale(S, sc[i]), w);
    } else if (FMT == QF_FMT_MXFP4) {
      mxfp4_decode8(cw[i], sc[i], w);
    } else {
      // sub-block j = e / 32 (e = 8 cc): its 6-bit scale and min from the header bytes 4-15
      const int j = cc >> 2, jj = j & 3, sh = 8 * jj;
      uint32_t ls, lm;
      if (j < 4) {
        ls = (hd[i].y >> sh) & 63u;
        lm = (hd[i].z >> sh) & 63u;
      } else {
        ls = ((hd[i].w >> sh) & 15u) | (((hd[i].y >> (sh + 6)) & 3u) << 4);
        lm = ((hd[i].w >> (sh + 4)) & 15u) | (((hd[i].z >> (sh + 6)) & 3u) << 4);
      }
      const float t1 = f16_value(hd[i].x & 0xFFFFu) * (float)ls;
      const float t2 = f16_value(hd[i].x >> 16) * (float)lm;
      const uint32_t qw[2] = {cw[i], sc[i]};
      q4k_decode8(qw, t1, t2, w);
    }
    tile[row * 32 + tslot(row, cc)] = make_uint4(w[0], w[1], w[2], w[3]);
  }
  __syncthreads();
  store_tile_transposed(tile, t, out, ldo, c0, r0, K, R);
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

// A contiguous tensor whose rows do not fill the workgroups' lanes (K / 8 chunks not a
// multiple of kThreads) is read as rows of 8 kThreads elements when its size allows (expert
// weights 3072 x 3072 and 3072 x 1536: a quarter of the lanes would idle).  Valid wherever
// the result does not depend on where rows break: the batched NVFP4 x_hat (16-element blocks
// along rows of a multiple of 16, one scale per tensor).
static void contiguous_row_view(int64_t& R, int64_t& K) {
  const int64_t row = 8 * kThreads;
  if ((K >> 3) % kThreads != 0 && (R * K) % row == 0) {
    R = R * K / row;
    K = row;
  }
}

// The next `count` reduction slots of the ring (one per tensor of a pass).
static uint32_t take_amax_slots(uint32_t count) {
  static std::atomic<uint32_t> next{0};
  return next.fetch_add(count, std::memory_order_relaxed) % kAmaxSlots;
}

// About one workgroup per CU over all E tensors, none idle.
static unsigned amax_flat_grid(int64_t n, int64_t E) {
  int64_t gx = 256 / E;
  if (gx < 1) gx = 1;
  const int64_t need = (n + kThreads * kAmaxFlatLoads - 1) / (kThreads * kAmaxFlatLoads);
  if (gx > need) gx = need;
  return (unsigned)(gx < 1 ? 1 : gx);
}

hipError_t launch_amax(const uint16_t* x, int64_t R, int64_t K, int64_t ldx, float* amax,
                       bool accumulate, hipStream_t s) {
  if (R == 0 || K == 0)
    return accumulate ? hipSuccess : launch_fill_f32(amax, 1, 0.0f, s);
  const uint32_t slot = take_amax_slots(1);
  if (ldx == K && K % 8 == 0) {
    const int64_t n = R * K / 8;
    hipLaunchKernelGGL(amax_flat_kernel, dim3(amax_flat_grid(n, 1)), dim3(kThreads), 0, s,
                       reinterpret_cast<const uint4*>(x), n, slot, amax, (int)accumulate);
  } else {
    const int64_t chunks = (K + 7) >> 3;
    int64_t gx = (chunks + kThreads - 1) / kThreads;
    if (gx > 64) gx = 64;
    int64_t gy = (R + kAmaxRows - 1) / kAmaxRows;
    const int64_t cap = 2048 / gx;
    if (gy > cap) gy = cap;
    if (gy < 1) gy = 1;
    hipLaunchKernelGGL(amax_rows_kernel, dim3((unsigned)gx, (unsigned)gy), dim3(kThreads), 0, s,
                       x, R, K, ldx, slot, amax, (int)accumulate);
  }
  return hipGetLastError();
}

hipError_t launch_amax_batched(const uint16_t* x, int64_t E, int64_t R, int64_t K, float* amax,
                               bool accumulate, hipStream_t s) {
  if (E == 0) return hipSuccess;
  if (R == 0 || K == 0)
    return accumulate ? hipSuccess : launch_fill_f32(amax, E, 0.0f, s);
  // tensors are contiguous, R * K apart; R * K is a multiple of 8 for the block formats
  const int64_t n = R * K / 8;
  const uint32_t slot0 = take_amax_slots((uint32_t)E);
  hipLaunchKernelGGL(amax_flat_kernel, dim3(amax_flat_grid(n, E), 1, (unsigned)E),
                     dim3(kThreads), 0, s, reinterpret_cast<const uint4*>(x), n, slot0, amax,
                     (int)accumulate);
  return hipGetLastError();
}

// Rows per thread of the NVFP4 and MXFP4 quantizers (even: NVFP4 pairs rows across lanes).
// At 14336 x 4096 two rows measured 42.6-42.9 against 43.6-43.7 us (NVFP4, given amax) and
// 40.8 against 41.5-41.6 us (MXFP4) for four, and eight rows 46.3-46.6 / 44.0-44.7 us.
constexpr int kRowsPerThread = 2;

hipError_t launch_nvfp4(const uint16_t* x, int64_t R, int64_t K, int64_t ldx, const float* g,
                        float* s_out, uint8_t* codes, uint8_t* scales, uint16_t* xhat,
                        hipStream_t s, bool stream_out) {
  if (R == 0 || K == 0) return hipSuccess;  // nothing to quantize; S is left to the caller
  if (stream_out)
    hipLaunchKernelGGL((nvfp4_kernel<kRowsPerThread, true>), row_grid(R, K, kRowsPerThread),
                       dim3(kThreads), 0, s, x, R, K, ldx, (int64_t)0, g, s_out, codes, scales,
                       xhat);
  else
    hipLaunchKernelGGL((nvfp4_kernel<kRowsPerThread, false>), row_grid(R, K, kRowsPerThread),
                       dim3(kThreads), 0, s, x, R, K, ldx, (int64_t)0, g, s_out, codes, scales,
                       xhat);
  return hipGetLastError();
}

hipError_t launch_nvfp4_batched(const uint16_t* x, int64_t E, int64_t R, int64_t K,
                                const float* g, float* s_out, uint8_t* codes, uint8_t* scales,
                                uint16_t* xhat, hipStream_t s) {
  if (E == 0 || R == 0 || K == 0) return hipSuccess;
  // Blocks of 16 lie along the contiguous rows and the scale g[z] covers the whole tensor, so
  // each (contiguous) tensor may be read as rows of 2048 elements: same blocks, same codes,
  // scales and x_hat at the same offsets, and every lane busy where K / 8 chunks would leave
  // some idle.
  contiguous_row_view(R, K);
  dim3 grid = row_grid(R, K, kRowsPerThread);
  grid.z = (unsigned)E;
  hipLaunchKernelGGL((nvfp4_kernel<kRowsPerThread, false>), grid, dim3(kThreads), 0, s, x, R, K, K,
                     R * K, g, s_out, codes, scales, xhat);
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
  if (K % 1024 == 0) {                      // whole wavefronts of 1024 elements per row
    const dim3 grid((unsigned)((K >> 4) / kThreads + ((K >> 4) % kThreads != 0)),
                    (unsigned)((R + 1) / 2), 1);
    hipLaunchKernelGGL((q4k16_kernel<2>), grid, dim3(kThreads), 0, s, x, R, K, ldx, packed, xhat);
  } else {
    hipLaunchKernelGGL((q4k_kernel<2, false>), row_grid(R, K, 2), dim3(kThreads), 0, s, x, R, K,
                       ldx, packed, xhat);
  }
  return hipGetLastError();
}

hipError_t launch_q4k_mse(const uint16_t* x, int64_t R, int64_t K, int64_t ldx, uint8_t* packed,
                          uint16_t* xhat, hipStream_t s) {
  if (R == 0 || K == 0) return hipSuccess;
  hipLaunchKernelGGL((q4k_kernel<1, true>), row_grid(R, K, 1), dim3(kThreads), 0, s, x, R, K, ldx,
                     packed, xhat);
  return hipGetLastError();
}

template <bool GROUPED>
hipError_t launch_quant_t_impl(int fmt, const uint16_t* x, int64_t R, int64_t K, int64_t ldx,
                               int64_t batch, int64_t xbs, const float* g, uint16_t* out,
                               int64_t ldo, int64_t obs, const int64_t* off, const int* kstart,
                               int E, int64_t ytiles, hipStream_t s) {
  // Plain dense transposes take the register-only form; the grouped ones (expert rows padded
  // to 64) keep the LDS tile, faster there (600 against 625 us for 262144 x 3072).
  if (fmt == QF_FMT_NONE && !GROUPED)
    return launch_transpose_bf16(x, R, K, ldx, out, ldo, batch, xbs, obs, s);
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

hipError_t launch_dequant_t(int fmt, const uint8_t* codes, const uint8_t* scales,
                            const float* S, int64_t R, int64_t K, uint16_t* out, int64_t ldo,
                            hipStream_t s, int64_t batch, int64_t obs) {
  if (R == 0 || K == 0 || batch == 0) return hipSuccess;
  const dim3 grid((unsigned)((K + kTC - 1) / kTC), (unsigned)((R + kTR - 1) / kTR),
                  (unsigned)batch);
  switch (fmt) {
#define QF_DQ(F)                                                                               \
  hipLaunchKernelGGL(dequant_t_kernel<F>, grid, dim3(kThreads), 0, s, codes, scales, S, R, K, \
                     out, ldo, obs);                                                           \
  break;
    case QF_FMT_NVFP4: QF_DQ(QF_FMT_NVFP4)
    case QF_FMT_MXFP4: QF_DQ(QF_FMT_MXFP4)
    case QF_FMT_Q4K: QF_DQ(QF_FMT_Q4K)
#undef QF_DQ
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
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
