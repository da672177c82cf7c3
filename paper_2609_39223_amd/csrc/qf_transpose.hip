// bf16 matrix transpose for gfx950: out[c][r] = in[r][c], optionally batched.
//
// The backward GEMMs of the quantization-aware layer run in NT form, which needs dY^T and the
// transposed operands.  Register-only form, no LDS: a 256-thread workgroup covers a 64 x 256
// tile, wavefront w its columns 64 w .. 64 w + 63, and lane 8 a + b loads rows 8 a .. 8 a + 7
// of column chunk b (8 lanes read 128 contiguous bytes of each row), transposes that 8 x 8
// block in registers and writes it as 8 output rows of 16 bytes (the 8 lanes with the same b
// write 128 contiguous bytes of each).  Non-temporal stores: the output is not read again by
// the launch.  Tile shapes from 32 x 512 to 256 x 256 through LDS (eight variants) measured
// 47-58 us at 14336 x 4096 against 47.5 us for this form, which needs no barrier.  (The grouped
// transposes of the expert layer keep the LDS tile of the transposing quantizer: this form
// measured 625 against 600 us there.)
// R and C must be multiples of 8 (16-byte chunks).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "qf_codecs.h"
#include "qf_internal.h"

namespace qf {
namespace {

using namespace codec;

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

// Tile of 64 input rows [r0, r_end) (rows past r_end read as zeros) and 256 columns from c0,
// written to output rows c0 .. and output columns from oc0, up to col_end.
__device__ __forceinline__ void transpose_tile(const uint16_t* __restrict__ in, int64_t ldi,
                                               int64_t r0, int64_t r_end, int64_t c0, int64_t C,
                                               uint16_t* __restrict__ out, int64_t ldo,
                                               int64_t oc0, int64_t col_end) {
  const int lane = threadIdx.x & 63, a = lane >> 3, b = lane & 7;
  const int64_t col = c0 + (threadIdx.x >> 6) * 64 + b * 8;
  uint32_t w[8][4];
#pragma unroll
  for (int i = 0; i < 8; ++i) {             // all eight loads first
    const int64_t row = r0 + a * 8 + i;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (row < r_end && col < C) v = *reinterpret_cast<const uint4*>(in + row * ldi + col);
    w[i][0] = v.x; w[i][1] = v.y; w[i][2] = v.z; w[i][3] = v.w;
  }
  const int64_t ocol = oc0 + a * 8;
  if (ocol >= col_end) return;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    if (col + j >= C) break;
    const uint4 o = block_row_transposed(w, j);
    __builtin_nontemporal_store(u32x4_t{o.x, o.y, o.z, o.w},
                                reinterpret_cast<u32x4_t*>(out + (col + j) * ldo + ocol));
  }
}

__global__ __launch_bounds__(256) void transpose_bf16_kernel(const uint16_t* __restrict__ in,
                                                             int64_t R, int64_t C, int64_t ldi,
                                                             uint16_t* __restrict__ out,
                                                             int64_t ldo, int64_t ibs,
                                                             int64_t obs) {
  const int64_t r0 = (int64_t)blockIdx.y * kTR;
  transpose_tile(in + (int64_t)blockIdx.z * ibs, ldi, r0, R, (int64_t)blockIdx.x * kTC, C,
                 out + (int64_t)blockIdx.z * obs, ldo, r0, R);
}

}  // namespace

hipError_t launch_transpose_bf16(const uint16_t* in, int64_t R, int64_t C, int64_t ldi,
                                 uint16_t* out, int64_t ldo, int64_t batch, int64_t ibs,
                                 int64_t obs, hipStream_t s) {
  if (R == 0 || C == 0 || batch == 0) return hipSuccess;
  const dim3 grid((unsigned)((C + kTC - 1) / kTC), (unsigned)((R + kTR - 1) / kTR),
                  (unsigned)batch);
  hipLaunchKernelGGL(transpose_bf16_kernel, grid, dim3(256), 0, s, in, R, C, ldi, out, ldo, ibs,
                     obs);
  return hipGetLastError();
}

}  // namespace qf
