// bf16 matrix transpose for gfx950: out[c][r] = in[r][c], optionally batched.
//
// The backward GEMMs of the quantization-aware layer run in NT form, which needs dY^T and the
// transposed quantized operands.  A 64 x 256 tile goes through LDS: rows are read with 16-byte
// loads (512 contiguous bytes per row), each lane then takes an 8 x 8 block out of LDS,
// transposes it in registers and writes 8 rows of 16 bytes; the 8 lanes that share an output
// row write 128 contiguous bytes.  LDS chunk c of tile row r lives at slot
// c ^ (((r >> 3) & 7) << 1), conflict-free for both the row writes and the block reads.
// R and C must be multiples of 8 (16-byte chunks).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "qf_internal.h"

namespace qf {
namespace {

constexpr int TR = 64, TC = 256, NT = 256;

__device__ __forceinline__ int slot(int r, int c) { return c ^ (((r >> 3) & 7) << 1); }

__global__ __launch_bounds__(NT) void transpose_bf16_kernel(const uint16_t* __restrict__ in,
                                                            int64_t R, int64_t C, int64_t ldi,
                                                            uint16_t* __restrict__ out,
                                                            int64_t ldo, int64_t ibs,
                                                            int64_t obs) {
  __shared__ uint4 tile[TR * (TC / 8)];
  const int t = threadIdx.x;
  const int64_t r0 = (int64_t)blockIdx.y * TR, c0 = (int64_t)blockIdx.x * TC;
  in += (int64_t)blockIdx.z * ibs;
  out += (int64_t)blockIdx.z * obs;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int id = i * NT + t;
    const int row = id >> 5, cc = id & 31;
    const int64_t gr = r0 + row, gc = c0 + cc * 8;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (gr < R && gc < C) v = *reinterpret_cast<const uint4*>(in + gr * ldi + gc);
    tile[row * 32 + slot(row, cc)] = v;
  }
  __syncthreads();
  const int rb = t & 7, cb = t >> 3;
  uint32_t w[8][4];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int row = rb * 8 + i;
    const uint4 v = tile[row * 32 + slot(row, cb)];
    w[i][0] = v.x; w[i][1] = v.y; w[i][2] = v.z; w[i][3] = v.w;
  }
  const int64_t orow0 = c0 + cb * 8, ocol = r0 + rb * 8;
  if (ocol >= R) return;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    if (orow0 + j >= C) break;
    uint32_t o[4];
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      const uint32_t lo = w[2 * d][j >> 1], hi = w[2 * d + 1][j >> 1];
      o[d] = (j & 1) ? ((lo >> 16) | (hi & 0xFFFF0000u)) : ((lo & 0xFFFFu) | (hi << 16));
    }
    *reinterpret_cast<uint4*>(out + (orow0 + j) * ldo + ocol) = make_uint4(o[0], o[1], o[2], o[3]);
  }
}

}  // namespace

hipError_t launch_transpose_bf16(const uint16_t* in, int64_t R, int64_t C, int64_t ldi,
                                 uint16_t* out, int64_t ldo, int64_t batch, int64_t ibs,
                                 int64_t obs, hipStream_t s) {
  if (R == 0 || C == 0 || batch == 0) return hipSuccess;
  const dim3 grid((unsigned)((C + TC - 1) / TC), (unsigned)((R + TR - 1) / TR), (unsigned)batch);
  hipLaunchKernelGGL(transpose_bf16_kernel, grid, dim3(NT), 0, s, in, R, C, ldi, out, ldo, ibs,
                     obs);
  return hipGetLastError();
}

}  // namespace qf
