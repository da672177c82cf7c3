// Device-side tables for the grouped (mixture-of-experts) layer: per-expert tile prefixes and
// expert orders, computed from the device row offsets so the host never reads them.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "qf_internal.h"

namespace qf {
namespace {

constexpr int BM = 256;   // row tile of the NT GEMM's grouped-rows mode

__global__ void grouped_prep_kernel(const int64_t* __restrict__ off, int E, int* tile_start,
                                    int* order, int* kstart) {
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
  }
}

}  // namespace

hipError_t launch_grouped_prep(const int64_t* off, int64_t E, int* tile_start, int* order,
                               int* kstart, hipStream_t s) {
  hipLaunchKernelGGL(grouped_prep_kernel, dim3(1), dim3(1024), 0, s, off, (int)E, tile_start,
                     order, kstart);
  return hipGetLastError();
}

}  // namespace qf
