// Engine-native export helpers (QATFactory Sec. 3.5 "Engine-native checkpoint export";
// Sec. 3.2.3 "Engine-specific scale sharing"): the NVFP4 scalars of a fused projection and the
// header of the weight-sync payload.  The codes and block scales come from the quantizer
// kernels, written straight into the caller's buffers (or into a payload's sections).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "qf.h"
#include "qf_internal.h"

namespace qf {
namespace {

// weight_scale_2 = g / 2688 (the tied tensor decode scale); input_scale = a / 2688 from the
// running activation amax (the decode scale the activation quantizer uses for that amax).
__global__ void export_scalars_kernel(const float* __restrict__ g, const float* __restrict__ a,
                                      float* __restrict__ ws2, float* __restrict__ is) {
  if (threadIdx.x != 0) return;
  if (ws2) *ws2 = *g / 2688.0f;
  if (is) *is = *a / 2688.0f;
}

// 64-byte payload header written with four 16-byte vector stores.
__global__ void payload_header_kernel(uint4* __restrict__ hdr, uint4 w0, uint4 w1, uint4 w2,
                                      uint4 w3) {
  const int t = threadIdx.x;
  if (t < 4) hdr[t] = t == 0 ? w0 : (t == 1 ? w1 : (t == 2 ? w2 : w3));
}

}  // namespace

hipError_t launch_export_scalars(const float* g, const float* a, float* ws2, float* is,
                                 hipStream_t s) {
  hipLaunchKernelGGL(export_scalars_kernel, dim3(1), dim3(64), 0, s, g, a, ws2, is);
  return hipGetLastError();
}

hipError_t launch_payload_header(void* payload, const uint32_t words[16], hipStream_t s) {
  const uint4 w0 = make_uint4(words[0], words[1], words[2], words[3]);
  const uint4 w1 = make_uint4(words[4], words[5], words[6], words[7]);
  const uint4 w2 = make_uint4(words[8], words[9], words[10], words[11]);
  const uint4 w3 = make_uint4(words[12], words[13], words[14], words[15]);
  hipLaunchKernelGGL(payload_header_kernel, dim3(1), dim3(64), 0, s,
                     reinterpret_cast<uint4*>(payload), w0, w1, w2, w3);
  return hipGetLastError();
}

}  // namespace qf
