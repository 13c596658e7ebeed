// Workspace header of an empty batch: with B = 0 no decode kernel runs, so
// this one-thread kernel records B = 0 for ctcbeam_query_status.
#include "ctcbeam_internal.h"

namespace ctcbeam {
namespace {
__global__ void ws_header_kernel(uint32_t* hdr, int B) {
  if (threadIdx.x == 0) write_ws_header(hdr, B);
}
}  // namespace

hipError_t launch_ws_header(uint32_t* hdr, int B, hipStream_t stream) {
  hipLaunchKernelGGL(ws_header_kernel, dim3(1), dim3(64), 0, stream, hdr, B);
  return hipGetLastError();
}
}  // namespace ctcbeam
