// Header writer of a saved pipeline state (the ring a pipelined step depends
// on, Sec. VI-A: every worker keeps the latest gradient of each partition it
// holds).  The header travels as a kernel argument, so saving needs no host
// buffer that outlives the call and stays asynchronous on the caller's stream.
#include <hip/hip_runtime.h>

#include "pgc_kernels.h"

namespace pgc {
namespace {

constexpr int kHeaderWords = static_cast<int>(kStateHeaderBytes / 8);

__global__ __launch_bounds__(kHeaderWords)
void write_state_header_kernel(StateHeader h, uint64_t* out) {
  const int i = threadIdx.x;
  const uint64_t* src = reinterpret_cast<const uint64_t*>(&h);
  out[i] = i < static_cast<int>(sizeof(StateHeader) / 8) ? src[i] : 0;
}

}  // namespace

hipError_t launch_write_state_header(const StateHeader& h, void* out, hipStream_t s) {
  hipLaunchKernelGGL(write_state_header_kernel, dim3(1), dim3(kHeaderWords), 0, s, h,
                     static_cast<uint64_t*>(out));
  return hipGetLastError();
}

}  // namespace pgc
