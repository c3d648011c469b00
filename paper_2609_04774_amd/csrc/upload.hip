// The launch tables' upload.  Each cp_attn_partial call copies its
// descriptors, work list and split list (a few KB to a few hundred KB) from
// the library's pinned host staging into the caller's workspace.  A copy
// engine transfer (hipMemcpyAsync) makes the compute queue wait for the copy
// engine's completion signal before the attention kernel starts, about 17 us
// per call on this GPU; a kernel on the same stream reads the staging over
// the bus instead and hands over like any two kernels do (about 7 us in
// all).  16 bytes per thread.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace cpattn {

namespace {

__global__ __launch_bounds__(256) void upload_tables_kernel(uint4* __restrict__ dst, const uint4* __restrict__ src,
                                                            size_t n16) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n16) dst[i] = src[i];
}

}  // namespace

int launch_upload(void* dst, const void* src, size_t bytes, void* stream) {
  if (bytes == 0) return CP_OK;
  if (bytes % 16 || (uintptr_t)dst % 16 || (uintptr_t)src % 16)
    return fail(CP_ERR_INVALID, "table upload: sizes and addresses must be multiples of 16 bytes");
  const size_t n16 = bytes / 16;
  hipLaunchKernelGGL(upload_tables_kernel, dim3((unsigned)((n16 + 255) / 256)), dim3(256), 0, (hipStream_t)stream,
                     static_cast<uint4*>(dst), static_cast<const uint4*>(src), n16);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(CP_ERR_HIP, std::string("table upload launch: ") + hipGetErrorString(e));
  return CP_OK;
}

}  // namespace cpattn
