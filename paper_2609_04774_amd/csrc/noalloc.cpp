// cp_attn_partial_noalloc: the partial attention for callers that cannot
// allocate (code under HIP graph capture, tight serving loops, harnesses that
// forbid allocation).  Same planning and kernels as cp_attn_partial; the
// device scratch -- the descriptor copy, the work list and the split-walk
// piece slots -- is a file-scope device array of the library instead of a
// caller workspace, and the tables go up by a plain copy from host memory
// instead of the pinned staging ring (which allocates on first use).
//
// Each GPU the library runs on holds its own copy of `scratch` until the
// process ends.  Host code never uses the array's name as an address: at a
// device's first call the address of that device's copy is fetched with
// hipGetSymbolAddress (with the device current) and kept per device, and
// that pointer is what the kernels receive.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <mutex>
#include <string>
#include <vector>

#include "internal.h"

using namespace cpattn;

namespace {

constexpr size_t kScratchBytes = CP_NOALLOC_SCRATCH_BYTES;

__device__ __attribute__((aligned(256))) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
unsigned char* g_scratch[kMaxDevices] = {};

// The current device's copy of `scratch` (fetched once per device).
int scratch_of_current_device(unsigned char** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(CP_ERR_HIP, std::string("cp_attn_partial_noalloc: hipGetDevice: ") +
                                                   hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices)
    return fail(CP_ERR_UNSUPPORTED, "cp_attn_partial_noalloc: device index beyond 63");
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(CP_ERR_HIP, std::string("cp_attn_partial_noalloc: hipGetSymbolAddress(scratch): ") +
                                  hipGetErrorString(e));
    g_scratch[dev] = static_cast<unsigned char*>(p);
  }
  *out = g_scratch[dev];
  return CP_OK;
}

}  // namespace

extern "C" int cp_attn_partial_noalloc(const cp_partial_desc* descs, int32_t n_descs, int32_t n_heads_q,
                                       int32_t n_heads_kv, int32_t head_dim, float softmax_scale, void* stream) {
  return guarded([&]() -> int {
    const char* who = "cp_attn_partial_noalloc";
    if (head_dim != CP_HEAD_DIM) return fail(CP_ERR_UNSUPPORTED, std::string(who) + ": head_dim must be 128");
    if (!(softmax_scale == softmax_scale)) return fail(CP_ERR_INVALID, std::string(who) + ": softmax_scale is NaN");
    // Plan as cp_attn_partial does; when the split-walk pieces would not fit
    // in the scratch, plan fewer (down to none): the result is the same
    // attention, only the work decomposition differs.
    Plan plan;
    Layout lay;
    int64_t target = kTargetPieces;
    for (;;) {
      const int st = build_plan(descs, n_descs, n_heads_q, n_heads_kv, target, &plan);
      if (st != CP_OK) return st;
      lay = layout_of(plan);
      if (lay.total <= kScratchBytes || plan.n_pieces == 0) break;
      target = target >= 4 ? target / 2 : 0;
    }
    if (plan.items.empty()) {
      clear_error();
      return CP_OK;
    }
    if (lay.total > kScratchBytes)
      return fail(CP_ERR_CAPACITY, std::string(who) + ": the launch's tables need " + std::to_string(lay.total) +
                                       " bytes, beyond the " + std::to_string(kScratchBytes) +
                                       "-byte scratch (use cp_attn_partial with a workspace)");
    unsigned char* ws = nullptr;
    int st = scratch_of_current_device(&ws);
    if (st != CP_OK) return st;
    std::vector<unsigned char> host;
    pack_tables(plan, lay, &host);
    // The scratch is shared by every call on this GPU: wait until the stream's
    // earlier work (an earlier call's kernels among it) is done before
    // overwriting the tables, then copy them from pageable host memory (a
    // synchronous copy in HIP).  Every piece slot is written by the kernel
    // before it is read, so nothing needs clearing.
    hipError_t e = hipStreamSynchronize((hipStream_t)stream);
    if (e != hipSuccess) return fail(CP_ERR_HIP, std::string(who) + ": hipStreamSynchronize: " + hipGetErrorString(e));
    e = hipMemcpyAsync(ws, host.data(), lay.pieces, hipMemcpyHostToDevice, (hipStream_t)stream);
    if (e != hipSuccess) return fail(CP_ERR_HIP, std::string(who) + ": hipMemcpyAsync (tables): " + hipGetErrorString(e));
    const float scale = softmax_scale > 0.f ? softmax_scale : 1.f / std::sqrt((float)head_dim);
    st = launch_partial(partial_params(plan, lay, ws, n_heads_q, n_heads_kv, scale), stream);
    if (st == CP_OK) clear_error();
    return st;
  });
}
