// Exact log-sum-exp merge of partial attention outputs (HBM-bound).
//
// Partials over disjoint key sets S_i of the same (token, head) row combine
// into attention over their union because sum_{j in S} e^{x_j} =
// sum_i e^{LSE_i}:  LSE = M + ln sum_i e^{LSE_i - M} with M = max_i LSE_i,
// O = sum_i e^{LSE_i - LSE} O_i.  A partial with LSE_i = -inf weighs 0.
// Optionally each rank-local row is written to its place in the original
// sequence order (the restore step of paper Sec. 2.1).
//
// Layout: one (token, head) row of 128 fp32 is read by 32 lanes as float4,
// so a wave64 merges two rows and a 256-thread block eight; every partial's
// row is one fully coalesced 512-byte read.
#include <hip/hip_runtime.h>

#include <cmath>

#include "internal.h"

namespace cpattn {

namespace {

constexpr int kRowsPerBlock = 8;

__device__ inline uint32_t pack_bf16x2(float a, float b) {
  // Round-to-nearest-even conversion; gfx950 emits v_cvt_pk_bf16_f32.
  __bf16 x = (__bf16)a, y = (__bf16)b;
  return (uint32_t)__builtin_bit_cast(uint16_t, x) | ((uint32_t)__builtin_bit_cast(uint16_t, y) << 16);
}

__global__ __launch_bounds__(256) void lse_merge_kernel(MergeParams p) {
  const int64_t row = (int64_t)blockIdx.x * kRowsPerBlock + (threadIdx.x >> 5);
  const int lane = threadIdx.x & 31;
  const int64_t n_rows = p.n_tokens * p.n_heads;
  if (row >= n_rows) return;
  const int64_t tok = row / p.n_heads;
  const int head = (int)(row - tok * p.n_heads);

  float l[CP_MAX_MERGE_PARTS];
  float m = -INFINITY;
#pragma unroll
  for (int i = 0; i < CP_MAX_MERGE_PARTS; ++i) {
    if (i < p.n_parts) {
      l[i] = p.lse[i][row];
      m = fmaxf(m, l[i]);
    }
  }
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  float lse_out = -INFINITY;
  if (m != -INFINITY) {
    float w[CP_MAX_MERGE_PARTS];
    float total = 0.f;
#pragma unroll
    for (int i = 0; i < CP_MAX_MERGE_PARTS; ++i) {
      if (i < p.n_parts) {
        w[i] = (l[i] == -INFINITY) ? 0.f : expf(l[i] - m);
        total += w[i];
      }
    }
    const float inv = 1.f / total;
    lse_out = m + logf(total);
#pragma unroll
    for (int i = 0; i < CP_MAX_MERGE_PARTS; ++i) {
      if (i < p.n_parts && w[i] != 0.f) {
        const float4 o = reinterpret_cast<const float4*>(p.o[i] + row * kHeadDim)[lane];
        const float c = w[i] * inv;
        acc.x += c * o.x;
        acc.y += c * o.y;
        acc.z += c * o.z;
        acc.w += c * o.w;
      }
    }
  }
  int64_t dst_tok = tok;
  if (p.restore) dst_tok = (tok < p.first_len) ? p.first_dst + tok : p.second_dst + (tok - p.first_len);
  const int64_t dst = dst_tok * p.n_heads + head;
  if (p.out_bf16) {
    uint2 v;
    v.x = pack_bf16x2(acc.x, acc.y);
    v.y = pack_bf16x2(acc.z, acc.w);
    reinterpret_cast<uint2*>(static_cast<uint16_t*>(p.o_out) + dst * kHeadDim)[lane] = v;
  } else {
    reinterpret_cast<float4*>(static_cast<float*>(p.o_out) + dst * kHeadDim)[lane] = acc;
  }
  if (p.lse_out && lane == 0) p.lse_out[dst] = lse_out;
}

}  // namespace

int launch_merge(const MergeParams& p, void* stream) {
  const int64_t n_rows = p.n_tokens * p.n_heads;
  if (n_rows == 0) return CP_OK;
  const int64_t blocks = (n_rows + kRowsPerBlock - 1) / kRowsPerBlock;
  if (blocks > 0x7fffffffLL) return fail(CP_ERR_UNSUPPORTED, "cp_attn_merge: too many rows for one launch");
  hipLaunchKernelGGL(lse_merge_kernel, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(CP_ERR_HIP, std::string("cp_attn_merge launch: ") + hipGetErrorString(e));
  return CP_OK;
}

}  // namespace cpattn
