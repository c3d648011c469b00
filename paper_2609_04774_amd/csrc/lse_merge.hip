// Exact log-sum-exp merge of partial attention outputs (HBM-bound).
//
// Partials over disjoint key sets S_i of the same (token, head) row combine
// into attention over their union because sum_{j in S} e^{x_j} =
// sum_i e^{LSE_i}:  LSE = M + ln sum_i e^{LSE_i - M} with M = max_i LSE_i,
// O = sum_i e^{LSE_i - LSE} O_i.  A partial with LSE_i = -inf weighs 0.
// Optionally each rank-local row is written to its place in the original
// sequence order (the restore step of paper Sec. 2.1).
//
// Layout: one (token, head) row of 128 fp32 is read by 32 lanes as float4
// (every partial's row is one fully coalesced 512-byte read); each 32-lane
// group merges two rows, a 256-thread block sixteen.
#include <hip/hip_runtime.h>

#include <cmath>

#include "internal.h"

namespace cpattn {

namespace {

constexpr int kRowsPerGroup = 2;                      // rows merged by one 32-lane group
constexpr int kRowsPerBlock = 8 * kRowsPerGroup;       // 256 threads = 8 groups
constexpr int kPartsInFlight = 4;                      // partials whose O loads are issued together

typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ inline uint32_t pack_bf16x2(float a, float b) {
  // Round-to-nearest-even conversion; gfx950 emits v_cvt_pk_bf16_f32.
  __bf16 x = (__bf16)a, y = (__bf16)b;
  return (uint32_t)__builtin_bit_cast(uint16_t, x) | ((uint32_t)__builtin_bit_cast(uint16_t, y) << 16);
}

// Each 32-lane group merges two rows: first every partial's LSE of both rows
// (so their latencies overlap), then the partial O rows that carry weight,
// all in flight together.  O is read and written with non-temporal hints:
// every byte is touched once, and streaming it past the caches measured
// about 20% faster than plain loads and stores on the 4-partial merge of the
// 32K shard.
__global__ __launch_bounds__(256) void lse_merge_kernel(MergeParams p) {
  const int lane = threadIdx.x & 31;
  const int64_t n_rows = p.n_tokens * p.n_heads;
  const int64_t row0 = (int64_t)blockIdx.x * kRowsPerBlock + kRowsPerGroup * (threadIdx.x >> 5);
  if (row0 >= n_rows) return;

  float l[kRowsPerGroup][CP_MAX_MERGE_PARTS];
#pragma unroll
  for (int i = 0; i < CP_MAX_MERGE_PARTS; ++i) {
    if (i < p.n_parts) {
#pragma unroll
      for (int r = 0; r < kRowsPerGroup; ++r) l[r][i] = row0 + r < n_rows ? p.lse[i][row0 + r] : -INFINITY;
    }
  }
  // Weights c = e^{LSE_i - M} / sum_k e^{LSE_k - M} (0 for a -inf partial and
  // for rows where every partial is -inf).
  float c[kRowsPerGroup][CP_MAX_MERGE_PARTS];
  float lse_out[kRowsPerGroup];
#pragma unroll
  for (int r = 0; r < kRowsPerGroup; ++r) {
    float m = -INFINITY;
#pragma unroll
    for (int i = 0; i < CP_MAX_MERGE_PARTS; ++i)
      if (i < p.n_parts) m = fmaxf(m, l[r][i]);
    float total = 0.f;
#pragma unroll
    for (int i = 0; i < CP_MAX_MERGE_PARTS; ++i) {
      if (i < p.n_parts) {
        c[r][i] = (m == -INFINITY || l[r][i] == -INFINITY) ? 0.f : expf(l[r][i] - m);
        total += c[r][i];
      }
    }
    lse_out[r] = -INFINITY;
    if (m != -INFINITY) {
      const float inv = 1.f / total;
      lse_out[r] = m + logf(total);
#pragma unroll
      for (int i = 0; i < CP_MAX_MERGE_PARTS; ++i)
        if (i < p.n_parts) c[r][i] *= inv;
    }
  }
  // Partials are taken kPartsInFlight at a time: all their O loads are
  // issued before any is used, so a lane has up to kPartsInFlight x
  // kRowsPerGroup 16-byte loads in flight.  The O of a partial of weight 0
  // (LSE = -inf) is not read.
  f32x4 acc[kRowsPerGroup];
#pragma unroll
  for (int r = 0; r < kRowsPerGroup; ++r) acc[r] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int i0 = 0; i0 < CP_MAX_MERGE_PARTS; i0 += kPartsInFlight) {
    if (i0 < p.n_parts) {
      f32x4 o[kPartsInFlight][kRowsPerGroup];
#pragma unroll
      for (int j = 0; j < kPartsInFlight; ++j) {
#pragma unroll
        for (int r = 0; r < kRowsPerGroup; ++r) {
          o[j][r] = f32x4{0.f, 0.f, 0.f, 0.f};
          if (i0 + j < p.n_parts && c[r][i0 + j] != 0.f)
            o[j][r] = __builtin_nontemporal_load(
                reinterpret_cast<const f32x4*>(p.o[i0 + j] + (row0 + r) * kHeadDim) + lane);
        }
      }
#pragma unroll
      for (int j = 0; j < kPartsInFlight; ++j) {
        if (i0 + j < p.n_parts) {
#pragma unroll
          for (int r = 0; r < kRowsPerGroup; ++r) acc[r] += c[r][i0 + j] * o[j][r];
        }
      }
    }
  }
#pragma unroll
  for (int r = 0; r < kRowsPerGroup; ++r) {
    const int64_t row = row0 + r;
    if (row >= n_rows) break;
    const int64_t tok = row / p.n_heads;
    const int head = (int)(row - tok * p.n_heads);
    int64_t dst_tok = tok;
    if (p.restore) dst_tok = (tok < p.first_len) ? p.first_dst + tok : p.second_dst + (tok - p.first_len);
    const int64_t dst = dst_tok * p.n_heads + head;
    if (p.out_bf16) {
      uint2 v;
      v.x = pack_bf16x2(acc[r][0], acc[r][1]);
      v.y = pack_bf16x2(acc[r][2], acc[r][3]);
      reinterpret_cast<uint2*>(static_cast<uint16_t*>(p.o_out) + dst * kHeadDim)[lane] = v;
    } else {
      __builtin_nontemporal_store(acc[r], reinterpret_cast<f32x4*>(static_cast<float*>(p.o_out) + dst * kHeadDim) + lane);
    }
    if (p.lse_out && lane == 0) p.lse_out[dst] = lse_out[r];
  }
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
