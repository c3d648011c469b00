// KV-cache steps around the attention, all pure row copies (HBM-bound):
//
//  * Paged write-back (paper Sec. 2.2, 7.1, 8): a CP rank's new K/V rows go
//    to their token positions in the block-16 paged cache, position p at
//    physical block block_table[p / 16], slot p % 16.
//  * Re-sharding between CP degrees (Sec. 6.2, 7.2): each row of a
//    destination rank is fetched from the source rank that holds the same
//    global position under the source degree.
//  * Paged gather (Sec. 2.2, 7.1, 7.2): positions of a request read back out
//    of the paged cache into contiguous rows.
//
// A workgroup takes 4 rows, one wave per row; each lane moves
// 16-byte pieces with plain vector loads and stores, so a row's bytes are
// read and written in fully coalesced 1 KiB wavefront accesses.  Row indices are derived in
// closed form from the zigzag plans; no index table is read except the
// block table.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace cpattn {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kRowsPerGroup = 4;  // rows copied by one workgroup, one wave per row

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// One wave copies one row: lane l moves 16-byte pieces l, l+64, ...; four
// loads are in flight before their stores.
__device__ __forceinline__ void copy_row(const unsigned char* __restrict__ src, unsigned char* __restrict__ dst,
                                         int64_t row_bytes, int lane) {
  const int64_t n = row_bytes >> 4;
  const u32x4* s = reinterpret_cast<const u32x4*>(src);
  u32x4* d = reinterpret_cast<u32x4*>(dst);
  int64_t i = lane;
  for (; i + 192 < n; i += 256) {
    const u32x4 a = s[i], b = s[i + 64], c = s[i + 128], e = s[i + 192];
    d[i] = a;
    d[i + 64] = b;
    d[i + 128] = c;
    d[i + 192] = e;
  }
  for (; i < n; i += 64) d[i] = s[i];
}

// Global position of a rank's local row t: chunk 0's rows, then chunk 1's.
__device__ __forceinline__ int64_t row_position(const int64_t (&q_begin)[2], const int64_t (&q_len)[2], int64_t t) {
  return t < q_len[0] ? q_begin[0] + t : q_begin[1] + (t - q_len[0]);
}

__global__ __launch_bounds__(kThreads) void kv_writeback_kernel(WritebackParams p) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int k = wave; k < kRowsPerGroup; k += kWaves) {
    const int64_t t = (int64_t)blockIdx.x * kRowsPerGroup + k;
    if (t >= p.n_rows) break;
    const int64_t pos = row_position(p.q_begin, p.q_len, t);
    const int64_t blk = p.block_table[pos / kBlockTokens];
    if (blk < 0 || blk >= p.n_blocks) continue;  // outside the cache: nothing is written
    const int64_t dst = (blk * kBlockTokens + pos % kBlockTokens) * p.row_bytes;
    copy_row(p.k_rows + t * p.row_bytes, p.k_cache + dst, p.row_bytes, lane);
    copy_row(p.v_rows + t * p.row_bytes, p.v_cache + dst, p.row_bytes, lane);
  }
}

__global__ __launch_bounds__(kThreads) void repartition_kernel(RepartitionParams p) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int k = wave; k < kRowsPerGroup; k += kWaves) {
    const int64_t t = (int64_t)blockIdx.x * kRowsPerGroup + k;
    if (t >= p.n_rows) break;
    // Source rank of the row's global position: suffix chunk c at the source
    // degree belongs to rank c (c < C) or 2C-1-c; its local row follows that
    // rank's first chunk when c is its second chunk.
    const int64_t i = row_position(p.dst_q_begin, p.dst_q_len, t) - p.P;
    const int64_t c = i / p.s_src;
    const int64_t C = p.C_src;
    const int64_t r = c < C ? c : 2 * C - 1 - c;
    int64_t local = i - c * p.s_src;
    if (c != r) {
      const int64_t first = p.R - r * p.s_src;  // rows of rank r's first chunk
      local += first < 0 ? 0 : (first > p.s_src ? p.s_src : first);
    }
    copy_row(p.src[r] + local * p.row_bytes, p.dst + t * p.row_bytes, p.row_bytes, lane);
  }
}

// Where suffix index i sits at degree C with chunk length s: the rank holding
// its chunk c (rank c or 2C-1-c) and the local row there (after that rank's
// first chunk when c is its second).
struct RankRow {
  int64_t rank, row;
};

__device__ __forceinline__ RankRow rank_row(int64_t i, int64_t C, int64_t s, int64_t R) {
  const int64_t c = i / s;
  const int64_t r = c < C ? c : 2 * C - 1 - c;
  int64_t local = i - c * s;
  if (c != r) {
    const int64_t first = R - r * s;  // rows of rank r's first chunk
    local += first < 0 ? 0 : (first > s ? s : first);
  }
  return RankRow{r, local};
}

// One wave per (set, suffix index): the row moves from its source rank to its
// destination rank.
__global__ __launch_bounds__(kThreads) void repartition_all_kernel(RepartitionAllParams p) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int k = wave; k < kRowsPerGroup; k += kWaves) {
    const int64_t t = (int64_t)blockIdx.x * kRowsPerGroup + k;
    if (t >= p.n_sets * p.R) break;
    const int set = t >= p.R ? 1 : 0;
    const int64_t i = t - set * p.R;
    const RankRow from = rank_row(i, p.C_src, p.s_src, p.R);
    const RankRow to = rank_row(i, p.C_dst, p.s_dst, p.R);
    copy_row(p.src[set][from.rank] + from.row * p.row_bytes, p.dst[set][to.rank] + to.row * p.row_bytes,
             p.row_bytes, lane);
  }
}

// One wave gathers one row of K and one of V out of the paged cache: per
// round, up to four 16-byte pieces of each (lane l takes pieces l, l+64, ...)
// are loaded before any is stored, with non-temporal hints (every byte is
// moved once).  A NULL source (a block-table entry outside the cache) writes
// zeros.
__device__ __forceinline__ void gather_row_pair(const unsigned char* ks, const unsigned char* vs,
                                                unsigned char* kd, unsigned char* vd, int64_t row_bytes,
                                                int lane) {
  const int64_t n = row_bytes >> 4;
  for (int64_t base = 0; base < n; base += 4 * 64) {
    u32x4 kv[4], vv[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int64_t i = base + lane + 64 * k;
      kv[k] = vv[k] = u32x4{0u, 0u, 0u, 0u};
      if (i < n && ks) {
        kv[k] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(ks) + i);
        vv[k] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(vs) + i);
      }
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int64_t i = base + lane + 64 * k;
      if (i < n) {
        __builtin_nontemporal_store(kv[k], reinterpret_cast<u32x4*>(kd) + i);
        __builtin_nontemporal_store(vv[k], reinterpret_cast<u32x4*>(vd) + i);
      }
    }
  }
}

__global__ __launch_bounds__(kThreads) void kv_gather_kernel(GatherParams p) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int k = wave; k < kRowsPerGroup; k += kWaves) {
    const int64_t t = (int64_t)blockIdx.x * kRowsPerGroup + k;
    if (t >= p.n_rows) break;
    const int64_t pos = p.pos_begin + t;
    const int64_t blk = p.block_table[pos / kBlockTokens];
    const bool inside = blk >= 0 && blk < p.n_blocks;
    const int64_t src = (blk * kBlockTokens + pos % kBlockTokens) * p.row_bytes;
    gather_row_pair(inside ? p.k_cache + src : nullptr, inside ? p.v_cache + src : nullptr,
                    p.k_rows + t * p.row_bytes, p.v_rows + t * p.row_bytes, p.row_bytes, lane);
  }
}

}  // namespace

int launch_repartition_all(const RepartitionAllParams& p, void* stream) {
  const int64_t rows = p.n_sets * p.R;
  if (rows == 0) return CP_OK;
  const int64_t groups = (rows + kRowsPerGroup - 1) / kRowsPerGroup;
  hipLaunchKernelGGL(repartition_all_kernel, dim3((unsigned)groups), dim3(kThreads), 0, (hipStream_t)stream, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(CP_ERR_HIP, std::string("cp_repartition_all launch: ") + hipGetErrorString(e));
  return CP_OK;
}

int launch_gather(const GatherParams& p, void* stream) {
  if (p.n_rows == 0) return CP_OK;
  const int64_t groups = (p.n_rows + kRowsPerGroup - 1) / kRowsPerGroup;
  hipLaunchKernelGGL(kv_gather_kernel, dim3((unsigned)groups), dim3(kThreads), 0, (hipStream_t)stream, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(CP_ERR_HIP, std::string("cp_kv_gather launch: ") + hipGetErrorString(e));
  return CP_OK;
}

int launch_writeback(const WritebackParams& p, void* stream) {
  if (p.n_rows == 0) return CP_OK;
  const int64_t groups = (p.n_rows + kRowsPerGroup - 1) / kRowsPerGroup;
  hipLaunchKernelGGL(kv_writeback_kernel, dim3((unsigned)groups), dim3(kThreads), 0, (hipStream_t)stream, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(CP_ERR_HIP, std::string("cp_kv_writeback launch: ") + hipGetErrorString(e));
  return CP_OK;
}

int launch_repartition(const RepartitionParams& p, void* stream) {
  if (p.n_rows == 0) return CP_OK;
  const int64_t groups = (p.n_rows + kRowsPerGroup - 1) / kRowsPerGroup;
  hipLaunchKernelGGL(repartition_kernel, dim3((unsigned)groups), dim3(kThreads), 0, (hipStream_t)stream, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(CP_ERR_HIP, std::string("cp_repartition launch: ") + hipGetErrorString(e));
  return CP_OK;
}

}  // namespace cpattn
