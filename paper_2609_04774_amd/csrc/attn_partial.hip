// Partial causal attention of one CP rank's zigzag rows, bf16 MFMA on gfx950.
//
// What is computed (paper Sec. 2.1 / 2.2): for every query row at global
// position p and head h, over the keys j of the descriptor's key set with
// j <= p:  x_j = scale * q.k_j,  LSE = ln sum_j e^{x_j},
// O = sum_j e^{x_j - LSE} v_j, with grouped KV head h / (Hq/Hkv).
//
// How (FlashAttention-2 style online softmax, Dao 2023, with the running
// max/sum recurrence of Milakov & Gimelshein 2018):
//   * A workgroup (4 wave64s) owns 256 (query, head) rows that share one KV
//     head: `heads_per_wg` query heads x `q_per_wg` consecutive positions, so
//     every K/V tile staged in LDS is reused by all of them.  Each wave owns
//     two blocks of 32 rows.
//   * Keys are visited in tiles of 64 along each key range (paged prefix,
//     then the suffix ranges).  Tiles past the workgroup's last query are
//     never visited; only tiles that cross the diagonal or a range end are
//     masked.
//   * Scores are computed transposed, S^T = K Q^T, with
//     v_mfma_f32_32x32x16_bf16: a lane then holds one query's column, so the
//     row max and row sum are in-lane plus one exchange with lane ^ 32, and
//     the probabilities feed O^T += V^T P^T directly from registers.  V^T
//     fragments come from the row-major V tile through ds_read_b64_tr_b16.
//   * LDS rows are 256 bytes; 16-byte chunks are XOR-swizzled by the row so
//     that both the K reads (8 rows, one chunk) and the transposed V reads
//     (4 rows, two chunks) hit distinct banks.
#include <hip/hip_runtime.h>

#include <cmath>

#include "internal.h"

namespace cpattn {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kTileKeys = 64;
constexpr int kRowBytes = kHeadDim * 2;
constexpr int kTileBytes = kTileKeys * kRowBytes;

__device__ __forceinline__ int swz(int key) { return ((key & 3) << 1) | ((key >> 2) & 1); }
__device__ __forceinline__ int lds_off(int key, int chunk) {
  return key * kRowBytes + ((chunk ^ swz(key)) << 4);
}

__device__ __forceinline__ s16x4 ds_read_tr16(const unsigned char* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(p));
}

__global__ __launch_bounds__(kThreads, 1) void attn_partial_kernel(PartialParams p) {
  __shared__ __attribute__((aligned(16))) unsigned char smem[2 * kTileBytes];
  unsigned char* const sk = smem;
  unsigned char* const sv = smem + kTileBytes;

  const WorkItem it = p.items[blockIdx.x];
  const DevDesc& d = p.descs[it.desc];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int half = lane >> 5;
  const int l32 = lane & 31;

  const int64_t q_begin = d.q_begin[it.chunk];
  const int64_t q_len = d.q_len[it.chunk];
  const int64_t loff = d.local_off[it.chunk];
  const int Hq = p.Hq;
  const int Hkv = p.Hkv;
  const int kvh = it.head_group / p.groups_per_kv;
  const int head0 = kvh * (Hq / Hkv) + (it.head_group % p.groups_per_kv) * p.heads_per_wg;
  const int qblocks_per_head = p.q_per_wg >> 5;
  const int64_t qb0 = (int64_t)it.q_block * p.q_per_wg;
  const int64_t wg_last = (qb0 + p.q_per_wg < q_len ? qb0 + p.q_per_wg : q_len) - 1;
  const int64_t wg_pos_hi = q_begin + wg_last;

  int head_b[2];
  int64_t qidx_b[2];
  int64_t pos_b[2];
  bool valid_b[2];
  int64_t wave_lo = INT64_MAX, wave_hi = -1;
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    const int bi = 2 * wave + b;
    head_b[b] = head0 + bi / qblocks_per_head;
    const int qo = (bi % qblocks_per_head) * 32;
    qidx_b[b] = qb0 + qo + l32;
    valid_b[b] = qidx_b[b] < q_len;
    pos_b[b] = valid_b[b] ? q_begin + qidx_b[b] : -1;
    const int64_t blo = qb0 + qo, bhi = (qb0 + qo + 31 < wg_last ? qb0 + qo + 31 : wg_last);
    if (blo <= wg_last) {
      wave_lo = (q_begin + blo < wave_lo) ? q_begin + blo : wave_lo;
      wave_hi = (q_begin + bhi > wave_hi) ? q_begin + bhi : wave_hi;
    }
  }
  const bool wave_active = wave_hi >= 0;

  // Query fragments (B operand of S^T = K Q^T): lane holds 8 consecutive
  // head-dim values of its query, for each of the 8 steps of 16 along D.
  bf16x8 qf[2][8];
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    const uint16_t* qrow = d.q + ((loff + qidx_b[b]) * Hq + head_b[b]) * kHeadDim + half * 8;
#pragma unroll
    for (int ds = 0; ds < 8; ++ds) {
      if (valid_b[b]) {
        qf[b][ds] = *reinterpret_cast<const bf16x8*>(qrow + ds * 16);
      } else {
        qf[b][ds] = bf16x8{};
      }
    }
  }

  f32x16 o[4][2];
#pragma unroll
  for (int db = 0; db < 4; ++db)
#pragma unroll
    for (int b = 0; b < 2; ++b) o[db][b] = f32x16{};
  float m_run[2] = {-INFINITY, -INFINITY};
  float l_run[2] = {0.f, 0.f};
  const float sl2 = p.scale_log2;

  for (int seg = 0; seg <= d.n_seg; ++seg) {
    int64_t lo, hi;
    const bool paged = (seg == 0);
    if (paged) {
      lo = 0;
      hi = d.prefix_keys;
    } else {
      lo = d.seg_lo[seg - 1];
      hi = d.seg_hi[seg - 1];
    }
    const int64_t hi_vis = (hi < wg_pos_hi + 1) ? hi : wg_pos_hi + 1;
    const uint16_t* kbase = paged ? d.k_cache : d.k_new;
    const uint16_t* vbase = paged ? d.v_cache : d.v_new;
    for (int64_t t0 = lo; t0 < hi_vis; t0 += kTileKeys) {
      // Stage K and V tiles: 64 keys x 16 chunks of 16 bytes each; zero rows
      // past the visible end so no memory outside the key range is read.
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int idx = tid + kThreads * i;
        const int key = idx >> 4;
        const int c = idx & 15;
        const int64_t pos = t0 + key;
        u32x4 kv = u32x4{0u, 0u, 0u, 0u};
        u32x4 vv = u32x4{0u, 0u, 0u, 0u};
        if (pos < hi_vis) {
          int64_t row;
          if (paged) {
            const int64_t blk = d.block_table[pos >> 4];
            row = (blk * kBlockTokens + (pos & (kBlockTokens - 1))) * Hkv + kvh;
          } else {
            row = (pos - d.P) * Hkv + kvh;
          }
          kv = *reinterpret_cast<const u32x4*>(kbase + row * kHeadDim + c * 8);
          vv = *reinterpret_cast<const u32x4*>(vbase + row * kHeadDim + c * 8);
        }
        *reinterpret_cast<u32x4*>(sk + lds_off(key, c)) = kv;
        *reinterpret_cast<u32x4*>(sv + lds_off(key, c)) = vv;
      }
      __syncthreads();

      if (wave_active && t0 <= wave_hi) {
        const bool need_mask = (t0 + kTileKeys > hi) || (t0 + kTileKeys - 1 > wave_lo);
        f32x16 s[2][2];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int b = 0; b < 2; ++b) s[kb][b] = f32x16{};
#pragma unroll
        for (int ds = 0; ds < 8; ++ds) {
#pragma unroll
          for (int kb = 0; kb < 2; ++kb) {
            const bf16x8 kf = *reinterpret_cast<const bf16x8*>(sk + lds_off(kb * 32 + l32, 2 * ds + half));
#pragma unroll
            for (int b = 0; b < 2; ++b)
              s[kb][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[b][ds], s[kb][b], 0, 0, 0);
          }
        }
        if (need_mask) {
#pragma unroll
          for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              const int64_t kp = t0 + kb * 32 + (r >> 2) * 8 + half * 4 + (r & 3);
#pragma unroll
              for (int b = 0; b < 2; ++b)
                if (kp >= hi || kp > pos_b[b]) s[kb][b][r] = -INFINITY;
            }
        }
        // Online softmax per query column; the two lane halves hold disjoint
        // keys of the same query and agree on the running max.
#pragma unroll
        for (int b = 0; b < 2; ++b) {
          float mx = -INFINITY;
#pragma unroll
          for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kb][b][r]);
          mx = fmaxf(mx, __shfl_xor(mx, 32));
          const float m_new = fmaxf(m_run[b], mx);
          const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
          const float alpha = __builtin_amdgcn_exp2f((m_run[b] - m_use) * sl2);
          m_run[b] = m_new;
          const float neg = -m_use * sl2;
          float rs = 0.f;
#pragma unroll
          for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              const float e = __builtin_amdgcn_exp2f(__builtin_fmaf(s[kb][b][r], sl2, neg));
              s[kb][b][r] = e;
              rs += e;
            }
          l_run[b] = l_run[b] * alpha + rs;
#pragma unroll
          for (int db = 0; db < 4; ++db) o[db][b] *= alpha;
        }
        // P^T fragments: k-step ks covers keys 16ks..16ks+15 of the tile; slot
        // t of lane half h is key 16ks + (t/4)*8 + 4h + t%4, which is exactly
        // accumulator register 8*(ks%2) + t of key block ks/2.
        bf16x8 pf[2][4];
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
          for (int ks = 0; ks < 4; ++ks)
#pragma unroll
            for (int t = 0; t < 8; ++t) pf[b][ks][t] = (__bf16)s[ks >> 1][b][8 * (ks & 1) + t];
        // O^T += V^T P^T.  The transposed read gives lane (group g, index i)
        // the four keys kbase..kbase+3 of column d0 + i, where the group's 16
        // lanes read rows kbase + i/4 at columns d0 + 4*(i%4).
        const int grp = lane >> 4;
        const int gi = lane & 15;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
          const int row1 = ks * 16 + half * 4 + (gi >> 2);
          const int row2 = row1 + 8;
#pragma unroll
          for (int db = 0; db < 4; ++db) {
            const int dcol = db * 32 + (grp & 1) * 16 + 4 * (gi & 3);
            const int c = dcol >> 3;
            const int e = (dcol & 7) * 2;
            const s16x4 lo4 = ds_read_tr16(sv + row1 * kRowBytes + ((c ^ swz(row1)) << 4) + e);
            const s16x4 hi4 = ds_read_tr16(sv + row2 * kRowBytes + ((c ^ swz(row2)) << 4) + e);
            const s16x8 v8 = __builtin_shufflevector(lo4, hi4, 0, 1, 2, 3, 4, 5, 6, 7);
            const bf16x8 vf = __builtin_bit_cast(bf16x8, v8);
#pragma unroll
            for (int b = 0; b < 2; ++b)
              o[db][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[b][ks], o[db][b], 0, 0, 0);
          }
        }
      }
      __syncthreads();
    }
  }

  // Normalise and store: O^T register r of d-block db is head-dim
  // db*32 + (r/4)*8 + 4*half + r%4 of this lane's query.
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    const float lt = l_run[b] + __shfl_xor(l_run[b], 32);
    const bool live = (m_run[b] != -INFINITY) && (lt > 0.f);
    const float inv = live ? 1.f / lt : 0.f;
    if (valid_b[b]) {
      float* orow = d.o + ((loff + qidx_b[b]) * Hq + head_b[b]) * kHeadDim;
#pragma unroll
      for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          float4 v;
          v.x = o[db][b][4 * q4 + 0] * inv;
          v.y = o[db][b][4 * q4 + 1] * inv;
          v.z = o[db][b][4 * q4 + 2] * inv;
          v.w = o[db][b][4 * q4 + 3] * inv;
          *reinterpret_cast<float4*>(orow + db * 32 + q4 * 8 + half * 4) = v;
        }
      if (half == 0) d.lse[(loff + qidx_b[b]) * Hq + head_b[b]] = live ? m_run[b] * p.scale + logf(lt) : -INFINITY;
    }
  }
}

}  // namespace

int launch_partial(const PartialParams& p, void* stream) {
  if (p.n_items == 0) return CP_OK;
  hipLaunchKernelGGL(attn_partial_kernel, dim3((unsigned)p.n_items), dim3(kThreads), 0, (hipStream_t)stream, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(CP_ERR_HIP, std::string("cp_attn_partial launch: ") + hipGetErrorString(e));
  return CP_OK;
}

}  // namespace cpattn
