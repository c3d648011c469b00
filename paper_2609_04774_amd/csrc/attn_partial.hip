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
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kTileKeys = 64;
constexpr bf16x2 kOnes = {(__bf16)1.0f, (__bf16)1.0f};
constexpr int kRowBytes = kHeadDim * 2;
constexpr int kTileBytes = kTileKeys * kRowBytes;

// 16-byte chunk swizzle of a 256-byte LDS row (64 banks x 4 bytes on gfx950):
// rows 0..15 get 16 distinct XOR masks, and any 4 rows r0..r0+3 (r0 % 4 == 0)
// differ in mask bits 2-3 -- so the 16-row K reads and the 4-row x 4-chunk
// transposed V reads each touch every bank once.
__device__ __forceinline__ int swz(int key) { return ((key & 3) << 2) | ((key >> 2) & 3); }
__device__ __forceinline__ int lds_off(int key, int chunk) {
  return key * kRowBytes + ((chunk ^ swz(key)) << 4);
}

__device__ __forceinline__ s16x4 ds_read_tr16(const unsigned char* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(p));
}

// Key ranges of one work item: the paged prefix (if read) and up to two
// suffix ranges, each clipped to the workgroup's last query position.  At
// most three; selected by a wave-uniform index.
struct Ranges {
  int64_t lo[3], hi[3], vis[3];
  int paged0;  // range 0 is the paged prefix
  int n;
};

struct Cursor {
  int r;       // range index
  int64_t t0;  // first key position of the tile
};

__device__ __forceinline__ int64_t sel3(const int64_t (&a)[3], int i) { return i == 0 ? a[0] : (i == 1 ? a[1] : a[2]); }

__device__ __forceinline__ void advance(Cursor& c, const Ranges& rg) {
  c.t0 += kTileKeys;
  if (c.t0 >= sel3(rg.vis, c.r)) {
    ++c.r;
    c.t0 = sel3(rg.lo, c.r);
  }
}

// One global_load_lds_dwordx4: lane l's 16 bytes at sbase + voff land at LDS
// byte m0 + 16*l.  Issued as inline assembly so the compiler does not treat
// every later LDS read as depending on it (it cannot tell the two buffers
// apart); the kernel waits for these loads itself (vmcnt) before the barrier
// that publishes a tile.
__device__ __forceinline__ void dma16(const void* sbase, uint32_t voff, uint32_t lds_base) {
  asm volatile(
      "s_mov_b32 m0, %0\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, %2\n\t" ::"s"(lds_base),
      "v"(voff), "s"(sbase)
      : "memory", "m0");
}

__device__ __forceinline__ uint32_t lds_addr(const unsigned char* p) {
  return (uint32_t)(uintptr_t)((const __attribute__((address_space(3))) unsigned char*)p);
}

// Issues this wave's share of one K/V tile straight into LDS.  Wave w fills
// tile rows RPW*w .. RPW*w + RPW-1; lane l of load i carries row
// RPW*w + 4i + l/16, physical chunk l%16, i.e. logical chunk (l%16) ^ swz(row).
// The address is a wave-uniform base (tile start, KV head) plus a per-lane
// offset `lane_off[i]` = row_in_tile * row_stride + 16 * logical chunk.  Rows
// past the visible end read a clamped, in-range row; those keys are masked
// in the scores.
template <int RPW>
__device__ __forceinline__ void issue_tile(const Cursor& c, const Ranges& rg, const DevDesc& d, int kvh,
                                           int row_stride, int wave, const uint32_t (&lane_off)[RPW / 4],
                                           const int (&lane_row)[RPW / 4], uint32_t sk, uint32_t sv) {
  const int64_t vis = sel3(rg.vis, c.r);
  const bool paged = (c.r == 0) && rg.paged0;
  const int row0 = wave * RPW;
  const unsigned char* kb;
  const unsigned char* vb;
  int clamp_row = 1 << 30;  // last readable row of this tile, relative to its first row
  if (paged) {
    // Prefix tiles start at multiples of 64 keys, so this wave's rows lie in
    // logical cache block t0/16 + row0/16 (clamped to the last block); the
    // lane offsets use the row within the tile, so step back by the block's
    // first tile row.
    int64_t lb = (c.t0 >> 4) + (row0 >> 4);
    const int64_t last = ((vis + kBlockTokens - 1) >> 4) - 1;
    lb = lb < last ? lb : last;
    const int64_t blk =
        __builtin_amdgcn_readfirstlane(((const __attribute__((address_space(1))) int32_t*)d.block_table)[lb]);
    const int64_t base = (blk * kBlockTokens - (row0 & ~(kBlockTokens - 1))) * row_stride + kvh * (kHeadDim * 2);
    kb = reinterpret_cast<const unsigned char*>(d.k_cache) + base;
    vb = reinterpret_cast<const unsigned char*>(d.v_cache) + base;
  } else {
    const int64_t base = (c.t0 - d.P) * row_stride + kvh * (kHeadDim * 2);
    kb = reinterpret_cast<const unsigned char*>(d.k_new) + base;
    vb = reinterpret_cast<const unsigned char*>(d.v_new) + base;
    if (c.t0 + kTileKeys > vis) clamp_row = (int)(vis - 1 - c.t0);
  }
#pragma unroll
  for (int i = 0; i < RPW / 4; ++i) {
    uint32_t off = lane_off[i];
    if (lane_row[i] > clamp_row) off = off - (uint32_t)((lane_row[i] - clamp_row) * row_stride);
    const uint32_t lrow = (uint32_t)((row0 + 4 * i) * kRowBytes);
    dma16(kb, off, sk + lrow);
    dma16(vb, off, sv + lrow);
  }
}

// Clamps a wave-uniform offset to a range where 32-bit arithmetic with a
// lane's query index (< 2^16) cannot overflow; results are clamped to a tile.
__device__ __forceinline__ int clamp_i32(int64_t x) {
  return (int)(x < -(1 << 24) ? -(1 << 24) : (x > (1 << 24) ? (1 << 24) : x));
}

__device__ __forceinline__ float xmax32(float x) {
  // Max with the lane 32 apart (the other half of the same query's keys).
  auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(unsigned, x), __builtin_bit_cast(unsigned, x),
                                            false, false);
  return __builtin_fmaxf(__builtin_bit_cast(float, (unsigned)r[0]), __builtin_bit_cast(float, (unsigned)r[1]));
}

__device__ __forceinline__ float xsum32(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(unsigned, x), __builtin_bit_cast(unsigned, x),
                                            false, false);
  return __builtin_bit_cast(float, (unsigned)r[0]) + __builtin_bit_cast(float, (unsigned)r[1]);
}

// Running max is only moved when it grows by more than 2^8 in the exponent
// (per wave); until then probabilities are taken against the stale max and
// stay below 256, which bf16 and the fp32 sums hold exactly as well.
constexpr float kLazyRescaleLog2 = 8.f;

// s_waitcnt immediate for vmcnt(0) with expcnt/lgkmcnt left at their maxima
// (gfx9 encoding: vmcnt[3:0], expcnt[6:4], lgkmcnt[11:8], vmcnt_hi[15:14]).
constexpr int kWaitVmcnt0 = 0x0F70;

// Per-lane LDS byte offsets of the fragments, relative to a K or V tile.
//   K (A operand of S^T = K Q^T): lane reads tile row 32kb + l32, logical
//   chunk 2ds + half.  swz(row) only depends on l32, so key block kb is a
//   constant +8192 and only the 8 steps ds need their own offset.
//   V (A operand of O^T += V^T P^T, transposed 64-bit reads): for k-step ks
//   and head-dim block db the group's 16 lanes read rows
//   kbase + i/4 (kbase = 16ks + 4half, +8 for the second half of the slots) at
//   columns d0 + 4(i%4), d0 = 32db + 16(group&1).  swz of those rows does not
//   depend on ks, so ks is a constant +4096 and 4 db x 2 halves need offsets.
struct FragOffsets {
  uint32_t krow;  // tile row l32 (key block 0): l32 * 256
  uint32_t kx;    // swz(l32), the XOR applied to K chunk indices
  uint32_t v[4][2];
};

__device__ __forceinline__ FragOffsets frag_offsets(int lane) {
  FragOffsets f;
  const int l32 = lane & 31, half = lane >> 5, grp = lane >> 4, gi = lane & 15;
  f.krow = (uint32_t)(l32 * kRowBytes);
  f.kx = (uint32_t)(swz(l32) ^ half);
  const int row1 = half * 4 + (gi >> 2);
  const int row2 = row1 + 8;
#pragma unroll
  for (int db = 0; db < 4; ++db) {
    const int dcol = db * 32 + (grp & 1) * 16 + 4 * (gi & 3);
    const int c = dcol >> 3;
    const int e = (dcol & 7) * 2;
    f.v[db][0] = (uint32_t)(row1 * kRowBytes + ((c ^ swz(row1)) << 4) + e);
    f.v[db][1] = (uint32_t)(row2 * kRowBytes + ((c ^ swz(row2)) << 4) + e);
  }
  return f;
}

// S^T = K Q^T for one 64-key tile: s[kb][b] holds keys 32kb..32kb+31 (rows)
// against the 32 queries of block b (columns).  K fragments come from the
// LDS tile (row l32 of key block kb, chunk 2ds+half); the query fragments
// qf[b][ds] stay in registers for the whole work item.
template <int NB>
__device__ __forceinline__ void qk_tile(const unsigned char* sk, const FragOffsets& fo, const bf16x8 (&qf)[NB][8],
                                        f32x16 (&s)[2][NB]) {
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int b = 0; b < NB; ++b) s[kb][b] = f32x16{};
#pragma unroll
  for (int ds = 0; ds < 8; ++ds) {
    const uint32_t off = fo.krow + (((uint32_t)(2 * ds) ^ fo.kx) << 4);
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const bf16x8 kf = *reinterpret_cast<const bf16x8*>(sk + off + kb * 32 * kRowBytes);
#pragma unroll
      for (int b = 0; b < NB; ++b)
        s[kb][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[b][ds], s[kb][b], 0, 0, 0);
    }
  }
}

// Masks keys at tile offsets >= lim[b]; accumulator register r of key block
// kb is tile key 32kb + (r/4)*8 + 4*half + r%4.
template <int NB>
__device__ __forceinline__ void mask_tile(f32x16 (&s)[2][NB], int half, const int (&lim)[NB]) {
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int off = kb * 32 + (r >> 2) * 8 + half * 4 + (r & 3);
#pragma unroll
      for (int b = 0; b < NB; ++b)
        if (off >= lim[b]) s[kb][b][r] = -INFINITY;
    }
}

// Online softmax, first half: the running max of each query column (the two
// lane halves hold disjoint keys of the same query and always agree on it)
// and the factor alpha that moves O and the row sums from the old max to
// the new one.  Returns -max * scale * log2(e), the exponent offset.
template <int NB>
__device__ __forceinline__ void softmax_max(const f32x16 (&s)[2][NB], float (&m_run)[NB], float (&l_run)[NB],
                                            float (&lb_run)[NB], float (&alpha)[NB], float (&neg)[NB], float sl2) {
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    float mx = s[0][b][0];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = __builtin_fmaxf(mx, s[kb][b][r]);
    mx = xmax32(mx);
    const float m_new = __builtin_fmaxf(m_run[b], mx);
    const bool grow = (m_new - m_run[b]) * sl2 > kLazyRescaleLog2;
    const float m_upd = grow ? m_new : m_run[b];
    alpha[b] = (m_upd == -INFINITY) ? 1.f : __builtin_amdgcn_exp2f((m_run[b] - m_upd) * sl2);
    m_run[b] = m_upd;
    l_run[b] *= alpha[b];
    lb_run[b] *= alpha[b];
    neg[b] = (m_upd == -INFINITY) ? 0.f : -m_upd * sl2;
  }
}

// Online softmax, second half: the probabilities of the tile, rounded to
// bf16 once for the PV product, as P^T fragments.  Two row sums: the fp32 one
// gives the LSE, the sum of the rounded values (v_dot2 against (1, 1))
// normalises O, so that O's numerator and denominator use the same weights
// (exact for a single dominant key).  Fragment ks covers tile keys
// 16ks..16ks+15; its slot t of lane half h is key 16ks + (t/4)*8 + 4h + t%4,
// i.e. accumulator register 8*(ks%2) + t of key block ks/2.
template <int NB>
__device__ __forceinline__ void softmax_probs(const f32x16 (&s)[2][NB], const float (&neg)[NB], float (&l_run)[NB],
                                              float (&lb_run)[NB], bf16x8 (&pf)[NB][4], float sl2) {
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    float rs = 0.f;
    float rsb = 0.f;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      bf16x2 pp[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const float e0 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[ks >> 1][b][8 * (ks & 1) + 2 * t], sl2, neg[b]));
        const float e1 =
            __builtin_amdgcn_exp2f(__builtin_fmaf(s[ks >> 1][b][8 * (ks & 1) + 2 * t + 1], sl2, neg[b]));
        pp[t] = bf16x2{(__bf16)e0, (__bf16)e1};
        rs += e0 + e1;
        rsb = __builtin_amdgcn_fdot2_f32_bf16(pp[t], kOnes, rsb, false);
      }
      pf[b][ks] = __builtin_shufflevector(__builtin_shufflevector(pp[0], pp[1], 0, 1, 2, 3),
                                          __builtin_shufflevector(pp[2], pp[3], 0, 1, 2, 3), 0, 1, 2, 3, 4, 5, 6,
                                          7);
    }
    l_run[b] += rs;
    lb_run[b] += rsb;
  }
}

// O^T += V^T P^T for one tile.  The transposed V read gives lane (group g,
// index i) the four keys kbase..kbase+3 of column d0 + i (see FragOffsets).
template <int NB>
__device__ __forceinline__ void pv_tile(const unsigned char* sv, const FragOffsets& fo, const bf16x8 (&pf)[NB][4],
                                        f32x16 (&o)[4][NB]) {
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) {
#pragma unroll
    for (int db = 0; db < 4; ++db) {
      const s16x4 lo4 = ds_read_tr16(sv + fo.v[db][0] + ks * 16 * kRowBytes);
      const s16x4 hi4 = ds_read_tr16(sv + fo.v[db][1] + ks * 16 * kRowBytes);
      const s16x8 v8 = __builtin_shufflevector(lo4, hi4, 0, 1, 2, 3, 4, 5, 6, 7);
      const bf16x8 vf = __builtin_bit_cast(bf16x8, v8);
#pragma unroll
      for (int b = 0; b < NB; ++b) o[db][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[b][ks], o[db][b], 0, 0, 0);
    }
  }
}

// MFMA phase M_j of one wave: O += V_{j-1}^T P_{j-1}, then S_j = K_j Q^T,
// then the mask of
// S_j: keys at tile offsets >= lim are past the key range end (hi) or after
// the lane's query (position q0 + qrel) and get -inf.
template <int NB>
__device__ __forceinline__ void mfma_phase(const unsigned char* sv_prev, const bf16x8 (&pf)[NB][4],
                                           const unsigned char* sk, const bf16x8 (&qf)[NB][8], const FragOffsets& fo,
                                           int64_t t0, int64_t hi, int64_t q0, bool wave_active, int64_t wave_lo,
                                           int64_t wave_hi, const int (&qrel)[NB], const bool (&valid)[NB],
                                           f32x16 (&o)[4][NB], f32x16 (&s)[2][NB]) {
  // Straight-line on purpose (one scheduling region): before the first tile
  // P is zero against tile 0's finite V, and a tile past the wave's last
  // query is multiplied anyway and then fully masked.
  const bool live = wave_active && t0 <= wave_hi;
  pv_tile<NB>(sv_prev, fo, pf, o);
  qk_tile<NB>(sk, fo, qf, s);
  // Read-ahead: four V fragments (two transposed reads each) ahead of the
  // PV MFMAs; the first four d-steps of K (two reads each) under the last four
  // PV MFMAs; then one K read per QK MFMA, which keeps K eight MFMAs ahead.
  static_assert(NB == 1, "schedule written for one 32-row block per wave");
  __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
  if (!live || (t0 + kTileKeys > hi) || (t0 + kTileKeys - 1 > wave_lo)) {
    // lim = min(pos + 1, hi) - t0 in 32 bits from two clamped uniform offsets.
    const int a32 = clamp_i32(q0 + 1 - t0);
    const int b32 = clamp_i32(hi - t0);
    int lim[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      int e = qrel[b] + a32 < b32 ? qrel[b] + a32 : b32;
      e = e < 0 ? 0 : (e > kTileKeys ? kTileKeys : e);
      lim[b] = (live && valid[b]) ? e : 0;
    }
    mask_tile<NB>(s, (threadIdx.x & 32) ? 1 : 0, lim);
  }
}

// VALU phase V_j: softmax of S_j, rescale of O to the new running max (O
// holds every tile up to j-1 at this point), probabilities P_j.
template <int NB>
__device__ __forceinline__ void valu_phase(const f32x16 (&s)[2][NB], float (&m_run)[NB], float (&l_run)[NB],
                                           float (&lb_run)[NB], bf16x8 (&pf)[NB][4], f32x16 (&o)[4][NB], float sl2) {
  float alpha[NB], neg[NB];
  softmax_max<NB>(s, m_run, l_run, lb_run, alpha, neg, sl2);
  bool rescale = false;
#pragma unroll
  for (int b = 0; b < NB; ++b) rescale |= alpha[b] != 1.f;
  if (__any(rescale)) {
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int db = 0; db < 4; ++db) o[db][b] *= alpha[b];
  }
  softmax_probs<NB>(s, neg, l_run, lb_run, pf, sl2);
}

// Barrier j+1 of the tile loop: this wave's loads of tile j+1 are complete
// (so after the barrier everyone's are), and every wave is past its reads of
// K_j and V_{j-1}, whose buffers tile j+2 then reuses.
template <int RPW>
__device__ __forceinline__ void barrier_and_prefetch(int j, int n_tiles, Cursor& lc, const Ranges& rg,
                                                     const DevDesc& d, int kvh, int row_stride, int wave,
                                                     const uint32_t (&lane_off)[RPW / 4],
                                                     const int (&lane_row)[RPW / 4], uint32_t lk0, uint32_t lv0) {
  __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
  __syncthreads();
  if (j + 2 < n_tiles) {
    advance(lc, rg);
    issue_tile<RPW>(lc, rg, d, kvh, row_stride, wave, lane_off, lane_row, lk0 + ((j + 2) % 2) * kTileBytes,
                    lv0 + ((j + 2) % 3) * kTileBytes);
  }
}

// NB = blocks of 32 rows per wave; 8/NB waves cover the workgroup's 256 rows.
template <int NB>
__global__ __launch_bounds__(64 * (8 / NB), 1) void attn_partial_kernel(const DevDesc* __restrict__ descs,
                                                                        const WorkItem* __restrict__ items,
                                                                        PartialParams p) {
  constexpr int kWaves = 8 / NB;
  constexpr int kRPW = kTileKeys / kWaves;  // tile rows each wave loads
  // LDS: two K tile buffers, then three V tile buffers.
  __shared__ __attribute__((aligned(1024))) unsigned char smem[5 * kTileBytes];

  const WorkItem it = items[blockIdx.x];
  const DevDesc& d = descs[it.desc];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int half = lane >> 5;
  const int l32 = lane & 31;

  const int64_t q_begin = it.chunk ? d.q_begin[1] : d.q_begin[0];
  const int64_t q_len = it.chunk ? d.q_len[1] : d.q_len[0];
  const int64_t loff = it.chunk ? d.local_off[1] : d.local_off[0];
  const int Hq = p.Hq;
  const int Hkv = p.Hkv;
  const int kvh = it.head_group / p.groups_per_kv;
  const int head0 = kvh * (Hq / Hkv) + (it.head_group % p.groups_per_kv) * p.heads_per_wg;
  const int qblocks_per_head = p.q_per_wg >> 5;
  const int64_t qb0 = (int64_t)it.q_block * p.q_per_wg;
  const int64_t wg_last = (qb0 + p.q_per_wg < q_len ? qb0 + p.q_per_wg : q_len) - 1;
  const int64_t wg_pos_hi = q_begin + wg_last;

  int head_b[NB];
  int qrel_b[NB];  // query index relative to the workgroup's first query
  bool valid_b[NB];
  int64_t wave_lo = INT64_MAX, wave_hi = -1;
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const int bi = NB * wave + b;
    head_b[b] = head0 + bi / qblocks_per_head;
    const int qo = (bi % qblocks_per_head) * 32;
    qrel_b[b] = qo + l32;
    valid_b[b] = qb0 + qrel_b[b] < q_len;
    const int64_t blo = qb0 + qo, bhi = (qb0 + qo + 31 < wg_last ? qb0 + qo + 31 : wg_last);
    if (blo <= wg_last) {
      wave_lo = (q_begin + blo < wave_lo) ? q_begin + blo : wave_lo;
      wave_hi = (q_begin + bhi > wave_hi) ? q_begin + bhi : wave_hi;
    }
  }
  const bool wave_active = wave_hi >= 0;

  // Key ranges and the number of 64-key tiles over all of them.
  Ranges rg;
  rg.n = 0;
  rg.paged0 = 0;
  int n_tiles = 0;
#pragma unroll
  for (int i = 0; i < 3; ++i) rg.lo[i] = rg.hi[i] = rg.vis[i] = 0;
  if (d.prefix_keys > 0) {
    rg.lo[0] = 0;
    rg.hi[0] = rg.vis[0] = d.prefix_keys;
    rg.paged0 = 1;
    rg.n = 1;
    n_tiles += (int)((d.prefix_keys + kTileKeys - 1) / kTileKeys);
  }
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    if (s < d.n_seg) {
      const int64_t lo = s ? d.seg_lo[1] : d.seg_lo[0];
      const int64_t hi = s ? d.seg_hi[1] : d.seg_hi[0];
      const int64_t vis = hi < wg_pos_hi + 1 ? hi : wg_pos_hi + 1;
      if (vis > lo) {
        if (rg.n == 0) {
          rg.lo[0] = lo; rg.hi[0] = hi; rg.vis[0] = vis;
        } else if (rg.n == 1) {
          rg.lo[1] = lo; rg.hi[1] = hi; rg.vis[1] = vis;
        } else {
          rg.lo[2] = lo; rg.hi[2] = hi; rg.vis[2] = vis;
        }
        ++rg.n;
        n_tiles += (int)((vis - lo + kTileKeys - 1) / kTileKeys);
      }
    }
  }

  Cursor cc{0, rg.lo[0]};
  Cursor lc = cc;
  // Per-lane part of the tile load addresses (see issue_tile).
  const int row_stride = Hkv * kHeadDim * 2;
  uint32_t lane_off[kRPW / 4];
  int lane_row[kRPW / 4];
#pragma unroll
  for (int i = 0; i < kRPW / 4; ++i) {
    const int row = wave * kRPW + 4 * i + (lane >> 4);
    lane_row[i] = row;
    lane_off[i] = (uint32_t)(row * row_stride + (((lane & 15) ^ swz(row)) << 4));
  }
  const uint32_t lds0 = lds_addr(smem);
  unsigned char* const sk0 = smem;                    // K buffer b at sk0 + b * kTileBytes (b < 2)
  unsigned char* const sv0 = smem + 2 * kTileBytes;   // V buffer b at sv0 + b * kTileBytes (b < 3)
  const uint32_t lk0 = lds0, lv0 = lds0 + 2 * kTileBytes;
  if (n_tiles > 0) issue_tile<kRPW>(lc, rg, d, kvh, row_stride, wave, lane_off, lane_row, lk0, lv0);

  // Query fragments (B operand of S^T = K Q^T): lane holds 8 consecutive
  // head-dim values of its query, for each of the 8 steps of 16 along D.
  // Rows past the chunk's end are zero and masked out of every tile.
  bf16x8 qf[NB][8];
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const __attribute__((address_space(1))) bf16x8* qrow =
        (const __attribute__((address_space(1))) bf16x8*)(d.q + ((loff + qb0 + qrel_b[b]) * Hq + head_b[b]) * kHeadDim +
                                                          half * 8);
#pragma unroll
    for (int ds = 0; ds < 8; ++ds) qf[b][ds] = valid_b[b] ? qrow[2 * ds] : bf16x8{};
  }

  // Query rows and tile 0 land before the first barrier of the loop.
  __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);

  f32x16 o[4][NB];
  float m_run[NB], l_run[NB], lb_run[NB];  // running max; sums of fp32 / bf16-rounded probabilities
#pragma unroll
  for (int b = 0; b < NB; ++b) {
#pragma unroll
    for (int db = 0; db < 4; ++db) o[db][b] = f32x16{};
    m_run[b] = -INFINITY;
    l_run[b] = 0.f;
    lb_run[b] = 0.f;
  }
  const float sl2 = p.scale_log2;

  // Two groups, one instruction stream, shifted barriers.  Every wave runs
  // M_0 V_0 M_1 V_1 ... M_n with M_j = {O += V_{j-1}^T P_{j-1}, S_j = K_j Q^T}
  // on the matrix cores and V_j = {softmax of S_j -> P_j} on the VALU.  Waves
  // 0..3 meet the per-tile barrier after V_j, waves 4..7 after M_j, so between
  // two barriers group 0 runs M_j then V_j while group 1 runs V_{j-1} then
  // M_j.  Wave w shares its SIMD with wave w +- 4, so each SIMD pairs one
  // wave's MFMA phase with the other's softmax.  Tile j+1 is issued right
  // after barrier j and awaited before barrier j+1; two K buffers and three V
  // buffers (V_{j-1} is read during interval j).
  const int group = wave >> 2;
  const FragOffsets fo = frag_offsets(lane);
  f32x16 s[2][NB];
  bf16x8 pf[NB][4];
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) pf[b][ks] = bf16x8{};

  // Barrier 0: tile 0 and the query rows are in LDS; tile 1 streams in.
  __syncthreads();
  if (n_tiles > 1) {
    advance(lc, rg);
    issue_tile<kRPW>(lc, rg, d, kvh, row_stride, wave, lane_off, lane_row, lk0 + kTileBytes, lv0 + kTileBytes);
  }
  for (int j = 0; j < n_tiles; ++j) {
    const int64_t t0 = cc.t0;
    const int64_t hi = sel3(rg.hi, cc.r);
    advance(cc, rg);
    mfma_phase<NB>(sv0 + (j >= 1 ? (j - 1) % 3 : 0) * kTileBytes, pf, sk0 + (j % 2) * kTileBytes, qf, fo, t0, hi,
                   q_begin + qb0, wave_active, wave_lo, wave_hi, qrel_b, valid_b, o, s);
    if (group == 1) barrier_and_prefetch<kRPW>(j, n_tiles, lc, rg, d, kvh, row_stride, wave, lane_off, lane_row, lk0, lv0);
    valu_phase<NB>(s, m_run, l_run, lb_run, pf, o, sl2);
    if (group == 0) barrier_and_prefetch<kRPW>(j, n_tiles, lc, rg, d, kvh, row_stride, wave, lane_off, lane_row, lk0, lv0);
  }
  if (n_tiles > 0) pv_tile<NB>(sv0 + ((n_tiles - 1) % 3) * kTileBytes, fo, pf, o);

  // Normalise and store: O^T register r of d-block db is head-dim
  // db*32 + (r/4)*8 + 4*half + r%4 of this lane's query.
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const float lt = xsum32(l_run[b]);
    const float ltb = xsum32(lb_run[b]);
    const bool live = (m_run[b] != -INFINITY) && (lt > 0.f) && (ltb > 0.f);
    const float inv = live ? 1.f / ltb : 0.f;
    if (valid_b[b]) {
      const int64_t row = loff + qb0 + qrel_b[b];
      float* orow = d.o + (row * Hq + head_b[b]) * kHeadDim;
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
      if (half == 0) d.lse[row * Hq + head_b[b]] = live ? m_run[b] * p.scale + logf(lt) : -INFINITY;
    }
  }
}

}  // namespace

int launch_partial(const PartialParams& p, void* stream) {
  if (p.n_items == 0) return CP_OK;
  hipLaunchKernelGGL(attn_partial_kernel<1>, dim3((unsigned)p.n_items), dim3(512), 0, (hipStream_t)stream,
                     p.descs, p.items, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(CP_ERR_HIP, std::string("cp_attn_partial launch: ") + hipGetErrorString(e));
  return CP_OK;
}

}  // namespace cpattn
