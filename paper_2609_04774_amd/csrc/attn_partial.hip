// Partial causal attention of one CP rank's zigzag rows, bf16 MFMA on gfx950.
//
// What is computed (paper Sec. 2.1 / 2.2): for every query row at global
// position p and head h, over the keys j of the descriptor's key set with
// j <= p:  x_j = scale * q.k_j,  LSE = ln sum_j e^{x_j},
// O = sum_j e^{x_j - LSE} v_j, with grouped KV head h / (Hq/Hkv).
//
// How (FlashAttention-2 style online softmax, Dao 2023, with the running
// max/sum recurrence of Milakov & Gimelshein 2018):
//   * A workgroup of 8 wave64s (two per SIMD) owns 128 NB (query, head) rows
//     that share one KV head: `heads_per_wg` query heads x `q_per_wg`
//     consecutive positions.  Each wave owns NB blocks of 16 rows, so every
//     K and V fragment read from LDS feeds NB MFMAs.  The kernel comes in two
//     shapes, NB = 3 (384 rows: fewer LDS bytes per FLOP) and NB = 2 (256
//     rows: more, shorter work items); the host plan picks one per launch.
//     Two waves
//     per SIMD let one wave's vector and scalar work issue while the other's
//     matrix work runs (a single wave issues one instruction at a time,
//     whatever its type); the 256 registers per lane this leaves a wave hold
//     all of its state in VGPRs.
//   * Keys are visited in tiles of 32 along each key range (paged prefix,
//     then the suffix ranges).  Tiles past the workgroup's last query are
//     never visited; only tiles that cross the diagonal or a range end are
//     masked.  A work item that sees no key writes its empty result and exits.
//   * Scores are computed transposed, S^T = K Q^T, with
//     v_mfma_f32_16x16x32_bf16: a lane then holds 8 keys of one query per
//     16-row block (the other 24 are in lanes l ^ 16, l ^ 32, l ^ 48), and
//     the probabilities feed O^T += V^T P^T directly from registers.  V^T
//     fragments come from the key-major V tile through ds_read_b64_tr_b16.
//     The sum of the bf16-rounded probabilities, which normalises O, is one
//     more MFMA per block over the same P fragments.
//   * Each row goes where the descriptor says: the rank's local row, or its
//     suffix index (the restore to sequence order in the kernel's stores).
//   * Software pipeline: iteration j runs O += V_{j-1}^T P_{j-1}, the
//     softmax of S_j and S_{j+1} = K_{j+1} Q^T -- three independent streams
//     -- as one fixed sequence of MFMA slots with the softmax dealt out
//     between them.  Iterations go in pairs that share one workgroup barrier
//     and swap the two score register sets; each iteration loads tile j+5
//     into LDS.
//   * LDS tiles are stored by 16-key halves and 16-byte columns: column c of
//     a half holds head-dim chunk c (8 values) of its 16 keys, key k at slot
//     k ^ 8(c % 2).  The K reads (16 keys, one column per 16 lanes) and the
//     transposed V reads (8 keys, two columns per 32 lanes) then hit every
//     bank once, and each lane's fragment addresses differ only by
//     constants, so the 24 LDS reads of one tile's 16 fragments need two
//     address registers.
#include <hip/hip_runtime.h>

#include <cmath>

#include "internal.h"

namespace cpattn {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = 8;                    // wave64s per workgroup, two per SIMD
constexpr int kBlockRows = 16;               // a wave holds NB (2 or 3) blocks of 16 query rows
constexpr int kTileKeys = 32;
constexpr int kBufs = 8;                     // LDS tile buffers, each for K and for V
constexpr int kAhead = 5;                    // the iteration of tile j loads tile j + kAhead
constexpr int kRowBytes = kHeadDim * 2;
constexpr int kTileBytes = kTileKeys * kRowBytes;

// LDS byte offset of head-dim chunk c (16 bytes) of tile key `key` within a
// tile buffer (64 banks x 4 bytes on gfx950).  A half (16 keys) is 16
// columns of 256 bytes; in column c, key k sits at slot k ^ 8(c % 2).  Any 16
// keys of one column fill 256 bytes (every bank once), and keys k0..k0+7
// (k0 % 8 == 0) of two columns 2c, 2c + 1 occupy 16 distinct slots.
constexpr int kHalfBytes = 16 * kRowBytes;
constexpr int kColBytes = 16 * 16;
__device__ __forceinline__ int lds_off(int key, int c) {
  return (key >> 4) * kHalfBytes + c * kColBytes + (((key & 15) ^ (8 * (c & 1))) << 4);
}

__device__ __forceinline__ s16x4 ds_read_tr16(const unsigned char* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(p));
}

// The key tiles of one work item: three ranges in a fixed order -- A, the
// paged prefix; B and C, the suffix ranges -- each walked in 32-key tiles from
// `lo` up to `vis` (one past the last key a query of the work item can see);
// `hi` is the range's end, used for masking.  An unused range has no tiles.
// Positions are below 2^30 (the host checks), so all of this is 32-bit
// scalar arithmetic, and a tile is found from its index with selects only.
// (Plain fields, no arrays: a select between array elements would become an
// indexed load from scratch memory.)
struct TileWalk {
  int hiA;                 // range A is [0, hiA), all visible
  int loB, hiB, visB;
  int loC, hiC, visC;
  int firstB, firstC;      // index of the first tile of ranges B and C
  int n;                   // tiles over all ranges
};

struct Tile {
  int t0;    // first key position
  int hi;    // end of the tile's range
  int vis;   // visible end of the tile's range
  bool paged;
};

// A select of two values (never of two variables' addresses, which would
// put both variables in scratch memory).
__device__ __forceinline__ int sel(bool c, int a, int b) { return c ? a : b; }

__device__ __forceinline__ Tile tile_at(const TileWalk w, int t) {
  const bool gB = t >= w.firstB, gC = t >= w.firstC;
  Tile x;
  const int lo = gC ? w.loC : (gB ? w.loB : 0);
  const int f = gC ? w.firstC : (gB ? w.firstB : 0);
  x.t0 = lo + (t - f) * kTileKeys;
  x.hi = gC ? w.hiC : (gB ? w.hiB : w.hiA);
  x.vis = gC ? w.visC : (gB ? w.visB : w.hiA);
  x.paged = !gB;
  return x;
}

// Descriptor fields the loop needs, read once into registers: the tile loads
// are inline assembly with a memory clobber, after which the compiler would
// otherwise load them again from the descriptor on every tile.
struct KvSource {
  const unsigned char* k_new;
  const unsigned char* v_new;
  const unsigned char* k_cache;
  const unsigned char* v_cache;
  const int32_t* block_table;
  int P;
  uint32_t n_blocks;
};

// Source of a cache block whose block-table entry lies outside the cache:
// 256 zero bytes, read by every row of the block (the per-lane offset is then
// only the 16-byte column, below 256), so such keys and values are zeros and
// nothing outside the cache is read.
__device__ __attribute__((aligned(256))) unsigned char g_zero_row[kHeadDim * 2];

// One global_load_lds_dwordx4: lane l's 16 bytes at sbase + voff land at LDS
// byte m0 + 16*l.  Issued as inline assembly so the compiler does not treat
// every later LDS read as depending on it (it cannot tell the two buffers
// apart); the kernel waits for these loads itself (vmcnt) before the barrier
// that publishes a tile.  The LDS address is an input operand bound to m0, so
// the compiler writes m0 itself and knows what it holds; the asm only reads
// it, after the one wait state an m0 write needs before an LDS-DMA load.  The
// base and the LDS address are wave-uniform; the lane reads place them in
// scalar registers however the compiler carried them.
__device__ __forceinline__ void dma16(const void* sbase, uint32_t voff, uint32_t lds_base) {
  const uint64_t b = (uint64_t)(uintptr_t)sbase;
  const uint64_t bs = ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(b >> 32)) << 32) |
                      (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)b);
  asm volatile(
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %0, %1\n\t" ::"v"(voff), "s"((const void*)(uintptr_t)bs),
      "{m0}"(__builtin_amdgcn_readfirstlane((int)lds_base))
      : "memory");
}

__device__ __forceinline__ uint32_t lds_addr(const unsigned char* p) {
  return (uint32_t)(uintptr_t)((const __attribute__((address_space(3))) unsigned char*)p);
}

// This wave's share of one K/V tile load, prepared ahead of the slots that
// issue it: 1 KB of K and 1 KB of V, i.e. four LDS columns (4g .. 4g+3, g =
// wave % 4) of tile half wave / 4.  Lane l fills slot l % 16 of column
// 4g + l/16, so it carries that column's chunk of half key (l % 16) ^ 8((l/16) % 2)
// (see lds_off).  The address is a wave-uniform base (tile start, KV head)
// plus a per-lane offset `lane_off` = row_in_tile * row_stride + 16 * column.
// In the last tile of a suffix range, rows past the visible end read the
// last visible row instead (in range; those keys are masked).
static_assert(kWaves * 4 * kColBytes == kTileBytes, "eight waves, 1 KB of the tile each");
struct TileLoad {
  const unsigned char* kb;
  const unsigned char* vb;
  uint32_t off;
  uint32_t lk, lv;  // LDS destinations
};

__device__ __forceinline__ TileLoad prep_tile(const Tile& x, const KvSource& src, int kvh, int row_stride, int wave,
                                              uint32_t lane_off, int lane_row, uint32_t lane_col, uint32_t sk,
                                              uint32_t sv) {
  const int row0 = (wave >> 2) * 16;  // first tile row of this wave's half
  const uint32_t dst = (uint32_t)((wave >> 2) * kHalfBytes + (wave & 3) * 4 * kColBytes);
  TileLoad t;
  t.off = lane_off;
  t.lk = sk + dst;
  t.lv = sv + dst;
  if (x.paged) {
    // Prefix tiles start at multiples of 32 keys, so this wave's half is
    // logical cache block t0/16 + row0/16 (clamped to the last block); the
    // lane offsets use the row within the tile, so step back by the half's
    // first tile row.  Wave-uniform index: a scalar load.
    int lb = (x.t0 >> 4) + (row0 >> 4);
    const int last = ((x.vis + kBlockTokens - 1) >> 4) - 1;
    lb = lb < last ? lb : last;
    const int32_t blk = ((const __attribute__((address_space(4))) int32_t*)src.block_table)[lb];
    if ((uint32_t)blk < src.n_blocks) {
      const int64_t base = ((int64_t)blk * kBlockTokens - row0) * row_stride + kvh * (kHeadDim * 2);
      t.kb = src.k_cache + base;
      t.vb = src.v_cache + base;
    } else {
      t.kb = g_zero_row;
      t.vb = g_zero_row;
      t.off = lane_col;
    }
  } else {
    const int64_t base = (int64_t)(x.t0 - src.P) * row_stride + kvh * (kHeadDim * 2);
    t.kb = src.k_new + base;
    t.vb = src.v_new + base;
    if (x.t0 + kTileKeys > x.vis) {
      const int clamp_row = x.vis - 1 - x.t0;
      const int r = lane_row < clamp_row ? lane_row : clamp_row;
      t.off = __umul24((uint32_t)r, (uint32_t)row_stride) + lane_col;
    }
  }
  return t;
}

// Load q (0: K, 1: V) of a prepared tile.
__device__ __forceinline__ void issue_load(const TileLoad& t, int q) {
  if (q & 1)
    dma16(t.vb, t.off, t.lv);
  else
    dma16(t.kb, t.off, t.lk);
}

__device__ __forceinline__ void issue_tile(const TileLoad& t) {
  issue_load(t, 0);
  issue_load(t, 1);
}

// max(a, b, c) in one v_maximum3_f32 (NaN-propagating maximum).  fmaxf on
// values the compiler cannot prove canonical -- the scores come out of
// inline assembly -- would cost an extra canonicalising max per operand.
__device__ __forceinline__ float max3(float a, float b, float c) {
  return __builtin_elementwise_maximum(__builtin_elementwise_maximum(a, b), c);
}

// Max / sum over the four lanes that hold one query (l, l ^ 16, l ^ 32, l ^
// 48: the four row groups of a 16x16 result), by two lane-swap exchanges.
__device__ __forceinline__ float swap16_max(float x) {
  auto r = __builtin_amdgcn_permlane16_swap(__builtin_bit_cast(unsigned, x), __builtin_bit_cast(unsigned, x),
                                            false, false);
  return __builtin_elementwise_maximum(__builtin_bit_cast(float, (unsigned)r[0]),
                                      __builtin_bit_cast(float, (unsigned)r[1]));
}

__device__ __forceinline__ float swap32_max(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(unsigned, x), __builtin_bit_cast(unsigned, x),
                                            false, false);
  return __builtin_elementwise_maximum(__builtin_bit_cast(float, (unsigned)r[0]),
                                      __builtin_bit_cast(float, (unsigned)r[1]));
}

__device__ __forceinline__ float swap16_sum(float x) {
  auto r = __builtin_amdgcn_permlane16_swap(__builtin_bit_cast(unsigned, x), __builtin_bit_cast(unsigned, x),
                                            false, false);
  return __builtin_bit_cast(float, (unsigned)r[0]) + __builtin_bit_cast(float, (unsigned)r[1]);
}

__device__ __forceinline__ float swap32_sum(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(unsigned, x), __builtin_bit_cast(unsigned, x),
                                            false, false);
  return __builtin_bit_cast(float, (unsigned)r[0]) + __builtin_bit_cast(float, (unsigned)r[1]);
}

__device__ __forceinline__ float quad_max(float x) { return swap32_max(swap16_max(x)); }
__device__ __forceinline__ float quad_sum(float x) { return swap32_sum(swap16_sum(x)); }

// Probabilities of a tile are taken against the running max m of the tiles
// before it, without looking at the tile's own scores first: p = 2^(x - m).
// They stay exact relative to each other whatever their size (fp32 and bf16
// keep 24 and 8 significant bits at any exponent), so m only has to move
// when p could overflow.  A tile whose fp32 sum of a lane's 8 probabilities
// of one query exceeds 2^16 (a score more than ~2^13 above m, or the first
// visible key of a query) is redone exactly: its scores recomputed from the
// K tile still in LDS, their max taken, O and the sums rescaled, the
// probabilities taken against the new max.  With probabilities below 2^16
// nothing overflows for any |v| below 2^100.
constexpr float kMaxTileSum = 65536.f;
// The running max is kept in units of the exponent (score * scale * log2 e)
// and starts at a finite "nothing seen" value far below any real score's:
// a query's first visible key then always overflows the check above (2^(x +
// 1e30) = inf) and sets it exactly, a fully masked tile (scores -inf)
// yields probabilities exp2(-inf) = 0 against it, and no lane needs a -inf
// special case.
constexpr float kNoMax = -1e30f;

constexpr float kLn2 = 0.69314718055994531f;

// Per-lane LDS byte offsets of the fragments in buffer 0 (buffer b adds
// b * kTileBytes: one scalar-plus-vector add per offset and tile; the rest
// are instruction immediates).  Lane l = 16g + i.
//   K (A operand of S^T = K Q^T, 16 keys x 32 head-dims): for key half kb
//   and head-dim step ds the lane reads key i of half kb, chunk c = 4ds + g:
//   K(kb, ds) = k + kb * 4096 + ds * 1024 (c % 2 = g % 2 for every ds).
//   V (A operand of O^T += V^T P^T, 16 head-dims x 32 keys, transposed
//   64-bit reads): for head-dim block db the group's 16 lanes read keys
//   16r + 4g + i/4 (r = 0, 1: the fragment's two 8-byte halves, one per key
//   half) at head-dims 16db + 4(i % 4), i.e. chunk c = 2db + (i % 4)/2, byte
//   8(i % 2) of it; lane i receives head-dim 16db + i of those 4 keys.
//   c % 2 = (i % 4)/2 for every db, so V(db, r) = v + r * 4096 + db * 512
//   (v includes the start of the V buffers, kBufs * kTileBytes).
// The P^T operand of a lane (query i, k = 8g .. 8g+7) then holds keys
// 4g .. 4g+3 of half 0 and of half 1 -- exactly the scores the lane holds
// (rows 4g .. 4g+3 of the two S^T results), so P never leaves the lane.
struct FragOffsets {
  uint32_t k;
  uint32_t v;
};

__device__ __forceinline__ FragOffsets frag_offsets(int lane) {
  FragOffsets f;
  const int g = lane >> 4, i = lane & 15;
  f.k = (uint32_t)lds_off(i, g);
  f.v = (uint32_t)(kBufs * kTileBytes + lds_off(4 * g + (i >> 2), (i & 3) >> 1) + 8 * (i & 1));
  return f;
}

__device__ __forceinline__ const unsigned char* k_frag_addr(const unsigned char* sk, const FragOffsets& fo, int q) {
  // q = 2 ds + kb (the order the region walks the eight K fragments)
  return sk + fo.k + (q & 1) * kHalfBytes + (q >> 1) * 4 * kColBytes;
}

__device__ __forceinline__ bf16x8 v_frag(const unsigned char* sv, const FragOffsets& fo, int db) {
  const int c = db * 2 * kColBytes;
  const s16x4 lo4 = ds_read_tr16(sv + fo.v + c);
  const s16x4 hi4 = ds_read_tr16(sv + fo.v + kHalfBytes + c);
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo4, hi4, 0, 1, 2, 3, 4, 5, 6, 7));
}

__device__ __forceinline__ f32x4 mfma16(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Scores of one tile: s[kb][b] = S^T of key half kb and query block b;
// register r of it is key 16kb + 4g + r of the tile.
template <int NB>
using Scores = f32x4[2][NB];

// One step of S^T = K Q^T (K fragment q = 2ds + kb) for the NB blocks.
// Every operand lives in VGPRs, and the compiler sees the instructions, so
// it keeps the matrix-core hazards (result reads, operand overwrites) itself.
template <int NB>
__device__ __forceinline__ void qk_step(Scores<NB>& s, const bf16x8& k, const bf16x8 (&qf)[NB][4], int q) {
  const int kb = q & 1, ds = q >> 1;
#pragma unroll
  for (int b = 0; b < NB; ++b) s[kb][b] = mfma16(k, qf[b][ds], ds == 0 ? f32x4{} : s[kb][b]);
}

// S^T = K Q^T for one 32-key tile (the prologue's first tile, and redos).
template <int NB>
__device__ __forceinline__ void qk_tile(const unsigned char* sk, const FragOffsets& fo, const bf16x8 (&qf)[NB][4],
                                        Scores<NB>& s) {
#pragma unroll
  for (int q = 0; q < 8; ++q) qk_step(s, *reinterpret_cast<const bf16x8*>(k_frag_addr(sk, fo, q)), qf, q);
}

// O^T += V^T P^T for one 32-key tile (the last one), with the bf16 row sums.
template <int NB>
__device__ __forceinline__ void pv_tile(const unsigned char* sv, const FragOffsets& fo, const bf16x8 (&pf)[NB],
                                        f32x4 (&o)[8][NB], const bf16x8& ones, f32x4 (&psum)[NB]) {
#pragma unroll
  for (int db = 0; db < 8; ++db) {
    const bf16x8 vf = v_frag(sv, fo, db);
#pragma unroll
    for (int b = 0; b < NB; ++b) o[db][b] = mfma16(vf, pf[b], o[db][b]);
  }
#pragma unroll
  for (int b = 0; b < NB; ++b) psum[b] = mfma16(ones, pf[b], psum[b]);
}

// Masks keys at tile offsets >= lim[b]; register r of s[kb][b] is tile key
// 16kb + 4g + r.
template <int NB>
__device__ __forceinline__ void mask_tile(Scores<NB>& s, int g, const int (&lim)[NB]) {
  // Compare the constant part of the offset with lim - 4g, so that no
  // per-register offsets need to be kept in registers.
  int limg[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) limg[b] = lim[b] - 4 * g;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int b = 0; b < NB; ++b)
        if (16 * kb + r >= limg[b]) s[kb][b][r] = -INFINITY;
}

// Keys at tile offsets >= lim are past the range end (hi) or after the
// lane's query (position q0 + qrel).  A tile past the wave's last query is
// masked entirely.
template <int NB>
__device__ __forceinline__ void tile_limits(const Tile& x, int q0, bool wave_active, int wave_hi,
                                            const int (&qrel)[NB], const bool (&valid)[NB], int (&lim)[NB]) {
  const bool live = wave_active && x.t0 <= wave_hi;
  const int a = q0 + 1 - x.t0;
  const int h = x.hi - x.t0;
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    int e = qrel[b] + a < h ? qrel[b] + a : h;
    e = e < 0 ? 0 : (e > kTileKeys ? kTileKeys : e);
    lim[b] = (live && valid[b]) ? e : 0;
  }
}

// One iteration's matrix and vector work as a fixed sequence of 16 slots,
// each with one LDS fragment and NB MFMAs (one per query block): slots 0-7
// add P_{j-1} V_{j-1} (V fragment = head-dim block slot), slots 8-15 compute
// S_{j+1} = K_{j+1} Q^T (K fragment slot - 8); slots 2, 4 (and 6) also take
// block (slot - 2)/2's bf16 row sums.  The softmax of S_j is cut into units
// of roughly equal VALU time and dealt out over the slots, so that every
// MFMA has vector work to overlap with.  LDS fragments are read a few slots
// ahead (kLookahead: about 100 cycles of MFMA work) in one continuous stream:
// the region's last slots read the next iteration's first V fragments (of
// tile j, published since before this pair of iterations), so no iteration
// starts by waiting for a fresh LDS read.  The two loads of tile j+5 (K rows,
// then V rows) go out at slots 1 and 9.  Scheduling barriers keep the slots
// in this order.  The other wave on the same SIMD runs the same sequence
// shifted in time, so one wave's vector and scalar work issues while the
// other's matrix work runs.
//
// Units: 4 NB times (two exponentials, one pack-and-sum) for score pairs,
// against the running max (see kMaxTileSum), in the order of kUnitOrder
// below.  The overflow check, and the exact redo of a tile in the rare case
// that it fails, follow the region.
constexpr int kSlots = 16;
template <int NB>
constexpr int kLookahead = NB == 2 ? 3 : 2;

// Forces `x` to be computed before this point: an empty volatile asm that
// reads it stays in program order with the scheduling barriers, so the
// value's producers cannot sink past the slot they were written in.
template <typename T>
__device__ __forceinline__ void pin(const T& x) {
  asm volatile("" ::"v"(x));
}

template <int NB>
struct SoftmaxState {
  float rs[NB];      // fp32 sum of this tile's probabilities, per block
  bf16x2 pp[NB][4];  // bf16 pairs: [half 0 regs 0-1, 2-3, half 1 regs 0-1, 2-3]
};

// Pair t of block b's 8 scores (t = 2 kb + r/2, registers r, r+1 of half
// kb, already exponentiated): rounded to bf16 once (the P operand of O += V
// P), and added to the block's fp32 sum (the LSE's).  The sum of the
// bf16-rounded values, which normalises O, is taken by an MFMA over the P
// fragments (psum in the kernel): a dot-product instruction here would share
// the matrix pipes with the tile's MFMAs and cost far more issue time.
template <int NB>
__device__ __forceinline__ void pack_and_sum(int b, int t, const Scores<NB>& s, SoftmaxState<NB>& st) {
  const int kb = t >> 1, r = 2 * (t & 1);
  const bf16x2 pp = bf16x2{(__bf16)s[kb][b][r], (__bf16)s[kb][b][r + 1]};
  st.pp[b][t] = pp;
  if (t == 0)
    st.rs[b] = s[kb][b][r] + s[kb][b][r + 1];
  else
    st.rs[b] += s[kb][b][r] + s[kb][b][r + 1];
  pin(st.rs[b]);
  pin(pp);
}

// The order of the units: the exponentials of every block but the last
// come first, then, once slot 8 starts (after the region's last use of the
// previous P), the pack-and-sums, the last block's units interleaved with
// its packs.  Each block's bf16 pairs are thereby produced after the
// registers of its previous P are free, and land in them directly.
struct Unit {
  int b, t, kind;  // block, pair, kind (0, 1: one exponential each; 2: pack and sum)
};
template <int NB>
struct UnitOrder {
  Unit u[12 * NB];
  constexpr UnitOrder() : u{} {
    int n = 0;
    for (int b = 0; b + 1 < NB; ++b)
      for (int t = 0; t < 4; ++t)
        for (int k = 0; k < 2; ++k) u[n++] = Unit{b, t, k};
    const int last = NB - 1;
    int te = 0;  // the last block's pairs whose exponentials are placed
    for (; n < 6 * NB; ++te) {
      u[n++] = Unit{last, te, 0};
      u[n++] = Unit{last, te, 1};
    }
    for (int b = 0; b + 1 < NB; ++b)
      for (int t = 0; t < 4; ++t) u[n++] = Unit{b, t, 2};
    for (int t = 0; t < 4; ++t) {
      if (t >= te) {
        u[n++] = Unit{last, t, 0};
        u[n++] = Unit{last, t, 1};
      }
      u[n++] = Unit{last, t, 2};
    }
  }
};
template <int NB>
constexpr UnitOrder<NB> kUnitOrder{};

template <int NB>
__device__ __forceinline__ void softmax_unit(int u, Scores<NB>& s, SoftmaxState<NB>& st, const float (&m_run)[NB],
                                             float sl2) {
  const int b = kUnitOrder<NB>.u[u].b, t = kUnitOrder<NB>.u[u].t, kind = kUnitOrder<NB>.u[u].kind;
  if (kind < 2) {
    const int kb = t >> 1, r = 2 * (t & 1) + kind;
    const float x = __builtin_amdgcn_exp2f(__builtin_fmaf(s[kb][b][r], sl2, -m_run[b]));
    pin(x);
    s[kb][b][r] = x;
  } else {
    pack_and_sum(b, t, s, st);
  }
}

// Max of block b's scores of one query (a lane's 8 and the three other
// lanes' 24), in exponent units.
template <int NB>
__device__ __forceinline__ float tile_max(const Scores<NB>& s, int b, float sl2) {
  float mx = max3(__builtin_elementwise_maximum(s[0][b][0], s[0][b][1]), s[0][b][2], s[0][b][3]);
  mx = max3(max3(mx, s[1][b][0], s[1][b][1]), s[1][b][2], s[1][b][3]);
  return quad_max(mx) * sl2;
}

// Fragment g of the region: g < 8 is V^T fragment (head-dim block g), g >=
// 8 is K fragment g - 8.
__device__ __forceinline__ bf16x8 load_frag(int g, const unsigned char* sv, const unsigned char* sk,
                                            const FragOffsets& fo) {
  if (g < 8) return v_frag(sv, fo, g);
  return *reinterpret_cast<const bf16x8*>(k_frag_addr(sk, fo, g - 8));
}

// s_in: S_j (masked), turned into its probabilities against m_run (their
// bf16 pairs and sums in st); s_out: receives S_{j+1}.  pf: P_{j-1}, added
// into O.
template <int NB>
__device__ __forceinline__ void pipelined_region(const unsigned char* sv, const unsigned char* sk,
                                                 const unsigned char* sv_next, const FragOffsets& fo,
                                                 const bf16x8 (&qf)[NB][4], const bf16x8 (&pf)[NB],
                                                 f32x4 (&o)[8][NB], Scores<NB>& s_in, Scores<NB>& s_out,
                                                 const float (&m_run)[NB], float sl2, const TileLoad& ld,
                                                 SoftmaxState<NB>& st, bf16x8 (&pre)[kLookahead<NB>], const bf16x8& ones,
                                                 f32x4 (&psum)[NB]) {
  bf16x8 fr[16];
#pragma unroll
  for (int g = 0; g < kLookahead<NB>; ++g) fr[g] = pre[g];
#pragma unroll
  for (int slot = 0; slot < kSlots; ++slot) {
    const int g = slot + kLookahead<NB>;
    if (g < 16)
      fr[g] = load_frag(g, sv, sk, fo);
    else
      pre[g - 16] = load_frag(g - 16, sv_next, sk, fo);  // the next iteration's first V fragments
    if ((slot & 7) == 1) issue_load(ld, slot >> 3);
    if (slot < 8) {
#pragma unroll
      for (int b = 0; b < NB; ++b) o[slot][b] = mfma16(fr[slot], pf[b], o[slot][b]);
      if (slot >= 2 && (slot & 1) == 0 && (slot - 2) / 2 < NB) {
        const int b = (slot - 2) / 2;
        psum[b] = mfma16(ones, pf[b], psum[b]);
      }
    } else {
      qk_step(s_out, fr[slot], qf, slot - 8);
    }
#pragma unroll
    for (int u = (slot * 12 * NB) / kSlots; u < ((slot + 1) * 12 * NB) / kSlots; ++u)
      softmax_unit(u, s_in, st, m_run, sl2);
    __builtin_amdgcn_sched_barrier(0);
  }
}

// The exact redo of tile j (rare; see kMaxTileSum): s holds S_j, recomputed
// and masked by the caller.  Each block's running max moves to the max of
// the tile where that is higher, O and the running sums are rescaled by
// 2^(m_old - m_new) (exactly 1 where it did not move, 0 before a query's
// first visible key), and the tile's probabilities are taken against the
// new max.
template <int NB>
__device__ __forceinline__ void exact_softmax(Scores<NB>& s, float (&m_run)[NB], float (&l_run)[NB],
                                              f32x4 (&psum)[NB], f32x4 (&o)[8][NB], float sl2, SoftmaxState<NB>& st) {
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const float m_new = __builtin_elementwise_maximum(tile_max(s, b, sl2), m_run[b]);
    const float alpha = __builtin_amdgcn_exp2f(m_run[b] - m_new);
    l_run[b] *= alpha;
    psum[b] *= alpha;
#pragma unroll
    for (int db = 0; db < 8; ++db) o[db][b] *= alpha;
    m_run[b] = m_new;
  }
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int t = 0; t < 4; ++t) {
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        const int kb = t >> 1, r = 2 * (t & 1) + k;
        s[kb][b][r] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[kb][b][r], sl2, -m_run[b]));
      }
      pack_and_sum(b, t, s, st);
    }
}

// s_waitcnt immediates (gfx9 encoding: vmcnt[3:0], expcnt[6:4], lgkmcnt[11:8],
// vmcnt_hi[15:14]) waiting until at most N of this wave's vector-memory
// operations are outstanding.
constexpr int kLoadsPerTile = 2;  // K and V loads of one tile per wave
constexpr int kWaitVm(int n) { return 0x0F70 | n; }

template <int NB>
__global__ __launch_bounds__(64 * kWaves, 1) void attn_partial_kernel(const DevDesc* __restrict__ descs,
                                                                     const WorkItem* __restrict__ items,
                                                                     PartialParams p) {
  // LDS: kBufs K tile buffers, then kBufs V tile buffers; tile t uses buffer
  // t % kBufs of each.
  __shared__ __attribute__((aligned(1024))) unsigned char smem[2 * kBufs * kTileBytes];

  const WorkItem it = items[blockIdx.x];
  const DevDesc& d = descs[it.desc];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g4 = lane >> 4;   // row group of the 16x16 results
  const int l16 = lane & 15;  // query of the lane within a block

  // Positions are below 2^30 (checked on the host): 32 bits suffice.
  const int q_begin = (int)(it.chunk ? d.q_begin[1] : d.q_begin[0]);
  const int q_len = (int)(it.chunk ? d.q_len[1] : d.q_len[0]);
  const int64_t loff = it.chunk ? d.local_off[1] : d.local_off[0];  // Q row of the chunk's first query
  const int64_t ooff = it.chunk ? d.o_off[1] : d.o_off[0];          // its O / LSE row
  const int Hq = p.Hq;
  const int Hkv = p.Hkv;
  const int kvh = it.head_group / p.groups_per_kv;
  const int head0 = kvh * (Hq / Hkv) + (it.head_group % p.groups_per_kv) * p.heads_per_wg;
  const int qblocks_per_head = p.q_per_wg / kBlockRows;
  const int qb0 = it.q_block * p.q_per_wg;
  const int wg_last = (qb0 + p.q_per_wg < q_len ? qb0 + p.q_per_wg : q_len) - 1;
  const int wg_pos_hi = q_begin + wg_last;

  int head_b[NB];
  int qrel_b[NB];  // query index relative to the workgroup's first query
  bool valid_b[NB];
  int wave_lo = INT32_MAX, wave_hi = -1;
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const int bi = NB * wave + b;
    head_b[b] = head0 + bi / qblocks_per_head;
    const int qo = (bi % qblocks_per_head) * kBlockRows;
    qrel_b[b] = qo + l16;
    valid_b[b] = qb0 + qrel_b[b] < q_len;
    const int blo = qb0 + qo, bhi = (qb0 + qo + kBlockRows - 1 < wg_last ? qb0 + qo + kBlockRows - 1 : wg_last);
    if (blo <= wg_last) {
      wave_lo = (q_begin + blo < wave_lo) ? q_begin + blo : wave_lo;
      wave_hi = (q_begin + bhi > wave_hi) ? q_begin + bhi : wave_hi;
    }
  }
  const bool wave_active = wave_hi >= 0;

  // Key ranges (prefix, then the suffix ranges clipped to the workgroup's
  // last query) and their tiles.
  TileWalk tw;
  {
    const int nA = (d.prefix_keys + kTileKeys - 1) / kTileKeys;  // 0 when the prefix is not read
    tw.hiA = d.prefix_keys;
    tw.loB = (int)d.seg_lo[0];
    tw.hiB = (int)d.seg_hi[0];
    tw.visB = tw.hiB < wg_pos_hi + 1 ? tw.hiB : wg_pos_hi + 1;
    tw.loC = (int)d.seg_lo[1];
    tw.hiC = (int)d.seg_hi[1];
    tw.visC = tw.hiC < wg_pos_hi + 1 ? tw.hiC : wg_pos_hi + 1;
    const int nB = (d.n_seg > 0 && tw.visB > tw.loB) ? (tw.visB - tw.loB + kTileKeys - 1) / kTileKeys : 0;
    const int nC = (d.n_seg > 1 && tw.visC > tw.loC) ? (tw.visC - tw.loC + kTileKeys - 1) / kTileKeys : 0;
    tw.firstB = nA;
    tw.firstC = nA + nB;
    tw.n = nA + nB + nC;
  }
  const int n_tiles = tw.n;
  // This workgroup's share of the walk: all of it, or one piece.
  const int t_first = it.t_end < 0 ? 0 : it.t_begin;
  const int t_stop = it.t_end < 0 ? n_tiles : it.t_end;

  // A work item that sees no key at all (a KV shard entirely after its
  // queries) only writes its rows' empty result: O = 0, LSE = -inf.  The whole
  // workgroup takes this exit together (n_tiles is the workgroup's).
  if (n_tiles == 0) {
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      if (!valid_b[b]) continue;
      const int64_t row = ooff + qb0 + qrel_b[b];
      float* orow = d.o + (row * Hq + head_b[b]) * kHeadDim;
#pragma unroll
      for (int db = 0; db < 8; ++db)
        *reinterpret_cast<float4*>(orow + db * 16 + g4 * 4) = float4{0.f, 0.f, 0.f, 0.f};
      if (g4 == 0) d.lse[row * Hq + head_b[b]] = -INFINITY;
    }
    return;
  }

  // Within each range, the tiles from some index on need masking (they pass
  // the range end, cross the diagonal or start after the wave's last query);
  // the ones before are entirely visible to every query of the wave.  So a
  // tile needs masking exactly when its index lies in [mA, firstB),
  // [mB, firstC) or [mC, n).
  auto first_masked = [&](int first, int n, int lo, int hi) {
    if (!wave_active) return first;
    int k = ((wave_hi - lo) >> 5) + 1;                    // starts after the last query
    const int kd = ((wave_lo - lo - (kTileKeys - 1)) >> 5) + 1;  // crosses the diagonal
    const int kp = (hi - lo) >> 5;                        // passes the range end
    k = k < kd ? k : kd;
    k = k < kp ? k : kp;
    k = k < 0 ? 0 : (k > n ? n : k);
    return first + k;
  };
  static_assert(kTileKeys == 32, "tile index = key offset >> 5");
  const int mask_a = first_masked(0, tw.firstB, 0, tw.hiA);
  const int mask_b = first_masked(tw.firstB, tw.firstC - tw.firstB, tw.loB, tw.hiB);
  const int mask_c = first_masked(tw.firstC, tw.n - tw.firstC, tw.loC, tw.hiC);

  KvSource src;
  src.k_new = reinterpret_cast<const unsigned char*>(d.k_new);
  src.v_new = reinterpret_cast<const unsigned char*>(d.v_new);
  src.k_cache = reinterpret_cast<const unsigned char*>(d.k_cache);
  src.v_cache = reinterpret_cast<const unsigned char*>(d.v_cache);
  src.block_table = d.block_table;
  src.P = (int)d.P;
  src.n_blocks = (uint32_t)d.n_blocks;

  // Per-lane part of the tile load addresses (see prep_tile): column
  // 4(wave % 4) + lane / 16 of half wave / 4, slot lane % 16.
  const int row_stride = Hkv * kHeadDim * 2;
  const int lane_row = (wave >> 2) * 16 + ((lane & 15) ^ (8 * ((lane >> 4) & 1)));
  const uint32_t lane_col = (uint32_t)((4 * (wave & 3) + (lane >> 4)) * 16);
  const uint32_t lane_off = (uint32_t)(lane_row * row_stride) + lane_col;
  const uint32_t lds0 = lds_addr(smem);
  const uint32_t lk0 = lds0, lv0 = lds0 + kBufs * kTileBytes;
  // Tile t's load into buffer `buf` (= t % kBufs).  t past the last tile
  // loads the last tile again, into a buffer nobody reads, so that every
  // iteration issues the same loads and the waits can count them.
  auto load_of = [&](int t, int buf) {
    const int tt = t < n_tiles ? t : n_tiles - 1;
    return prep_tile(tile_at(tw, tt), src, kvh, row_stride, wave, lane_off, lane_row, lane_col,
                     lk0 + buf * kTileBytes, lv0 + buf * kTileBytes);
  };
  if (n_tiles > 0) issue_tile(load_of(t_first, t_first & (kBufs - 1)));

  // Query fragments (B operand of S^T = K Q^T, 32 head-dims x 16 queries):
  // lane 16g + i holds 8 consecutive head-dim values (8g .. 8g+7 of step ds)
  // of query i of each block, for each of the 4 steps of 32 along D.  Rows
  // past the chunk's end are zero and masked out of every tile.
  bf16x8 qf[NB][4];
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const int64_t qrow_i = loff + (valid_b[b] ? qb0 + qrel_b[b] : qb0);
    const __attribute__((address_space(1))) bf16x8* qrow =
        (const __attribute__((address_space(1))) bf16x8*)(d.q + (qrow_i * Hq + head_b[b]) * kHeadDim + g4 * 8);
#pragma unroll
    for (int ds = 0; ds < 4; ++ds) {
      const bf16x8 v = qrow[4 * ds];
      qf[b][ds] = valid_b[b] ? v : bf16x8{};
    }
  }
  // Query fragments and the first tile have landed (the builtin form lets
  // the compiler's own wait tracking see it); then the next kAhead-1 tiles
  // stream in.
  __builtin_amdgcn_s_waitcnt(kWaitVm(0));

  // Load cursor.  Within a suffix range a tile's rows are the previous
  // tile's plus 32, so the common tile load only advances two pointers.
  // The full computation is left to the tiles of the paged prefix (a block
  // lookup each), the first and the (possibly clamped) last tile of each
  // suffix range, and the repeats past the last tile; `cur_full` is the
  // next such tile.
  const int64_t tile_step = (int64_t)kTileKeys * row_stride;
  auto next_full = [fB = tw.firstB, fC = tw.firstC, n = n_tiles](int t) {
    if (t + 1 < fB) return t + 1;
    int f = n;
    f = sel(fB > t && fB < f, fB, f);
    f = sel(fC - 1 > t && fC - 1 < f, fC - 1, f);
    f = sel(fC > t && fC < f, fC, f);
    f = sel(n - 1 > t && n - 1 < f, n - 1, f);
    return sel(f > t, f, t + 1);
  };
  TileLoad cur = {};
  int cur_full = 0;
  if (n_tiles > 0) {
    for (int t = t_first + 1; t < t_first + kAhead; ++t) {
      cur = load_of(t, t & (kBufs - 1));
      issue_tile(cur);
    }
    cur_full = next_full(t_first + kAhead - 1);
  }
  const uint32_t wave_dst = (uint32_t)((wave >> 2) * kHalfBytes + (wave & 3) * 4 * kColBytes);

  const FragOffsets fo = frag_offsets(lane);
  const float sl2 = p.scale_log2;
  f32x4 o[8][NB];
  float m_run[NB];                            // running max (exponent units)
  float l_run[NB];                            // sum of the fp32 probabilities (lane's keys)
  // Sums of the bf16-rounded probabilities, by a 16x16x32 MFMA with an
  // all-ones A over each block's P fragment: every row of psum[b] holds the
  // sum over the tile's 32 keys of the lane's query, so every lane has its
  // query's full sum.
  f32x4 psum[NB];
  bf16x8 ones;
#pragma unroll
  for (int e = 0; e < 8; ++e) ones[e] = (__bf16)1.0f;
  bf16x8 pf[NB];                              // P of the previous tile
#pragma unroll
  for (int b = 0; b < NB; ++b) {
#pragma unroll
    for (int db = 0; db < 8; ++db) o[db][b] = f32x4{};
    m_run[b] = kNoMax;
    l_run[b] = 0.f;
    psum[b] = f32x4{};
    pf[b] = bf16x8{};
  }
  // Scores of the current tile alternate between two register sets.
  Scores<NB> sa, sb;
  const int q0 = q_begin + qb0;

  // The first iteration's P V step reads the V buffer before the first
  // tile's (its P is zero): fill that buffer with zeros so that the product
  // is zero too.  (No load writes it before the second pair's barrier.)
  static_assert(kTileBytes == 64 * kWaves * 16, "one 16-byte store per thread");
  *reinterpret_cast<u32x4*>(smem + (kBufs + ((t_first + kBufs - 1) & (kBufs - 1))) * kTileBytes + 16 * tid) =
      u32x4{};
  __syncthreads();  // the first tile is in LDS for everyone
  // A tile needs masking exactly when its index lies in [mA, firstB),
  // [mB, firstC) or [mC, n) (the thresholds below).  The tests between
  // regions (mask, cursor, overflow) are marked with their common outcome so
  // that it falls through: a taken branch costs the wave a fresh instruction
  // fetch, about 1 % of the launch.
  auto masked_tile = [&](int j) {
    return ((j >= mask_a) & (j < tw.firstB)) | ((j >= mask_b) & (j < tw.firstC)) | (j >= mask_c);
  };
  auto mask_if_needed = [&](int j, Scores<NB>& s) {
    if (__builtin_expect(masked_tile(j), 0)) {
      int lim[NB];
      tile_limits(tile_at(tw, j), q0, wave_active, wave_hi, qrel_b, valid_b, lim);
      mask_tile(s, g4, lim);
    }
  };
  bf16x8 pre[kLookahead<NB>];
  if (n_tiles > 0 && wave_active) {
#pragma unroll
    for (int g = 0; g < kLookahead<NB>; ++g)
      pre[g] = load_frag(g, smem + ((t_first + kBufs - 1) & (kBufs - 1)) * kTileBytes, smem, fo);
    // The first tile's scores, and the running max seeded with their max (so
    // that the first iteration's probabilities need no redo).
    qk_tile(smem + (t_first & (kBufs - 1)) * kTileBytes, fo, qf, sa);
    mask_if_needed(t_first, sa);
#pragma unroll
    for (int b = 0; b < NB; ++b) m_run[b] = __builtin_elementwise_maximum(tile_max(sa, b, sl2), kNoMax);
  }

  // Iteration j (tile buffer B = j % kBufs): mask
  // S_j, then the region (S_{j+1} from K buffer B+1, softmax of S_j, P_{j-1}
  // V_{j-1} from V buffer B-1, loads of tile j+kAhead into buffer
  // B+kAhead), then O's rescale if the max moved.  The last iteration
  // computes scores of the tile after its own from the repeated last tile
  // (finite data, unused).
  // This wave's share of the load that iteration j issues (tile j+kAhead).
  auto next_load = [&](int j) {
    const int t = j + kAhead, buf = t & (kBufs - 1);
    TileLoad ld;
    if (__builtin_expect(t >= cur_full, 0)) {
      ld = load_of(t, buf);
      cur_full = next_full(t);
    } else {
      ld.kb = cur.kb + tile_step;
      ld.vb = cur.vb + tile_step;
      ld.off = lane_off;
      ld.lk = lk0 + buf * kTileBytes + wave_dst;
      ld.lv = lv0 + buf * kTileBytes + wave_dst;
    }
    cur = ld;
    return ld;
  };
  auto iteration = [&](int j, Scores<NB>& s_in, Scores<NB>& s_out) {
    const int B = j & (kBufs - 1);
    mask_if_needed(j, s_in);
    const TileLoad ld = next_load(j);
    SoftmaxState<NB> st;
    pipelined_region(smem + ((B + kBufs - 1) % kBufs) * kTileBytes, smem + ((B + 1) % kBufs) * kTileBytes,
                     smem + B * kTileBytes, fo, qf, pf, o, s_in, s_out, m_run, sl2, ld, st, pre, ones, psum);
    // Rare: some lane's probabilities were too large (its max grew by more
    // than ~2^13, or it saw its first key).  Redo the tile exactly; its K
    // tile is still in buffer B (tile j + 8 is loaded three iterations on).
    bool ok = true;
#pragma unroll
    for (int b = 0; b < NB; ++b) ok = ok && st.rs[b] <= kMaxTileSum;
    if (__builtin_expect(__builtin_amdgcn_ballot_w64(!ok) != 0, 0)) {
      qk_tile(smem + B * kTileBytes, fo, qf, s_in);
      mask_if_needed(j, s_in);
      exact_softmax(s_in, m_run, l_run, psum, o, sl2, st);
    }
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      l_run[b] += st.rs[b];
      pf[b] = __builtin_shufflevector(__builtin_shufflevector(st.pp[b][0], st.pp[b][1], 0, 1, 2, 3),
                                      __builtin_shufflevector(st.pp[b][2], st.pp[b][3], 0, 1, 2, 3), 0, 1, 2, 3,
                                      4, 5, 6, 7);
    }
  };

  // Iterations go in pairs behind one barrier.  At a pair's start every tile
  // up to j+2 must have landed (both iterations read the K tile after their
  // own); the two tiles issued after those may still be in flight.  After the
  // barrier every wave is also done with the iterations before the pair, the
  // last readers of the buffers its loads reuse (tile j+5 takes tile j-3's).
  // A wave with no query row in the work item (a query block cut short at a
  // chunk's end) computes nothing: it only loads its share of every tile and
  // keeps the workgroup's barriers.
  if (wave_active) {
    for (int j = t_first; j < t_stop; j += 2) {
      __builtin_amdgcn_s_waitcnt(kWaitVm(2 * kLoadsPerTile));
      __syncthreads();
      iteration(j, sa, sb);
      if (j + 1 >= t_stop) break;
      iteration(j + 1, sb, sa);
    }
  } else {
    for (int j = t_first; j < t_stop; j += 2) {
      __builtin_amdgcn_s_waitcnt(kWaitVm(2 * kLoadsPerTile));
      __syncthreads();
      issue_tile(next_load(j));
      if (j + 1 >= t_stop) break;
      issue_tile(next_load(j + 1));
    }
  }
  // No tile load may still be writing LDS when the workgroup ends.
  __builtin_amdgcn_s_waitcnt(kWaitVm(0));
  if (n_tiles > 0 && wave_active) pv_tile(smem + ((t_stop - 1) & (kBufs - 1)) * kTileBytes, fo, pf, o, ones, psum);

  // Normalise and store: O^T register r of (db, b) is head-dim 16db + 4g + r
  // of this lane's query of block b.
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const float lt = quad_sum(l_run[b]);
    const float ltb = psum[b][0];
    const bool live = (m_run[b] > 0.5f * kNoMax) && (lt > 0.f) && (ltb > 0.f);
    const float inv = live ? 1.f / ltb : 0.f;
    const float lse = live ? m_run[b] * kLn2 + logf(lt) : -INFINITY;
    float* orow;
    float* lrow;
    if (it.piece >= 0) {
      // One piece of a split walk: its partial over its keys goes to the
      // piece slot (row 16 * block + query of the work item).
      unsigned char* slot = p.pieces + (size_t)it.piece * piece_bytes(kWaves * kBlockRows * NB);
      const int r = (NB * wave + b) * kBlockRows + l16;
      orow = reinterpret_cast<float*>(slot) + (size_t)r * kHeadDim;
      lrow = reinterpret_cast<float*>(slot + piece_o_bytes(kWaves * kBlockRows * NB)) + r;
    } else {
      if (!valid_b[b]) continue;
      const int64_t row = ooff + qb0 + qrel_b[b];
      orow = d.o + (row * Hq + head_b[b]) * kHeadDim;
      lrow = d.lse + row * Hq + head_b[b];
    }
#pragma unroll
    for (int db = 0; db < 8; ++db) {
      float4 v;
      v.x = o[db][b][0] * inv;
      v.y = o[db][b][1] * inv;
      v.z = o[db][b][2] * inv;
      v.w = o[db][b][3] * inv;
      *reinterpret_cast<float4*>(orow + db * 16 + g4 * 4) = v;
    }
    if (g4 == 0) *lrow = lse;
  }
}

// Exact combination of a split work item's pieces (disjoint key sets of the
// same rows): LSE = M + ln sum_k e^{LSE_k - M}, O = sum_k e^{LSE_k - LSE} O_k,
// a piece with LSE_k = -inf weighing 0 (and not read).  Each row of the item
// is written to the descriptor's output where the unsplit item would have
// written it.  32 lanes per row (float4 each), 8 rows per 256-thread block,
// rows_per_wg / 8 blocks per split item.
constexpr int kMergeRowsPerBlock = 8;

__global__ __launch_bounds__(256) void split_merge_kernel(const DevDesc* __restrict__ descs,
                                                          const SplitItem* __restrict__ splits, PartialParams p) {
  const int blocks_per_item = p.rows_per_wg / kMergeRowsPerBlock;
  const size_t slot_bytes = piece_bytes(p.rows_per_wg), o_bytes = piece_o_bytes(p.rows_per_wg);
  const SplitItem sp = splits[blockIdx.x / blocks_per_item];
  const int r = (blockIdx.x % blocks_per_item) * kMergeRowsPerBlock + (threadIdx.x >> 5);
  const int lane = threadIdx.x & 31;
  const DevDesc& d = descs[sp.desc];
  // The row's place, as the attention kernel assigns it (block bi, query l16).
  const int bi = r >> 4, l16 = r & 15;
  const int qblocks_per_head = p.q_per_wg >> 4;
  const int kvh = sp.head_group / p.groups_per_kv;
  const int head = kvh * (p.Hq / p.Hkv) + (sp.head_group % p.groups_per_kv) * p.heads_per_wg + bi / qblocks_per_head;
  const int qrel = (bi % qblocks_per_head) * 16 + l16;
  const int64_t qb0 = (int64_t)sp.q_block * p.q_per_wg;
  const int64_t q_len = sp.chunk ? d.q_len[1] : d.q_len[0];
  if (qb0 + qrel >= q_len) return;
  const int64_t row = (sp.chunk ? d.o_off[1] : d.o_off[0]) + qb0 + qrel;

  float m = -INFINITY;
  for (int k = 0; k < sp.n_pieces; ++k) {
    const unsigned char* slot = p.pieces + (size_t)(sp.first_piece + k) * slot_bytes;
    m = fmaxf(m, reinterpret_cast<const float*>(slot + o_bytes)[r]);
  }
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  float lse = -INFINITY;
  if (m != -INFINITY) {
    float total = 0.f;
    for (int k = 0; k < sp.n_pieces; ++k) {
      const unsigned char* slot = p.pieces + (size_t)(sp.first_piece + k) * slot_bytes;
      const float lk = reinterpret_cast<const float*>(slot + o_bytes)[r];
      if (lk == -INFINITY) continue;
      const float w = expf(lk - m);
      total += w;
      const float4 v = reinterpret_cast<const float4*>(slot)[(size_t)r * (kHeadDim / 4) + lane];
      acc.x += w * v.x;
      acc.y += w * v.y;
      acc.z += w * v.z;
      acc.w += w * v.w;
    }
    const float inv = 1.f / total;
    acc.x *= inv;
    acc.y *= inv;
    acc.z *= inv;
    acc.w *= inv;
    lse = m + logf(total);
  }
  reinterpret_cast<float4*>(d.o + (row * p.Hq + head) * kHeadDim)[lane] = acc;
  if (lane == 0) d.lse[row * p.Hq + head] = lse;
}

}  // namespace

int launch_partial(const PartialParams& p, void* stream) {
  if (p.n_items == 0) return CP_OK;
  if (p.rows_per_wg == kWaves * kBlockRows * 3)
    hipLaunchKernelGGL(attn_partial_kernel<3>, dim3((unsigned)p.n_items), dim3(64 * kWaves), 0, (hipStream_t)stream,
                       p.descs, p.items, p);
  else if (p.rows_per_wg == kWaves * kBlockRows * 2)
    hipLaunchKernelGGL(attn_partial_kernel<2>, dim3((unsigned)p.n_items), dim3(64 * kWaves), 0, (hipStream_t)stream,
                       p.descs, p.items, p);
  else
    return fail(CP_ERR_INVALID, "cp_attn_partial: unsupported workgroup shape");
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(CP_ERR_HIP, std::string("cp_attn_partial launch: ") + hipGetErrorString(e));
  if (p.n_splits > 0) {
    const unsigned blocks = (unsigned)p.n_splits * (unsigned)(p.rows_per_wg / kMergeRowsPerBlock);
    hipLaunchKernelGGL(split_merge_kernel, dim3(blocks), dim3(256), 0, (hipStream_t)stream, p.descs, p.splits, p);
    e = hipGetLastError();
    if (e != hipSuccess) return fail(CP_ERR_HIP, std::string("cp_attn_partial merge launch: ") + hipGetErrorString(e));
  }
  return CP_OK;
}

}  // namespace cpattn
