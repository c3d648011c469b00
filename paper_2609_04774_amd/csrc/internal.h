// Internal declarations shared by the host ABI code and the HIP kernels of
// libcpattn.  Not part of the public C ABI (that is include/cp_attn.h).
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <new>
#include <string>
#include <vector>

#include "cp_attn.h"

namespace cpattn {

// Records a failure reason for cp_last_error() and returns `status`.
int fail(int status, const std::string& why);
// The same without allocating: `why` must be a string literal.
int fail_static(int status, const char* why) noexcept;
void clear_error();

// Runs the body of an extern "C" entry point: a C++ exception thrown by the
// host code (std::bad_alloc from a container, say) becomes CP_ERR_HOST
// instead of crossing the C boundary, which would terminate the caller.
template <class F>
int guarded(F&& body) noexcept {
  try {
    return body();
  } catch (const std::bad_alloc&) {
    return fail_static(CP_ERR_HOST, "out of host memory");
  } catch (...) {
    return fail_static(CP_ERR_HOST, "internal error (C++ exception in the host code)");
  }
}

// Re-derives a plan from (P, R, C, rank); shared by cp_shard_plan and the
// descriptor checks of cp_attn_partial / cp_attn_merge.
int make_plan(int64_t P, int64_t R, int32_t C, int32_t rank, cp_rank_plan* out);
bool plan_equal(const cp_rank_plan& a, const cp_rank_plan& b);

// ---------------------------------------------------------------------------
// Partial attention: what one launch consumes.

constexpr int kHeadDim = 128;
constexpr int kBlockTokens = 16;
// (query, head) rows per workgroup: 8 waves of 2 or 3 blocks of 16 rows,
// chosen per launch by the host plan.
constexpr int kRowsSmall = 256;
constexpr int kRowsLarge = 384;

// One descriptor as the kernel reads it.  Key sets are expressed as global
// positions: the prefix [0, prefix_keys) through the block table, then up to
// two suffix ranges [seg_lo, seg_hi) read from k_new / v_new row (pos - P).
// A block-table entry outside [0, n_blocks) names no cache block: its 16
// keys and values read as zeros.
struct DevDesc {
  const uint16_t* q;
  const uint16_t* k_new;
  const uint16_t* v_new;
  const uint16_t* k_cache;
  const uint16_t* v_cache;
  const int32_t* block_table;
  float* o;
  float* lse;
  int64_t P;
  int64_t R;
  int64_t q_begin[2];
  int64_t q_len[2];
  int64_t local_off[2];  // Q row of each chunk's first query
  int64_t o_off[2];      // O / LSE row of each chunk's first query
  int64_t seg_lo[2];
  int64_t seg_hi[2];
  int32_t n_seg;
  int32_t prefix_keys;
  int32_t n_blocks;     // blocks of k_cache / v_cache (at most 2^31 - 1)
  int32_t reserved;
};

// One workgroup's unit: a block of query positions of one chunk of one
// descriptor, for one group of query heads sharing a KV head, over the key
// tiles [t_begin, t_end) of its walk (t_end < 0: the whole walk).  A work item
// whose walk is split over several workgroups ("pieces") writes each piece's
// partial result to piece slot `piece` of the workspace; the pieces are then
// merged into the descriptor's output (split_merge).  piece < 0: the item
// writes its rows directly.
struct WorkItem {
  int32_t desc;
  int32_t chunk;
  int32_t q_block;
  int32_t head_group;
  int32_t t_begin;
  int32_t t_end;
  int32_t piece;
  int32_t reserved;
};

// A work item that was split: its pieces occupy slots [first_piece,
// first_piece + n_pieces).
struct SplitItem {
  int32_t desc;
  int32_t chunk;
  int32_t q_block;
  int32_t head_group;
  int32_t first_piece;
  int32_t n_pieces;
};

// Workspace of one piece of a work item of `rows` rows: fp32 O of its rows
// (row = 16 * block + query), then their LSE.
__host__ __device__ constexpr size_t piece_o_bytes(int rows) { return (size_t)rows * kHeadDim * 4; }
__host__ __device__ constexpr size_t piece_bytes(int rows) { return piece_o_bytes(rows) + (size_t)rows * 4; }

struct PartialParams {
  const DevDesc* descs;
  const WorkItem* items;
  int32_t n_items;
  int32_t Hq;
  int32_t Hkv;
  int32_t heads_per_wg;   // query heads of one KV head handled by one workgroup
  int32_t q_per_wg;       // query positions per workgroup (heads_per_wg * q_per_wg = rows_per_wg)
  int32_t groups_per_kv;  // (Hq / Hkv) / heads_per_wg
  float scale_log2;       // softmax scale * log2(e)
  float scale;            // softmax scale
  int32_t rows_per_wg;    // 256 or 384 (8 waves of two or three 16-row blocks)
  unsigned char* pieces;  // piece slots (kPieceBytes each), or null when nothing is split
  const SplitItem* splits;
  int32_t n_splits;
};

int launch_partial(const PartialParams& p, void* stream);

// Copies `bytes` (a multiple of 16) from pinned host memory mapped into the
// device's address space to device memory, with a kernel on `stream`
// (upload.hip).
int launch_upload(void* dst, const void* src, size_t bytes, void* stream);

// Host planning of one cp_attn_partial launch (cp_attn.cpp), shared by the
// entry points that take a caller workspace and the one that uses the
// library's own scratch.
struct Shape {
  int rows_per_wg, heads_per_wg, q_per_wg, groups_per_kv;
};

struct Plan {
  std::vector<DevDesc> descs;
  std::vector<WorkItem> items;
  std::vector<SplitItem> splits;
  int64_t n_pieces = 0;
  Shape shape;
};

// Key walks of launches with few work items are split into about
// `target_pieces` pieces (0: never split).
constexpr int64_t kTargetPieces = 1024;
int build_plan(const cp_partial_desc* descs, int32_t n_descs, int32_t Hq, int32_t Hkv, int64_t target_pieces,
               Plan* out);

// Workspace layout: descriptors | work items | split items | piece slots.
// The first `pieces` bytes are uploaded from the host; the piece slots are
// written by the kernel before they are read.
struct Layout {
  size_t items, splits, pieces, total;
};
Layout layout_of(const Plan& plan);
void pack_tables(const Plan& plan, const Layout& lay, std::vector<unsigned char>* host);
PartialParams partial_params(const Plan& plan, const Layout& lay, unsigned char* ws, int32_t Hq, int32_t Hkv,
                             float scale);

// ---------------------------------------------------------------------------
// LSE merge.

struct MergeParams {
  const float* o[CP_MAX_MERGE_PARTS];
  const float* lse[CP_MAX_MERGE_PARTS];
  int32_t n_parts;
  int32_t n_heads;
  int64_t n_tokens;
  void* o_out;
  float* lse_out;
  int32_t out_bf16;
  int32_t restore;        // 1: map local row t to its suffix index
  int64_t first_len;      // rows of the rank's first chunk
  int64_t first_dst;      // suffix index of the first chunk's first row
  int64_t second_dst;     // suffix index of the second chunk's first row
};

int launch_merge(const MergeParams& p, void* stream);

// ---------------------------------------------------------------------------
// KV-cache steps after the attention: paged write-back, re-sharding and the
// paged gather.

struct WritebackParams {
  const unsigned char* k_rows;  // [n_rows][row_bytes]
  const unsigned char* v_rows;
  unsigned char* k_cache;       // [n_blocks][16][row_bytes]
  unsigned char* v_cache;
  const int32_t* block_table;
  int64_t n_blocks;
  int64_t row_bytes;            // Hkv * D * 2, a multiple of 16
  int64_t q_begin[2];           // global position of each chunk's first row
  int64_t q_len[2];             // rows of each chunk (chunk 0's rows come first)
  int64_t n_rows;
};

int launch_writeback(const WritebackParams& p, void* stream);

struct RepartitionParams {
  const unsigned char* src[CP_MAX_DEGREE];  // source rank r's rows
  unsigned char* dst;
  int64_t row_bytes;
  int64_t P, R;
  int64_t s_src;                // chunk length at the source degree
  int32_t C_src;
  int64_t dst_q_begin[2];       // the destination rank's chunks (global positions)
  int64_t dst_q_len[2];
  int64_t n_rows;
};

int launch_repartition(const RepartitionParams& p, void* stream);

// Every destination rank of up to two row sets in one launch: row i of the
// suffix (global position P + i) of set k goes from its source rank to its
// destination rank, both found in closed form from the two zigzag plans.
struct RepartitionAllParams {
  const unsigned char* src[2][CP_MAX_DEGREE];
  unsigned char* dst[2][CP_MAX_DEGREE];
  int64_t row_bytes;
  int64_t R;
  int64_t s_src, s_dst;         // chunk lengths at the two degrees
  int32_t C_src, C_dst;
  int32_t n_sets;
};

int launch_repartition_all(const RepartitionAllParams& p, void* stream);

struct GatherParams {
  const unsigned char* k_cache;  // [n_blocks][16][row_bytes]
  const unsigned char* v_cache;
  const int32_t* block_table;
  int64_t n_blocks;
  int64_t row_bytes;             // Hkv * D * 2, a multiple of 16
  int64_t pos_begin;             // position of output row 0
  int64_t n_rows;
  unsigned char* k_rows;         // [n_rows][row_bytes]
  unsigned char* v_rows;
};

int launch_gather(const GatherParams& p, void* stream);

}  // namespace cpattn
