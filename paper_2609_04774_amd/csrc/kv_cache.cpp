// Host side of the KV-cache steps after the attention: argument checks and
// kernel parameters for cp_kv_writeback, cp_repartition and cp_kv_gather
// (include/cp_attn.h).
#include <cstdint>
#include <cstring>
#include <string>

#include "internal.h"

using namespace cpattn;

namespace {

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

}  // namespace

extern "C" int cp_kv_writeback(const cp_rank_plan* plan, const void* k_rows, const void* v_rows, int32_t n_heads_kv,
                               int32_t head_dim, void* k_cache, void* v_cache, int64_t n_blocks,
                               const int32_t* block_table, int64_t table_len, void* stream) {
  return guarded([&]() -> int {
    const std::string who = "cp_kv_writeback: ";
    if (!plan) return fail(CP_ERR_INVALID, who + "plan is NULL");
    cp_rank_plan ref;
    if (make_plan(plan->prefix_len, plan->new_len, plan->C, plan->rank, &ref) != CP_OK || !plan_equal(ref, *plan))
      return fail(CP_ERR_INVALID, who + "plan does not match cp_shard_plan");
    if (plan->prefix_len % CP_KV_BLOCK_TOKENS)
      return fail(CP_ERR_INVALID, who + "prefix_len must be a multiple of 16");
    if (n_heads_kv < 1 || head_dim < 8 || head_dim % 8)
      return fail(CP_ERR_INVALID, who + "n_heads_kv must be >= 1 and head_dim a positive multiple of 8");
    const int64_t total = plan->prefix_len + plan->new_len;
    if (table_len < (total + CP_KV_BLOCK_TOKENS - 1) / CP_KV_BLOCK_TOKENS)
      return fail(CP_ERR_INVALID, who + "block table shorter than ceil((P + R) / 16)");
    if (n_blocks < 0) return fail(CP_ERR_INVALID, who + "n_blocks < 0");
    if (plan->n_rows > 0) {
      if (!k_rows || !v_rows || !k_cache || !v_cache || !block_table)
        return fail(CP_ERR_INVALID, who + "rows, caches and block table are required");
      if (!aligned(k_rows, 16) || !aligned(v_rows, 16) || !aligned(k_cache, 16) || !aligned(v_cache, 16) ||
          !aligned(block_table, 4))
        return fail(CP_ERR_INVALID, who + "rows/caches must be 16-byte and the block table 4-byte aligned");
    }
    WritebackParams p;
    std::memset(&p, 0, sizeof(p));
    p.k_rows = static_cast<const unsigned char*>(k_rows);
    p.v_rows = static_cast<const unsigned char*>(v_rows);
    p.k_cache = static_cast<unsigned char*>(k_cache);
    p.v_cache = static_cast<unsigned char*>(v_cache);
    p.block_table = block_table;
    p.n_blocks = n_blocks;
    p.row_bytes = (int64_t)n_heads_kv * head_dim * 2;
    for (int c = 0; c < 2; ++c) {
      p.q_begin[c] = plan->chunk[c].q_begin;
      p.q_len[c] = plan->chunk[c].q_len;
    }
    p.n_rows = plan->n_rows;
    const int st = launch_writeback(p, stream);
    if (st == CP_OK) clear_error();
    return st;
  });
}

extern "C" int cp_repartition(int64_t P, int64_t R, int32_t C_src, const void* const* src_rows, int32_t C_dst,
                              int32_t dst_rank, void* dst_rows, int64_t row_bytes, void* stream) {
  return guarded([&]() -> int {
    const std::string who = "cp_repartition: ";
    if (C_src < 1 || C_src > CP_MAX_DEGREE || C_dst < 1 || C_dst > CP_MAX_DEGREE)
      return fail(CP_ERR_INVALID, who + "degrees must be 1..64");
    if (dst_rank < 0 || dst_rank >= C_dst) return fail(CP_ERR_INVALID, who + "dst_rank out of range");
    if (row_bytes <= 0 || row_bytes % 16) return fail(CP_ERR_INVALID, who + "row_bytes must be a positive multiple of 16");
    if (P < 0 || R < 0) return fail(CP_ERR_INVALID, who + "P and R must be >= 0");
    if (P + R > ((int64_t)1 << 31)) return fail(CP_ERR_UNSUPPORTED, who + "positions beyond 2^31");
    cp_rank_plan dst;
    if (make_plan(P, R, C_dst, dst_rank, &dst) != CP_OK) return fail(CP_ERR_INVALID, who + "invalid (P, R, C_dst)");
    RepartitionParams p;
    std::memset(&p, 0, sizeof(p));
    if (dst.n_rows > 0) {
      if (!src_rows) return fail(CP_ERR_INVALID, who + "src_rows is NULL");
      if (!dst_rows || !aligned(dst_rows, 16)) return fail(CP_ERR_INVALID, who + "dst_rows NULL or not 16-byte aligned");
      for (int r = 0; r < C_src; ++r) {
        cp_rank_plan src;
        if (make_plan(P, R, C_src, r, &src) != CP_OK) return fail(CP_ERR_INVALID, who + "invalid (P, R, C_src)");
        if (src.n_rows > 0 && (!src_rows[r] || !aligned(src_rows[r], 16)))
          return fail(CP_ERR_INVALID, who + "source rank " + std::to_string(r) + " rows NULL or not 16-byte aligned");
        p.src[r] = static_cast<const unsigned char*>(src_rows[r]);
      }
      cp_rank_plan src0;
      make_plan(P, R, C_src, 0, &src0);
      p.s_src = src0.chunk_len;
    }
    p.dst = static_cast<unsigned char*>(dst_rows);
    p.row_bytes = row_bytes;
    p.P = P;
    p.R = R;
    p.C_src = C_src;
    for (int c = 0; c < 2; ++c) {
      p.dst_q_begin[c] = dst.chunk[c].q_begin;
      p.dst_q_len[c] = dst.chunk[c].q_len;
    }
    p.n_rows = dst.n_rows;
    const int st = launch_repartition(p, stream);
    if (st == CP_OK) clear_error();
    return st;
  });
}

extern "C" int cp_repartition_all(int64_t P, int64_t R, int32_t C_src, const void* const* src_rows, int32_t C_dst,
                                  void* const* dst_rows, int32_t n_sets, int64_t row_bytes, void* stream) {
  return guarded([&]() -> int {
    const std::string who = "cp_repartition_all: ";
    if (C_src < 1 || C_src > CP_MAX_DEGREE || C_dst < 1 || C_dst > CP_MAX_DEGREE)
      return fail(CP_ERR_INVALID, who + "degrees must be 1..64");
    if (n_sets < 1 || n_sets > 2) return fail(CP_ERR_INVALID, who + "n_sets must be 1 or 2");
    if (row_bytes <= 0 || row_bytes % 16)
      return fail(CP_ERR_INVALID, who + "row_bytes must be a positive multiple of 16");
    if (P < 0 || R < 0) return fail(CP_ERR_INVALID, who + "P and R must be >= 0");
    if (P + R > ((int64_t)1 << 31)) return fail(CP_ERR_UNSUPPORTED, who + "positions beyond 2^31");
    if (R > 0 && (!src_rows || !dst_rows)) return fail(CP_ERR_INVALID, who + "src_rows / dst_rows is NULL");
    RepartitionAllParams p;
    std::memset(&p, 0, sizeof(p));
    cp_rank_plan pl;
    for (int k = 0; k < n_sets && R > 0; ++k) {
      for (int r = 0; r < C_src; ++r) {
        if (make_plan(P, R, C_src, r, &pl) != CP_OK) return fail(CP_ERR_INVALID, who + "invalid (P, R, C_src)");
        const void* ptr = src_rows[k * C_src + r];
        if (pl.n_rows > 0 && (!ptr || !aligned(ptr, 16)))
          return fail(CP_ERR_INVALID, who + "source set " + std::to_string(k) + " rank " + std::to_string(r) +
                                          " rows NULL or not 16-byte aligned");
        p.src[k][r] = static_cast<const unsigned char*>(ptr);
        p.s_src = pl.chunk_len;
      }
      for (int r = 0; r < C_dst; ++r) {
        if (make_plan(P, R, C_dst, r, &pl) != CP_OK) return fail(CP_ERR_INVALID, who + "invalid (P, R, C_dst)");
        void* ptr = dst_rows[k * C_dst + r];
        if (pl.n_rows > 0 && (!ptr || !aligned(ptr, 16)))
          return fail(CP_ERR_INVALID, who + "destination set " + std::to_string(k) + " rank " + std::to_string(r) +
                                          " rows NULL or not 16-byte aligned");
        p.dst[k][r] = static_cast<unsigned char*>(ptr);
        p.s_dst = pl.chunk_len;
      }
    }
    p.row_bytes = row_bytes;
    p.R = R;
    p.C_src = C_src;
    p.C_dst = C_dst;
    p.n_sets = n_sets;
    const int st = launch_repartition_all(p, stream);
    if (st == CP_OK) clear_error();
    return st;
  });
}

extern "C" int cp_kv_gather(const void* k_cache, const void* v_cache, int64_t n_blocks, const int32_t* block_table,
                            int64_t table_len, int64_t pos_begin, int64_t n_tokens, int32_t n_heads_kv,
                            int32_t head_dim, void* k_rows, void* v_rows, void* stream) {
  return guarded([&]() -> int {
    const std::string who = "cp_kv_gather: ";
    if (pos_begin < 0 || n_tokens < 0) return fail(CP_ERR_INVALID, who + "pos_begin and n_tokens must be >= 0");
    if (pos_begin + n_tokens > ((int64_t)1 << 31)) return fail(CP_ERR_UNSUPPORTED, who + "positions beyond 2^31");
    if (n_heads_kv < 1 || head_dim < 8 || head_dim % 8)
      return fail(CP_ERR_INVALID, who + "n_heads_kv must be >= 1 and head_dim a positive multiple of 8");
    if (n_blocks < 0) return fail(CP_ERR_INVALID, who + "n_blocks < 0");
    if (table_len < (pos_begin + n_tokens + CP_KV_BLOCK_TOKENS - 1) / CP_KV_BLOCK_TOKENS)
      return fail(CP_ERR_INVALID, who + "block table shorter than ceil((pos_begin + n_tokens) / 16)");
    if (n_tokens > 0) {
      if (!k_rows || !v_rows || !k_cache || !v_cache || !block_table)
        return fail(CP_ERR_INVALID, who + "rows, caches and block table are required");
      if (!aligned(k_rows, 16) || !aligned(v_rows, 16) || !aligned(k_cache, 16) || !aligned(v_cache, 16) ||
          !aligned(block_table, 4))
        return fail(CP_ERR_INVALID, who + "rows/caches must be 16-byte and the block table 4-byte aligned");
    }
    GatherParams p;
    std::memset(&p, 0, sizeof(p));
    p.k_cache = static_cast<const unsigned char*>(k_cache);
    p.v_cache = static_cast<const unsigned char*>(v_cache);
    p.block_table = block_table;
    p.n_blocks = n_blocks;
    p.row_bytes = (int64_t)n_heads_kv * head_dim * 2;
    p.pos_begin = pos_begin;
    p.n_rows = n_tokens;
    p.k_rows = static_cast<unsigned char*>(k_rows);
    p.v_rows = static_cast<unsigned char*>(v_rows);
    const int st = launch_gather(p, stream);
    if (st == CP_OK) clear_error();
    return st;
  });
}
