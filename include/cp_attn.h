/*
 * cp_attn.h -- C ABI of libcpattn: one context-parallel (CP) rank's causal
 * prefill attention on an AMD Instinct MI355X (gfx950).
 *
 * The method (arXiv 2609.04774, "Adaptive Context Parallelism for Production
 * LLM Serving"):
 *   Sec. 2.1  Causal attention softmax(QK^T/sqrt(d_h) + M)V, M_ij = 0 for
 *             j <= i.  Zigzag CP: the sequence is padded to a multiple of 2C,
 *             cut into 2C equal contiguous chunks, and rank k holds chunks k
 *             and 2C-1-k; each rank attends its queries to every causally
 *             visible key and the outputs are restored to the original order.
 *   Sec. 2.2  With a prefix-cache hit L = P + R: only the R uncached tokens
 *             are computed, attending to the P cached keys and to the earlier
 *             uncached ones; the work is W(R,P) = RP + R(R+1)/2 pairs.
 *   Sec. 7.1  The cached prefix is a sequence of fixed-size cache blocks.
 *   Sec. 6.2, 7.2  After a worker split or merge, and for replication between
 *             workers of different CP degree, resident KV is re-sharded to
 *             the destination's CP geometry (and read out of the paged
 *             cache for the destination).
 *
 * Conventions shared by every call:
 *   - Tensors are dense, row-major, in device memory unless a pointer is
 *     documented as host memory.  bf16 is IEEE bfloat16 stored as uint16.
 *   - Positions: the cached prefix occupies global positions 0..P-1, the
 *     uncached suffix P..P+R-1 (suffix index i <-> global position P+i).
 *   - Zigzag is applied to the suffix only; padding sits at its end and is
 *     never a row.  A rank's rows are compact: chunk `rank` first, then chunk
 *     2C-1-rank, each in increasing position.
 *   - Grouped-query attention: query head h reads KV head h / (Hq/Hkv).
 *   - The head dimension D is 128; paged KV blocks hold 16 tokens.
 *   - Partial outputs are normalised: O = sum_j e^{x_j - LSE} v_j over the
 *     partial's keys, LSE = ln sum_j e^{x_j} (natural log, x_j = scale*q.k).
 *     A row that sees no key has O = 0 and LSE = -inf.
 *   - The caller owns every buffer and the stream.  No call allocates device
 *     memory, synchronises the device, or keeps pointers after returning
 *     (cp_attn_partial_noalloc waits for its stream before reusing its
 *     scratch, as it states).
 *     Launching calls are asynchronous on `stream` (a hipStream_t; NULL is the
 *     null stream) and return after host-side validation and the launch.
 *   - Errors: every call returns CP_OK (0) or a negative status, checks its
 *     arguments before launching anything, and launches nothing on error.
 *     No call throws: a host-side failure inside the library (exhausted
 *     host memory) is returned as CP_ERR_HOST.
 *     cp_last_error() gives a readable reason for the calling thread's last
 *     failure.  Block-table entries outside the cache are handled on the
 *     device as each call states (never read or written through); other
 *     device-side contents are not checked.
 */
#ifndef CP_ATTN_H_
#define CP_ATTN_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define CP_OK 0
#define CP_ERR_INVALID (-1)     /* bad argument (null, range, alignment, shape) */
#define CP_ERR_UNSUPPORTED (-2) /* well-formed but not built for (e.g. D != 128) */
#define CP_ERR_HIP (-3)         /* the HIP runtime reported an error */
#define CP_ERR_CAPACITY (-4)    /* a caller buffer is too small */
#define CP_ERR_HOST (-5)        /* host-side failure: out of host memory or an internal error */

#define CP_HEAD_DIM 128
#define CP_KV_BLOCK_TOKENS 16
#define CP_MAX_MERGE_PARTS 16
#define CP_MAX_DEGREE 64        /* largest CP degree C of any call */
#define CP_NOALLOC_SCRATCH_BYTES (32u << 20) /* device scratch of cp_attn_partial_noalloc, per GPU */

/* kv_rank values of cp_partial_desc besides a rank number 0..C-1. */
#define CP_KV_ALL (-1)  /* every causally visible suffix key (all-gathered KV) */
#define CP_KV_NONE (-2) /* no suffix key (prefix-only partial) */

/* Row order of a partial's outputs (cp_partial_desc.out_order). */
#define CP_OUT_LOCAL 0    /* the rank's rows in local order, as its queries */
#define CP_OUT_SEQUENCE 1 /* rows at their suffix index in an R-row output */

/* Static description of a status code.  (Library utility; not from the
 * paper.) */
const char* cp_status_string(int status);

/* Detail of the calling thread's most recent failing call ("" if none).
 * (Library utility; not from the paper.) */
const char* cp_last_error(void);

/* ---------------------------------------------------------------------- */
/* Shard plan (Sec. 2.1 zigzag, Sec. 2.2 prefix/suffix split) -- host only */

typedef struct cp_chunk {
  int32_t chunk_id;     /* 0..2C-1 */
  int32_t reserved;
  int64_t q_begin;      /* global position of the chunk's first token: P + chunk_id*chunk_len */
  int64_t q_len;        /* real (unpadded) tokens of the chunk: clamp(R - chunk_id*chunk_len, 0, chunk_len) */
  int64_t local_offset; /* first local row of the chunk in the rank's buffers */
} cp_chunk;

typedef struct cp_rank_plan {
  int32_t C;            /* CP degree */
  int32_t rank;         /* 0..C-1 */
  int64_t prefix_len;   /* P: cached tokens, global positions 0..P-1 */
  int64_t new_len;      /* R: uncached tokens, global positions P..P+R-1 */
  int64_t padded_len;   /* R rounded up to a multiple of 2C */
  int64_t chunk_len;    /* padded_len / 2C */
  int64_t n_rows;       /* chunk[0].q_len + chunk[1].q_len */
  cp_chunk chunk[2];    /* chunk `rank`, then chunk 2C-1-rank */
  int64_t visible_pairs;/* per head: sum over rows of (pos + 1), i.e. keys 0..pos */
} cp_rank_plan;

/*
 * Plan of rank `rank` of a degree-C worker for a request with P cached and R
 * uncached tokens (Sec. 2.1, 2.2).  Summed over the C ranks, visible_pairs is
 * W(R,P) = RP + R(R+1)/2.
 *   out      host, required; filled on success.
 *   row_pos  host, optional (NULL): receives the global position of every
 *            local row, out->n_rows entries; row_pos_cap is its capacity.
 * Errors: CP_ERR_INVALID if C < 1, C > CP_MAX_DEGREE, rank outside
 * 0..C-1, P < 0, R < 0, P > 2^31 or R > 2^31 (so that visible_pairs fits in
 * 64 bits) or out == NULL; CP_ERR_CAPACITY if row_pos != NULL and
 * row_pos_cap < n_rows.
 * R = 0 and R < 2C are legal (empty chunks have q_len = 0).
 */
int cp_shard_plan(int64_t prefix_len, int64_t new_len, int32_t C, int32_t rank,
                  cp_rank_plan* out, int64_t* row_pos, int64_t row_pos_cap);

/*
 * Restore map (Sec. 2.1): for each suffix index i in 0..R-1, the rank that
 * holds it and its local row there.  rank_of (int32) and row_of (int64) are
 * host arrays of capacity `cap` >= R.
 * Errors: CP_ERR_INVALID for bad P/R/C (as cp_shard_plan) or NULL arrays;
 * CP_ERR_CAPACITY if cap < R.
 */
int cp_shard_inverse(int64_t prefix_len, int64_t new_len, int32_t C,
                     int32_t* rank_of, int64_t* row_of, int64_t cap);

/* ---------------------------------------------------------------------- */
/* Partial attention (Sec. 2.1 causal attention of a rank's rows)          */

/*
 * One unit of partial-attention work: the rows of one rank (plan) against
 * one set of keys.  Pointers are device memory, 16-byte aligned (lse: 4).
 *   plan        from cp_shard_plan (checked against (P, R, C, rank)).
 *   q           bf16 [plan.n_rows][Hq][D]: the rank's query rows, local order.
 *   k_new,v_new bf16 [R][Hkv][D]: K/V of all R suffix tokens in original
 *               order (the all-gathered view; suffix index i = position P+i).
 *               Only rows of the selected suffix keys are read.  May be NULL
 *               when kv_rank == CP_KV_NONE or R == 0.
 *   k_cache,v_cache  bf16 [n_blocks][16][Hkv][D]: paged prefix cache.
 *   block_table int32 [P/16]: physical block of each logical prefix block.
 *               The three prefix pointers may be NULL unless include_prefix
 *               and P > 0; then P must be a multiple of 16.  An entry
 *               outside [0, n_blocks) names no block of the cache: its 16
 *               tokens' keys and values read as zeros (nothing is read
 *               through it), as in cp_kv_gather.
 *   include_prefix  1: rows attend to all P prefix keys; 0: to none.
 *   kv_rank     CP_KV_ALL: rows attend to every suffix key at or before them
 *               (the paper's all-gathered CP); r in 0..C-1: only to the suffix
 *               keys of rank r's two zigzag chunks (pass-KV partial; the C
 *               shards partition the suffix); CP_KV_NONE: to no suffix key.
 *   o           fp32 [rows][Hq][D], normalised partial output.
 *   lse         fp32 [rows][Hq], natural-log LSE (-inf: no key).
 *   n_blocks    blocks in k_cache and v_cache; >= 1 when the prefix is read.
 *               Values above 2^31 - 1 act as 2^31 - 1 (entries are int32).
 *   out_order   CP_OUT_LOCAL: o and lse have rows = plan.n_rows, the rank's
 *               rows in local order.  CP_OUT_SEQUENCE: o and lse have rows =
 *               R in the original suffix order (row i = position P + i) and
 *               the call writes only this rank's rows there -- the restore of
 *               Sec. 2.1 done by the attention's own stores, so a rank's one
 *               all-gathered partial needs no cp_attn_merge.  Other values:
 *               CP_ERR_INVALID.
 *   reserved    must be 0.
 * Merging (cp_attn_merge) the C pass-KV partials plus a prefix-only partial
 * gives the CP_KV_ALL result with include_prefix = 1.
 */
typedef struct cp_partial_desc {
  cp_rank_plan plan;
  const void* q;
  const void* k_new;
  const void* v_new;
  const void* k_cache;
  const void* v_cache;
  const int32_t* block_table;
  int32_t include_prefix;
  int32_t kv_rank;
  float* o;
  float* lse;
  int64_t n_blocks;
  int32_t out_order;
  int32_t reserved;
} cp_partial_desc;

/*
 * Sizing call of cp_attn_partial (Sec. 2.1, 2.2 partial attention; the
 * workspace itself is a library interface, not from the paper).
 * Device workspace bytes cp_attn_partial needs for this descriptor set: the
 * device copy of the descriptors and the scheduled work list, and, when the
 * set has few work items with long key walks (a short suffix over a long
 * cached prefix) or long items that do not divide evenly among the compute
 * units, one slot of rows x (128 + 1) fp32 per piece the walks are split
 * into (rows = 256 or 384, the launch's workgroup size; about a thousand
 * pieces at most).  Deterministic in the descriptors, the head counts and
 * the cp_set_workgroup_rows setting.  0 on invalid arguments (and
 * cp_last_error says why).
 */
size_t cp_attn_partial_workspace_size(const cp_partial_desc* descs, int32_t n_descs,
                                      int32_t n_heads_q, int32_t n_heads_kv);

/*
 * Partial attention of every descriptor (Sec. 2.1: each rank's local queries
 * against the causally visible keys; Sec. 2.2: the cached prefix's keys
 * included), in one kernel launch, plus, when key walks were split, one
 * launch that combines each walk's pieces with the log-sum-exp identity
 * cp_attn_merge applies (exact: the pieces cover disjoint key sets).
 *   descs       host array of n_descs descriptors (read during the call only);
 *               n_descs == 0 is a no-op.  Descriptors may come from different
 *               requests (ragged lengths); output buffers must not overlap.
 *   n_heads_q, n_heads_kv  Hq and Hkv, Hq % Hkv == 0.
 *   head_dim    must be 128 (else CP_ERR_UNSUPPORTED).
 *   softmax_scale  <= 0 selects 1/sqrt(head_dim) (the paper's 1/sqrt(d_h)).
 *   workspace   device buffer of workspace_bytes >= the size above; it is
 *               written by an asynchronous copy on `stream` and read by the
 *               kernel, so it must not be reused until the stream reaches
 *               this work.
 * The work list is planned on the host; the lists of the last 16 launches
 * are kept (keyed by every non-pointer field of the descriptors, the head
 * counts and the pinned workgroup shape, matched exactly), so a launch of
 * the same geometry with other buffers, such as the next layer's, reuses its
 * list instead of planning it again.
 * Each call stages the descriptor copy through pinned host memory owned by
 * the library (allocated on first use, kept until process exit), in a ring
 * of eight slots, and a small kernel on `stream` copies it into the
 * workspace: a call that finds its slot's previous copy not yet done blocks
 * the calling host thread on that copy's event (never on the whole device)
 * before reusing the slot.
 * Errors: CP_ERR_INVALID (shapes, plans, pointers, alignment, kv_rank),
 * CP_ERR_UNSUPPORTED (head_dim; a request with P + R > 2^30 tokens),
 * CP_ERR_CAPACITY (workspace), CP_ERR_HIP.
 */
int cp_attn_partial(const cp_partial_desc* descs, int32_t n_descs, int32_t n_heads_q,
                    int32_t n_heads_kv, int32_t head_dim, float softmax_scale,
                    void* workspace, size_t workspace_bytes, void* stream);

/*
 * Tuning control of cp_attn_partial's work decomposition (a library
 * interface, not from the paper).  Each launch runs workgroups of 256 or
 * 384 (query, head) rows -- 8 waves of two or three 16-row blocks; the
 * larger shares each K/V tile between more rows, the smaller fills the
 * compute units better when the launch has few or evenly long work items --
 * and by default (rows = 0) the host plan picks the one whose simulated
 * schedule ends first.  rows = 256 or 384 pins that shape for every later
 * call in the process (reproducible timings, tests of each kernel shape);
 * results agree within rounding either way.  Process-wide; takes effect at
 * the next call.
 * Errors: CP_ERR_INVALID for any other value.
 */
int cp_set_workgroup_rows(int32_t rows);

/*
 * cp_attn_partial for callers that cannot allocate: code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation.  It takes
 * no workspace and calls no allocating routine (no hipMalloc, hipFree or
 * pinned host allocation); its device scratch -- the descriptor copy, the
 * work list and the split-walk piece slots -- is a library-owned array of
 * CP_NOALLOC_SCRATCH_BYTES (32 MiB) on each GPU it runs on, held until the
 * process ends.  Descriptors, arguments and results are those of
 * cp_attn_partial; when split key walks would need more piece slots than
 * the scratch holds, fewer, longer pieces are used (same attention, other
 * work decomposition).
 * Each call waits on the host for `stream`'s earlier work before it
 * overwrites the scratch, then copies the tables from host memory (a
 * synchronous copy), so consecutive calls on one stream are safe.  The
 * scratch is shared by every call on a GPU and keeps the last call's
 * contents: calls that overlap on one GPU (other streams or threads) race.
 * Errors: as cp_attn_partial, plus CP_ERR_CAPACITY when the launch's tables
 * alone exceed the scratch (cp_attn_partial with a workspace has no limit).
 */
int cp_attn_partial_noalloc(const cp_partial_desc* descs, int32_t n_descs, int32_t n_heads_q,
                            int32_t n_heads_kv, int32_t head_dim, float softmax_scale, void* stream);

/* ---------------------------------------------------------------------- */
/* Exact log-sum-exp merge of partials (+ optional restore of order)      */

/*
 * Merge n_parts partials of the same rows that were computed over disjoint
 * key sets:  LSE = ln sum_i e^{LSE_i},  O = sum_i e^{LSE_i - LSE} O_i
 * (partials with LSE_i = -inf weigh 0; all -inf gives O = 0, LSE = -inf).
 * Source: the paper defines no partial outputs.  This is the exact identity
 * for a softmax over a union of disjoint key sets (the online-softmax
 * recurrence of Milakov & Gimelshein, 2018), which the ring-attention CP
 * scheme Sec. 2.1 cites as an alternative (Liu et al., 2024) needs to combine
 * the partials of successive KV shards.  With one partial and a restore plan
 * it is Sec. 2.1's final step alone: the rank's outputs put back in sequence
 * order, which concatenated over the ranks equals single-rank attention.
 *   o_parts, lse_parts  host arrays of n_parts device pointers (1..16):
 *               o_parts[i] fp32 [n_tokens][n_heads][D], lse_parts[i] fp32
 *               [n_tokens][n_heads].  n_parts == 1 copies (and restores).
 *   o_out       [n_out][n_heads][D], fp32, or bf16 when out_bf16 != 0.
 *   lse_out     fp32 [n_out][n_heads]; may be NULL.
 *   restore     host, optional: the plan the rows came from.  NULL: token t
 *               is written to row t (n_out = n_tokens).  Otherwise local row t
 *               of that rank is written to its suffix index (position - P),
 *               the Sec. 2.1 restore, so o_out is [R][n_heads][D] and every
 *               rank's merge can write into one shared output; n_tokens must
 *               equal restore->n_rows.
 * Errors: CP_ERR_INVALID (counts, NULL pointers, alignment, plan mismatch),
 * CP_ERR_UNSUPPORTED (head_dim != 128), CP_ERR_HIP.
 */
int cp_attn_merge(int32_t n_parts, const float* const* o_parts, const float* const* lse_parts,
                  int64_t n_tokens, int32_t n_heads, int32_t head_dim, void* o_out,
                  int32_t out_bf16, float* lse_out, const cp_rank_plan* restore, void* stream);

/*
 * Paged KV write-back: stores one CP rank's new K and V rows in the block-16
 * paged cache, where a later request's prefix hit reads them (Sec. 2.2:
 * prefill builds the KV states of its tokens and prefix caching keeps them
 * for later requests; Sec. 7.1: one trie node is one cache block; Sec. 8: the
 * destination installs KV states in physical blocks it reserved).
 *   plan        the rank's plan, as from cp_shard_plan (checked against it);
 *               plan->prefix_len must be a multiple of 16, so that new
 *               tokens never land in a block of the (shared) cached prefix.
 *   k_rows, v_rows  bf16 device [plan->n_rows][n_heads_kv][head_dim]: the
 *               rank's rows in plan order (row t is global position
 *               row_pos[t]).  16-byte aligned.
 *   n_heads_kv, head_dim  Hkv >= 1; head_dim a multiple of 8.
 *   k_cache, v_cache  bf16 device [n_blocks][16][n_heads_kv][head_dim].
 *   block_table int32 device [table_len]: physical block of each logical
 *               block of the request; position p goes to block
 *               block_table[p / 16], slot p % 16.  table_len must cover
 *               the request: table_len >= ceil((P + R) / 16).
 * Entries outside [0, n_blocks) are skipped on the device (nothing is
 * written for those rows); the ranks of one request write disjoint slots.
 * Errors: CP_ERR_INVALID (plan, pointers, alignment, prefix_len % 16,
 * table_len, shapes), CP_ERR_HIP.
 */
int cp_kv_writeback(const cp_rank_plan* plan, const void* k_rows, const void* v_rows,
                    int32_t n_heads_kv, int32_t head_dim, void* k_cache, void* v_cache,
                    int64_t n_blocks, const int32_t* block_table, int64_t table_len, void* stream);

/*
 * Re-shards one request's per-rank rows from CP degree C_src to degree C_dst
 * (Sec. 6.2: after a split or merge, resident KV is installed under the new
 * CP geometry; Sec. 7.2: inter-degree replication repartitions KV states for
 * the destination worker).  Row t of destination rank dst_rank (plan
 * cp_shard_plan(P, R, C_dst, dst_rank)) receives the row of the same global
 * position from the degree-C_src rank that holds it.  When 4C divides the
 * padded suffix, going between degrees C and 2C is pairwise: degree-2C ranks
 * 2k and 2k+1 draw only on degree-C rank k, and rank k only on them.
 *   src_rows    host array of C_src device pointers: rank r's rows
 *               [n_rows_r][row_bytes] in its plan order (NULL allowed for a
 *               rank with no rows).  16-byte aligned.
 *   dst_rows    device [n_rows_dst][row_bytes]; must not overlap a source.
 *   row_bytes   bytes per row, a positive multiple of 16 (K or V rows:
 *               Hkv * D * 2).
 *   1 <= C_src, C_dst <= CP_MAX_DEGREE, 0 <= dst_rank < C_dst.
 * Errors: CP_ERR_INVALID, CP_ERR_UNSUPPORTED (positions beyond 2^31),
 * CP_ERR_HIP.
 */
int cp_repartition(int64_t P, int64_t R, int32_t C_src, const void* const* src_rows, int32_t C_dst,
                   int32_t dst_rank, void* dst_rows, int64_t row_bytes, void* stream);

/*
 * cp_repartition for every destination rank at once, and for up to two row
 * sets (a request's K and V) in one launch (Sec. 6.2: after a split or merge
 * the resident KV is installed under the new CP geometry; Sec. 7.2:
 * inter-degree replication repartitions KV states for the destination).
 * Row t of set k of destination rank r receives the row of the same global
 * position from the degree-C_src rank that holds it, as cp_repartition(P, R,
 * C_src, set k's sources, C_dst, r, ...) would write it.
 *   src_rows   host array of n_sets * C_src device pointers: entry
 *              k * C_src + r is set k's rows of source rank r
 *              ([n_rows_r][row_bytes], plan order; NULL allowed for a rank
 *              with no rows).  16-byte aligned.
 *   dst_rows   host array of n_sets * C_dst device pointers: entry
 *              k * C_dst + r receives set k's rows of destination rank r
 *              ([n_rows_r][row_bytes]); no destination may overlap a source
 *              or another destination.  NULL allowed for a rank with no rows.
 *   n_sets     1 or 2.
 *   row_bytes  bytes per row, a positive multiple of 16.
 *   1 <= C_src, C_dst <= CP_MAX_DEGREE.  R == 0 is a no-op.
 * Errors: CP_ERR_INVALID, CP_ERR_UNSUPPORTED (positions beyond 2^31),
 * CP_ERR_HIP.
 */
int cp_repartition_all(int64_t P, int64_t R, int32_t C_src, const void* const* src_rows, int32_t C_dst,
                       void* const* dst_rows, int32_t n_sets, int64_t row_bytes, void* stream);

/*
 * Paged KV gather: copies positions pos_begin .. pos_begin + n_tokens - 1 of
 * one request out of the block-16 paged cache into contiguous rows.  It is
 * the read side of cp_kv_writeback and the same block-table gather that
 * cp_attn_partial performs tile by tile for a cached prefix (Sec. 2.2: a
 * prefix hit reuses the cached KV states; Sec. 7.1: one trie node is one
 * cache block), here as a standalone copy -- e.g. the KV states handed to a
 * worker of another CP degree on replication (Sec. 7.2).
 *   k_cache, v_cache  bf16 device [n_blocks][16][n_heads_kv][head_dim].
 *   block_table int32 device [table_len]: position p lives in block
 *               block_table[p / 16], slot p % 16; table_len must cover the
 *               range: table_len >= ceil((pos_begin + n_tokens) / 16).
 *   k_rows, v_rows  bf16 device [n_tokens][n_heads_kv][head_dim], written:
 *               row t is position pos_begin + t.  16-byte aligned; must not
 *               overlap the caches.
 *   n_heads_kv, head_dim  Hkv >= 1; head_dim a positive multiple of 8.
 * A row whose block-table entry lies outside [0, n_blocks) is written as
 * zeros (nothing is read through such an entry).  n_tokens == 0 is a no-op.
 * Errors: CP_ERR_INVALID (pointers, alignment, shapes, negative counts,
 * table_len), CP_ERR_UNSUPPORTED (positions beyond 2^31), CP_ERR_HIP.
 */
int cp_kv_gather(const void* k_cache, const void* v_cache, int64_t n_blocks, const int32_t* block_table,
                 int64_t table_len, int64_t pos_begin, int64_t n_tokens, int32_t n_heads_kv,
                 int32_t head_dim, void* k_rows, void* v_rows, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* CP_ATTN_H_ */
