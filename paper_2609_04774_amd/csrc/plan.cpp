// Zigzag shard plan (paper Sec. 2.1) over the uncached suffix of a request
// with a cached prefix (Sec. 2.2), plus status/error reporting.
//
// Rule: pad R to a multiple of 2C, cut into 2C equal chunks of chunk_len;
// rank k holds chunks k and 2C-1-k.  Padding sits at the end of the suffix
// and is not a row, so chunk c holds clamp(R - c*chunk_len, 0, chunk_len)
// real tokens.  Rows of a rank are compact: chunk k's, then chunk 2C-1-k's.
// Integer arithmetic only; every value is exact.
#include <cstring>
#include <string>

#include "internal.h"

namespace cpattn {

static thread_local std::string g_last_error;
static thread_local const char* g_last_static = nullptr;  // set when the message is a literal

int fail(int status, const std::string& why) {
  g_last_static = nullptr;
  g_last_error = why;
  return status;
}

int fail_static(int status, const char* why) noexcept {
  g_last_static = why;
  return status;
}

void clear_error() {
  g_last_static = nullptr;
  g_last_error.clear();
}

static int64_t clamp64(int64_t x, int64_t lo, int64_t hi) { return x < lo ? lo : (x > hi ? hi : x); }

// Sum of (pos + 1) over pos in [lo, lo + n): keys 0..pos are visible to the
// query at pos.  Evaluated as n*lo + n(n+1)/2 in 128-bit to avoid overflow.
static int64_t pairs_of_range(int64_t lo, int64_t n) {
  __int128 v = (__int128)n * lo + ((__int128)n * (n + 1)) / 2;
  return (int64_t)v;
}

int make_plan(int64_t P, int64_t R, int32_t C, int32_t rank, cp_rank_plan* out) {
  if (!out) return fail(CP_ERR_INVALID, "cp_shard_plan: out is NULL");
  if (C < 1) return fail(CP_ERR_INVALID, "cp_shard_plan: C must be >= 1");
  if (C > CP_MAX_DEGREE) return fail(CP_ERR_INVALID, "cp_shard_plan: C must be <= CP_MAX_DEGREE (64)");
  if (rank < 0 || rank >= C) return fail(CP_ERR_INVALID, "cp_shard_plan: rank outside 0..C-1");
  if (P < 0 || R < 0) return fail(CP_ERR_INVALID, "cp_shard_plan: negative prefix or suffix length");
  // P, R <= 2^31 keeps visible_pairs (< R P + R^2) below 2^63.
  if (R > ((int64_t)1 << 31) || P > ((int64_t)1 << 31))
    return fail(CP_ERR_INVALID, "cp_shard_plan: prefix or suffix beyond 2^31 tokens");
  const int64_t two_c = 2 * (int64_t)C;
  const int64_t s = (R + two_c - 1) / two_c;
  cp_rank_plan p;
  std::memset(&p, 0, sizeof(p));
  p.C = C;
  p.rank = rank;
  p.prefix_len = P;
  p.new_len = R;
  p.padded_len = s * two_c;
  p.chunk_len = s;
  const int64_t ids[2] = {rank, two_c - 1 - rank};
  int64_t rows = 0, pairs = 0;
  for (int i = 0; i < 2; ++i) {
    const int64_t start = ids[i] * s;
    const int64_t len = clamp64(R - start, 0, s);
    p.chunk[i].chunk_id = (int32_t)ids[i];  // below 2 * CP_MAX_DEGREE
    p.chunk[i].q_begin = P + start;
    p.chunk[i].q_len = len;
    p.chunk[i].local_offset = rows;
    rows += len;
    pairs += pairs_of_range(P + start, len);
  }
  p.n_rows = rows;
  p.visible_pairs = pairs;
  *out = p;
  return CP_OK;
}

bool plan_equal(const cp_rank_plan& a, const cp_rank_plan& b) {
  if (a.C != b.C || a.rank != b.rank || a.prefix_len != b.prefix_len || a.new_len != b.new_len ||
      a.padded_len != b.padded_len || a.chunk_len != b.chunk_len || a.n_rows != b.n_rows ||
      a.visible_pairs != b.visible_pairs)
    return false;
  for (int i = 0; i < 2; ++i) {
    if (a.chunk[i].chunk_id != b.chunk[i].chunk_id || a.chunk[i].q_begin != b.chunk[i].q_begin ||
        a.chunk[i].q_len != b.chunk[i].q_len || a.chunk[i].local_offset != b.chunk[i].local_offset)
      return false;
  }
  return true;
}

}  // namespace cpattn

using namespace cpattn;

extern "C" const char* cp_status_string(int status) {
  switch (status) {
    case CP_OK: return "ok";
    case CP_ERR_INVALID: return "invalid argument";
    case CP_ERR_UNSUPPORTED: return "unsupported configuration";
    case CP_ERR_HIP: return "HIP runtime error";
    case CP_ERR_CAPACITY: return "buffer too small";
    case CP_ERR_HOST: return "host-side failure";
    default: return "unknown status";
  }
}

extern "C" const char* cp_last_error(void) { return g_last_static ? g_last_static : g_last_error.c_str(); }

extern "C" int cp_shard_plan(int64_t prefix_len, int64_t new_len, int32_t C, int32_t rank,
                             cp_rank_plan* out, int64_t* row_pos, int64_t row_pos_cap) {
  return guarded([&]() -> int {
    cp_rank_plan p;
    int st = make_plan(prefix_len, new_len, C, rank, &p);
    if (st != CP_OK) return st;
    if (!out) return fail(CP_ERR_INVALID, "cp_shard_plan: out is NULL");
    if (row_pos) {
      if (row_pos_cap < p.n_rows) return fail(CP_ERR_CAPACITY, "cp_shard_plan: row_pos_cap < n_rows");
      int64_t r = 0;
      for (int i = 0; i < 2; ++i)
        for (int64_t t = 0; t < p.chunk[i].q_len; ++t) row_pos[r++] = p.chunk[i].q_begin + t;
    }
    *out = p;
    clear_error();
    return CP_OK;
  });
}

extern "C" int cp_shard_inverse(int64_t prefix_len, int64_t new_len, int32_t C, int32_t* rank_of,
                                int64_t* row_of, int64_t cap) {
  return guarded([&]() -> int {
    if (!rank_of || !row_of) return fail(CP_ERR_INVALID, "cp_shard_inverse: NULL output array");
    if (C < 1) return fail(CP_ERR_INVALID, "cp_shard_inverse: C must be >= 1");
    cp_rank_plan p;
    int st = make_plan(prefix_len, new_len, C, 0, &p);
    if (st != CP_OK) return st;
    if (cap < new_len) return fail(CP_ERR_CAPACITY, "cp_shard_inverse: cap < R");
    // Walk each rank's rows and record where every suffix index went.
    for (int32_t r = 0; r < C; ++r) {
      make_plan(prefix_len, new_len, C, r, &p);
      for (int i = 0; i < 2; ++i) {
        const int64_t base = p.chunk[i].q_begin - prefix_len;
        for (int64_t t = 0; t < p.chunk[i].q_len; ++t) {
          rank_of[base + t] = r;
          row_of[base + t] = p.chunk[i].local_offset + t;
        }
      }
    }
    clear_error();
    return CP_OK;
  });
}
