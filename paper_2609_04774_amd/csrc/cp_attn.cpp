// Host side of the C ABI: argument checks, the per-launch work list, the
// staging of descriptors into the caller's workspace, and the launches.
//
// Work list.  Every descriptor contributes, per non-empty chunk of its rank,
// ceil(q_len / q_per_wg) query blocks times (Hkv * groups_per_kv) head
// groups.  Items are ordered longest first (visible keys per item), which
// makes the hardware's in-order workgroup dispatch an LPT schedule, and are
// interleaved so that item i lands on XCD i % 8 with all items of one KV head
// group on the same XCD: the workgroups streaming one head's K/V share that
// XCD's L2.
//
// Split key walks.  When a launch has few work items (a short suffix over a
// long cached prefix: few query rows, many keys each), the GPU's 256 compute
// units would mostly idle.  Then each item's walk of key tiles is cut into
// pieces of at least kMinPieceTiles tiles, aiming at about kTargetPieces
// pieces in all; each piece is its own workgroup and writes a partial result
// (O, LSE over its keys) to the workspace, and split_merge combines an item's
// pieces exactly (the same log-sum-exp combination as cp_attn_merge).
//
// Workgroup shape.  The attention kernel runs 256- or 384-row workgroups; the
// work list is built for both and the one whose simulated schedule ends first
// is launched (balance cuts and the estimate below).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <atomic>
#include <mutex>
#include <numeric>
#include <queue>
#include <string>
#include <vector>

#include "internal.h"

using namespace cpattn;

namespace {

constexpr int kXcds = 8;
constexpr size_t kItemsAlign = 256;

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

int gcd_int(int a, int b) {
  while (b) {
    int t = a % b;
    a = b;
    b = t;
  }
  return a;
}

Shape shape_for(int Hq, int Hkv, int rows) {
  const int G = Hq / Hkv;
  Shape s;
  s.rows_per_wg = rows;
  s.heads_per_wg = gcd_int(G, 8);
  s.q_per_wg = rows / s.heads_per_wg;
  s.groups_per_kv = G / s.heads_per_wg;
  return s;
}

int check_heads(int32_t Hq, int32_t Hkv, const char* who) {
  if (Hq < 1 || Hkv < 1) return fail(CP_ERR_INVALID, std::string(who) + ": head counts must be >= 1");
  if (Hq % Hkv) return fail(CP_ERR_INVALID, std::string(who) + ": n_heads_q must be a multiple of n_heads_kv");
  if (Hq > 4096) return fail(CP_ERR_UNSUPPORTED, std::string(who) + ": more than 4096 query heads");
  return CP_OK;
}

// Validates one descriptor and converts it to the kernel's form.
int to_dev(const cp_partial_desc& x, int idx, DevDesc* out) {
  const std::string who = "cp_attn_partial: desc " + std::to_string(idx) + ": ";
  const cp_rank_plan& pl = x.plan;
  cp_rank_plan ref;
  if (make_plan(pl.prefix_len, pl.new_len, pl.C, pl.rank, &ref) != CP_OK)
    return fail(CP_ERR_INVALID, who + "plan has invalid (P, R, C, rank)");
  if (!plan_equal(ref, pl)) return fail(CP_ERR_INVALID, who + "plan does not match cp_shard_plan(P, R, C, rank)");
  if (pl.n_rows > ((int64_t)1 << 31)) return fail(CP_ERR_UNSUPPORTED, who + "more than 2^31 rows");
  const int64_t P = pl.prefix_len, R = pl.new_len;
  // The kernel walks key and query positions in 32-bit arithmetic.
  if (P + R > ((int64_t)1 << 30)) return fail(CP_ERR_UNSUPPORTED, who + "sequence beyond 2^30 tokens");
  if (x.kv_rank < CP_KV_NONE || x.kv_rank >= pl.C) return fail(CP_ERR_INVALID, who + "kv_rank out of range");
  if (x.include_prefix != 0 && x.include_prefix != 1) return fail(CP_ERR_INVALID, who + "include_prefix must be 0 or 1");
  if (x.out_order != CP_OUT_LOCAL && x.out_order != CP_OUT_SEQUENCE)
    return fail(CP_ERR_INVALID, who + "out_order must be CP_OUT_LOCAL or CP_OUT_SEQUENCE");
  if (x.reserved != 0) return fail(CP_ERR_INVALID, who + "reserved must be 0");
  if (pl.n_rows > 0) {
    if (!x.q || !x.o || !x.lse) return fail(CP_ERR_INVALID, who + "q, o and lse are required");
    if (!aligned(x.q, 16) || !aligned(x.o, 16) || !aligned(x.lse, 4))
      return fail(CP_ERR_INVALID, who + "q/o must be 16-byte and lse 4-byte aligned");
  }
  const bool use_suffix = x.kv_rank != CP_KV_NONE && R > 0;
  if (use_suffix && pl.n_rows > 0) {
    if (!x.k_new || !x.v_new) return fail(CP_ERR_INVALID, who + "k_new and v_new are required");
    if (!aligned(x.k_new, 16) || !aligned(x.v_new, 16))
      return fail(CP_ERR_INVALID, who + "k_new/v_new must be 16-byte aligned");
  }
  const bool use_prefix = x.include_prefix && P > 0;
  if (use_prefix && pl.n_rows > 0) {
    if (P % CP_KV_BLOCK_TOKENS) return fail(CP_ERR_INVALID, who + "prefix_len must be a multiple of 16 when the prefix is read");
    if (!x.k_cache || !x.v_cache || !x.block_table)
      return fail(CP_ERR_INVALID, who + "k_cache, v_cache and block_table are required");
    if (!aligned(x.k_cache, 16) || !aligned(x.v_cache, 16) || !aligned(x.block_table, 4))
      return fail(CP_ERR_INVALID, who + "k_cache/v_cache must be 16-byte and block_table 4-byte aligned");
    if (P > INT32_MAX) return fail(CP_ERR_UNSUPPORTED, who + "prefix beyond 2^31 tokens");
    if (x.n_blocks < 1) return fail(CP_ERR_INVALID, who + "n_blocks must be >= 1 when the prefix is read");
  }
  DevDesc d;
  std::memset(&d, 0, sizeof(d));
  d.q = static_cast<const uint16_t*>(x.q);
  d.k_new = static_cast<const uint16_t*>(x.k_new);
  d.v_new = static_cast<const uint16_t*>(x.v_new);
  d.k_cache = static_cast<const uint16_t*>(x.k_cache);
  d.v_cache = static_cast<const uint16_t*>(x.v_cache);
  d.block_table = x.block_table;
  d.o = x.o;
  d.lse = x.lse;
  d.P = P;
  d.R = R;
  for (int i = 0; i < 2; ++i) {
    d.q_begin[i] = pl.chunk[i].q_begin;
    d.q_len[i] = pl.chunk[i].q_len;
    d.local_off[i] = pl.chunk[i].local_offset;
    // Sequence order: the chunk's first query is suffix index q_begin - P.
    d.o_off[i] = x.out_order == CP_OUT_SEQUENCE ? pl.chunk[i].q_begin - P : pl.chunk[i].local_offset;
  }
  d.prefix_keys = use_prefix ? (int32_t)P : 0;
  // Entries are int32: a cache of more blocks than that holds every entry.
  d.n_blocks = use_prefix ? (int32_t)std::min<int64_t>(x.n_blocks, INT32_MAX) : 0;
  d.n_seg = 0;
  if (use_suffix) {
    if (x.kv_rank == CP_KV_ALL) {
      d.seg_lo[0] = P;
      d.seg_hi[0] = P + R;
      d.n_seg = 1;
    } else {
      // Rank kv_rank's own suffix keys: its chunks kv_rank and 2C-1-kv_rank.
      const int64_t s = pl.chunk_len;
      const int64_t ids[2] = {x.kv_rank, 2 * (int64_t)pl.C - 1 - x.kv_rank};
      for (int i = 0; i < 2; ++i) {
        const int64_t lo = ids[i] * s;
        const int64_t hi = std::min(R, lo + s);
        if (hi > lo) {
          d.seg_lo[d.n_seg] = P + lo;
          d.seg_hi[d.n_seg] = P + hi;
          ++d.n_seg;
        }
      }
    }
  }
  *out = d;
  return CP_OK;
}

constexpr int64_t kSplitBelowItems = 512;  // split only launches with fewer non-empty items
constexpr int64_t kMinPieceTiles = 32;     // 1024 keys: the prologue and merge stay small
constexpr int64_t kMaxPieces = 64;
constexpr int kComputeUnits = 256;         // 8 XCDs x 32 compute units
constexpr int64_t kItemSetupTiles = 16;    // a workgroup's set-up and stores, in tile times
constexpr int64_t kMinBalancePiece = 256;  // tiles of the smaller part of a balance cut
constexpr double kBalanceSlack = 1.03;

// Balance cuts.  The hardware dispatches workgroups in list order to
// whichever compute unit frees up first, so a list sorted longest first is an
// LPT schedule -- but when the long items are not a multiple of the compute
// units (384-row items of a 4096-row chunk: 344 of them for 256 units), the
// last round of long items runs on a few units while the rest idle.  This
// simulates that schedule (item time = its tiles + kItemSetupTiles) and, when
// its makespan exceeds the ideal (total / units) by more than kBalanceSlack,
// tries two ways of cutting items into pieces:
//  * fill: the same schedule, where an item that would push the least loaded
//    unit past the ideal gives that unit only the tiles that fill it up, its
//    remaining tiles going back into the queue as a later item;
//  * even: the longest items are placed whole while the least loaded unit
//    takes them within the bound; each item left that can be cut in two is
//    cut into equal pieces, m units' worth of pieces in all (m = 1 .. 4),
//    dealt in proportion to the items' lengths.
// Each candidate is scored by the schedule that the dispatch makes of it (all
// pieces sorted longest first), and the one that ends first is kept; fewer
// pieces win a tie.  Every piece keeps at least kMinBalancePiece tiles (each
// costs a set-up, and its rows a merge).  Fill suits a few long items over a
// round of shorter ones (the 32K prompt's rank 0, whose short chunk's items
// fill the gaps); even suits rounds of equally long items (a prompt behind a
// long cached prefix), where fill's remainders are too long for the room
// they find.  Returns each item's interior cut points (tile indices,
// ascending) in `cuts` (indexed by the items' numbers, allocated only when a
// cut is made).
struct ItemTiles {
  int64_t item;   // the item's number in the launch
  int64_t tiles;  // its key walk
};

// Makespan of list scheduling `lens` (sorted longest first) onto units whose
// loads start at `loads`.
int64_t list_schedule(const std::vector<int64_t>& loads, const std::vector<int64_t>& lens) {
  std::priority_queue<int64_t, std::vector<int64_t>, std::greater<int64_t>> units(loads.begin(), loads.end());
  int64_t makespan = *std::max_element(loads.begin(), loads.end());
  for (int64_t len : lens) {
    const int64_t t = units.top() + len + kItemSetupTiles;
    units.pop();
    units.push(t);
    makespan = std::max(makespan, t);
  }
  return makespan;
}

typedef std::vector<std::vector<int32_t>> Cuts;  // per item (position in the list): cut points

// The fill candidate (see balance_cuts).
Cuts fill_cuts(const std::vector<ItemTiles>& items, int n_units, int64_t ideal, int64_t limit) {
  struct Seg {
    int64_t len;
    size_t idx;
    int32_t t0;
  };
  Cuts c(items.size());
  std::priority_queue<int64_t, std::vector<int64_t>, std::greater<int64_t>> units;
  for (int u = 0; u < n_units; ++u) units.push(0);
  auto longer = [](const Seg& a, const Seg& b) { return a.len < b.len || (a.len == b.len && a.idx > b.idx); };
  std::priority_queue<Seg, std::vector<Seg>, decltype(longer)> queue(longer);
  for (size_t i = 0; i < items.size(); ++i) queue.push(Seg{items[i].tiles, i, 0});
  while (!queue.empty()) {
    const Seg s = queue.top();
    queue.pop();
    const int64_t load = units.top();
    units.pop();
    int64_t take = s.len;
    if (load + s.len + kItemSetupTiles > limit && (int64_t)c[s.idx].size() + 1 < kMaxPieces) {
      // Fill this unit up to the ideal, or give it the smallest piece when
      // it is there already.
      const int64_t room = ideal - load - kItemSetupTiles;
      if (s.len >= 2 * kMinBalancePiece) take = std::min(std::max(room, kMinBalancePiece), s.len - kMinBalancePiece);
    }
    units.push(load + take + kItemSetupTiles);
    if (take < s.len) {
      c[s.idx].push_back(s.t0 + (int32_t)take);
      queue.push(Seg{s.len - take, s.idx, s.t0 + (int32_t)take});
    }
  }
  for (std::vector<int32_t>& v : c) std::sort(v.begin(), v.end());
  return c;
}

// The even candidate for m units' worth of pieces (see balance_cuts); no cut
// when it makes none.
Cuts even_cuts(const std::vector<ItemTiles>& items, int n_units, int64_t limit, int m) {
  Cuts c(items.size());
  std::vector<size_t> order(items.size());
  for (size_t i = 0; i < items.size(); ++i) order[i] = i;
  std::sort(order.begin(), order.end(), [&](size_t a, size_t b) {
    return items[a].tiles > items[b].tiles || (items[a].tiles == items[b].tiles && a < b);
  });
  // The longest items, each while the least loaded unit takes it within the
  // limit.
  std::priority_queue<int64_t, std::vector<int64_t>, std::greater<int64_t>> units;
  for (int u = 0; u < n_units; ++u) units.push(0);
  size_t n_whole = 0;
  for (; n_whole < order.size(); ++n_whole) {
    const int64_t t = units.top() + items[order[n_whole]].tiles + kItemSetupTiles;
    if (t > limit) break;
    units.pop();
    units.push(t);
  }
  std::vector<size_t> big;  // the rest that can be cut in two
  int64_t big_tiles = 0;
  for (size_t k = n_whole; k < order.size(); ++k)
    if (items[order[k]].tiles >= 2 * kMinBalancePiece) {
      big.push_back(order[k]);
      big_tiles += items[order[k]].tiles;
    }
  const int64_t target = (int64_t)m * n_units;
  if (target <= (int64_t)big.size()) return c;
  // Pieces in proportion to the lengths (largest remainders first), each
  // item's at most its length allows.
  std::vector<int64_t> n_pieces(big.size());
  std::vector<std::pair<double, size_t>> frac;
  int64_t dealt = 0;
  for (size_t i = 0; i < big.size(); ++i) {
    const int64_t len = items[big[i]].tiles;
    const double share = (double)target * (double)len / (double)big_tiles;
    const int64_t most = std::min<int64_t>(kMaxPieces, len / kMinBalancePiece);
    n_pieces[i] = std::max<int64_t>(1, std::min<int64_t>(most, (int64_t)share));
    dealt += n_pieces[i];
    if (n_pieces[i] < most) frac.push_back(std::make_pair(share - (double)n_pieces[i], i));
  }
  std::stable_sort(frac.begin(), frac.end(), [](const std::pair<double, size_t>& x, const std::pair<double, size_t>& y) {
    return x.first > y.first;
  });
  for (size_t f = 0; f < frac.size() && dealt < target; ++f, ++dealt) ++n_pieces[frac[f].second];
  for (size_t i = 0; i < big.size(); ++i) {
    const int64_t len = items[big[i]].tiles;
    for (int64_t k = 1; k < n_pieces[i]; ++k) c[big[i]].push_back((int32_t)(len * k / n_pieces[i]));
  }
  return c;
}

// The dispatch's schedule of a candidate: makespan and piece count.
std::pair<int64_t, int64_t> score_cuts(const std::vector<ItemTiles>& items, const Cuts& c, int n_units) {
  std::vector<int64_t> lens;
  int64_t pieces = 0;
  for (size_t i = 0; i < items.size(); ++i) {
    int32_t prev = 0;
    for (int32_t x : c[i]) {
      lens.push_back(x - prev);
      prev = x;
    }
    lens.push_back(items[i].tiles - prev);
    if (!c[i].empty()) pieces += (int64_t)c[i].size() + 1;
  }
  std::sort(lens.begin(), lens.end(), std::greater<int64_t>());
  return std::make_pair(list_schedule(std::vector<int64_t>(n_units, 0), lens), pieces);
}

void balance_cuts(const std::vector<ItemTiles>& items, int n_units, size_t n_items_total, Cuts* cuts) {
  if (items.empty()) return;
  int64_t total = 0, longest = 0;
  for (const ItemTiles& it : items) {
    total += it.tiles + kItemSetupTiles;
    longest = std::max(longest, it.tiles);
  }
  const int64_t ideal = (total + n_units - 1) / n_units;
  const int64_t limit = (int64_t)(ideal * kBalanceSlack);
  // List scheduling ends within one item of the even spread: when the longest
  // item fits in the slack, no schedule needs cuts (and none is simulated).
  if (ideal + longest + kItemSetupTiles <= limit) return;
  const Cuts none(items.size());
  std::pair<int64_t, int64_t> best = score_cuts(items, none, n_units);
  if (best.first <= limit) return;
  Cuts chosen;
  auto consider = [&](Cuts c) {
    const std::pair<int64_t, int64_t> sc = score_cuts(items, c, n_units);
    if (sc.first < best.first || (sc.first == best.first && sc.second < best.second)) {
      best = sc;
      chosen.swap(c);
    }
  };
  consider(fill_cuts(items, n_units, ideal, limit));
  for (int m = 1; m <= 4; ++m) consider(even_cuts(items, n_units, limit, m));
  if (chosen.empty()) return;
  for (size_t i = 0; i < items.size(); ++i) {
    if (chosen[i].empty()) continue;
    if (cuts->empty()) cuts->resize(n_items_total);
    (*cuts)[(size_t)items[i].item] = chosen[i];
  }
}

// Key tiles of one work item's walk, exactly as the kernel counts them: the
// paged prefix, then each suffix range clipped to the item's last query.
int64_t item_tiles(const DevDesc& d, int chunk, int64_t qb, int q_per_wg) {
  constexpr int64_t T = 32;
  const int64_t last = std::min(qb * q_per_wg + q_per_wg, d.q_len[chunk]) - 1;
  const int64_t vis_end = d.q_begin[chunk] + last + 1;
  int64_t n = (d.prefix_keys + T - 1) / T;
  for (int s = 0; s < d.n_seg; ++s) {
    const int64_t vis = std::min(d.seg_hi[s], vis_end);
    if (vis > d.seg_lo[s]) n += (vis - d.seg_lo[s] + T - 1) / T;
  }
  return n;
}

int64_t item_keys(const DevDesc& d, int chunk, int64_t qb, int q_per_wg) {
  const int64_t last = std::min(qb * q_per_wg + q_per_wg, d.q_len[chunk]) - 1;
  const int64_t pos_hi = d.q_begin[chunk] + last;
  int64_t keys = d.prefix_keys;
  for (int s = 0; s < d.n_seg; ++s) keys += std::max<int64_t>(0, std::min(d.seg_hi[s], pos_hi + 1) - d.seg_lo[s]);
  return keys;
}

// The work list of one launch for one workgroup shape: items, split items and
// piece count into *out (whose descriptors are set).
int plan_items(int32_t Hq, int32_t Hkv, int rows, int64_t target_pieces, Plan* out) {
  out->shape = shape_for(Hq, Hkv, rows);
  const Shape& sh = out->shape;
  const int n_descs = (int)out->descs.size();
  const int n_groups = Hkv * sh.groups_per_kv;
  struct Cand {
    int64_t cost;
    WorkItem w;
  };
  // Query blocks of every descriptor and chunk, with their tile counts.
  struct Block {
    int32_t desc, chunk, q_block;
    int64_t keys, tiles;
  };
  std::vector<Block> blocks;
  int64_t nonempty = 0, all_tiles = 0, max_tiles = 0;
  for (int i = 0; i < n_descs; ++i) {
    const DevDesc& d = out->descs[i];
    for (int c = 0; c < 2; ++c) {
      if (d.q_len[c] == 0) continue;
      const int64_t nqb = (d.q_len[c] + sh.q_per_wg - 1) / sh.q_per_wg;
      for (int64_t qb = 0; qb < nqb; ++qb) {
        const int64_t tiles = item_tiles(d, c, qb, sh.q_per_wg);
        blocks.push_back(Block{i, c, (int32_t)qb, item_keys(d, c, qb, sh.q_per_wg), tiles});
        if (tiles > 0) nonempty += n_groups;
        all_tiles += tiles * n_groups;
        max_tiles = std::max(max_tiles, tiles);
      }
    }
  }
  // Splitting pays when the longest walk is long against the piece size (the
  // pieces' set-up and the merge pass are not free).
  int64_t piece_tiles = 0;  // 0: no splitting in this launch
  if (target_pieces > 0 && nonempty > 0 && nonempty < kSplitBelowItems && max_tiles >= 4 * kMinPieceTiles)
    piece_tiles = std::max<int64_t>(kMinPieceTiles, (all_tiles + target_pieces - 1) / target_pieces);
  // Cut points of each item's walk (item = block * n_groups + head group):
  // equal pieces when few items split for occupancy, else balance cuts.
  std::vector<std::vector<int32_t>> cuts;
  if (piece_tiles) {
    cuts.resize(blocks.size() * n_groups);
    for (size_t bi = 0; bi < blocks.size(); ++bi) {
      const int64_t n = std::min<int64_t>(kMaxPieces, blocks[bi].tiles / piece_tiles);
      for (int g = 0; g < n_groups; ++g)
        for (int64_t k = 1; k < n; ++k) cuts[bi * n_groups + g].push_back((int32_t)(blocks[bi].tiles * k / n));
    }
  } else if (target_pieces > 0) {
    // With the head groups a multiple of the XCDs, each XCD's list is its own
    // schedule on its 32 compute units; otherwise the lists share the units
    // (the interleave below moves items between XCDs) and one schedule over
    // all of them is the closer model.
    const int n_sched = n_groups % kXcds == 0 ? kXcds : 1;
    std::vector<ItemTiles> sched;
    for (int x = 0; x < n_sched; ++x) {
      sched.clear();
      for (size_t bi = 0; bi < blocks.size(); ++bi)
        if (blocks[bi].tiles > 0)
          for (int g = x; g < n_groups; g += n_sched) sched.push_back(ItemTiles{(int64_t)(bi * n_groups + g), blocks[bi].tiles});
      balance_cuts(sched, kComputeUnits / n_sched, blocks.size() * n_groups, &cuts);
    }
  }
  out->splits.clear();
  out->n_pieces = 0;
  std::vector<std::vector<Cand>> per_xcd(kXcds);
  int64_t total = 0;
  for (size_t bi = 0; bi < blocks.size(); ++bi) {
    const Block& b = blocks[bi];
    for (int g = 0; g < n_groups; ++g) {
      const std::vector<int32_t>* c = cuts.empty() ? nullptr : &cuts[bi * n_groups + g];
      if (!c || c->empty()) {
        per_xcd[g % kXcds].push_back(Cand{b.keys, WorkItem{b.desc, b.chunk, b.q_block, g, 0, -1, -1, 0}});
        ++total;
        continue;
      }
      const int64_t n_pieces = (int64_t)c->size() + 1;
      out->splits.push_back(SplitItem{b.desc, b.chunk, b.q_block, g, (int32_t)out->n_pieces, (int32_t)n_pieces});
      for (int64_t k = 0; k < n_pieces; ++k) {
        const int32_t t0 = k == 0 ? 0 : (*c)[k - 1];
        const int32_t t1 = k + 1 == n_pieces ? (int32_t)b.tiles : (*c)[k];
        per_xcd[g % kXcds].push_back(
            Cand{(int64_t)(t1 - t0) * 32, WorkItem{b.desc, b.chunk, b.q_block, g, t0, t1, (int32_t)(out->n_pieces + k), 0}});
        ++total;
      }
      out->n_pieces += n_pieces;
    }
  }
  if (total > 0x7fffffffLL) return fail(CP_ERR_UNSUPPORTED, "cp_attn_partial: work list beyond 2^31 workgroups");
  for (auto& v : per_xcd)
    std::stable_sort(v.begin(), v.end(), [](const Cand& a, const Cand& b) { return a.cost > b.cost; });
  out->items.clear();
  out->items.reserve((size_t)total);
  std::vector<size_t> head(kXcds, 0);
  for (int64_t i = 0; i < total; ++i) {
    int x = (int)(i % kXcds);
    if (head[x] == per_xcd[x].size()) {
      // This XCD's list ran dry: take the costliest remaining item anywhere.
      int best = -1;
      for (int y = 0; y < kXcds; ++y)
        if (head[y] < per_xcd[y].size() && (best < 0 || per_xcd[y][head[y]].cost > per_xcd[best][head[best]].cost))
          best = y;
      x = best;
    }
    out->items.push_back(per_xcd[x][head[x]++].w);
  }
  return CP_OK;
}

// Estimated time (microseconds) of a planned launch: the in-order dispatch
// of its work list simulated on each XCD's 32 compute units (list item i on
// XCD i % 8), an item taking its tiles times the shape's time per tile plus
// a fixed set-up, then the split merge's traffic.  The 384-row shape's tile
// is 1.5 times the 256-row one's work at kLargeTileGain times its rate.  The
// three constants are fitted to both shapes' times on 136 rank launches (the
// prompts of 4K-32K tokens at C = 1-8 with and without a 16K prefix, and five
// larger shapes), timed alternately in one process.
constexpr double kSmallTileUs = 0.90;   // a 256-row x 32-key tile on one compute unit
constexpr double kLargeTileGain = 1.06;
constexpr double kItemSetupUs = 8.0;
constexpr double kMergeBytesPerUs = 5.0e6;

double estimate_us(const Plan& plan) {
  const double tile_us = plan.shape.rows_per_wg == kRowsLarge ? kSmallTileUs * 1.5 / kLargeTileGain : kSmallTileUs;
  std::vector<std::priority_queue<double, std::vector<double>, std::greater<double>>> units(kXcds);
  for (auto& q : units)
    for (int u = 0; u < kComputeUnits / kXcds; ++u) q.push(0.0);
  double makespan = 0.0;
  for (size_t i = 0; i < plan.items.size(); ++i) {
    const WorkItem& w = plan.items[i];
    const int64_t tiles = w.t_end >= 0 ? (int64_t)(w.t_end - w.t_begin)
                                       : item_tiles(plan.descs[w.desc], w.chunk, w.q_block, plan.shape.q_per_wg);
    auto& q = units[i % kXcds];
    const double t = q.top() + tiles * tile_us + kItemSetupUs;
    q.pop();
    q.push(t);
    makespan = std::max(makespan, t);
  }
  if (plan.n_pieces) {
    // Pieces written and read back, the merged rows written.
    const double bytes = (double)piece_bytes(plan.shape.rows_per_wg) * (2.0 * plan.n_pieces + plan.splits.size());
    makespan += bytes / kMergeBytesPerUs + kItemSetupUs;
  }
  return makespan;
}

// Bounds (microseconds) of one shape's schedule before any item is cut: the
// launch's work spread evenly over the compute units (every XCD gets the same
// share of each block when the head groups are a multiple of the XCDs, and the
// interleave spreads them otherwise), and that plus the longest item (list
// scheduling ends within one item of the even spread).
// `splits` tells whether the launch has few enough items to be split for
// occupancy, which the bounds do not model.
struct Bounds {
  double lo, hi;
  bool splits;
};

Bounds shape_bounds(const std::vector<DevDesc>& descs, int32_t Hq, int32_t Hkv, int rows) {
  const Shape sh = shape_for(Hq, Hkv, rows);
  const int n_groups = Hkv * sh.groups_per_kv;
  const double tile_us = rows == kRowsLarge ? kSmallTileUs * 1.5 / kLargeTileGain : kSmallTileUs;
  double work = 0.0;  // microseconds over all items
  int64_t nonempty = 0, max_tiles = 0;
  for (const DevDesc& d : descs)
    for (int c = 0; c < 2; ++c)
      for (int64_t qb = 0; qb * sh.q_per_wg < d.q_len[c]; ++qb) {
        const int64_t tiles = item_tiles(d, c, qb, sh.q_per_wg);
        work += (tiles * tile_us + kItemSetupUs) * n_groups;
        if (tiles > 0) nonempty += n_groups;
        max_tiles = std::max(max_tiles, tiles);
      }
  const double lo = work / kComputeUnits;
  Bounds b;
  b.lo = lo;
  b.hi = lo + max_tiles * tile_us + kItemSetupUs;
  b.splits = nonempty < kSplitBelowItems;
  return b;
}

// Work-group shape forced by cp_set_workgroup_rows (0: chosen per launch).
std::atomic<int> g_forced_rows{0};

}  // namespace

extern "C" int cp_set_workgroup_rows(int32_t rows) {
  if (rows != 0 && rows != kRowsSmall && rows != kRowsLarge)
    return fail_static(CP_ERR_INVALID, "cp_set_workgroup_rows: rows must be 0, 256 or 384");
  g_forced_rows.store(rows);
  clear_error();
  return CP_OK;
}

namespace cpattn {

// Work lists of recent launches.  A layer after layer of the same shapes
// plans the same list (the work list depends on the descriptors' positions,
// chunks and key ranges and on the heads, never on their buffers), so the
// list of a launch whose key matches is reused instead of planned again:
// the key holds every non-pointer field of the converted descriptors, the
// head counts, the piece target and the pinned shape, and matches exactly.
struct CachedPlan {
  std::vector<int64_t> key;
  std::vector<WorkItem> items;
  std::vector<SplitItem> splits;
  int64_t n_pieces;
  Shape shape;
};
constexpr size_t kPlanCacheSize = 16;
static std::mutex g_plan_cache_mu;
static std::vector<CachedPlan> g_plan_cache;  // most recent last
static size_t g_plan_cache_hits = 0;

static std::vector<int64_t> plan_key(const std::vector<DevDesc>& descs, int32_t Hq, int32_t Hkv, int64_t target_pieces,
                                     int forced) {
  std::vector<int64_t> k = {Hq, Hkv, target_pieces, forced, (int64_t)descs.size()};
  for (const DevDesc& d : descs) {
    const int64_t f[] = {d.P, d.R, d.q_begin[0], d.q_begin[1], d.q_len[0], d.q_len[1], d.local_off[0], d.local_off[1],
                         d.o_off[0], d.o_off[1], d.seg_lo[0], d.seg_lo[1], d.seg_hi[0], d.seg_hi[1], d.n_seg,
                         d.prefix_keys, d.n_blocks, d.reserved};
    k.insert(k.end(), f, f + sizeof(f) / sizeof(f[0]));
  }
  return k;
}

static int plan_uncached(int32_t Hq, int32_t Hkv, int64_t target_pieces, int forced, Plan* out);

int build_plan(const cp_partial_desc* descs, int32_t n_descs, int32_t Hq, int32_t Hkv, int64_t target_pieces,
               Plan* out) {
  int st = check_heads(Hq, Hkv, "cp_attn_partial");
  if (st != CP_OK) return st;
  if (n_descs < 0) return fail(CP_ERR_INVALID, "cp_attn_partial: n_descs < 0");
  if (n_descs > 0 && !descs) return fail(CP_ERR_INVALID, "cp_attn_partial: descs is NULL");
  out->descs.resize(n_descs);
  for (int i = 0; i < n_descs; ++i) {
    st = to_dev(descs[i], i, &out->descs[i]);
    if (st != CP_OK) return st;
  }
  const int forced = g_forced_rows.load();
  std::vector<int64_t> key = plan_key(out->descs, Hq, Hkv, target_pieces, forced);
  {
    std::lock_guard<std::mutex> lock(g_plan_cache_mu);
    for (size_t i = g_plan_cache.size(); i-- > 0;) {
      const CachedPlan& c = g_plan_cache[i];
      if (c.key != key) continue;
      out->items = c.items;
      out->splits = c.splits;
      out->n_pieces = c.n_pieces;
      out->shape = c.shape;
      ++g_plan_cache_hits;
      return CP_OK;
    }
  }
  st = plan_uncached(Hq, Hkv, target_pieces, forced, out);
  if (st != CP_OK) return st;
  std::lock_guard<std::mutex> lock(g_plan_cache_mu);
  if (g_plan_cache.size() == kPlanCacheSize) g_plan_cache.erase(g_plan_cache.begin());
  g_plan_cache.push_back(CachedPlan{std::move(key), out->items, out->splits, out->n_pieces, out->shape});
  return CP_OK;
}

// The work list of a launch whose descriptors are converted (out->descs).
static int plan_uncached(int32_t Hq, int32_t Hkv, int64_t target_pieces, int forced, Plan* out) {
  int st;
  // The workgroup shape: two or three 16-row blocks per wave.  The larger
  // shares every K/V fragment between more rows (faster per tile) but makes
  // fewer, longer work items, which fill the compute units worse; plan both
  // and keep the one whose simulated schedule ends first.
  if (forced) return plan_items(Hq, Hkv, forced, target_pieces, out);
  // When the bounds already decide (one shape's worst case ends before the
  // other's best), only the winner is planned.
  const Bounds bs = shape_bounds(out->descs, Hq, Hkv, kRowsSmall);
  const Bounds bl = shape_bounds(out->descs, Hq, Hkv, kRowsLarge);
  if (!bs.splits && !bl.splits) {
    if (bl.hi < bs.lo) return plan_items(Hq, Hkv, kRowsLarge, target_pieces, out);
    if (bs.hi < bl.lo) return plan_items(Hq, Hkv, kRowsSmall, target_pieces, out);
  }
  Plan small;
  small.descs = out->descs;
  st = plan_items(Hq, Hkv, kRowsSmall, target_pieces, &small);
  if (st != CP_OK) return st;
  st = plan_items(Hq, Hkv, kRowsLarge, target_pieces, out);
  if (st != CP_OK) return st;
  if (estimate_us(small) < estimate_us(*out)) *out = std::move(small);
  return CP_OK;
}

static size_t align_up(size_t x) { return (x + kItemsAlign - 1) / kItemsAlign * kItemsAlign; }

Layout layout_of(const Plan& plan) {
  Layout l;
  l.items = align_up(plan.descs.size() * sizeof(DevDesc));
  l.splits = align_up(l.items + plan.items.size() * sizeof(WorkItem));
  l.pieces = align_up(l.splits + plan.splits.size() * sizeof(SplitItem));
  l.total = l.pieces + (size_t)plan.n_pieces * piece_bytes(plan.shape.rows_per_wg);
  return l;
}

void pack_tables(const Plan& plan, const Layout& lay, std::vector<unsigned char>* host) {
  host->assign(lay.pieces, 0);
  std::memcpy(host->data(), plan.descs.data(), plan.descs.size() * sizeof(DevDesc));
  std::memcpy(host->data() + lay.items, plan.items.data(), plan.items.size() * sizeof(WorkItem));
  if (!plan.splits.empty())
    std::memcpy(host->data() + lay.splits, plan.splits.data(), plan.splits.size() * sizeof(SplitItem));
}

PartialParams partial_params(const Plan& plan, const Layout& lay, unsigned char* ws, int32_t Hq, int32_t Hkv,
                             float scale) {
  PartialParams p;
  std::memset(&p, 0, sizeof(p));
  p.descs = reinterpret_cast<const DevDesc*>(ws);
  p.items = reinterpret_cast<const WorkItem*>(ws + lay.items);
  p.n_items = (int32_t)plan.items.size();
  p.Hq = Hq;
  p.Hkv = Hkv;
  p.heads_per_wg = plan.shape.heads_per_wg;
  p.q_per_wg = plan.shape.q_per_wg;
  p.groups_per_kv = plan.shape.groups_per_kv;
  p.scale = scale;
  p.scale_log2 = scale * 1.4426950408889634f;
  p.rows_per_wg = plan.shape.rows_per_wg;
  p.pieces = plan.n_pieces ? ws + lay.pieces : nullptr;
  p.splits = reinterpret_cast<const SplitItem*>(ws + lay.splits);
  p.n_splits = (int32_t)plan.splits.size();
  return p;
}

}  // namespace cpattn

namespace {

// Pinned host staging for the descriptor/work-list upload, mapped into the
// device's address space and coherent (the device reads it over the bus,
// never from a cached copy): the upload kernel reads it (upload.hip).  A slot
// is reused only after the upload that read it has completed (its event).
struct Slot {
  void* host = nullptr;
  void* mapped = nullptr;  // the same memory as the device addresses it
  size_t cap = 0;
  hipEvent_t ev = nullptr;
  int device = -1;
  bool pending = false;
};
constexpr int kSlots = 8;
std::mutex g_stage_mu;
Slot g_slots[kSlots];
int g_next_slot = 0;

int stage_and_copy(const void* src, size_t bytes, void* dst, hipStream_t stream) {
  std::lock_guard<std::mutex> lock(g_stage_mu);
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(CP_ERR_HIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
  Slot& s = g_slots[g_next_slot];
  g_next_slot = (g_next_slot + 1) % kSlots;
  if (s.pending) {
    e = hipEventSynchronize(s.ev);
    if (e != hipSuccess) return fail(CP_ERR_HIP, std::string("hipEventSynchronize: ") + hipGetErrorString(e));
    s.pending = false;
  }
  if (s.ev && s.device != dev) {
    (void)hipEventDestroy(s.ev);
    s.ev = nullptr;
  }
  if (!s.ev) {
    e = hipEventCreateWithFlags(&s.ev, hipEventDisableTiming);
    if (e != hipSuccess) return fail(CP_ERR_HIP, std::string("hipEventCreate: ") + hipGetErrorString(e));
    s.device = dev;
  }
  if (s.cap < bytes) {
    if (s.host) (void)hipHostFree(s.host);
    s.host = nullptr;
    s.mapped = nullptr;
    s.cap = 0;
    const size_t cap = std::max<size_t>(bytes, 64 * 1024);
    e = hipHostMalloc(&s.host, cap, hipHostMallocMapped | hipHostMallocPortable | hipHostMallocCoherent);
    if (e != hipSuccess) return fail(CP_ERR_HIP, std::string("hipHostMalloc (staging): ") + hipGetErrorString(e));
    e = hipHostGetDevicePointer(&s.mapped, s.host, 0);
    if (e != hipSuccess) return fail(CP_ERR_HIP, std::string("hipHostGetDevicePointer (staging): ") + hipGetErrorString(e));
    s.cap = cap;
  }
  std::memcpy(s.host, src, bytes);
  const int up = cpattn::launch_upload(dst, s.mapped, bytes, stream);
  if (up != CP_OK) return up;
  e = hipEventRecord(s.ev, stream);
  if (e != hipSuccess) return fail(CP_ERR_HIP, std::string("hipEventRecord: ") + hipGetErrorString(e));
  s.pending = true;
  return CP_OK;
}

}  // namespace

extern "C" size_t cp_attn_partial_workspace_size(const cp_partial_desc* descs, int32_t n_descs,
                                                 int32_t n_heads_q, int32_t n_heads_kv) {
  size_t total = 0;
  const int st = guarded([&]() -> int {
    Plan plan;
    const int s = build_plan(descs, n_descs, n_heads_q, n_heads_kv, kTargetPieces, &plan);
    if (s == CP_OK) total = layout_of(plan).total;
    return s;
  });
  if (st != CP_OK) return 0;
  clear_error();
  return total;
}

extern "C" int cp_attn_partial(const cp_partial_desc* descs, int32_t n_descs, int32_t n_heads_q,
                               int32_t n_heads_kv, int32_t head_dim, float softmax_scale, void* workspace,
                               size_t workspace_bytes, void* stream) {
  return guarded([&]() -> int {
    if (head_dim != CP_HEAD_DIM) return fail(CP_ERR_UNSUPPORTED, "cp_attn_partial: head_dim must be 128");
    if (!(softmax_scale == softmax_scale)) return fail(CP_ERR_INVALID, "cp_attn_partial: softmax_scale is NaN");
    Plan plan;
    int st = build_plan(descs, n_descs, n_heads_q, n_heads_kv, kTargetPieces, &plan);
    if (st != CP_OK) return st;
    if (plan.items.empty()) {
      clear_error();
      return CP_OK;
    }
    const Layout lay = layout_of(plan);
    if (!workspace) return fail(CP_ERR_INVALID, "cp_attn_partial: workspace is NULL");
    if (!aligned(workspace, 256)) return fail(CP_ERR_INVALID, "cp_attn_partial: workspace must be 256-byte aligned");
    if (workspace_bytes < lay.total)
      return fail(CP_ERR_CAPACITY, "cp_attn_partial: workspace needs " + std::to_string(lay.total) + " bytes");
    // Only the tables are uploaded; the piece slots are written by the kernel.
    std::vector<unsigned char> host;
    pack_tables(plan, lay, &host);
    st = stage_and_copy(host.data(), lay.pieces, workspace, (hipStream_t)stream);
    if (st != CP_OK) return st;
    const float scale = softmax_scale > 0.f ? softmax_scale : 1.f / std::sqrt((float)head_dim);
    st = launch_partial(partial_params(plan, lay, static_cast<unsigned char*>(workspace), n_heads_q, n_heads_kv, scale),
                        stream);
    if (st == CP_OK) clear_error();
    return st;
  });
}

extern "C" int cp_attn_merge(int32_t n_parts, const float* const* o_parts, const float* const* lse_parts,
                             int64_t n_tokens, int32_t n_heads, int32_t head_dim, void* o_out, int32_t out_bf16,
                             float* lse_out, const cp_rank_plan* restore, void* stream) {
  return guarded([&]() -> int {
    if (head_dim != CP_HEAD_DIM) return fail(CP_ERR_UNSUPPORTED, "cp_attn_merge: head_dim must be 128");
    if (n_parts < 1 || n_parts > CP_MAX_MERGE_PARTS) return fail(CP_ERR_INVALID, "cp_attn_merge: n_parts must be 1..16");
    if (!o_parts || !lse_parts) return fail(CP_ERR_INVALID, "cp_attn_merge: o_parts/lse_parts is NULL");
    if (n_tokens < 0 || n_heads < 1) return fail(CP_ERR_INVALID, "cp_attn_merge: n_tokens < 0 or n_heads < 1");
    if (out_bf16 != 0 && out_bf16 != 1) return fail(CP_ERR_INVALID, "cp_attn_merge: out_bf16 must be 0 or 1");
    MergeParams p;
    std::memset(&p, 0, sizeof(p));
    if (n_tokens > 0) {
      for (int i = 0; i < n_parts; ++i) {
        if (!o_parts[i] || !lse_parts[i]) return fail(CP_ERR_INVALID, "cp_attn_merge: NULL partial pointer");
        if (!aligned(o_parts[i], 16) || !aligned(lse_parts[i], 4))
          return fail(CP_ERR_INVALID, "cp_attn_merge: partial O must be 16-byte, LSE 4-byte aligned");
        p.o[i] = o_parts[i];
        p.lse[i] = lse_parts[i];
      }
      if (!o_out) return fail(CP_ERR_INVALID, "cp_attn_merge: o_out is NULL");
      if (!aligned(o_out, 16)) return fail(CP_ERR_INVALID, "cp_attn_merge: o_out must be 16-byte aligned");
      if (lse_out && !aligned(lse_out, 4)) return fail(CP_ERR_INVALID, "cp_attn_merge: lse_out must be 4-byte aligned");
    }
    if (restore) {
      cp_rank_plan ref;
      if (make_plan(restore->prefix_len, restore->new_len, restore->C, restore->rank, &ref) != CP_OK ||
          !plan_equal(ref, *restore))
        return fail(CP_ERR_INVALID, "cp_attn_merge: restore plan does not match cp_shard_plan");
      if (restore->n_rows != n_tokens) return fail(CP_ERR_INVALID, "cp_attn_merge: n_tokens != restore->n_rows");
      p.restore = 1;
      p.first_len = restore->chunk[0].q_len;
      p.first_dst = restore->chunk[0].q_begin - restore->prefix_len;
      p.second_dst = restore->chunk[1].q_begin - restore->prefix_len;
    }
    p.n_parts = n_parts;
    p.n_heads = n_heads;
    p.n_tokens = n_tokens;
    p.o_out = o_out;
    p.lse_out = lse_out;
    p.out_bf16 = out_bf16;
    int st = launch_merge(p, stream);
    if (st == CP_OK) clear_error();
    return st;
  });
}
