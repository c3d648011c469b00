// Host-only check of the attention work list (tests/test_planner.py builds and
// runs it; no GPU is touched).  It includes the planner's source so that the
// internal plan can be inspected, builds the plan of several launches (named
// ones and 60 seeded random ones) in each workgroup shape and checks:
//   * every (descriptor, chunk, query block, head group) of the launch is
//     scheduled exactly once: whole, or as pieces whose tile ranges cover its
//     key walk [0, tiles) in order, one slot per piece, described by exactly
//     one split item;
//   * pieces keep the minimum sizes of their policy (at least 32 tiles when a
//     launch with few items is split for occupancy, 256 for balance cuts,
//     whether they fill units up or cut items evenly);
//   * the work list holds nothing else, and the workspace layout holds one
//     slot of the shape's size per piece;
//   * a launch planned again is served from the plan cache with the list a
//     fresh plan gives, and a launch that differs is planned anew.
// Prints "ok <cases>" on success, else the first failure, and exits non-zero.
#include "../paper_2609_04774_amd/csrc/cp_attn.cpp"

#include <cstdio>
#include <map>
#include <tuple>

namespace cpattn {
// The check never launches anything.
int launch_partial(const PartialParams&, void*) { return 1; }
int launch_merge(const MergeParams&, void*) { return 1; }
int launch_upload(void*, const void*, size_t, void*) { return 1; }
}  // namespace cpattn

namespace {

int failures = 0;

void expect(bool ok, const std::string& what) {
  if (!ok && failures++ == 0) std::printf("FAIL %s\n", what.c_str());
}

struct Launch {
  std::string name;
  std::vector<cp_partial_desc> descs;
  int Hq, Hkv;
};

cp_partial_desc desc(int64_t P, int64_t R, int C, int rank, int kv_rank, int include_prefix) {
  cp_partial_desc d{};
  make_plan(P, R, C, rank, &d.plan);
  void* f = reinterpret_cast<void*>(0x100000);
  d.q = d.k_new = d.v_new = d.k_cache = d.v_cache = f;
  d.o = d.lse = static_cast<float*>(f);
  d.block_table = static_cast<const int32_t*>(f);
  d.n_blocks = 1 << 20;
  d.include_prefix = include_prefix;
  d.kv_rank = kv_rank;
  return d;
}

void check(const Launch& l, int rows) {
  const std::string who = l.name + " rows " + std::to_string(rows);
  cp_set_workgroup_rows(rows);
  Plan plan;
  const int st = build_plan(l.descs.data(), (int32_t)l.descs.size(), l.Hq, l.Hkv, kTargetPieces, &plan);
  expect(st == CP_OK, who + ": build_plan failed");
  if (st != CP_OK) return;
  const Shape& sh = plan.shape;
  expect(rows == 0 || sh.rows_per_wg == rows, who + ": pinned shape not used");
  expect(sh.rows_per_wg == kRowsSmall || sh.rows_per_wg == kRowsLarge, who + ": unknown shape");
  expect(sh.heads_per_wg * sh.q_per_wg == sh.rows_per_wg && sh.q_per_wg % 16 == 0, who + ": shape arithmetic");
  const int n_groups = l.Hkv * sh.groups_per_kv;
  // Expected items: (desc, chunk, q_block, group) -> tiles.
  typedef std::tuple<int, int, int, int> Key;
  std::map<Key, int64_t> expected;
  for (int i = 0; i < (int)plan.descs.size(); ++i)
    for (int c = 0; c < 2; ++c) {
      const int64_t q_len = plan.descs[i].q_len[c];
      for (int64_t qb = 0; qb * sh.q_per_wg < q_len; ++qb)
        for (int g = 0; g < n_groups; ++g)
          expected[Key(i, c, (int)qb, g)] = item_tiles(plan.descs[i], c, qb, sh.q_per_wg);
    }
  std::map<Key, int> whole;
  std::map<Key, std::vector<std::pair<int, int>>> pieces;  // (t_begin, slot)
  std::map<int, std::pair<int, int>> slot_range;           // slot -> (t_begin, t_end)
  std::map<int, Key> slot_item;
  for (const WorkItem& w : plan.items) {
    const Key k(w.desc, w.chunk, w.q_block, w.head_group);
    expect(expected.count(k) == 1, who + ": item outside the launch");
    if (w.piece < 0) {
      expect(w.t_end < 0, who + ": whole item with a tile range");
      ++whole[k];
    } else {
      expect(w.piece < plan.n_pieces, who + ": piece slot out of range");
      expect(slot_range.count(w.piece) == 0, who + ": piece slot used twice");
      slot_range[w.piece] = {w.t_begin, w.t_end};
      slot_item[w.piece] = k;
      pieces[k].push_back({w.t_begin, w.piece});
    }
  }
  expect((int64_t)slot_range.size() == plan.n_pieces, who + ": piece count");
  int64_t min_piece = INT64_MAX;
  std::map<Key, int> split_of;
  for (const SplitItem& s : plan.splits) {
    const Key k(s.desc, s.chunk, s.q_block, s.head_group);
    expect(split_of.count(k) == 0, who + ": item split twice");
    split_of[k] = 1;
    expect(s.n_pieces >= 2 && s.n_pieces <= kMaxPieces, who + ": pieces per split item");
    int64_t t = 0;
    for (int p = s.first_piece; p < s.first_piece + s.n_pieces; ++p) {
      expect(slot_range.count(p) == 1 && slot_item[p] == k, who + ": split item's slots");
      if (!slot_range.count(p)) return;
      expect(slot_range[p].first == t && slot_range[p].second > t, who + ": pieces do not tile the walk");
      min_piece = std::min<int64_t>(min_piece, slot_range[p].second - slot_range[p].first);
      t = slot_range[p].second;
    }
    expect(expected.count(k) && t == expected[k], who + ": pieces do not end at the walk's end");
  }
  for (const auto& e : expected) {
    const bool is_whole = whole.count(e.first) != 0, is_split = split_of.count(e.first) != 0;
    expect(is_whole != is_split, who + ": item scheduled " + (is_whole ? "twice" : "never"));
    if (is_whole) expect(whole[e.first] == 1, who + ": whole item listed twice");
    if (is_split) expect((int)pieces[e.first].size() >= 2, who + ": split item with one piece");
  }
  if (!plan.splits.empty()) expect(min_piece >= kMinPieceTiles, who + ": piece below 32 tiles");
  const Layout lay = layout_of(plan);
  expect(lay.total == lay.pieces + (size_t)plan.n_pieces * piece_bytes(sh.rows_per_wg), who + ": workspace layout");
}

}  // namespace

int main() {
  std::vector<Launch> launches;
  for (int r = 0; r < 4; ++r)
    launches.push_back({"32K C=4 rank " + std::to_string(r), {desc(0, 32768, 4, r, CP_KV_ALL, 1)}, 32, 8});
  launches.push_back({"prefix hit 48K+16K C=2", {desc(49152, 16384, 2, 0, CP_KV_ALL, 1)}, 32, 8});
  {
    Launch l{"pass-KV 32K C=4", {}, 32, 8};
    for (int s = 0; s < 4; ++s) l.descs.push_back(desc(0, 32768, 4, 0, s, 0));
    launches.push_back(l);
  }
  {
    Launch l{"70B pass-KV 128K C=8", {}, 64, 8};
    for (int s = 0; s < 8; ++s) l.descs.push_back(desc(0, 131072, 8, 0, s, 0));
    launches.push_back(l);
  }
  launches.push_back({"few rows over a long prefix", {desc(65536, 64, 1, 0, CP_KV_ALL, 1)}, 32, 8});
  launches.push_back({"ragged GQA 3", {desc(96, 1000, 3, 1, CP_KV_ALL, 1)}, 12, 4});
  launches.push_back({"MHA", {desc(0, 8192, 2, 1, CP_KV_ALL, 1)}, 16, 16});
  {
    Launch l{"mixed requests", {}, 32, 8};
    const int64_t lens[][2] = {{4096, 0}, {20000, 8192}, {700, 0}, {40000, 0}, {3000, 1024}};
    const int degrees[] = {1, 2, 1, 4, 2};
    for (int i = 0; i < 5; ++i)
      for (int r = 0; r < degrees[i]; ++r)
        l.descs.push_back(desc(lens[i][1], lens[i][0] - lens[i][1], degrees[i], r, CP_KV_ALL, 1));
    launches.push_back(l);
  }
  // Random launches (fixed seed): prompts of 1..64K new tokens behind 0..64K
  // cached ones, degree 1..8, one all-gathered partial or a rank's pass-KV
  // partials, several head layouts.
  uint64_t rng = 0x9e3779b97f4a7c15ULL;
  auto next = [&](uint64_t n) {
    rng ^= rng << 13;
    rng ^= rng >> 7;
    rng ^= rng << 17;
    return (int64_t)(rng % n);
  };
  const int heads[][2] = {{32, 8}, {64, 8}, {12, 4}, {16, 16}, {8, 2}};
  for (int i = 0; i < 60; ++i) {
    const int C = 1 << next(4);
    const int64_t R = 2 * C + next(65536 - 2 * C);
    const int64_t P = 16 * next(4097);
    const int rank = (int)next(C);
    const int* h = heads[next(5)];
    Launch l{"random " + std::to_string(i), {}, h[0], h[1]};
    if (next(2))
      l.descs.push_back(desc(P, R, C, rank, CP_KV_ALL, 1));
    else
      for (int sh = 0; sh < C; ++sh) l.descs.push_back(desc(P, R, C, rank, sh, sh == 0));
    launches.push_back(l);
  }
  int cases = 0;
  for (const Launch& l : launches)
    for (int rows : {0, kRowsSmall, kRowsLarge}) {
      check(l, rows);
      ++cases;
    }
  // Balance cuts alone: the 32K rank-0 launch in 384-row items is cut, every
  // piece of at least 256 tiles.
  cp_set_workgroup_rows(kRowsLarge);
  Plan p;
  const cp_partial_desc d0 = desc(0, 32768, 4, 0, CP_KV_ALL, 1);
  build_plan(&d0, 1, 32, 8, kTargetPieces, &p);
  expect(!p.splits.empty(), "32K rank 0 in 384-row items has no balance cuts");
  for (const WorkItem& w : p.items)
    if (w.piece >= 0) expect(w.t_end - w.t_begin >= kMinBalancePiece, "balance piece below 256 tiles");
  // A prompt behind a long cached prefix (every item about equally long, 2.7
  // per compute unit in 384-row items) is cut into even pieces: more than
  // the fill cuts' one per item left over, none below 256 tiles, and the
  // dispatch's schedule within 3 % of the even spread.
  const cp_partial_desc dp = desc(49152, 16384, 2, 0, CP_KV_ALL, 1);
  build_plan(&dp, 1, 32, 8, kTargetPieces, &p);
  expect(p.n_pieces > 352, "prefix launch in 384-row items should be cut evenly");
  int64_t work = 0;
  std::vector<int64_t> lens;
  for (const WorkItem& w : p.items) {
    const int64_t t = w.piece >= 0 ? w.t_end - w.t_begin : item_tiles(p.descs[w.desc], w.chunk, w.q_block, p.shape.q_per_wg);
    if (w.piece >= 0) expect(t >= kMinBalancePiece, "even piece below 256 tiles");
    work += t + kItemSetupTiles;
    lens.push_back(t);
  }
  std::sort(lens.begin(), lens.end(), std::greater<int64_t>());
  const int64_t spread = work / kComputeUnits;
  expect(list_schedule(std::vector<int64_t>(kComputeUnits, 0), lens) <= spread * 103 / 100,
         "prefix launch's schedule more than 3 % past the even spread");
  // The plan cache: a launch planned again (its buffers moved) gets the work
  // list that planning it afresh gives, from the cache; another rank, head
  // layout or pinned shape is planned anew.
  {
    cp_set_workgroup_rows(0);
    cp_partial_desc a = desc(16384, 16384, 4, 1, CP_KV_ALL, 1);
    Plan first, again, fresh;
    build_plan(&a, 1, 32, 8, kTargetPieces, &first);
    a.q = a.k_new = reinterpret_cast<void*>(0x200000);  // other buffers, same geometry
    const size_t hits = g_plan_cache_hits;
    build_plan(&a, 1, 32, 8, kTargetPieces, &again);
    expect(g_plan_cache_hits == hits + 1, "plan cache: an identical launch is not served from the cache");
    expect(again.descs[0].q == reinterpret_cast<const uint16_t*>(0x200000), "plan cache: stale buffer pointers");
    fresh.descs = again.descs;
    plan_uncached(32, 8, kTargetPieces, 0, &fresh);
    bool same = fresh.items.size() == again.items.size() && fresh.splits.size() == again.splits.size() &&
                fresh.n_pieces == again.n_pieces && fresh.shape.rows_per_wg == again.shape.rows_per_wg;
    for (size_t i = 0; same && i < fresh.items.size(); ++i)
      same = std::memcmp(&fresh.items[i], &again.items[i], sizeof(WorkItem)) == 0;
    for (size_t i = 0; same && i < fresh.splits.size(); ++i)
      same = std::memcmp(&fresh.splits[i], &again.splits[i], sizeof(SplitItem)) == 0;
    expect(same, "plan cache: the cached work list differs from a fresh plan");
    const cp_partial_desc b2 = desc(16384, 16384, 4, 2, CP_KV_ALL, 1);
    Plan other;
    build_plan(&b2, 1, 32, 8, kTargetPieces, &other);
    build_plan(&a, 1, 64, 8, kTargetPieces, &other);
    cp_set_workgroup_rows(kRowsSmall);
    build_plan(&a, 1, 32, 8, kTargetPieces, &other);
    expect(g_plan_cache_hits == hits + 1, "plan cache: a different launch was served from the cache");
    expect(other.shape.rows_per_wg == kRowsSmall, "plan cache: the pinned shape was not planned");
    cp_set_workgroup_rows(0);
  }
  // The per-launch choice keeps 384 rows for that launch and 256 for few
  // long walks.
  cp_set_workgroup_rows(0);
  build_plan(&d0, 1, 32, 8, kTargetPieces, &p);
  expect(p.shape.rows_per_wg == kRowsLarge, "32K rank 0 should run 384-row workgroups");
  const cp_partial_desc d1 = desc(65536, 64, 1, 0, CP_KV_ALL, 1);
  build_plan(&d1, 1, 32, 8, kTargetPieces, &p);
  expect(p.shape.rows_per_wg == kRowsSmall, "few long walks should run 256-row workgroups");
  if (failures) return 1;
  std::printf("ok %d\n", cases);
  return 0;
}
