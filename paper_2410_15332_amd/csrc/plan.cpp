// Host planner of the link step: integer work only, no device calls.
//
// Builds, for a batch of requests, the selected set S (LegoLink-k, Sec. 4.2:
// the first k tokens of every chunk but the first, plus the suffix; k < 0 =
// every token, Sec. 2.3), the linked block tables (chunks concatenated in
// order, then the suffix), the request-private blocks that receive recomputed
// K/V (copy-on-write when a block also keeps cached rows), and the attention
// work decomposition (query tiles x split-KV key ranges).
#include <algorithm>
#include <cstring>
#include <functional>
#include <vector>

#include "plan_internal.h"
#include "status.h"

namespace epic {

epic_status validate_attn_cfg(const epic_attn_cfg* cfg) {
  EPIC_CHECK_ARG(cfg != nullptr, "attention config is NULL");
  if (cfg->num_kv_heads <= 0 || cfg->num_q_heads <= 0 || cfg->num_q_heads % cfg->num_kv_heads != 0)
    return fail(EPIC_ERR_INVALID_ARG, "num_q_heads (%d) must be a positive multiple of num_kv_heads (%d)",
                cfg->num_q_heads, cfg->num_kv_heads);
  const int G = cfg->num_q_heads / cfg->num_kv_heads;
  if ((G & (G - 1)) != 0 || G > kTileRowsSmall)
    return fail(EPIC_ERR_UNSUPPORTED, "query heads per KV head (%d) must be a power of two <= %d", G,
                kTileRowsSmall);
  if (cfg->head_dim != 64 && cfg->head_dim != 128)
    return fail(EPIC_ERR_UNSUPPORTED, "head_dim %d not supported (64 or 128)", cfg->head_dim);
  if (cfg->block_size != kBlock)
    return fail(EPIC_ERR_UNSUPPORTED, "block_size %d not supported (16)", cfg->block_size);
  if (cfg->kv_split_blocks < 0)
    return fail(EPIC_ERR_INVALID_ARG, "kv_split_blocks %d < 0", cfg->kv_split_blocks);
  if (cfg->tile_rows != 0 && !valid_tile_rows(cfg->tile_rows))
    return fail(EPIC_ERR_UNSUPPORTED, "tile_rows %d (expected 0, %d, %d or %d)", cfg->tile_rows, kTileRowsTiny,
                kTileRowsSmall, kTileRowsLarge);
  if (cfg->tile_rows == kTileRowsTiny && G > kTileRowsTiny)
    return fail(EPIC_ERR_UNSUPPORTED, "tile_rows %d needs at most %d query heads per KV head (%d)", kTileRowsTiny,
                kTileRowsTiny, G);
  if (!(cfg->softmax_scale >= 0.0f)) return fail(EPIC_ERR_INVALID_ARG, "softmax_scale must be >= 0");
  return EPIC_OK;
}

namespace {

int cdiv(int64_t a, int64_t b) { return static_cast<int>((a + b - 1) / b); }

struct ReqShape {
  int64_t n_chunk_tokens = 0;
  int n_s = 0, n_lb = 0, n_priv = 0, n_rerot = 0;
};

// Re-rotation applies to the cached rows of chunks after the first (chunk 0 sits
// at offset 0, where the compile rotation is already the linked one).
bool rerotates(const epic_link_request& r, int j) { return r.rerotate != 0 && r.k >= 0 && j > 0; }

// Number of tokens of chunk j that belong to S.
int selected_in_chunk(const epic_link_request& r, int j) {
  if (r.k < 0) return r.chunk_len[j];
  if (j == 0) return 0;  // the first chunk is never recomputed
  return std::min(r.k, r.chunk_len[j]);
}

epic_status validate_request(const epic_link_request& r, int idx, ReqShape* sh) {
  EPIC_CHECK_ARG(r.num_chunks >= 0, "request %d: num_chunks %d < 0", idx, r.num_chunks);
  EPIC_CHECK_ARG(r.suffix_len >= 0, "request %d: suffix_len %d < 0", idx, r.suffix_len);
  EPIC_CHECK_ARG(r.rerotate == 0 || r.rerotate == 1, "request %d: rerotate %d (0 or 1)", idx, r.rerotate);
  if (r.num_chunks > 0) {
    EPIC_CHECK_ARG(r.chunk_len && r.chunk_block_off && r.chunk_blocks,
                   "request %d: chunk arrays are NULL", idx);
    EPIC_CHECK_ARG(r.chunk_block_off[0] == 0, "request %d: chunk_block_off[0] != 0", idx);
  }
  *sh = ReqShape{};
  for (int j = 0; j < r.num_chunks; ++j) {
    const int L = r.chunk_len[j];
    EPIC_CHECK_ARG(L >= 1, "request %d chunk %d: length %d < 1", idx, j, L);
    const int nb = r.chunk_block_off[j + 1] - r.chunk_block_off[j];
    EPIC_CHECK_ARG(nb == cdiv(L, kBlock), "request %d chunk %d: %d blocks given, %d needed", idx, j, nb,
                   cdiv(L, kBlock));
    sh->n_chunk_tokens += L;
    const int sel = selected_in_chunk(r, j);
    sh->n_s += sel;
    sh->n_lb += nb;
    if (rerotates(r, j)) {
      sh->n_priv += nb;                                   // every block: a rotated copy
      sh->n_rerot += sel >= L ? 0 : nb - sel / kBlock;    // those that keep a cached row
    } else {
      sh->n_priv += cdiv(sel, kBlock);
    }
  }
  sh->n_s += r.suffix_len;
  sh->n_lb += cdiv(r.suffix_len, kBlock);
  sh->n_priv += cdiv(r.suffix_len, kBlock);
  EPIC_CHECK_ARG(sh->n_chunk_tokens + r.suffix_len < (int64_t(1) << 30), "request %d: too many tokens", idx);
  return EPIC_OK;
}

// Linked positions of S for one request, ascending.
void select_positions(const epic_link_request& r, std::vector<int32_t>* pos) {
  int64_t off = 0;
  for (int j = 0; j < r.num_chunks; ++j) {
    const int sel = selected_in_chunk(r, j);
    for (int t = 0; t < sel; ++t) pos->push_back(static_cast<int32_t>(off + t));
    off += r.chunk_len[j];
  }
  for (int t = 0; t < r.suffix_len; ++t) pos->push_back(static_cast<int32_t>(off + t));
}

// Linked block table of one request: (pos0, len) of each block in position order.
void linked_blocks(const epic_link_request& r, std::vector<int32_t>* pos0, std::vector<int32_t>* len) {
  int64_t off = 0;
  for (int j = 0; j < r.num_chunks; ++j) {
    for (int t = 0; t < r.chunk_len[j]; t += kBlock) {
      pos0->push_back(static_cast<int32_t>(off + t));
      len->push_back(std::min(kBlock, r.chunk_len[j] - t));
    }
    off += r.chunk_len[j];
  }
  for (int t = 0; t < r.suffix_len; t += kBlock) {
    pos0->push_back(static_cast<int32_t>(off + t));
    len->push_back(std::min(kBlock, r.suffix_len - t));
  }
}

struct Tile {
  int req, row0, nrows, nblk;
};

// S positions and linked-block first positions of one request.
struct ReqRows {
  std::vector<int32_t> pos, p0;
};

// Query tiles: consecutive S rows of one request, rows_per_tile at a time.  A
// tile needs the linked blocks whose first position is <= its last row's position.
void make_tiles(const std::vector<ReqRows>& rr, int rows_per_tile, std::vector<Tile>* tiles) {
  int row_base = 0;
  for (size_t b = 0; b < rr.size(); ++b) {
    const std::vector<int32_t>& pos = rr[b].pos;
    const std::vector<int32_t>& p0 = rr[b].p0;
    for (size_t r0 = 0; r0 < pos.size(); r0 += rows_per_tile) {
      const int n = static_cast<int>(std::min<size_t>(rows_per_tile, pos.size() - r0));
      const int32_t last = pos[r0 + n - 1];
      const int nblk = static_cast<int>(std::upper_bound(p0.begin(), p0.end(), last) - p0.begin());
      tiles->push_back(Tile{static_cast<int>(b), row_base + static_cast<int>(r0), n, nblk});
    }
    row_base += static_cast<int>(pos.size());
  }
}

// Work items of a split, in launch order: longest key range first, so the
// dispatcher's greedy fill of freed workgroup slots ends with the short items;
// among equal lengths segment-major (all first segments, then all second
// segments, ...) and tiles with the longest key range first, so workgroups that
// start together read the same KV blocks through their XCD's L2.  Each entry:
// (tile, segment).
std::vector<std::pair<int, int>> item_order(const std::vector<Tile>& tiles, int split) {
  std::vector<int> order(tiles.size());
  for (size_t t = 0; t < tiles.size(); ++t) order[t] = static_cast<int>(t);
  std::stable_sort(order.begin(), order.end(), [&](int x, int y) { return tiles[x].nblk > tiles[y].nblk; });
  int max_splits = 1;
  for (const Tile& t : tiles) max_splits = std::max(max_splits, cdiv(t.nblk, split));
  std::vector<std::pair<int, int>> items;
  for (int seg = 0; seg < max_splits; ++seg)
    for (int t : order)
      if (seg < std::max(1, cdiv(tiles[t].nblk, split))) items.emplace_back(t, seg);
  auto blocks = [&](const std::pair<int, int>& it) {
    return std::min(tiles[it.first].nblk, (it.second + 1) * split) - it.second * split;
  };
  std::stable_sort(items.begin(), items.end(),
                   [&](const std::pair<int, int>& x, const std::pair<int, int>& y) { return blocks(x) > blocks(y); });
  return items;
}

// Kernel shape of a tile size: workgroup slots per launch round, and the time of
// one 64-key step of one workgroup and its fixed prologue / epilogue charge, in
// steps (the split search compares splits of one shape only).
// A split item also writes its fp32 partial tile, which the combine reads back.
struct TileShape {
  int rows, slots;
  double step_cost, item_overhead, partial_cost;
};
constexpr TileShape kShapeLarge{kTileRowsLarge, 256, 1.0, 3.0, 4.0};   // one 8-wavefront workgroup per CU, 256 CUs
constexpr TileShape kShapeSmall{kTileRowsSmall, 512, 1.0, 2.0, 4.0};   // two 4-wavefront workgroups per CU
constexpr TileShape kShapeTiny{kTileRowsTiny, 768, 1.0, 2.0, 1.0};      // three 4-wavefront workgroups per CU

// Estimated duration of the attention launch for a split: the items (times the
// KV heads, head-minor as in the grid) are dealt in launch order to the
// workgroup slots, each to the slot that frees up first -- as the hardware
// dispatcher does -- and an item costs its steps plus a fixed prologue /
// epilogue charge.
double estimate_makespan(const std::vector<Tile>& tiles, int split, int hkv, const TileShape& sh) {
  std::vector<double> slots(sh.slots, 0.0);   // min-heap of slot finish times
  double makespan = 0.0;
  for (const auto& [t, seg] : item_order(tiles, split)) {
    const int blocks = std::min(tiles[t].nblk, (seg + 1) * split) - seg * split;
    const bool partial = tiles[t].nblk > split;
    const double cost = cdiv(std::max(blocks, 1), kKvTileBlocks) * sh.step_cost + sh.item_overhead +
                        (partial ? sh.partial_cost : 0.0);
    for (int g = 0; g < hkv; ++g) {
      std::pop_heap(slots.begin(), slots.end(), std::greater<double>());
      slots.back() += cost;
      makespan = std::max(makespan, slots.back());
      std::push_heap(slots.begin(), slots.end(), std::greater<double>());
    }
  }
  return makespan;
}

// Key blocks per split-KV work item: among splits max_nblk / n (n from 1 to 128
// in about geometric steps, rounded up to whole 4-block tiles, never below 64
// blocks, because every split writes and re-reads a tile of fp32 partial
// results), the one with the shortest estimated launch, where a finer split
// must be 3% shorter to win (fewer partials).  *time receives that estimate.
int split_blocks(const epic_attn_cfg* cfg, const std::vector<Tile>& tiles, const TileShape& sh, double* time) {
  const int hkv = cfg->num_kv_heads;
  if (cfg->kv_split_blocks > 0) {
    const int split = std::max(kKvTileBlocks, cfg->kv_split_blocks / kKvTileBlocks * kKvTileBlocks);
    *time = estimate_makespan(tiles, split, hkv, sh);
    return split;
  }
  constexpr int kMinSplit = 64;
  constexpr int64_t kMaxRounds = 16;   // past this many dispatch rounds, splitting cannot balance better
  int max_nblk = kKvTileBlocks;
  for (const Tile& t : tiles) max_nblk = std::max(max_nblk, t.nblk);
  auto n_items = [&](int split) {
    int64_t n = 0;
    for (const Tile& t : tiles) n += std::max(1, cdiv(t.nblk, split));
    return n;
  };
  const int whole = cdiv(max_nblk, kKvTileBlocks) * kKvTileBlocks;
  int best = whole;
  double best_time = estimate_makespan(tiles, whole, hkv, sh);
  if (n_items(whole) * hkv < kMaxRounds * sh.slots) {
    int prev = whole;
    static constexpr int kParts[] = {2, 3, 4, 5, 6, 7, 8, 10, 12, 14, 16, 20, 24, 28, 32, 40, 48, 56, 64, 96, 128};
    for (const int n : kParts) {
      const int split = std::max(kMinSplit, cdiv(cdiv(max_nblk, n), kKvTileBlocks) * kKvTileBlocks);
      if (split >= prev) continue;
      prev = split;
      if (n_items(split) * hkv > kMaxRounds * sh.slots) break;
      const double t = estimate_makespan(tiles, split, hkv, sh);
      if (t < best_time * 0.97) {               // finer splits must pay for their partials clearly
        best_time = t;
        best = split;
      }
      if (split == kMinSplit) break;
    }
  }
  *time = best_time;
  return best;
}

int64_t align16(int64_t n) { return (n + 15) & ~int64_t(15); }

}  // namespace

}  // namespace epic

using namespace epic;

namespace {

// Tile size and split-KV split for these S rows; fills s->tile_rows, n_tiles,
// n_work, n_partials.  256-row tiles share each staged K/V block between twice
// the rows, which pays when their rows need nearly the same keys and the tiles
// still balance over the CUs.  Take them when they cost at most 5% more
// (row x 64-key) steps than 128-row tiles, their estimated launch is at most
// kLargeEdge times that of 128-row tiles (each estimate in its own kernel's
// steps: the 8-wavefront kernel runs a 256-row step in about 1/1.07-1/1.13 of
// the time two 4-wavefront workgroups take for two 128-row steps, measured), and
// they give every CU a workgroup.
void choose_tiles(const std::vector<ReqRows>& rr, const epic_attn_cfg* cfg, epic_plan_sizes* s,
                  std::vector<Tile>* tiles_out, int* split_out) {
  const int G = cfg->num_q_heads / cfg->num_kv_heads;
  std::vector<Tile>& tiles = *tiles_out;
  // 16-row tiles (the decode kernel) when every request has at most 16 / G S rows:
  // a 128-row tile would hold almost only empty rows
  bool few_rows = G <= kTileRowsTiny;
  size_t any_rows = 0;
  for (const ReqRows& r : rr) {
    few_rows = few_rows && r.pos.size() <= static_cast<size_t>(kTileRowsTiny / G);
    any_rows += r.pos.size();
  }
  if (cfg->tile_rows == kTileRowsTiny || (cfg->tile_rows == 0 && few_rows && any_rows > 0)) {
    make_tiles(rr, kTileRowsTiny / G, &tiles);
    s->tile_rows = kTileRowsTiny;
    double est = 0.0;
    const int split = split_blocks(cfg, tiles, kShapeTiny, &est);
    *split_out = split;
    int64_t n_work = 0, n_part = 0;
    for (const Tile& t : tiles) {
      const int ns = std::max(1, cdiv(t.nblk, split));
      n_work += ns;
      if (ns > 1) n_part += ns;
    }
    s->n_tiles = static_cast<int32_t>(tiles.size());
    s->n_work = static_cast<int32_t>(n_work);
    s->n_partials = static_cast<int32_t>(n_part);
    return;
  }
  std::vector<Tile> small, large;
  make_tiles(rr, kTileRowsSmall / G, &small);
  make_tiles(rr, kTileRowsLarge / G, &large);
  auto row_steps = [](const std::vector<Tile>& ts, int rows) {
    int64_t n = 0;
    for (const Tile& t : ts) n += int64_t(cdiv(t.nblk, kKvTileBlocks)) * rows;
    return n;
  };
  constexpr double kLargeEdge = 1.07;
  double est = 0.0, est_small = 0.0;
  int split = split_blocks(cfg, large, kShapeLarge, &est);
  int64_t large_items = 0;
  for (const Tile& t : large) large_items += std::max(1, cdiv(t.nblk, split));
  bool use_large = cfg->tile_rows == kTileRowsLarge;
  int split_small = 0;
  if (cfg->tile_rows == 0 && row_steps(large, kTileRowsLarge) * 100 <= row_steps(small, kTileRowsSmall) * 105 &&
      large_items * cfg->num_kv_heads >= kShapeLarge.slots) {
    split_small = split_blocks(cfg, small, kShapeSmall, &est_small);
    use_large = est <= kLargeEdge * est_small;
  }
  if (use_large) {
    tiles.swap(large);
    s->tile_rows = kTileRowsLarge;
  } else {
    tiles.swap(small);
    s->tile_rows = kTileRowsSmall;
    split = split_small > 0 ? split_small : split_blocks(cfg, tiles, kShapeSmall, &est);
  }
  *split_out = split;
  int64_t n_work = 0, n_part = 0;
  for (const Tile& t : tiles) {
    const int ns = std::max(1, cdiv(t.nblk, split));
    n_work += ns;
    if (ns > 1) n_part += ns;
  }
  s->n_tiles = static_cast<int32_t>(tiles.size());
  s->n_work = static_cast<int32_t>(n_work);
  s->n_partials = static_cast<int32_t>(n_part);
}

void finish_sizes(epic_plan_sizes* s) {
  s->total_ints = 3 * align16(s->n_s) + 2 * align16(s->batch + 1) + 3 * align16(s->n_linked_blocks) +
                  3 * align16(s->n_private) + align16(int64_t(s->n_private) * kBlock) +
                  align16(4 * int64_t(s->n_tiles)) + align16(kWorkInts * int64_t(s->n_work));
}

// Attention tiles and split-KV work items of a plan whose S rows and linked
// tables are written.  Work items go in item_order's launch order (longest key
// range first; among equal lengths key segment first, so that workgroups that
// start together read the same KV blocks through their XCD's L2).
epic_status write_work(const std::vector<Tile>& tiles, int split, const epic_plan_sizes& chk, epic_plan* plan) {
  int part = 0;
  for (size_t t = 0; t < tiles.size(); ++t) {
    const int ns = std::max(1, cdiv(tiles[t].nblk, split));
    plan->tiles[4 * t + 0] = tiles[t].row0;
    plan->tiles[4 * t + 1] = tiles[t].nrows;
    plan->tiles[4 * t + 2] = ns > 1 ? part : -1;
    plan->tiles[4 * t + 3] = ns;
    if (ns > 1) part += ns;
  }
  // work items in launch order
  int w = 0;
  for (const auto& [t, seg] : item_order(tiles, split)) {
    const int ns = plan->tiles[4 * t + 3];
    const int base = plan->blk_off[tiles[t].req];
    const int b0 = base + seg * split;
    const int b1 = base + std::min(tiles[t].nblk, (seg + 1) * split);
    // Leading KV tiles (kKvTileBlocks blocks each) that need no mask: all
    // blocks full and every key at or before the tile's first row.
    const int32_t first_pos = plan->s_pos[tiles[t].row0];
    int n_fast = 0;
    for (int b = b0; b + kKvTileBlocks <= b1; b += kKvTileBlocks) {
      bool ok = true;
      for (int i = 0; i < kKvTileBlocks; ++i) ok = ok && plan->block_len[b + i] == kBlock;
      const int last = b + kKvTileBlocks - 1;
      ok = ok && plan->block_pos0[last] + kBlock - 1 <= first_pos;
      if (!ok) break;
      ++n_fast;
    }
    int32_t* wk = plan->work + int64_t(kWorkInts) * w;
    wk[0] = static_cast<int32_t>(t);
    wk[1] = b0;
    wk[2] = b1;
    wk[3] = ns > 1 ? plan->tiles[4 * t + 2] + seg : -1;
    wk[4] = n_fast;
    wk[5] = wk[6] = wk[7] = 0;
    ++w;
  }
  if (w != chk.n_work || part != chk.n_partials)
    return fail(EPIC_ERR_INVALID_ARG, "internal planner inconsistency (work)");
  return EPIC_OK;
}

// Sizes of the link plan, plus its attention tiles and split (shared by the sizes
// query and the plan builder, so the split search runs once per call).
epic_status plan_shape(const epic_link_request* reqs, int32_t batch, const epic_attn_cfg* cfg, int32_t n_free,
                       epic_plan_sizes* out, std::vector<Tile>* tiles_out, int* split_out) {
  EPIC_CHECK_ARG(out != nullptr, "output sizes pointer is NULL");
  EPIC_CHECK_ARG(batch >= 0, "batch %d < 0", batch);
  EPIC_CHECK_ARG(batch == 0 || reqs != nullptr, "requests pointer is NULL");
  EPIC_CHECK_ARG(n_free >= 0, "n_free %d < 0", n_free);
  epic_status st = validate_attn_cfg(cfg);
  if (st != EPIC_OK) return st;
  epic_plan_sizes s{};
  s.batch = batch;
  int64_t n_s = 0, n_lb = 0, n_priv = 0, n_rerot = 0, max_pos = 0;
  for (int b = 0; b < batch; ++b) {
    ReqShape sh;
    st = validate_request(reqs[b], b, &sh);
    if (st != EPIC_OK) return st;
    n_s += sh.n_s;
    n_lb += sh.n_lb;
    n_priv += sh.n_priv;
    n_rerot += sh.n_rerot;
    max_pos = std::max<int64_t>(max_pos, sh.n_chunk_tokens + reqs[b].suffix_len);
  }
  EPIC_CHECK_ARG(n_s < (int64_t(1) << 30) && n_lb < (int64_t(1) << 30), "batch too large");
  if (n_priv > n_free)
    return fail(EPIC_ERR_NO_PRIVATE_BLOCKS, "plan needs %lld private blocks, %d free", (long long)n_priv, n_free);
  std::vector<ReqRows> rr(static_cast<size_t>(batch));
  for (int b = 0; b < batch; ++b) {
    std::vector<int32_t> ln;
    select_positions(reqs[b], &rr[b].pos);
    linked_blocks(reqs[b], &rr[b].p0, &ln);
  }
  choose_tiles(rr, cfg, &s, tiles_out, split_out);
  s.n_s = static_cast<int32_t>(n_s);
  s.n_linked_blocks = static_cast<int32_t>(n_lb);
  s.n_private = static_cast<int32_t>(n_priv);
  s.n_rerotated = static_cast<int32_t>(n_rerot);
  s.max_pos = static_cast<int32_t>(max_pos);
  finish_sizes(&s);
  *out = s;
  return EPIC_OK;
}

}  // namespace

extern "C" epic_status epic_plan_sizes_get(const epic_link_request* reqs, int32_t batch,
                                           const epic_attn_cfg* cfg, int32_t n_free,
                                           epic_plan_sizes* out) {
  clear_error();
  std::vector<Tile> tiles;
  int split = 0;
  return plan_shape(reqs, batch, cfg, n_free, out, &tiles, &split);
}

extern "C" epic_status epic_plan_layout(const epic_plan_sizes* s, int32_t* base, epic_plan* p) {
  clear_error();
  EPIC_CHECK_ARG(s && p, "NULL argument");
  int32_t* cur = base;
  auto take = [&](int64_t n) {
    int32_t* r = cur;
    cur += align16(n);
    return r;
  };
  p->s_pos = take(s->n_s);
  p->s_req = take(s->n_s);
  p->s_slot = take(s->n_s);
  p->s_off = take(s->batch + 1);
  p->linked_blocks = take(s->n_linked_blocks);
  p->block_pos0 = take(s->n_linked_blocks);
  p->block_len = take(s->n_linked_blocks);
  p->blk_off = take(s->batch + 1);
  p->priv_block = take(s->n_private);
  p->priv_src = take(s->n_private);
  p->priv_rows = take(int64_t(s->n_private) * kBlock);
  p->tiles = take(4 * int64_t(s->n_tiles));
  p->work = take(kWorkInts * int64_t(s->n_work));
  p->priv_rot = take(s->n_private);
  if (cur - base != s->total_ints) return fail(EPIC_ERR_INVALID_ARG, "plan sizes are inconsistent");
  return EPIC_OK;
}

extern "C" epic_status epic_plan_link(const epic_link_request* reqs, int32_t batch,
                                      const epic_attn_cfg* cfg, const int32_t* free_blocks,
                                      int32_t n_free, int32_t num_blocks,
                                      const epic_plan_sizes* sizes, epic_plan* plan) {
  clear_error();
  epic_plan_sizes chk;
  std::vector<Tile> tiles;
  int split = 0;
  epic_status st = plan_shape(reqs, batch, cfg, n_free, &chk, &tiles, &split);
  if (st != EPIC_OK) return st;
  EPIC_CHECK_ARG(sizes && plan, "NULL sizes or plan");
  EPIC_CHECK_ARG(std::memcmp(&chk, sizes, sizeof(chk)) == 0, "sizes do not match these requests");
  EPIC_CHECK_ARG(num_blocks > 0, "num_blocks %d <= 0", num_blocks);
  EPIC_CHECK_ARG(chk.n_private == 0 || free_blocks != nullptr, "free_blocks is NULL");

  // Block ids: chunk blocks and free blocks in range, free blocks distinct and unused by chunks.
  std::vector<uint8_t> used(static_cast<size_t>(num_blocks), 0);
  for (int b = 0; b < batch; ++b) {
    const epic_link_request& r = reqs[b];
    const int nb = r.num_chunks > 0 ? r.chunk_block_off[r.num_chunks] : 0;
    for (int i = 0; i < nb; ++i) {
      const int id = r.chunk_blocks[i];
      EPIC_CHECK_ARG(id >= 0 && id < num_blocks, "request %d: chunk block id %d out of range [0, %d)", b, id,
                     num_blocks);
      used[id] = 1;
    }
  }
  for (int i = 0; i < chk.n_private; ++i) {
    const int id = free_blocks[i];
    EPIC_CHECK_ARG(id >= 0 && id < num_blocks, "free block id %d out of range [0, %d)", id, num_blocks);
    EPIC_CHECK_ARG(used[id] == 0, "free block %d is a chunk block or listed twice", id);
    used[id] = 2;
  }

  const int bs = kBlock;
  int row = 0, lb = 0, pv = 0;
  for (int b = 0; b < batch; ++b) {
    const epic_link_request& r = reqs[b];
    plan->s_off[b] = row;
    plan->blk_off[b] = lb;
    int64_t off = 0;
    // chunk tokens
    for (int j = 0; j < r.num_chunks; ++j) {
      const int L = r.chunk_len[j];
      const int sel = selected_in_chunk(r, j);  // tokens [0, sel) of the chunk are in S
      const int32_t* cb = r.chunk_blocks + r.chunk_block_off[j];
      for (int i = 0; i * bs < L; ++i) {
        const int t0 = i * bs, len = std::min(bs, L - t0);
        plan->block_pos0[lb] = static_cast<int32_t>(off + t0);
        plan->block_len[lb] = len;
        if (t0 < sel || rerotates(r, j)) {
          const int id = free_blocks[pv];
          const bool keeps_cached = sel < t0 + len;  // some valid slot is not recomputed
          plan->priv_block[pv] = id;
          plan->priv_src[pv] = keeps_cached ? cb[i] : -1;
          plan->priv_rot[pv] = keeps_cached && rerotates(r, j) ? static_cast<int32_t>(off) : 0;
          for (int o = 0; o < bs; ++o) {
            const int t = t0 + o;
            int32_t rr = -1;
            if (t < sel) {
              rr = row++;
              plan->s_pos[rr] = static_cast<int32_t>(off + t);
              plan->s_req[rr] = b;
              plan->s_slot[rr] = id * bs + o;
            }
            plan->priv_rows[int64_t(pv) * bs + o] = rr;
          }
          plan->linked_blocks[lb] = id;
          ++pv;
        } else {
          plan->linked_blocks[lb] = cb[i];
        }
        ++lb;
      }
      off += L;
    }
    // suffix tokens: all new, all in S
    for (int t0 = 0; t0 < r.suffix_len; t0 += bs) {
      const int len = std::min(bs, r.suffix_len - t0);
      const int id = free_blocks[pv];
      plan->block_pos0[lb] = static_cast<int32_t>(off + t0);
      plan->block_len[lb] = len;
      plan->linked_blocks[lb] = id;
      plan->priv_block[pv] = id;
      plan->priv_src[pv] = -1;
      plan->priv_rot[pv] = 0;
      for (int o = 0; o < bs; ++o) {
        int32_t rr = -1;
        if (o < len) {
          rr = row++;
          plan->s_pos[rr] = static_cast<int32_t>(off + t0 + o);
          plan->s_req[rr] = b;
          plan->s_slot[rr] = id * bs + o;
        }
        plan->priv_rows[int64_t(pv) * bs + o] = rr;
      }
      ++pv;
      ++lb;
    }
  }
  plan->s_off[batch] = row;
  plan->blk_off[batch] = lb;
  if (row != chk.n_s || lb != chk.n_linked_blocks || pv != chk.n_private)
    return fail(EPIC_ERR_INVALID_ARG, "internal planner inconsistency");

  return write_work(tiles, split, chk, plan);
}

// ---------------------------------------------------------------- decode

namespace {

// One request of a decode plan: its blocks in the previous plan, its length there,
// the free slots of its last block when that block may take the new tokens, and
// the new blocks it needs.
struct DecodeReq {
  int a = 0, e = 0;        // linked blocks [a, e) of the previous plan
  int64_t n = 0;           // tokens linked so far
  int t = 0;               // new tokens
  int room = 0;            // new tokens that go into the last block
  int extra = 0;           // new blocks
};

epic_status decode_shape(const epic_plan_sizes* ps, const epic_plan* prev, const int32_t* new_tokens,
                         const epic_attn_cfg* cfg, int32_t n_free, epic_plan_sizes* out,
                         std::vector<Tile>* tiles_out, int* split_out, std::vector<DecodeReq>* dr_out) {
  EPIC_CHECK_ARG(ps && prev && out, "NULL previous plan, sizes or output");
  EPIC_CHECK_ARG(n_free >= 0, "n_free %d < 0", n_free);
  epic_status st = validate_attn_cfg(cfg);
  if (st != EPIC_OK) return st;
  const int batch = ps->batch;
  EPIC_CHECK_ARG(batch == 0 || (new_tokens && prev->blk_off && prev->linked_blocks && prev->block_pos0 &&
                                prev->block_len),
                 "NULL new_tokens or previous plan array");
  EPIC_CHECK_ARG(ps->n_private == 0 || prev->priv_block, "previous plan has no private block list");
  // blocks the previous step wrote: only those may take further tokens
  std::vector<int32_t> written(prev->priv_block, prev->priv_block + ps->n_private);
  std::sort(written.begin(), written.end());
  std::vector<DecodeReq>& dr = *dr_out;
  dr.assign(static_cast<size_t>(batch), DecodeReq{});
  std::vector<ReqRows> rr(static_cast<size_t>(batch));
  int64_t n_s = 0, n_lb = 0, n_priv = 0, n_take = 0, max_pos = 0;
  for (int b = 0; b < batch; ++b) {
    DecodeReq& d = dr[b];
    d.a = prev->blk_off[b];
    d.e = prev->blk_off[b + 1];
    EPIC_CHECK_ARG(0 <= d.a && d.a <= d.e && d.e <= ps->n_linked_blocks, "previous plan: bad blk_off at %d", b);
    d.t = new_tokens[b];
    EPIC_CHECK_ARG(d.t >= 0, "request %d: %d new tokens", b, d.t);
    for (int i = d.a; i < d.e; ++i) rr[b].p0.push_back(prev->block_pos0[i]);
    if (d.e > d.a) {
      const int last = d.e - 1, len = prev->block_len[last];
      d.n = int64_t(prev->block_pos0[last]) + len;
      if (len < kBlock && std::binary_search(written.begin(), written.end(), prev->linked_blocks[last]))
        d.room = std::min(d.t, kBlock - len);
    }
    d.extra = cdiv(d.t - d.room, kBlock);
    EPIC_CHECK_ARG(d.n + d.t < (int64_t(1) << 30), "request %d: too many tokens", b);
    for (int i = 0; i < d.extra; ++i) rr[b].p0.push_back(static_cast<int32_t>(d.n + d.room + int64_t(i) * kBlock));
    for (int i = 0; i < d.t; ++i) rr[b].pos.push_back(static_cast<int32_t>(d.n + i));
    n_s += d.t;
    n_lb += (d.e - d.a) + d.extra;
    n_priv += (d.room > 0 ? 1 : 0) + d.extra;
    n_take += d.extra;
    max_pos = std::max<int64_t>(max_pos, d.n + d.t);
  }
  EPIC_CHECK_ARG(n_s < (int64_t(1) << 30) && n_lb < (int64_t(1) << 30), "batch too large");
  if (n_take > n_free)
    return fail(EPIC_ERR_NO_PRIVATE_BLOCKS, "plan needs %lld new blocks, %d free", (long long)n_take, n_free);
  epic_plan_sizes s{};
  s.batch = batch;
  choose_tiles(rr, cfg, &s, tiles_out, split_out);
  s.n_s = static_cast<int32_t>(n_s);
  s.n_linked_blocks = static_cast<int32_t>(n_lb);
  s.n_private = static_cast<int32_t>(n_priv);
  s.max_pos = static_cast<int32_t>(max_pos);
  finish_sizes(&s);
  *out = s;
  return EPIC_OK;
}

}  // namespace

extern "C" epic_status epic_plan_decode_sizes(const epic_plan_sizes* prev_sizes, const epic_plan* prev,
                                              const int32_t* new_tokens, const epic_attn_cfg* cfg, int32_t n_free,
                                              epic_plan_sizes* out) {
  clear_error();
  std::vector<Tile> tiles;
  std::vector<DecodeReq> dr;
  int split = 0;
  return decode_shape(prev_sizes, prev, new_tokens, cfg, n_free, out, &tiles, &split, &dr);
}

extern "C" epic_status epic_plan_decode(const epic_plan_sizes* prev_sizes, const epic_plan* prev,
                                        const int32_t* new_tokens, const epic_attn_cfg* cfg,
                                        const int32_t* free_blocks, int32_t n_free, int32_t num_blocks,
                                        const epic_plan_sizes* sizes, epic_plan* plan) {
  clear_error();
  epic_plan_sizes chk;
  std::vector<Tile> tiles;
  std::vector<DecodeReq> dr;
  int split = 0;
  epic_status st = decode_shape(prev_sizes, prev, new_tokens, cfg, n_free, &chk, &tiles, &split, &dr);
  if (st != EPIC_OK) return st;
  EPIC_CHECK_ARG(sizes && plan, "NULL sizes or plan");
  EPIC_CHECK_ARG(std::memcmp(&chk, sizes, sizeof(chk)) == 0, "sizes do not match this previous plan");
  EPIC_CHECK_ARG(num_blocks > 0, "num_blocks %d <= 0", num_blocks);
  int64_t n_take = 0;
  for (const DecodeReq& d : dr) n_take += d.extra;
  EPIC_CHECK_ARG(n_take == 0 || free_blocks != nullptr, "free_blocks is NULL");
  // free blocks: in range, distinct, not linked by the previous plan
  std::vector<uint8_t> used(static_cast<size_t>(num_blocks), 0);
  for (int i = 0; i < prev_sizes->n_linked_blocks; ++i) {
    const int id = prev->linked_blocks[i];
    EPIC_CHECK_ARG(id >= 0 && id < num_blocks, "previous plan: block id %d out of range [0, %d)", id, num_blocks);
    used[id] = 1;
  }
  for (int64_t i = 0; i < n_take; ++i) {
    const int id = free_blocks[i];
    EPIC_CHECK_ARG(id >= 0 && id < num_blocks, "free block id %d out of range [0, %d)", id, num_blocks);
    EPIC_CHECK_ARG(used[id] == 0, "free block %d is already linked or listed twice", id);
    used[id] = 2;
  }
  const int bs = kBlock;
  int row = 0, lb = 0, pv = 0, fl = 0;
  auto add_row = [&](int b, int64_t pos, int id, int o) {
    plan->s_pos[row] = static_cast<int32_t>(pos);
    plan->s_req[row] = b;
    plan->s_slot[row] = id * bs + o;
    return row++;
  };
  for (int b = 0; b < chk.batch; ++b) {
    const DecodeReq& d = dr[b];
    plan->s_off[b] = row;
    plan->blk_off[b] = lb;
    for (int i = d.a; i < d.e; ++i, ++lb) {
      plan->linked_blocks[lb] = prev->linked_blocks[i];
      plan->block_pos0[lb] = prev->block_pos0[i];
      plan->block_len[lb] = prev->block_len[i] + (i == d.e - 1 ? d.room : 0);
    }
    int64_t pos = d.n;
    if (d.room > 0) {                          // the last block takes the first new tokens
      const int id = prev->linked_blocks[d.e - 1], len = prev->block_len[d.e - 1];
      plan->priv_block[pv] = id;
      plan->priv_src[pv] = id;                 // its earlier tokens stay: copied onto themselves
      plan->priv_rot[pv] = 0;
      for (int o = 0; o < bs; ++o)
        plan->priv_rows[int64_t(pv) * bs + o] = (o >= len && o < len + d.room) ? add_row(b, pos++, id, o) : -1;
      ++pv;
    }
    for (int i = 0; i < d.extra; ++i, ++lb, ++pv) {
      const int id = free_blocks[fl++];
      const int len = static_cast<int>(std::min<int64_t>(bs, d.n + d.t - pos));
      plan->linked_blocks[lb] = id;
      plan->block_pos0[lb] = static_cast<int32_t>(pos);
      plan->block_len[lb] = len;
      plan->priv_block[pv] = id;
      plan->priv_src[pv] = -1;
      plan->priv_rot[pv] = 0;
      for (int o = 0; o < bs; ++o) plan->priv_rows[int64_t(pv) * bs + o] = o < len ? add_row(b, pos++, id, o) : -1;
    }
  }
  plan->s_off[chk.batch] = row;
  plan->blk_off[chk.batch] = lb;
  if (row != chk.n_s || lb != chk.n_linked_blocks || pv != chk.n_private || fl != n_take)
    return fail(EPIC_ERR_INVALID_ARG, "internal planner inconsistency (decode)");
  return write_work(tiles, split, chk, plan);
}

// ---------------------------------------------------------------- compile

namespace {

// The compile step (Sec. 2.2) prefills every chunk alone; LegoLink-0 (Sec. 5.4)
// first prepends n_dummy dummy tokens to each chunk and afterwards drops their
// K/V.  Each chunk is one request of the plan: S = its n_dummy + L tokens at
// positions 0 .. n_dummy + L - 1, the dummies first.  Without dummies the
// chunk's own blocks are its linked (attention) blocks.  With dummies the
// attention reads n_dummy + L tokens from staging blocks taken from the free
// list, and the chunk's blocks are further private blocks outside the linked
// table that receive chunk token t at slot t (rows n_dummy + t).
epic_status compile_shape(const epic_compile_batch* cb, const epic_attn_cfg* cfg, int32_t n_free,
                          epic_plan_sizes* out, std::vector<Tile>* tiles_out, int* split_out,
                          int64_t* n_staging) {
  EPIC_CHECK_ARG(cb && out, "NULL compile batch or output sizes");
  EPIC_CHECK_ARG(n_free >= 0, "n_free %d < 0", n_free);
  epic_status st = validate_attn_cfg(cfg);
  if (st != EPIC_OK) return st;
  const int n = cb->num_chunks;
  EPIC_CHECK_ARG(n >= 0, "num_chunks %d < 0", n);
  EPIC_CHECK_ARG(cb->n_dummy >= 0 && cb->n_dummy <= (1 << 20), "n_dummy %d outside [0, 2^20]", cb->n_dummy);
  if (n > 0) {
    EPIC_CHECK_ARG(cb->chunk_len && cb->chunk_block_off && cb->chunk_blocks, "chunk arrays are NULL");
    EPIC_CHECK_ARG(cb->chunk_block_off[0] == 0, "chunk_block_off[0] != 0");
  }
  const int nd = cb->n_dummy;
  std::vector<ReqRows> rr(static_cast<size_t>(n));
  int64_t n_s = 0, n_lb = 0, n_priv = 0, stage = 0, max_pos = 0;
  for (int j = 0; j < n; ++j) {
    const int L = cb->chunk_len[j];
    EPIC_CHECK_ARG(L >= 1, "chunk %d: length %d < 1", j, L);
    EPIC_CHECK_ARG(int64_t(L) + nd < (int64_t(1) << 30), "chunk %d: too many tokens", j);
    const int nb = cb->chunk_block_off[j + 1] - cb->chunk_block_off[j];
    EPIC_CHECK_ARG(nb == cdiv(L, kBlock), "chunk %d: %d blocks given, %d needed", j, nb, cdiv(L, kBlock));
    const int total = nd + L, lb = cdiv(total, kBlock);
    for (int p = 0; p < total; ++p) rr[j].pos.push_back(p);
    for (int i = 0; i < lb; ++i) rr[j].p0.push_back(i * kBlock);
    n_s += total;
    n_lb += lb;
    n_priv += nb + (nd > 0 ? lb : 0);
    stage += nd > 0 ? lb : 0;
    max_pos = std::max<int64_t>(max_pos, total);
  }
  EPIC_CHECK_ARG(n_s < (int64_t(1) << 30) && n_priv < (int64_t(1) << 30), "batch too large");
  if (stage > n_free)
    return fail(EPIC_ERR_NO_PRIVATE_BLOCKS, "plan needs %lld staging blocks, %d free", (long long)stage, n_free);
  epic_plan_sizes s{};
  s.batch = n;
  choose_tiles(rr, cfg, &s, tiles_out, split_out);
  s.n_s = static_cast<int32_t>(n_s);
  s.n_linked_blocks = static_cast<int32_t>(n_lb);
  s.n_private = static_cast<int32_t>(n_priv);
  s.max_pos = static_cast<int32_t>(max_pos);
  finish_sizes(&s);
  *out = s;
  *n_staging = stage;
  return EPIC_OK;
}

}  // namespace

extern "C" epic_status epic_plan_compile_sizes(const epic_compile_batch* batch, const epic_attn_cfg* cfg,
                                               int32_t n_free, epic_plan_sizes* out) {
  clear_error();
  std::vector<Tile> tiles;
  int split = 0;
  int64_t stage = 0;
  return compile_shape(batch, cfg, n_free, out, &tiles, &split, &stage);
}

extern "C" epic_status epic_plan_compile(const epic_compile_batch* batch, const epic_attn_cfg* cfg,
                                         const int32_t* free_blocks, int32_t n_free, int32_t num_blocks,
                                         const epic_plan_sizes* sizes, epic_plan* plan) {
  clear_error();
  epic_plan_sizes chk;
  std::vector<Tile> tiles;
  int split = 0;
  int64_t stage = 0;
  epic_status st = compile_shape(batch, cfg, n_free, &chk, &tiles, &split, &stage);
  if (st != EPIC_OK) return st;
  EPIC_CHECK_ARG(sizes && plan, "NULL sizes or plan");
  EPIC_CHECK_ARG(std::memcmp(&chk, sizes, sizeof(chk)) == 0, "sizes do not match this compile batch");
  EPIC_CHECK_ARG(num_blocks > 0, "num_blocks %d <= 0", num_blocks);
  EPIC_CHECK_ARG(stage == 0 || free_blocks != nullptr, "free_blocks is NULL");
  const int n = batch->num_chunks, nd = batch->n_dummy, bs = kBlock;
  // every block is written: chunk blocks and staging blocks in range and all distinct
  std::vector<uint8_t> used(static_cast<size_t>(num_blocks), 0);
  const int n_chunk_blocks = n > 0 ? batch->chunk_block_off[n] : 0;
  for (int i = 0; i < n_chunk_blocks; ++i) {
    const int id = batch->chunk_blocks[i];
    EPIC_CHECK_ARG(id >= 0 && id < num_blocks, "chunk block id %d out of range [0, %d)", id, num_blocks);
    EPIC_CHECK_ARG(used[id] == 0, "chunk block %d is listed twice", id);
    used[id] = 1;
  }
  for (int64_t i = 0; i < stage; ++i) {
    const int id = free_blocks[i];
    EPIC_CHECK_ARG(id >= 0 && id < num_blocks, "free block id %d out of range [0, %d)", id, num_blocks);
    EPIC_CHECK_ARG(used[id] == 0, "free block %d is a chunk block or listed twice", id);
    used[id] = 2;
  }
  int row = 0, lb = 0, pv = 0, fl = 0;
  for (int j = 0; j < n; ++j) {
    const int L = batch->chunk_len[j], total = nd + L;
    const int32_t* cbk = batch->chunk_blocks + batch->chunk_block_off[j];
    const int row0 = row;
    plan->s_off[j] = row;
    plan->blk_off[j] = lb;
    // linked (attention) blocks: the chunk's own blocks, or staging blocks with dummies
    for (int i = 0; i * bs < total; ++i, ++lb, ++pv) {
      const int id = nd > 0 ? free_blocks[fl++] : cbk[i];
      const int len = std::min(bs, total - i * bs);
      plan->linked_blocks[lb] = id;
      plan->block_pos0[lb] = i * bs;
      plan->block_len[lb] = len;
      plan->priv_block[pv] = id;
      plan->priv_src[pv] = -1;
      plan->priv_rot[pv] = 0;
      for (int o = 0; o < bs; ++o) {
        int32_t r = -1;
        if (o < len) {
          r = row++;
          plan->s_pos[r] = i * bs + o;
          plan->s_req[r] = j;
          plan->s_slot[r] = id * bs + o;
        }
        plan->priv_rows[int64_t(pv) * bs + o] = r;
      }
    }
    // the chunk's cache without the dummies: chunk token t (row row0 + nd + t) at slot t
    if (nd > 0) {
      for (int i = 0; i * bs < L; ++i, ++pv) {
        plan->priv_block[pv] = cbk[i];
        plan->priv_src[pv] = -1;
        plan->priv_rot[pv] = 0;
        for (int o = 0; o < bs; ++o) {
          const int t = i * bs + o;
          plan->priv_rows[int64_t(pv) * bs + o] = t < L ? row0 + nd + t : -1;
        }
      }
    }
  }
  plan->s_off[n] = row;
  plan->blk_off[n] = lb;
  if (row != chk.n_s || lb != chk.n_linked_blocks || pv != chk.n_private || fl != stage)
    return fail(EPIC_ERR_INVALID_ARG, "internal planner inconsistency (compile)");
  return write_work(tiles, split, chk, plan);
}
