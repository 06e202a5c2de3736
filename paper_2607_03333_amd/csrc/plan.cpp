#include "plan.h"

#include <algorithm>
#include <climits>
#include <cstring>
#include <map>
#include <queue>

namespace spork {
namespace {

size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

// A context range [lo, hi) read by the rows of `threads`, through the block
// table of `table_thread` (all of them share those blocks).
struct Range {
  int32_t lo, hi;
  int32_t table_thread;
  std::vector<int32_t> threads;
};

// Relative cost of a 32-token stage of the 8-wave kernel by the row tiles
// its busiest SIMD holds (tile t is on SIMD t % 4), in 1/1024 of a full one:
// measured 1,236, 1,560, 1,773 and 2,211 cycles for 1 to 4 tiles.
constexpr int64_t kStageWeight8[5] = {0, 572, 722, 821, 1024};
int64_t stage_weight8(int32_t slice_tiles) { return kStageWeight8[std::min(4, (slice_tiles + 3) / 4)]; }

struct Unit {  // one token segment of one item, split over `slices` row slices
  int32_t item, lo, hi, slices;
  int64_t cost() const { return static_cast<int64_t>(hi - lo) * slices; }
};

// End of a unit cut from [lo, rest_hi) that asks for about `want` tokens
// (at least min_piece, at most kMaxUnitTokens): on a tile boundary, or the
// end of the range.
int32_t cut_piece(int32_t lo, int32_t rest_hi, int64_t want, int64_t min_piece) {
  want = std::min<int64_t>(std::max<int64_t>(want, min_piece), kMaxUnitTokens);
  const int64_t hi = (static_cast<int64_t>(lo) + want + kTileTokens - 1) / kTileTokens * kTileTokens;
  return hi >= rest_hi ? rest_hi : static_cast<int32_t>(hi);
}

}  // namespace

int32_t unit_table_span(int32_t tok_lo, int32_t tok_hi, int32_t block_size) {
  const int32_t tb0 = tok_lo / kTileTokens * kTileTokens;
  const int32_t span_end = tb0 + (tok_hi - tb0 + kTileTokens - 1) / kTileTokens * kTileTokens + 16;
  return span_end / block_size - tb0 / block_size + 1;
}

std::string build_plan(const BlockManager& bm, const PlanShape& shape, const int32_t* seqs,
                       const int32_t* n_rows, const int32_t* groups, int32_t n_threads,
                       int32_t n_cu, Plan* out) {
  if (shape.hq <= 0 || shape.hkv <= 0 || shape.hq % shape.hkv != 0)
    return "hq and hkv must be positive with hq a multiple of hkv";
  if (shape.head_dim <= 0 || shape.block_size <= 0) return "head_dim and block_size must be positive";
  if (shape.unit_tiles_max <= 0) return "unit_tiles_max must be positive";
  if (shape.block_size != bm.block_size()) return "shape.block_size differs from the cache's block size";
  if (n_threads <= 0) return "n_threads must be positive";
  if (n_cu <= 0) n_cu = 256;
  const int32_t bs = shape.block_size, hq = shape.hq, hkv = shape.hkv, gq = hq / hkv;

  std::vector<int32_t> len(n_threads), row_base(n_threads + 1, 0);
  for (int32_t t = 0; t < n_threads; ++t) {
    if (!bm.has(seqs[t])) return "unknown sequence id " + std::to_string(seqs[t]);
    len[t] = bm.length(seqs[t]);
    if (n_rows[t] < 1 || n_rows[t] > len[t])
      return "thread " + std::to_string(t) + ": n_rows must be in [1, sequence length]";
    row_base[t + 1] = row_base[t] + n_rows[t];
  }
  const int64_t total_rows = row_base[n_threads];
  if (total_rows * hq > INT32_MAX / 2) return "batch too large";

  // Fork groups in order of first appearance; -1 stands alone.
  std::vector<std::vector<int32_t>> members;
  std::map<int32_t, size_t> gid;
  for (int32_t t = 0; t < n_threads; ++t) {
    if (groups[t] < 0) {
      members.push_back({t});
      continue;
    }
    auto it = gid.find(groups[t]);
    if (it == gid.end()) {
      gid.emplace(groups[t], members.size());
      members.push_back({t});
    } else {
      members[it->second].push_back(t);
    }
  }

  Plan p;
  p.shape = shape;
  p.n_threads = n_threads;
  p.n_rows = static_cast<int32_t>(total_rows);
  p.n_groups = static_cast<int32_t>(members.size());

  // Ranges of each fork group: a prefix tree over the members' block tables.
  // `split(S, b)` takes members S that hold the same blocks [0, b) and whose
  // rows all see positions [0, b * bs); it sorts them by their block at index
  // b. A class of one member reads the rest of its context privately. A
  // larger class shares the longest run of blocks its members agree on,
  // capped so that every row of every member sees all of it, and then splits
  // again behind it. Staggered forks (probes forked at different points of
  // the main thread's chain of thought) give one nested level per fork point.
  std::vector<Range> ranges;
  std::vector<const std::vector<int32_t>*> tab(n_threads);
  for (int32_t t = 0; t < n_threads; ++t) tab[t] = &bm.table(seqs[t]);
  auto add_private = [&](int32_t t, int32_t lo) {
    if (len[t] > lo) {
      ranges.push_back({lo, len[t], t, {t}});
      p.private_tokens += len[t] - lo;
    }
  };
  std::function<void(const std::vector<int32_t>&, size_t)> split = [&](const std::vector<int32_t>& S, size_t b) {
    const int32_t lo = static_cast<int32_t>(b) * bs;
    std::vector<std::vector<int32_t>> classes;
    std::map<int32_t, size_t> by_block;
    for (int32_t t : S) {
      if (tab[t]->size() <= b) continue;  // no tokens at or past lo
      const auto it = by_block.find((*tab[t])[b]);
      if (it == by_block.end()) {
        by_block.emplace((*tab[t])[b], classes.size());
        classes.push_back({t});
      } else {
        classes[it->second].push_back(t);
      }
    }
    for (const auto& C : classes) {
      if (C.size() == 1) {
        add_private(C[0], lo);
        continue;
      }
      size_t e = b + 1;
      for (;; ++e) {
        bool same = true;
        for (int32_t t : C) same = same && tab[t]->size() > e && (*tab[t])[e] == (*tab[C[0]])[e];
        if (!same) break;
      }
      int64_t shared = static_cast<int64_t>(e) * bs;
      for (int32_t t : C) shared = std::min<int64_t>(shared, len[t] - n_rows[t] + 1);
      const int32_t P = static_cast<int32_t>(shared);
      if (P > lo) {
        ranges.push_back({lo, P, C[0], C});
        p.shared_tokens += P - lo;
      }
      if (P >= lo && static_cast<int64_t>(P) == static_cast<int64_t>(e) * bs) {
        split(C, e);
      } else {
        for (int32_t t : C) add_private(t, std::max(P, lo));
      }
    }
  };
  for (const auto& m : members) {
    for (int32_t t : m) p.flat_tokens += len[t];
    split(m, 0);
  }

  // Row tiles per workgroup: large row sets are split into near-equal slices
  // of at most unit_tiles_max tiles (8-wave plans: per range, below); every
  // workgroup of the launch is sized for the largest slice.
  int32_t row_tiles = 1;
  std::vector<int32_t> range_rows(ranges.size());
  for (size_t r = 0; r < ranges.size(); ++r) {
    int32_t rows = 0;
    for (int32_t t : ranges[r].threads) rows += n_rows[t] * gq;
    range_rows[r] = rows;
    const int32_t tiles = (rows + 15) / 16;
    p.max_range_tiles = std::max(p.max_range_tiles, tiles);
    const int32_t slices = (tiles + shape.unit_tiles_max - 1) / shape.unit_tiles_max;
    row_tiles = std::max(row_tiles, (tiles + slices - 1) / slices);
  }
  // 8-wave plans slice each range on its own: into the fewest slices of at
  // most unit_tiles_max tiles (or one more), with the tile counts whose
  // summed stage weights are least, larger slices first among equals (26
  // tiles as 16 + 10: a full stage and a three-tile one per 32 tokens, not
  // 13 + 13, two full ones; 20 tiles as 12 + 8, not 16 + 4).
  std::vector<std::vector<int32_t>> range_slice_tiles(ranges.size());
  if (shape.persistent && shape.waves == 8) {
    row_tiles = 1;
    for (size_t r = 0; r < ranges.size(); ++r) {
      const int32_t tiles = (range_rows[r] + 15) / 16;
      const int32_t s0 = (tiles + shape.unit_tiles_max - 1) / shape.unit_tiles_max;
      // A slice of class c (1..4) holds up to 4c tiles, c on its busiest
      // SIMD. For s0 and s0 + 1 slices, the counts of slices per class with
      // enough tiles and the least summed weight, more slices of the larger
      // classes first among equals; past 64 slices, full slices.
      const int32_t max_class = std::min(4, (shape.unit_tiles_max + 3) / 4);
      int64_t best = INT64_MAX;
      std::vector<int32_t> best_cls;
      for (int32_t sl = s0; sl <= std::min(s0 + 1, tiles) && sl <= 64; ++sl) {
        for (int32_t n4 = max_class >= 4 ? sl : 0; n4 >= 0; --n4)
          for (int32_t n3 = (max_class >= 3 ? sl - n4 : 0); n3 >= 0; --n3)
            for (int32_t n2 = (max_class >= 2 ? sl - n4 - n3 : 0); n2 >= 0; --n2) {
              const int32_t n1 = sl - n4 - n3 - n2;
              if (4 * (4 * n4 + 3 * n3 + 2 * n2 + n1) < tiles) continue;
              const int64_t cost = n4 * kStageWeight8[4] + n3 * kStageWeight8[3] + n2 * kStageWeight8[2] +
                                   n1 * kStageWeight8[1];
              if (cost < best) {
                best = cost;
                best_cls.assign(n4, 4);
                best_cls.insert(best_cls.end(), n3, 3);
                best_cls.insert(best_cls.end(), n2, 2);
                best_cls.insert(best_cls.end(), n1, 1);
              }
            }
      }
      if (best_cls.empty()) best_cls.assign(s0, max_class);  // slices of unit_tiles_max tiles, the last shorter
      std::vector<int32_t>& st = range_slice_tiles[r];
      int32_t done = 0;
      for (size_t i = 0; i < best_cls.size(); ++i) {
        const int32_t rest = static_cast<int32_t>(best_cls.size() - i - 1);  // slices still to fill, one tile each at least
        const int32_t n = std::min({4 * best_cls[i], shape.unit_tiles_max, tiles - done - rest});
        st.push_back(n);
        done += n;
        row_tiles = std::max(row_tiles, n);
      }
    }
  }
  const int32_t slice_rows = row_tiles * 16;
  p.row_tiles = row_tiles;

  // Items (range x KV head), their rows and the block tables. Each copied
  // table keeps kTableReserve free entries behind it for the blocks later
  // decode steps append (spork_plan_advance).
  std::vector<int32_t> table_off(n_threads, -1);
  std::vector<int32_t> tables;
  std::vector<ItemDesc> items;
  std::vector<RowDesc> rows;
  std::vector<Range*> item_range;
  std::vector<int32_t> item_rng;  // index of the item's range
  p.seqs.assign(seqs, seqs + n_threads);
  p.len = len;
  p.thread_items.assign(n_threads, {});
  p.thread_table.assign(n_threads, {});
  p.thread_table_off.assign(n_threads, -1);
  p.thread_table_cap.assign(n_threads, 0);
  for (size_t r = 0; r < ranges.size(); ++r) {
    Range& rg = ranges[r];
    const int32_t tt = rg.table_thread;
    if (table_off[tt] < 0) {
      table_off[tt] = static_cast<int32_t>(tables.size());
      const auto& tb = bm.table(seqs[tt]);
      tables.insert(tables.end(), tb.begin(), tb.end());
      tables.insert(tables.end(), kTableReserve, 0);
      p.thread_table[tt] = tb;
      p.thread_table_off[tt] = table_off[tt];
      p.thread_table_cap[tt] = static_cast<int32_t>(tb.size()) + kTableReserve;
    }
    const bool priv = rg.threads.size() == 1;
    for (int32_t h = 0; h < hkv; ++h) {
      ItemDesc it{};
      it.kv_head = h;
      it.table_off = table_off[tt];
      it.n_blocks = static_cast<int32_t>(bm.table(seqs[tt]).size());
      it.row_off = static_cast<int32_t>(rows.size());
      it.n_rows = range_rows[r];
      it.hi = rg.hi;
      it.grow = 0;
      it.thread = priv ? tt : -1;
      if (priv) p.thread_items[tt].push_back(static_cast<int32_t>(items.size()));
      for (int32_t t : rg.threads)
        for (int32_t q = 0; q < n_rows[t]; ++q)
          for (int32_t j = 0; j < gq; ++j)
            rows.push_back({(row_base[t] + q) * hq + h * gq + j, len[t] - n_rows[t] + q});
      items.push_back(it);
      item_range.push_back(&rg);
      item_rng.push_back(static_cast<int32_t>(r));
    }
  }
  p.n_items = static_cast<int32_t>(items.size());

  // Split-K. Items are cut into work units (token range x row slice).
  const int32_t per_cu = 2 * row_tiles <= shape.unit_tiles_max ? shape.units_per_cu_half : shape.units_per_cu;
  const int64_t n_wg = static_cast<int64_t>(n_cu) * std::max(1, per_cu);
  std::vector<int32_t> slices_of(items.size());
  const bool own_slices = shape.persistent && shape.waves == 8;  // per-range slice tiles (above)
  for (size_t it = 0; it < items.size(); ++it)
    slices_of[it] = own_slices ? static_cast<int32_t>(range_slice_tiles[item_rng[it]].size())
                               : (items[it].n_rows + slice_rows - 1) / slice_rows;
  std::vector<WaveDesc> waves;
  std::vector<int32_t> wg_off;
  auto desc = [&](int32_t item, int32_t lo, int32_t hi, int32_t s) {
    WaveDesc w{};
    w.item = item;
    w.tok_lo = lo;
    w.tok_hi = hi;
    if (own_slices) {
      const std::vector<int32_t>& st = range_slice_tiles[item_rng[item]];
      int32_t t0 = 0;
      for (int32_t j = 0; j < s; ++j) t0 += st[j];
      w.row0 = 16 * t0;
      w.nrows = std::min(16 * st[s], items[item].n_rows - w.row0);
    } else {
      w.row0 = s * slice_rows;
      w.nrows = std::min(slice_rows, items[item].n_rows - s * slice_rows);
    }
    return w;
  };
  if (shape.persistent) {
    // Persistent launch: n_wg resident workgroups. Units go on one list per
    // compute unit, shared by the workgroups resident on it (workgroups c and
    // c + n_wg/2 when two share a compute unit), which take the list's units
    // in order through an atomic cursor: the faster workgroup of the pair
    // (the one dispatched first wins the instruction arbiter by age) simply
    // takes more units. The compute units of one accelerator die stream at
    // about the same rate; the dies differ by a few percent (up to 13% on a
    // small decode batch), which a static plan cannot know, but a shared list
    // that every workgroup takes its last units from, to even that out at run
    // time, cost more than it recovered (its one cursor serialises the
    // takes), so the lists are balanced statically. A range with two row slices
    // puts both slices next to each other on one list, so the pair streams
    // its KV through one L2 at the same time.
    //
    // Lists are balanced by water-filling on cost, each unit also costing
    // kUnitOverheadTokens for its start-up: ranges shorter than half a list's
    // share go whole, longest first, to the least-loaded list; longer ranges
    // are cut so that each piece tops the least-loaded list up to the share,
    // a piece being at most one workgroup's share so that both workgroups of
    // a list find work. Each list runs longest unit first, so its last units
    // are short.
    //
    // Cost of a token: one per row slice in 4-wave plans, whose stages are
    // bound by HBM. The stages of 8-wave plans are bound by the matrix cores
    // of the SIMD that holds the most row tiles, so a token of a slice costs
    // stage_weight8(its tiles) / 1024 there.
    const int64_t wunit = shape.waves == 8 ? 1024 : 1;  // cost of a token of a full slice
    const int64_t ovh = kUnitOverheadTokens * wunit;    // start-up cost of a unit
    std::vector<int64_t> tok_cost(items.size());        // cost of a token of the item, all slices
    for (size_t it = 0; it < items.size(); ++it) {
      if (wunit == 1) {
        tok_cost[it] = slices_of[it];
        continue;
      }
      tok_cost[it] = 0;
      for (int32_t sl = 0; sl < slices_of[it]; ++sl)
        tok_cost[it] += stage_weight8((desc(static_cast<int32_t>(it), 0, 0, sl).nrows + 15) / 16);
    }
    const int64_t per_list = per_cu == 2 ? 2 : 1;
    const int64_t lanes = n_wg / per_list;
    std::vector<std::vector<WaveDesc>> lists(lanes);
    std::vector<int64_t> load(lanes, 0);
    // The least-loaded list (the lowest index among equals), kept in a heap.
    std::priority_queue<std::pair<int64_t, int64_t>, std::vector<std::pair<int64_t, int64_t>>, std::greater<>> heap;
    auto least = [&]() { return heap.top().second; };
    auto place = [&](int32_t item, int32_t lo, int32_t hi, int32_t slices) {
      const int64_t c = least();
      heap.pop();
      for (int32_t s = 0; s < slices; ++s) lists[c].push_back(desc(item, lo, hi, s));
      load[c] += static_cast<int64_t>(hi - lo) * tok_cost[item] + ovh * slices;
      heap.push({load[c], c});
    };
    std::vector<size_t> order(items.size());
    for (size_t i = 0; i < order.size(); ++i) order[i] = i;
    std::stable_sort(order.begin(), order.end(), [&](size_t x, size_t y) {
      return item_range[x]->hi - item_range[x]->lo > item_range[y]->hi - item_range[y]->lo;
    });
    // The share of a list: the fixed point of share = (cost of the tokens +
    // start-up cost of the units) / lanes, where a range cheaper than half
    // the share is one unit per slice and a longer one is cut into pieces
    // whose units cost share / max(slices, workgroups per list) each.
    int64_t tokens = 0;
    for (size_t it = 0; it < items.size(); ++it)
      tokens += static_cast<int64_t>(item_range[it]->hi - item_range[it]->lo) * tok_cost[it];
    auto unit_cost_share = [&](int64_t share) {
      int64_t units = 0;
      for (size_t it = 0; it < items.size(); ++it) {
        const int64_t len = item_range[it]->hi - item_range[it]->lo, sl = slices_of[it];
        const int64_t piece = std::max<int64_t>(
            kTileTokens, (share / std::max<int64_t>(sl, per_list) - ovh) * sl / tok_cost[it]);
        units += (len * tok_cost[it] + ovh * sl <= share / 2 ? 1 : (len + piece - 1) / piece) * sl;
      }
      return (tokens + ovh * units + lanes - 1) / lanes;
    };
    int64_t share = (tokens + lanes - 1) / lanes;
    for (int iter = 0; iter < 32; ++iter) {
      const int64_t next = unit_cost_share(share);
      if (next == share) break;
      share = (share + next + 1) / 2;
    }
    // Fill towards `level`; what is left once every list has reached it (the
    // estimate's unit count was short) goes out in short pieces, each with
    // its own start-up cost; the level is then raised by that overflow spread
    // over all lists and the fill repeated, keeping the lowest maximum.
    const int64_t min_piece =  // an eighth of a workgroup's share, 64..512 tokens
        std::min<int64_t>(kMinPieceTokens,
                          std::max<int64_t>(64, share / wunit / per_list / 8 / kTileTokens * kTileTokens));
    auto fill = [&](int64_t level, int64_t* overflow) {
      for (auto& l : lists) l.clear();
      std::fill(load.begin(), load.end(), 0);
      heap = {};
      for (int64_t c = 0; c < lanes; ++c) heap.push({0, c});
      *overflow = 0;
      for (int pass = 0; pass < 2; ++pass) {
        for (size_t it : order) {
          const Range& rg = *item_range[it];
          const int32_t slices = slices_of[it];
          const bool small = static_cast<int64_t>(rg.hi - rg.lo) * tok_cost[it] + ovh * slices <= share / 2;
          if (small != (pass == 0)) continue;
          for (int32_t lo = rg.lo; lo < rg.hi;) {
            int64_t want = kMaxUnitTokens;
            // a piece tops the list up, but is at most one workgroup's share
            if (!small)
              want = (std::min(level - load[least()], level / per_list * slices) - ovh * slices) / tok_cost[it];
            const int32_t hi = cut_piece(lo, rg.hi, want, min_piece);
            if (!small && want < min_piece) *overflow += static_cast<int64_t>(hi - lo) * tok_cost[it] + ovh * slices;
            place(static_cast<int32_t>(it), lo, hi, slices);
            lo = hi;
          }
        }
      }
      return *std::max_element(load.begin(), load.end());
    };
    std::vector<std::vector<WaveDesc>> best;
    int64_t best_max = INT64_MAX, level = share;
    for (int round = 0; round < 6; ++round) {
      int64_t overflow = 0;
      const int64_t mx = fill(level, &overflow);
      if (mx < best_max) {
        best_max = mx;
        best = lists;
      }
      if (overflow == 0) break;
      level += std::max<int64_t>(kTileTokens * wunit, (overflow + lanes - 1) / lanes);
    }
    lists.swap(best);
    wg_off.push_back(0);
    for (auto& l : lists) {
      // longest unit first; the row slices of a piece stay adjacent
      std::stable_sort(l.begin(), l.end(), [](const WaveDesc& x, const WaveDesc& y) {
        const int32_t lx = x.tok_hi - x.tok_lo, ly = y.tok_hi - y.tok_lo;
        if (lx != ly) return lx > ly;
        if (x.item != y.item) return x.item < y.item;
        if (x.tok_lo != y.tok_lo) return x.tok_lo < y.tok_lo;
        return x.row0 < y.row0;
      });
      waves.insert(waves.end(), l.begin(), l.end());
      wg_off.push_back(static_cast<int32_t>(waves.size()));
    }
    p.grid = static_cast<int32_t>(n_wg);
    p.n_lists = static_cast<int32_t>(lanes);
  } else {
    // One workgroup per unit: items cut into round(len / ideal) segments of
    // near-equal cost (ideal: the batch's cost over the resident workgroups),
    // longest first, each to the least-loaded die; workgroup ids are dealt to
    // the dies round-robin, so a unit's row slices stay on one die's L2.
    int64_t cost = 0;
    for (size_t it = 0; it < items.size(); ++it)
      cost += static_cast<int64_t>(item_range[it]->hi - item_range[it]->lo) * slices_of[it];
    const double ideal = std::max(1.0, static_cast<double>(cost) / static_cast<double>(n_wg));
    std::vector<Unit> units;
    for (size_t it = 0; it < items.size(); ++it) {
      const Range& rg = *item_range[it];
      const int64_t n = rg.hi - rg.lo;
      int64_t nseg = std::max<int64_t>(1, static_cast<int64_t>(static_cast<double>(n) / ideal + 0.5));
      nseg = std::max<int64_t>(nseg, (n + kMaxUnitTokens - 1) / kMaxUnitTokens);
      nseg = std::min<int64_t>(nseg, std::max<int64_t>(1, n / kTileTokens));
      int32_t lo = rg.lo;
      for (int64_t k = 1; k <= nseg; ++k) {
        int32_t hi = rg.hi;
        if (k < nseg) {
          const int64_t cut = rg.lo + n * k / nseg;
          hi = static_cast<int32_t>((cut + kTileTokens / 2) / kTileTokens * kTileTokens);
          if (hi <= lo || hi >= rg.hi) continue;
        }
        units.push_back({static_cast<int32_t>(it), lo, hi, slices_of[it]});
        lo = hi;
      }
    }
    std::stable_sort(units.begin(), units.end(),
                     [](const Unit& a, const Unit& b) { return a.hi - a.lo > b.hi - b.lo; });
    std::vector<std::vector<WaveDesc>> queue(kXcds);
    std::vector<int64_t> load(kXcds, 0);
    for (const Unit& u : units) {
      const int x = static_cast<int>(std::min_element(load.begin(), load.end()) - load.begin());
      load[x] += u.cost();
      for (int32_t s = 0; s < u.slices; ++s) queue[x].push_back(desc(u.item, u.lo, u.hi, s));
    }
    size_t depth = 0;
    for (const auto& q : queue) depth = std::max(depth, q.size());
    for (size_t d = 0; d < depth; ++d)
      for (int x = 0; x < kXcds; ++x)
        waves.push_back(d < queue[x].size() ? queue[x][d] : WaveDesc{-1, 0, 0, 0, 0, 0});
    for (size_t i = 0; i <= waves.size(); ++i) wg_off.push_back(static_cast<int32_t>(i));
    p.grid = static_cast<int32_t>(waves.size());
    p.n_lists = p.grid;
  }
  int32_t partial = 0;
  for (size_t u = 0; u < waves.size(); ++u) {
    WaveDesc& w = waves[u];
    if (w.item < 0) continue;
    // the bf16 kernel stages a 32-token block's entry twice
    if (unit_table_span(w.tok_lo, w.tok_hi, shape.block_size) * (shape.block_size == 32 ? 2 : 1) > kUnitTableEntries)
      return "internal: unit too long";
    w.partial = partial;
    partial += w.nrows;
    // the last unit of a private range is the one later decode steps extend
    const ItemDesc& it = items[w.item];
    if (it.thread >= 0 && w.tok_hi == it.hi) p.open_units.push_back(static_cast<int32_t>(u));
  }
  p.n_units = static_cast<int32_t>(waves.size());
  p.n_partials = partial;

  // Merge lists: the partial rows of every output (query row x query head).
  p.n_out = static_cast<int32_t>(total_rows * hq);
  std::vector<int32_t> count(p.n_out + 1, 0);
  for (const WaveDesc& w : waves) {
    if (w.item < 0) continue;
    for (int32_t i = 0; i < w.nrows; ++i) count[rows[items[w.item].row_off + w.row0 + i].qidx + 1]++;
  }
  for (int32_t o = 0; o < p.n_out; ++o) {
    if (count[o + 1] == 0) return "internal: output without a partial";
    count[o + 1] += count[o];
  }
  // Each unit row writes its partial result at its output's next merge
  // position, so the partials of an output sit next to each other and the
  // merge reads them without an index list.
  std::vector<int32_t> part_slot(partial);
  std::vector<int32_t> fill(count.begin(), count.end() - 1);
  for (const WaveDesc& w : waves) {
    if (w.item < 0) continue;
    for (int32_t i = 0; i < w.nrows; ++i)
      part_slot[w.partial + i] = fill[rows[items[w.item].row_off + w.row0 + i].qidx]++;
  }

  // Device image.
  size_t off = 0;
  auto place = [&](size_t bytes) {
    const size_t at = off;
    off = align256(off + bytes);
    return at;
  };
  p.off_waves = place(waves.size() * sizeof(WaveDesc));
  p.off_items = place(items.size() * sizeof(ItemDesc));
  p.off_rows = place(rows.size() * sizeof(RowDesc));
  p.off_tables = place(tables.size() * sizeof(int32_t));
  p.off_merge_off = place(count.size() * sizeof(int32_t));
  p.off_part_slot = place(part_slot.size() * sizeof(int32_t));
  p.off_wg_off = place(wg_off.size() * sizeof(int32_t));
  p.image.assign(off, 0);
  auto put = [&](size_t at, const void* src, size_t bytes) {
    if (bytes) std::memcpy(p.image.data() + at, src, bytes);
  };
  put(p.off_waves, waves.data(), waves.size() * sizeof(WaveDesc));
  put(p.off_items, items.data(), items.size() * sizeof(ItemDesc));
  put(p.off_rows, rows.data(), rows.size() * sizeof(RowDesc));
  put(p.off_tables, tables.data(), tables.size() * sizeof(int32_t));
  put(p.off_merge_off, count.data(), count.size() * sizeof(int32_t));
  put(p.off_part_slot, part_slot.data(), part_slot.size() * sizeof(int32_t));
  put(p.off_wg_off, wg_off.data(), wg_off.size() * sizeof(int32_t));
  p.grow.assign(n_threads, 0);

  // Control words: the list cursors and the cursor of the argmax units a
  // verify launch takes after its lists (persistent launches); then the
  // partial outputs and their (m, l) pairs.
  p.off_ws_cursors = 0;
  p.n_cursors = shape.persistent ? p.n_lists + 1 : 0;
  p.control_bytes = static_cast<size_t>(p.n_cursors) * kCursorStride * sizeof(int32_t);
  p.off_ws_o = p.control_bytes;
  p.off_ws_ml = p.off_ws_o + align256(static_cast<size_t>(partial) * shape.head_dim * shape.elem_bytes);
  p.workspace_bytes = p.off_ws_ml + align256(static_cast<size_t>(partial) * 2 * sizeof(float));
  *out = std::move(p);
  return "";
}

}  // namespace spork
