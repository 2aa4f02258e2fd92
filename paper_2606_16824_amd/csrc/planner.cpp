// Extend work planner (host).
//
// Work unit: one query tile (block_m packed rows of one sequence and kv head)
// over a contiguous range of keys.  A tile whose rows end at token t_last needs
// keys [0, Lp + t_last + 1) (bottom-right causal).  When there are too few
// tiles to fill the GPU, each tile's key range is split into chunks of about
// equal length ("split-K"); the chunks write unnormalised partials that a
// second kernel merges with a log-sum-exp weighting.
//
// Launch order is XCD-aware: the dispatcher hands workgroup i to XCD i % X, and
// each XCD has its own L2.  All tiles of one (sequence, kv head) read the same
// keys, so the work of a (sequence, kv head) that fills whole rounds of the GPU
// is dealt round by round across all XCDs (every XCD streams the same keys at
// the same time), and the rest of it is kept on one XCD (split into several
// bundles only when there are fewer bundles than XCDs), bundles spread over
// XCDs longest-processing-time first; the per-XCD queues are interleaved.
// Queues that run out early are padded with idle items so that later items
// still land on their XCD.
#include "planner.h"

#include <algorithm>
#include <climits>
#include <iterator>
#include <numeric>

namespace cw {
namespace {

constexpr int32_t MIN_CHUNK_TILES = 4;  // a chunk of fewer keys wastes the Q load

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

struct Tile {
  int32_t seq, kvh, q_row0, rows, kv_len, n_kt;
};

struct Bundle {
  std::vector<WorkItem> items;
  int64_t cost = 0;  // key tiles
};

void layout_workspace(ExtendPlan& plan, int32_t head_dim);

}  // namespace

ExtendPlan build_extend_plan(const int32_t* prefix_lens, const int32_t* suffix_lens,
                             int32_t num_seqs, int32_t num_kv_heads, int32_t gqa_group,
                             int32_t head_dim, int32_t block_m, int32_t wgs_per_cu,
                             int32_t num_cus, int32_t num_xcds, const Tuning& tuning,
                             const int32_t* cu_rows, const int32_t* bt_rows) {
  ExtendPlan plan;
  plan.seqs.resize(num_seqs);
  int64_t cu = 0;
  for (int32_t b = 0; b < num_seqs; ++b) {
    plan.seqs[b] = SeqInfo{prefix_lens[b], suffix_lens[b],
                           cu_rows ? cu_rows[b] : static_cast<int32_t>(cu), bt_rows ? bt_rows[b] : b};
    cu += suffix_lens[b];
  }

  // 1. query tiles, per sequence and kv head
  std::vector<Tile> tiles;
  int64_t total_kt = 0;
  for (int32_t b = 0; b < num_seqs; ++b) {
    const int64_t rows = int64_t(suffix_lens[b]) * gqa_group;
    for (int64_t r0 = 0; r0 < rows; r0 += block_m) {
      const int32_t nr = static_cast<int32_t>(std::min<int64_t>(block_m, rows - r0));
      const int64_t t_last = (r0 + nr - 1) / gqa_group;
      const int32_t kv_len = static_cast<int32_t>(prefix_lens[b] + t_last + 1);
      const int32_t n_kt = (kv_len + BLOCK_N - 1) / BLOCK_N;
      for (int32_t h = 0; h < num_kv_heads; ++h) {
        tiles.push_back(Tile{b, h, static_cast<int32_t>(r0), nr, kv_len, n_kt});
        total_kt += n_kt;
      }
    }
  }

  // 2. split-K: number of chunks per tile.  Automatic: when there are fewer
  // tiles than `target` workgroups (all resident at once), each tile gets
  // about n_kt / (total_kt / target) chunks, so chunks are of about equal
  // length and their count is close to the target.
  const int64_t target =
      tuning.target_wgs > 0 ? tuning.target_wgs : int64_t(std::max(1, wgs_per_cu)) * num_cus;
  double chunk_len = 0.0;  // 0: no split
  if (tuning.kv_chunk_tiles > 0) {
    chunk_len = tuning.kv_chunk_tiles;
  } else if (static_cast<int64_t>(tiles.size()) < target && !tiles.empty()) {
    chunk_len = std::max<double>(MIN_CHUNK_TILES, double(total_kt) / double(target));
  }
  auto n_chunks = [&](int32_t n_kt) -> int64_t {
    if (chunk_len <= 0.0) return 1;
    if (tuning.kv_chunk_tiles > 0) return std::max<int64_t>(1, (n_kt + tuning.kv_chunk_tiles - 1) / tuning.kv_chunk_tiles);
    const int64_t n = static_cast<int64_t>(double(n_kt) / chunk_len + 0.5);
    return std::max<int64_t>(1, std::min<int64_t>(n, n_kt / MIN_CHUNK_TILES));
  };

  // 3. work items grouped into bundles by (sequence, kv head)
  std::vector<Bundle> bundles;
  {
    int32_t cur_seq = -1, cur_kvh = -1;
    std::vector<std::vector<WorkItem>> chunk_major;  // [chunk][tile] inside a bundle
    auto flush = [&]() {
      if (chunk_major.empty()) return;
      Bundle bd;
      for (auto& v : chunk_major)
        for (auto& it : v) {
          bd.items.push_back(it);
          bd.cost += (it.kv_end - it.kv_begin + BLOCK_N - 1) / BLOCK_N;
        }
      bundles.push_back(std::move(bd));
      chunk_major.clear();
    };
    // tiles are ordered (seq, q tile, kvh); regroup them per (seq, kvh)
    std::vector<size_t> order(tiles.size());
    std::iota(order.begin(), order.end(), 0);
    std::stable_sort(order.begin(), order.end(), [&](size_t a, size_t c) {
      if (tiles[a].seq != tiles[c].seq) return tiles[a].seq < tiles[c].seq;
      return tiles[a].kvh < tiles[c].kvh;
    });
    for (size_t oi : order) {
      const Tile& t = tiles[oi];
      if (t.seq != cur_seq || t.kvh != cur_kvh) {
        flush();
        cur_seq = t.seq;
        cur_kvh = t.kvh;
      }
      const int64_t n_c = n_chunks(t.n_kt);
      int32_t part0 = -1;
      if (n_c > 1) {
        part0 = static_cast<int32_t>(plan.n_parts);
        plan.groups.push_back(CombineGroup{t.seq, t.kvh, t.q_row0, t.rows, part0,
                                           static_cast<int32_t>(n_c), 0, 0});
        plan.n_parts += n_c;
      }
      // chunk boundaries: equal shares of the tile's cost, a key tile that
      // reaches past the cached prefix (masked, read from the new tokens)
      // costing suffix_weight / 100 of a prefix tile (forced chunk sizes:
      // equal key counts)
      const int64_t n_pre = std::min<int64_t>(t.n_kt, prefix_lens[t.seq] / BLOCK_N);
      const int64_t wgt = tuning.kv_chunk_tiles > 0 ? 100 : std::max(1, tuning.suffix_weight);
      const int64_t total_cost = n_pre * 100 + (t.n_kt - n_pre) * wgt;
      // first key tile of each chunk, every chunk at least one tile long
      std::vector<int64_t> first(static_cast<size_t>(n_c) + 1);
      first[0] = 0;
      first[n_c] = t.n_kt;
      for (int64_t c = 1; c < n_c; ++c) {
        int64_t b = c * t.n_kt / n_c;
        if (wgt != 100) {
          const int64_t goal = c * total_cost / n_c;
          b = goal <= n_pre * 100 ? (goal + 99) / 100 : n_pre + (goal - n_pre * 100 + wgt - 1) / wgt;
        }
        first[c] = std::min(std::max(b, first[c - 1] + 1), t.n_kt - (n_c - c));
      }
      for (int64_t c = 0; c < n_c; ++c) {
        const int64_t kt0 = first[c], kt1 = first[c + 1];
        WorkItem it{t.seq, t.kvh, t.q_row0, static_cast<int32_t>(kt0 * BLOCK_N),
                    static_cast<int32_t>(std::min<int64_t>(kt1 * BLOCK_N, t.kv_len)),
                    n_c > 1 ? static_cast<int32_t>(part0 + c) : -1, t.rows, 0};
        if (static_cast<int64_t>(chunk_major.size()) <= c) chunk_major.resize(c + 1);
        chunk_major[c].push_back(it);
      }
    }
    flush();
  }

  // 4. Bundles that fill whole rounds of the GPU (R items per XCD, one per
  // resident workgroup slot): dealt across every XCD a round at a time, so all
  // XCDs stream the keys of the same (sequence, kv head) at once and what one
  // XCD's L2 has dropped is still in the memory-side cache for the others (a
  // bundle kept on one XCD for several rounds has all XCDs streaming different
  // heads, more than that cache holds).  The items of every other round run in
  // reverse order, so the slot that drew a short tile draws a long one next and
  // the slots of an XCD stay close together in the key stream.  Within a round
  // each XCD takes consecutive items (tiles of about equal length), rotating
  // over the round's blocks from one round to the next.
  const int32_t X = std::max(1, num_xcds);
  const int64_t R = std::max<int64_t>(1, int64_t(std::max(1, wgs_per_cu)) * num_cus / X);
  std::vector<std::vector<WorkItem>> queues(X);
  if (tuning.deal_rounds != 0) {
    int64_t round = 0;
    for (auto& bd : bundles) {
      const int64_t n_rounds = static_cast<int64_t>(bd.items.size()) / (R * X);
      for (int64_t r = 0; r < n_rounds; ++r, ++round)
        for (int32_t x = 0; x < X; ++x) {
          // XCD x takes block (x + round) % X of the round's X blocks of R
          // items: blocks later in a bundle hold longer tiles (more keys), and
          // the rotation gives every XCD each position in turn
          const auto b0 = bd.items.begin() + (r * X + (x + round) % X) * R;
          if (round & 1) queues[x].insert(queues[x].end(), std::make_reverse_iterator(b0 + R),
                                          std::make_reverse_iterator(b0));
          else queues[x].insert(queues[x].end(), b0, b0 + R);
        }
      if (n_rounds > 0) {
        bd.items.erase(bd.items.begin(), bd.items.begin() + n_rounds * R * X);
        bd.cost = 0;
        for (auto& w : bd.items) bd.cost += (w.kv_end - w.kv_begin + BLOCK_N - 1) / BLOCK_N;
      }
    }
    bundles.erase(std::remove_if(bundles.begin(), bundles.end(),
                                 [](const Bundle& b) { return b.items.empty(); }),
                  bundles.end());
  }

  // 5. enough bundles to occupy every XCD: halve the largest while possible
  while (static_cast<int32_t>(bundles.size()) < 2 * X) {
    auto it = std::max_element(bundles.begin(), bundles.end(),
                               [](const Bundle& a, const Bundle& c) { return a.items.size() < c.items.size(); });
    if (it == bundles.end() || it->items.size() < 2) break;
    Bundle hi;
    const size_t half = it->items.size() / 2;
    hi.items.assign(it->items.begin() + half, it->items.end());
    it->items.resize(half);
    it->cost = hi.cost = 0;
    for (auto& w : it->items) it->cost += (w.kv_end - w.kv_begin + BLOCK_N - 1) / BLOCK_N;
    for (auto& w : hi.items) hi.cost += (w.kv_end - w.kv_begin + BLOCK_N - 1) / BLOCK_N;
    bundles.push_back(std::move(hi));
  }

  // 6. LPT assignment of the other bundles to XCD queues (after the dealt
  // rounds, which every queue holds the same number of), then interleave
  std::stable_sort(bundles.begin(), bundles.end(),
                   [](const Bundle& a, const Bundle& c) { return a.cost > c.cost; });
  std::vector<int64_t> load(X, 0);
  for (auto& bd : bundles) {
    const int32_t x = static_cast<int32_t>(std::min_element(load.begin(), load.end()) - load.begin());
    load[x] += bd.cost;
    queues[x].insert(queues[x].end(), bd.items.begin(), bd.items.end());
  }
  size_t max_len = 0;
  for (auto& qv : queues) max_len = std::max(max_len, qv.size());
  const WorkItem idle{-1, 0, 0, 0, 0, -1, 0, 0};
  int32_t used_queues = 0;
  for (auto& qv : queues) used_queues += qv.empty() ? 0 : 1;
  for (size_t i = 0; i < max_len; ++i)
    for (int32_t x = 0; x < X; ++x) {
      if (i < queues[x].size()) plan.items.push_back(queues[x][i]);
      else if (used_queues > 1) plan.items.push_back(idle);
    }
  // trailing idle items launch nothing useful
  while (!plan.items.empty() && plan.items.back().seq < 0) plan.items.pop_back();

  // 7. workspace layout
  plan.part_rows = block_m;
  layout_workspace(plan, head_dim);
  return plan;
}

namespace {
void layout_workspace(ExtendPlan& plan, int32_t head_dim) {
  plan.off_seqs = 0;
  plan.off_items = align256(plan.off_seqs + plan.seqs.size() * sizeof(SeqInfo));
  plan.off_groups = align256(plan.off_items + plan.items.size() * sizeof(WorkItem));
  plan.meta_bytes = align256(plan.off_groups + plan.groups.size() * sizeof(CombineGroup));
  plan.off_part_o = plan.meta_bytes;
  // the partial O is stored in bf16 (2 bytes), the running max and sum in fp32
  plan.off_part_ml = align256(plan.off_part_o + size_t(plan.n_parts) * plan.part_rows * head_dim * 2);
  plan.total_bytes = align256(plan.off_part_ml + size_t(plan.n_parts) * plan.part_rows * 2 * sizeof(float));
}
}  // namespace

// Decode planning.  The cached prefix of each (sequence, kv head) is cut into
// chunks of whole decode tiles and whole pages (at most 64 pages, the kernel
// keeps one page id per lane).  Chunks are as long as one wave per resident
// slot allows (a decode wave streams its chunk at its share of HBM bandwidth;
// every wave pays one start-up latency for its page ids and first tile, so
// fewer, longer waves waste less), within the 64-page cap.  The new token's
// own key rides with the last chunk.
ExtendPlan build_decode_plan(const int32_t* prefix_lens, int32_t num_seqs, int32_t num_kv_heads,
                             int32_t gqa_group, int32_t head_dim, int32_t page_size,
                             int32_t keys_per_tile, int32_t waves_per_cu, int32_t num_cus,
                             const Tuning& tuning, const int32_t* cu_rows, const int32_t* bt_rows) {
  ExtendPlan plan;
  plan.part_rows = gqa_group;
  plan.seqs.resize(num_seqs);
  int64_t total_tiles = 0;
  for (int32_t b = 0; b < num_seqs; ++b) {
    plan.seqs[b] = SeqInfo{prefix_lens[b], 1, cu_rows ? cu_rows[b] : b, bt_rows ? bt_rows[b] : b};
    total_tiles += (int64_t(prefix_lens[b]) + keys_per_tile) / keys_per_tile * num_kv_heads;
  }
  const int64_t unit = std::max<int64_t>(keys_per_tile, page_size);  // chunk granule
  const int64_t max_chunk = int64_t(64) * page_size;                 // keys
  int64_t chunk;
  if (tuning.kv_chunk_tiles > 0) {
    chunk = int64_t(tuning.kv_chunk_tiles) * keys_per_tile;
  } else {
    const int64_t target = tuning.target_wgs > 0 ? tuning.target_wgs : int64_t(num_cus) * waves_per_cu;
    const int64_t tiles = std::max<int64_t>(2, (total_tiles + target - 1) / target);
    chunk = tiles * keys_per_tile;
  }
  chunk = std::min(max_chunk, std::max(unit, (chunk + unit - 1) / unit * unit));
  // Longest chunks first so that short tails fill in at the end: every chunk but
  // the last of a (sequence, kv head) has the full length, so the order is the
  // full-length chunks in build order, then the shorter last chunks by length
  // (stable), the same as a stable sort of all items by length.
  int64_t n_items = 0;
  for (int32_t b = 0; b < num_seqs; ++b) n_items += (int64_t(prefix_lens[b]) + chunk) / chunk;
  plan.items.reserve(size_t(n_items * num_kv_heads));
  std::vector<WorkItem> tails;
  tails.reserve(size_t(num_seqs) * num_kv_heads);
  for (int32_t b = 0; b < num_seqs; ++b) {
    const int64_t n = int64_t(prefix_lens[b]) + 1;  // keys including the new one
    const int64_t n_c = (n + chunk - 1) / chunk;
    for (int32_t h = 0; h < num_kv_heads; ++h) {
      int32_t part0 = -1;
      if (n_c > 1) {
        part0 = static_cast<int32_t>(plan.n_parts);
        plan.groups.push_back(CombineGroup{b, h, 0, gqa_group, part0, static_cast<int32_t>(n_c), 0, 0});
        plan.n_parts += n_c;
      }
      for (int64_t c = 0; c < n_c; ++c) {
        const WorkItem it{b, h, 0, static_cast<int32_t>(c * chunk),
                          static_cast<int32_t>(std::min(n, (c + 1) * chunk)),
                          n_c > 1 ? static_cast<int32_t>(part0 + c) : -1, gqa_group, 0};
        (it.kv_end - it.kv_begin == chunk ? plan.items : tails).push_back(it);
      }
    }
  }
  std::stable_sort(tails.begin(), tails.end(), [](const WorkItem& a, const WorkItem& c) {
    return (a.kv_end - a.kv_begin) > (c.kv_end - c.kv_begin);
  });
  plan.items.insert(plan.items.end(), tails.begin(), tails.end());
  layout_workspace(plan, head_dim);

  // the compact form: one record per sequence, the order of the last chunks
  plan.compact = true;
  plan.recs.resize(num_seqs);
  int32_t full_off = 0, part_off = 0, group_off = 0;
  std::vector<std::pair<int64_t, int32_t>> tail_len;  // (length, sequence)
  for (int32_t b = 0; b < num_seqs; ++b) {
    const int64_t n = int64_t(prefix_lens[b]) + 1;
    const int32_t nc = static_cast<int32_t>((n + chunk - 1) / chunk);
    const int32_t full = n % chunk == 0 ? nc : nc - 1;
    plan.recs[b] = DecodeRec{full_off, full, nc, static_cast<int32_t>(n), part_off, group_off};
    full_off += full * num_kv_heads;
    if (nc > 1) {
      part_off += nc * num_kv_heads;
      group_off += num_kv_heads;
    }
    if (full < nc) tail_len.emplace_back(n - int64_t(full) * chunk, b);
  }
  std::stable_sort(tail_len.begin(), tail_len.end(),
                   [](const std::pair<int64_t, int32_t>& a, const std::pair<int64_t, int32_t>& c) {
                     return a.first > c.first;
                   });
  for (const auto& t : tail_len) plan.tails.push_back(t.second);
  ExpandDesc& d = plan.desc;
  d.n_seqs = num_seqs;
  d.n_full = full_off;
  d.n_items = static_cast<int32_t>(plan.items.size());
  d.n_groups = static_cast<int32_t>(plan.groups.size());
  d.n_tails = static_cast<int32_t>(plan.tails.size());
  d.chunk = static_cast<int32_t>(chunk);
  d.hkv = num_kv_heads;
  d.rows = gqa_group;
  d.items_off = static_cast<uint32_t>(plan.off_items);
  d.groups_off = static_cast<uint32_t>(plan.off_groups);
  return plan;
}

void pack_plan_head(const ExtendPlan& plan, uint8_t* dst) {
  std::fill(dst, dst + plan.off_items, uint8_t(0));
  std::copy(reinterpret_cast<const uint8_t*>(plan.seqs.data()),
            reinterpret_cast<const uint8_t*>(plan.seqs.data() + plan.seqs.size()), dst + plan.off_seqs);
}

void pack_plan_meta(const ExtendPlan& plan, uint8_t* dst) {
  std::fill(dst, dst + plan.meta_bytes, uint8_t(0));
  std::copy(reinterpret_cast<const uint8_t*>(plan.seqs.data()),
            reinterpret_cast<const uint8_t*>(plan.seqs.data() + plan.seqs.size()), dst + plan.off_seqs);
  std::copy(reinterpret_cast<const uint8_t*>(plan.items.data()),
            reinterpret_cast<const uint8_t*>(plan.items.data() + plan.items.size()), dst + plan.off_items);
  std::copy(reinterpret_cast<const uint8_t*>(plan.groups.data()),
            reinterpret_cast<const uint8_t*>(plan.groups.data() + plan.groups.size()), dst + plan.off_groups);
}

}  // namespace cw
