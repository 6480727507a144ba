// Host-side validation and work planning for one mixed step (pure C++, no HIP).
#include "plan.h"

#include <algorithm>
#include <cmath>
#include <numeric>

namespace ppas {

namespace {
size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// decode cost / prefill cost above which the two kinds are interleaved
#ifndef PPAS_INTERLEAVE_RATIO
#define PPAS_INTERLEAVE_RATIO 0.5
#endif
constexpr double kInterleaveRatio = PPAS_INTERLEAVE_RATIO;
// largest decode cost, relative to the prefill cost, at which a step may use
// 32-position prefill tiles
#ifndef PPAS_LARGE_TILE_DECODE_SHARE
#define PPAS_LARGE_TILE_DECODE_SHARE 0.05
#endif
constexpr double kLargeTileDecodeShare = PPAS_LARGE_TILE_DECODE_SHARE;
// when interleaving, prefill advances at this multiple of the decode fraction
#ifndef PPAS_INTERLEAVE_BIAS
#define PPAS_INTERLEAVE_BIAS 1.0
#endif
// prefill items aimed at per compute unit when tiles need key splits
#ifndef PPAS_PREFILL_ITEMS_PER_CU
#define PPAS_PREFILL_ITEMS_PER_CU 2
#endif
int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
}  // namespace

ppas_status validate(const ppas_shape* shape, const ppas_seq* seqs, int32_t n_seqs,
                     const int32_t* bt_host, int32_t bt_stride, bool check_overlap) {
  if (!shape) return PPAS_EINVAL;
  const ppas_shape& s = *shape;
  if (s.n_q_heads <= 0 || s.n_kv_heads <= 0 || s.head_dim <= 0 || s.page_size <= 0 || s.num_pages <= 0)
    return PPAS_EINVAL;
  if (!std::isfinite(s.scale) || !(s.scale > 0.f)) return PPAS_EINVAL;
  if (s.n_q_heads % s.n_kv_heads != 0) return PPAS_EINVAL;
  if (s.n_q_heads / s.n_kv_heads != kGroup || s.head_dim != kHeadDim || s.page_size != kPage)
    return PPAS_EUNSUPPORTED;
  if (n_seqs < 0) return PPAS_EINVAL;
  if (n_seqs == 0) return PPAS_OK;
  if (!seqs) return PPAS_EINVAL;
  if (bt_stride <= 0) return PPAS_EINVAL;
  int64_t qs = 0;
  for (int32_t i = 0; i < n_seqs; ++i) {
    const ppas_seq& q = seqs[i];
    if (q.n_query < 1 || q.cached_len < 0) return PPAS_EINVAL;
    if (q.query_start != qs) return PPAS_EINVAL;
    const int64_t len = int64_t(q.cached_len) + q.n_query;
    if (len > INT32_MAX - 64) return PPAS_ERANGE;
    qs += q.n_query;
    if (qs > INT32_MAX) return PPAS_ERANGE;
    if (ceil_div(len, kPage) > bt_stride) return PPAS_EINVAL;
  }
  if (!bt_host) return PPAS_OK;
  for (int32_t i = 0; i < n_seqs; ++i) {
    const int64_t pages = ceil_div(int64_t(seqs[i].cached_len) + seqs[i].n_query, kPage);
    const int32_t* row = bt_host + int64_t(i) * bt_stride;
    for (int64_t j = 0; j < pages; ++j)
      if (row[j] < 0 || row[j] >= s.num_pages) return PPAS_ERANGE;
  }
  if (check_overlap) {
    // No (page, slot) may be written by two requests of the step. A request's new
    // positions form one run of slots per page it touches; sorting those runs by
    // (page, first slot) puts any two that share a page side by side, so the cost
    // follows the pages the step writes, not the size of the pool.
    struct Run {
      int32_t page, lo, hi;   // slots lo..hi of the page
    };
    std::vector<Run> runs;
    for (int32_t i = 0; i < n_seqs; ++i) {
      const int32_t* row = bt_host + int64_t(i) * bt_stride;
      const int64_t end = int64_t(seqs[i].cached_len) + seqs[i].n_query;
      for (int64_t p = seqs[i].cached_len; p < end;) {
        const int64_t lp = p / kPage;
        const int64_t stop = std::min(end, (lp + 1) * kPage);
        runs.push_back(Run{row[lp], int32_t(p % kPage), int32_t((stop - 1) % kPage)});
        p = stop;
      }
    }
    std::sort(runs.begin(), runs.end(),
              [](const Run& a, const Run& b) { return a.page != b.page ? a.page < b.page : a.lo < b.lo; });
    for (size_t k = 1; k < runs.size(); ++k)
      if (runs[k].page == runs[k - 1].page && runs[k].lo <= runs[k - 1].hi) return PPAS_EINVAL;
  }
  return PPAS_OK;
}

namespace {

struct Job {
  WorkItem item;
  double cost;
  int32_t order_key[4];
};

}  // namespace

void make_plan(const ppas_shape& shape, const ppas_seq* seqs, int32_t n_seqs, int num_cus, const PlanOpts& opts,
               Plan& plan) {
  plan.items.clear();
  plan.combine.clear();
  plan.part_slots = 0;
  const int hkv = shape.n_kv_heads;
  if (num_cus <= 0) num_cus = 256;

  // Total work, to size the key splits so that the launch has several
  // workgroups per compute unit: keys summed over prefill tiles (of either
  // size) and over decode rows.
  auto prefill_keys_for = [&](int32_t tile) {
    int64_t keys = 0;
    for (int32_t s = 0; s < n_seqs; ++s) {
      const ppas_seq& q = seqs[s];
      if (q.n_query == 1) continue;
      for (int32_t t0 = 0; t0 < q.n_query; t0 += tile) keys += int64_t(q.cached_len) + std::min(q.n_query, t0 + tile);
    }
    return keys * hkv;
  };
  int64_t decode_keys = 0, large_tiles = 0;
  for (int32_t s = 0; s < n_seqs; ++s) {
    const ppas_seq& q = seqs[s];
    if (q.n_query == 1)
      decode_keys += int64_t(q.cached_len + 1) * hkv;
    else
      large_tiles += ceil_div(q.n_query, kTilePosLarge) * hkv;
  }

  // Tile shape. The eight-wave kernel stages each K/V block once for 256 rows
  // instead of 128, which pays when the step's prefill alone fills the chip with
  // 32-position tiles (two per CU before any key split) and decode rows are a
  // small share of the work (a workgroup then holds a whole CU, so a prefill
  // tile no longer shares its CU with a decode item).
  int32_t tile = opts.tile_pos;
  if (tile != kTilePosSmall && tile != kTilePosLarge) {
    const int64_t small_keys = prefill_keys_for(kTilePosSmall);
    const bool big = large_tiles >= int64_t(2) * num_cus;
    const bool few_decodes = double(decode_keys) * 2.0 < kLargeTileDecodeShare * double(small_keys);
    tile = (big && few_decodes) ? kTilePosLarge : kTilePosSmall;
  }
  plan.tile_pos = tile;
  const int64_t prefill_keys = prefill_keys_for(tile);

  int64_t ksp = opts.prefill_split;
  if (ksp <= 0) {
    const int64_t target = int64_t(PPAS_PREFILL_ITEMS_PER_CU) * num_cus;
    ksp = std::max<int64_t>(256, ceil_div(prefill_keys, target));
  }
  ksp = std::max<int64_t>(kPrefillBlock, ceil_div(ksp, kPrefillBlock) * kPrefillBlock);
  int64_t ksd = opts.decode_split;
  if (ksd <= 0) {
    const int64_t target = int64_t(2) * num_cus;
    ksd = std::min<int64_t>(8192, std::max<int64_t>(512, ceil_div(decode_keys, target)));
  }
  ksd = std::max<int64_t>(kDecodeBlock, ceil_div(ksd, kDecodeBlock) * kDecodeBlock);
  ksd = std::min<int64_t>(ksd, kDecodeMaxKeys);

  // Prefill tiles load the matrix cores and decode items the memory system. When
  // the decode work is comparable to the prefill work, the two kinds are
  // interleaved in the launch order (below); otherwise decode goes last.
  const double tile_cost = double(tile) / kTilePosSmall;   // per key, relative to a 16-position tile
  const bool interleave = 2.0 * double(decode_keys) >= kInterleaveRatio * tile_cost * double(prefill_keys);

  // Key ranges of one tile or decode row. Decode rows, and prefill tiles of
  // interleaved steps, take pieces of `split` keys from key 0 (the last one
  // ragged: the short pieces fill the gaps between long items). Other prefill
  // tiles take round(keys / split) even pieces, so a step's items come close to
  // a whole number per workgroup slot. Prefill boundaries are multiples of the
  // 64-key block at or before the tile's first position, so every row sees a
  // key in every piece.
  //
  // A step of decode rows only (and no split size requested) cuts each row's keys
  // into even pieces instead, about one item per CU over the whole step: every
  // workgroup then streams from its own CU and all of them finish together
  // (measured on 48 rows of 20k-30k keys: 190 us with ~one item per CU against
  // 205 us with about two per CU, ragged). A piece never exceeds the page-id
  // capacity of a decode item.
  const bool decode_even = prefill_keys == 0 && decode_keys > 0 && opts.decode_split <= 0;
  auto piece_bounds = [&](int64_t kend, int64_t pos0, int kind) {
    std::vector<int64_t> b{0};
    if (kind == kKindDecode && decode_even) {
      const int64_t n = std::max<int64_t>(ceil_div(kend, int64_t(kDecodeMaxKeys - kDecodeBlock)),
                                          (kend * num_cus + decode_keys / 2) / decode_keys);
      for (int64_t k = 1; k < n; ++k) b.push_back(kend * k / n / kDecodeBlock * kDecodeBlock);
    } else if (kind == kKindDecode) {
      for (int64_t k = 1; k * ksd < kend; ++k) b.push_back(k * ksd);
    } else if (interleave) {
      for (int64_t k = 1; k * ksp <= pos0; ++k) b.push_back(k * ksp);
    } else {
      const int64_t n = std::max<int64_t>(1, (kend + ksp / 2) / ksp);
      const int64_t top = pos0 / kPrefillBlock * kPrefillBlock;
      for (int64_t k = 1; k < n; ++k) b.push_back(std::min(top, kend * k / n / kPrefillBlock * kPrefillBlock));
    }
    b.push_back(kend);
    b.erase(std::unique(b.begin(), b.end()), b.end());
    return b;
  };

  std::vector<Job> jobs;
  auto add_unit = [&](int32_t s, int32_t g, int32_t row0, int32_t pos0, int32_t npos, int kind) {
    const int64_t kend = int64_t(pos0) + npos;        // keys 0..kend-1 are visible to some row
    const std::vector<int64_t> bounds = piece_bounds(kend, pos0, kind);
    const int64_t nsplit = int64_t(bounds.size()) - 1;
    int32_t part = -1;
    if (nsplit > 1) {
      part = int32_t(plan.part_slots);
      plan.combine.push_back(CombineItem{row0, g, npos, int32_t(nsplit), part, 0, 0, 0});
      plan.part_slots += nsplit * int64_t(npos) * kGroup;
    }
    for (int64_t k = 0; k < nsplit; ++k) {
      const int64_t lo = bounds[size_t(k)], hi = bounds[size_t(k) + 1];
      Job j;
      j.item = WorkItem{s, g, row0, pos0, npos | (kind << 16), int32_t(lo), int32_t(hi),
                        part < 0 ? -1 : int32_t(part + k * int64_t(npos) * kGroup)};
      // relative cost: a prefill key of a 16-position tile costs 128 rows of MFMA
      // work (twice that in a 32-position tile), a decode key ~512 bytes of HBM
      // traffic; one decode key is about two prefill keys of a 16-position tile.
      j.cost = double(hi - lo) * (kind == kKindDecode ? 2.0 : tile_cost);
      j.order_key[0] = s;
      j.order_key[1] = g;
      j.order_key[2] = -pos0;
      j.order_key[3] = int32_t(k);
      jobs.push_back(j);
    }
  };
  for (int32_t s = 0; s < n_seqs; ++s) {
    const ppas_seq& q = seqs[s];
    for (int32_t g = 0; g < hkv; ++g) {
      if (q.n_query == 1) {
        add_unit(s, g, q.query_start, q.cached_len, 1, kKindDecode);
      } else {
        for (int32_t t0 = 0; t0 < q.n_query; t0 += tile)
          add_unit(s, g, q.query_start + t0, q.cached_len + t0, std::min(tile, q.n_query - t0), kKindPrefill);
      }
    }
  }

  // Longest first within each kind, in cost buckets of 256 keys; inside a bucket
  // keep items of the same request and KV head together so neighbours share keys
  // in one L2.
  auto lpt = [](const Job& a, const Job& b) {
    const int64_t ca = int64_t(a.cost) >> 8, cb = int64_t(b.cost) >> 8;
    if (ca != cb) return ca > cb;
    for (int i = 0; i < 4; ++i)
      if (a.order_key[i] != b.order_key[i]) return a.order_key[i] < b.order_key[i];
    return false;
  };
  std::vector<Job> pre, dec;
  for (const Job& j : jobs) ((j.item.npos_kind >> 16) == kKindDecode ? dec : pre).push_back(j);
  std::stable_sort(pre.begin(), pre.end(), lpt);
  std::stable_sort(dec.begin(), dec.end(), lpt);
  // Interleaved steps merge the two queues so that both advance at the same
  // fraction of their total work and finish together (prefill tiles load the
  // matrix cores, decode items the memory system); otherwise decode goes last
  // and fills the tail of the prefill rounds.
  double tot_p = 0, tot_d = 0;
  for (const Job& j : pre) tot_p += j.cost;
  for (const Job& j : dec) tot_d += j.cost;
  jobs.clear();
  size_t ip = 0, id = 0;
  double done_p = 0, done_d = 0;
  while (ip < pre.size() || id < dec.size()) {
    const bool take_p = id >= dec.size() ||
                        (ip < pre.size() && (!interleave || done_p * tot_d <= PPAS_INTERLEAVE_BIAS * done_d * tot_p));
    if (take_p) {
      done_p += pre[ip].cost;
      jobs.push_back(pre[ip++]);
    } else {
      done_d += dec[id].cost;
      jobs.push_back(dec[id++]);
    }
  }

  // Workgroup b of a launch runs on XCD b % 8. Hand each XCD runs of 8
  // consecutive items of the sorted list, with runs dealt round-robin so every XCD
  // gets the same mix of long and short items: within each block of 64 launch
  // slots, slot 8v + x takes sorted item 8x + v.
  const size_t n = jobs.size();
  plan.items.resize(n);
  const size_t full = n / 64 * 64;
  for (size_t b = 0; b < full; ++b) {
    const size_t x = b % 8, k = b / 8;
    const size_t src = ((k / 8) * 8 + x) * 8 + (k % 8);
    plan.items[b] = jobs[src].item;
  }
  for (size_t b = full; b < n; ++b) plan.items[b] = jobs[b].item;

  plan.off_combine = align_up(n * sizeof(WorkItem), 256);
  plan.list_bytes = plan.off_combine + plan.combine.size() * sizeof(CombineItem);
  plan.off_ml = 0;
  plan.off_acc = align_up(size_t(plan.part_slots) * 8, 256);
  plan.total = std::max<size_t>(256, align_up(plan.off_acc + size_t(plan.part_slots) * kHeadDim * 4, 256));
}

void make_append_items(const ppas_seq* seqs, int32_t n_seqs, std::vector<AppendItem>& items) {
  items.clear();
  for (int32_t s = 0; s < n_seqs; ++s) {
    const ppas_seq& q = seqs[s];
    const int32_t first = q.cached_len / kPage;
    const int32_t last = int32_t((int64_t(q.cached_len) + q.n_query - 1) / kPage);
    for (int32_t lp = first; lp <= last; ++lp)
      items.push_back(AppendItem{s, lp, q.cached_len, q.n_query, q.query_start, 0, 0, 0});
  }
}

}  // namespace ppas
