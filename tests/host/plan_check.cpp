// Host-side check of the step validator and the work planner, built with g++
// under AddressSanitizer and UndefinedBehaviorSanitizer by
// tests/test_host_sanitizers.py. It fuzzes valid steps (several CU counts and
// key-split settings) and checks the plan's invariants, then feeds invalid
// steps and checks each one's status code. Prints "ok" and returns 0 on success.
#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <map>
#include <numeric>
#include <utility>
#include <vector>

#include "plan.h"

using namespace ppas;

namespace {

int g_failures = 0;
#define CHECK(cond)                                                              \
  do {                                                                           \
    if (!(cond)) {                                                               \
      std::fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__, __LINE__, #cond); \
      if (++g_failures > 20) std::exit(1);                                       \
    }                                                                            \
  } while (0)

// splitmix64: a small deterministic generator for the fuzz cases
struct Rng {
  uint64_t s;
  uint64_t next() {
    uint64_t z = (s += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
  }
  int uniform(int lo, int hi) { return lo + int(next() % uint64_t(hi - lo + 1)); }   // inclusive
};

ppas_shape make_shape(int num_pages) {
  ppas_shape s;
  s.n_q_heads = 16;
  s.n_kv_heads = 2;
  s.head_dim = 128;
  s.page_size = 16;
  s.num_pages = num_pages;
  s.scale = 0.08838834764831845f;
  return s;
}

struct Step {
  std::vector<ppas_seq> seqs;
  std::vector<int32_t> bt;
  int stride = 1, pages = 1;
};

Step random_step(Rng& g) {
  Step st;
  const int n = g.uniform(0, 12);
  int32_t qs = 0;
  for (int i = 0; i < n; ++i) {
    ppas_seq q;
    const bool decode = g.uniform(0, 2) == 0;
    q.n_query = decode ? 1 : g.uniform(1, 300);
    q.cached_len = g.uniform(0, 3) == 0 ? g.uniform(0, 40000) : g.uniform(0, 3000);
    q.query_start = qs;
    qs += q.n_query;
    st.seqs.push_back(q);
  }
  int total = 0;
  for (const auto& q : st.seqs) {
    const int p = (q.cached_len + q.n_query + kPage - 1) / kPage;
    st.stride = std::max(st.stride, p);
    total += p;
  }
  st.pages = std::max(1, total + g.uniform(0, 5));
  std::vector<int32_t> perm(size_t(st.pages));
  std::iota(perm.begin(), perm.end(), 0);
  for (int i = st.pages - 1; i > 0; --i) std::swap(perm[size_t(i)], perm[size_t(g.uniform(0, i))]);
  st.bt.assign(size_t(std::max<size_t>(1, st.seqs.size())) * size_t(st.stride), -1);
  int at = 0;
  for (size_t i = 0; i < st.seqs.size(); ++i) {
    const int p = (st.seqs[i].cached_len + st.seqs[i].n_query + kPage - 1) / kPage;
    for (int j = 0; j < p; ++j) st.bt[i * size_t(st.stride) + size_t(j)] = perm[size_t(at++)];
  }
  return st;
}

// Every (row, KV head) sees keys 0..p exactly once over its items; every item
// gives each of its rows a visible key; split rows are merged once.
void check_plan(const Step& st, const Plan& plan) {
  const int hkv = 2;
  std::map<std::pair<int64_t, int>, std::vector<std::pair<int64_t, int64_t>>> cover;
  std::vector<char> slot_used(size_t(plan.part_slots), 0);
  for (const WorkItem& it : plan.items) {
    const int npos = it.npos_kind & 0xffff, kind = it.npos_kind >> 16;
    CHECK(it.seq >= 0 && size_t(it.seq) < st.seqs.size());
    if (it.seq < 0 || size_t(it.seq) >= st.seqs.size()) continue;
    const ppas_seq& q = st.seqs[size_t(it.seq)];
    CHECK(it.kvh >= 0 && it.kvh < hkv);
    CHECK(kind == (q.n_query == 1 ? kKindDecode : kKindPrefill));
    CHECK(npos >= 1 && npos <= plan.tile_pos);
    CHECK(plan.tile_pos == kTilePosSmall || plan.tile_pos == kTilePosLarge);
    CHECK(it.row0 >= q.query_start && it.row0 + npos <= q.query_start + q.n_query);
    CHECK(it.pos0 == q.cached_len + (it.row0 - q.query_start));
    CHECK(it.key_lo >= 0 && it.key_lo < it.key_hi && it.key_hi <= it.pos0 + npos);
    CHECK(it.key_lo <= it.pos0);   // every row of the item sees at least one key
    if (kind == kKindDecode) {
      CHECK(it.key_hi - it.key_lo <= kDecodeMaxKeys);
      CHECK(it.key_lo % kDecodeBlock == 0);
    } else {
      CHECK(it.key_lo % kPrefillBlock == 0);
    }
    if (it.part >= 0) {
      CHECK(int64_t(it.part) + npos * kGroup <= plan.part_slots);
      for (int r = 0; r < npos * kGroup && int64_t(it.part) + r < plan.part_slots; ++r) {
        CHECK(!slot_used[size_t(it.part + r)]);
        slot_used[size_t(it.part + r)] = 1;
      }
    }
    for (int r = 0; r < npos; ++r) {
      const int64_t p = it.pos0 + r;
      cover[{int64_t(it.row0 + r), it.kvh}].push_back({it.key_lo, std::min<int64_t>(it.key_hi, p + 1)});
    }
  }
  for (char u : slot_used) CHECK(u);
  int64_t rows = 0;
  for (const auto& q : st.seqs) rows += q.n_query;
  CHECK(int64_t(cover.size()) == rows * hkv);
  for (const auto& q : st.seqs)
    for (int i = 0; i < q.n_query; ++i)
      for (int g = 0; g < hkv; ++g) {
        auto r = cover[{int64_t(q.query_start + i), g}];
        std::sort(r.begin(), r.end());
        CHECK(!r.empty() && r.front().first == 0 && r.back().second == int64_t(q.cached_len) + i + 1);
        for (size_t k = 1; k < r.size(); ++k) CHECK(r[k - 1].second == r[k].first);
      }
  // combine items: one per split (row block, KV head), each split item accounted for
  int64_t comb_slots = 0;
  for (const CombineItem& c : plan.combine) {
    CHECK(c.nsplit >= 2 && c.npos >= 1 && c.npos <= plan.tile_pos);
    CHECK(c.part >= 0 && int64_t(c.part) + int64_t(c.nsplit) * c.npos * kGroup <= plan.part_slots);
    comb_slots += int64_t(c.nsplit) * c.npos * kGroup;
  }
  CHECK(comb_slots == plan.part_slots);
  // work-list and workspace layouts: ordered, aligned, large enough for every array
  CHECK(plan.off_combine >= plan.items.size() * sizeof(WorkItem) && plan.off_combine % 256 == 0);
  CHECK(plan.list_bytes == plan.off_combine + plan.combine.size() * sizeof(CombineItem));
  CHECK(plan.off_ml == 0);
  CHECK(plan.off_acc >= size_t(plan.part_slots) * 8 && plan.off_acc % 256 == 0);
  CHECK(plan.total >= plan.off_acc + size_t(plan.part_slots) * kHeadDim * 4);
  CHECK(plan.total >= 256 && plan.total % 256 == 0);
}

void fuzz() {
  Rng g{12345};
  const int cus[] = {1, 8, 80, 256, 304};
  const int32_t splits[][2] = {{0, 0}, {64, 32}, {128, 96}, {4096, 1 << 20}};
  for (int t = 0; t < 400; ++t) {
    const Step st = random_step(g);
    const ppas_shape sh = make_shape(st.pages);
    const int32_t n = int32_t(st.seqs.size());
    CHECK(validate(&sh, st.seqs.data(), n, st.bt.data(), st.stride, true) == PPAS_OK);
    const auto& sp = splits[t % 4];
    PlanOpts opts;
    opts.prefill_split = sp[0];
    opts.decode_split = sp[1];
    opts.tile_pos = (t / 4) % 3 == 0 ? 0 : (t / 4) % 3 == 1 ? kTilePosSmall : kTilePosLarge;
    Plan plan;
    make_plan(sh, st.seqs.data(), n, cus[t % 5], opts, plan);
    check_plan(st, plan);
    // the page-write list: one item per (request, touched logical page), in order
    std::vector<AppendItem> app;
    make_append_items(st.seqs.data(), n, app);
    size_t k = 0;
    for (int32_t s = 0; s < n; ++s) {
      const ppas_seq& q = st.seqs[size_t(s)];
      for (int32_t lp = q.cached_len / kPage; lp <= (q.cached_len + q.n_query - 1) / kPage; ++lp, ++k) {
        CHECK(k < app.size());
        if (k >= app.size()) break;
        CHECK(app[k].seq == s && app[k].lpage == lp && app[k].cached_len == q.cached_len &&
              app[k].n_query == q.n_query && app[k].query_start == q.query_start);
      }
    }
    CHECK(k == app.size());
  }
}

void invalid() {
  ppas_shape sh = make_shape(64);
  std::vector<ppas_seq> seqs = {{0, 10, 20}, {10, 1, 5}};
  std::vector<int32_t> bt = {0, 1, -1, 2, -1, -1};   // stride 3
  CHECK(validate(&sh, seqs.data(), 2, bt.data(), 3, true) == PPAS_OK);
  CHECK(validate(nullptr, seqs.data(), 2, bt.data(), 3, true) == PPAS_EINVAL);
  CHECK(validate(&sh, seqs.data(), -1, bt.data(), 3, true) == PPAS_EINVAL);
  CHECK(validate(&sh, nullptr, 2, bt.data(), 3, true) == PPAS_EINVAL);
  CHECK(validate(&sh, seqs.data(), 2, bt.data(), 0, true) == PPAS_EINVAL);
  CHECK(validate(&sh, seqs.data(), 2, bt.data(), 1, true) == PPAS_EINVAL);   // row too short
  {
    auto s2 = seqs;
    s2[1].query_start = 11;   // not contiguous
    CHECK(validate(&sh, s2.data(), 2, bt.data(), 3, true) == PPAS_EINVAL);
    s2 = seqs;
    s2[0].n_query = 0;
    CHECK(validate(&sh, s2.data(), 2, bt.data(), 3, true) == PPAS_EINVAL);
    s2 = seqs;
    s2[1].cached_len = -1;
    CHECK(validate(&sh, s2.data(), 2, bt.data(), 3, true) == PPAS_EINVAL);
    s2 = seqs;
    s2[0].cached_len = INT32_MAX - 70;
    CHECK(validate(&sh, s2.data(), 2, bt.data(), 3, false) == PPAS_ERANGE);
  }
  {
    auto b2 = bt;
    b2[1] = 64;   // page outside the pool
    CHECK(validate(&sh, seqs.data(), 2, b2.data(), 3, true) == PPAS_ERANGE);
    b2 = bt;
    b2[3] = 1;    // request 1 writes its slot 5 of page 1, which request 0 writes (positions 20..29)
    CHECK(validate(&sh, seqs.data(), 2, b2.data(), 3, true) == PPAS_EINVAL);
  }
  {
    ppas_shape s2 = sh;
    s2.head_dim = 64;
    CHECK(validate(&s2, seqs.data(), 2, bt.data(), 3, true) == PPAS_EUNSUPPORTED);
    s2 = sh;
    s2.n_q_heads = 12;   // groups of 6: a valid shape outside the compiled one
    CHECK(validate(&s2, seqs.data(), 2, bt.data(), 3, true) == PPAS_EUNSUPPORTED);
    s2 = sh;
    s2.n_q_heads = 15;   // heads not divisible into groups
    CHECK(validate(&s2, seqs.data(), 2, bt.data(), 3, true) == PPAS_EINVAL);
    s2 = sh;
    s2.scale = 0.f;
    CHECK(validate(&s2, seqs.data(), 2, bt.data(), 3, true) == PPAS_EINVAL);
    s2 = sh;
    s2.num_pages = 0;
    CHECK(validate(&s2, seqs.data(), 2, bt.data(), 3, true) == PPAS_EINVAL);
  }
  CHECK(validate(&sh, seqs.data(), 0, nullptr, 0, true) == PPAS_OK);   // empty step
  {
    // overlap checks by slot runs: one request whose logical pages 0 and 2 share a
    // physical page clashes on slots 0..7; two requests sharing a page on disjoint
    // slot runs (0..4 and 5..15) do not, on touching runs (0..5 and 5..15) they do
    std::vector<ppas_seq> one = {{0, 40, 0}};
    std::vector<int32_t> r = {5, 6, 5};
    CHECK(validate(&sh, one.data(), 1, r.data(), 3, true) == PPAS_EINVAL);
    CHECK(validate(&sh, one.data(), 1, r.data(), 3, false) == PPAS_OK);
    r = {5, 6, 7};
    CHECK(validate(&sh, one.data(), 1, r.data(), 3, true) == PPAS_OK);
    std::vector<ppas_seq> two = {{0, 5, 16}, {5, 11, 5}};
    std::vector<int32_t> t = {9, 9, 9, 8};   // stride 2: request 0 -> page 9 slots 0..4; request 1 -> page 9 slots 5..15
    CHECK(validate(&sh, two.data(), 2, t.data(), 2, true) == PPAS_OK);
    two[0].n_query = 6;
    two[1].query_start = 6;
    CHECK(validate(&sh, two.data(), 2, t.data(), 2, true) == PPAS_EINVAL);
  }
}

}  // namespace

int main() {
  fuzz();
  invalid();
  if (g_failures) {
    std::fprintf(stderr, "%d check(s) failed\n", g_failures);
    return 1;
  }
  std::printf("ok\n");
  return 0;
}
