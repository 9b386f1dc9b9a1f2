// CPU check of the launch planning (paper_2511_20982_amd/csrc/plan.hpp) at a
// given machine shape: the decode partition and its workspace slots, the
// prefill's XCD-aware work order and the automatic key-split count.
// Usage: plan_harness <cus> <xcds>; prints "ok <cases>" or the first failure.
#include <cstdio>
#include <cstdlib>
#include <random>
#include <set>
#include <vector>

#include "../paper_2511_20982_amd/csrc/plan.hpp"

using namespace dopd;

static int fail(const char* what, long a, long b) {
  std::printf("FAIL %s (%ld, %ld)\n", what, a, b);
  return 1;
}

// Walks the slices as the decode kernel does (a slice holds whole or partial
// spans of kDecSegCost + pairs units; pairs of one (r, c) inside a slice form
// a segment) and checks the workspace slots the segments write.
static int check_decode(const std::vector<int32_t>& ctx, int hkv, int split, int d,
                        const MachineShape& m) {
  const int n = (int)ctx.size(), g = 4;
  const int64_t total = decode_total_units(ctx.data(), n, hkv);
  const DecodeLayout L = decode_layout(g, hkv, d, ctx.data(), n, split, m);
  const int64_t nwg = L.nwg;
  if (split == 0 && nwg > (int64_t)kWgPerCu * m.cus) return fail("nwg above resident slots", nwg, m.cus);
  if (nwg < 1) return fail("no workgroup", nwg, total);
  if (L.part_ml_off % 256 || L.total % 256) return fail("layout alignment", L.part_ml_off, L.total);
  if (L.total < (size_t)L.slots * g * (d + 2) * 4) return fail("layout too small", L.total, L.slots);
  if (dec_slice_begin(0, total, nwg) != 0 || dec_slice_begin(nwg, total, nwg) != total)
    return fail("slices do not cover the units", 0, total);
  for (int64_t b = 0; b < nwg; ++b)
    if (dec_slice_begin(b, total, nwg) > dec_slice_begin(b + 1, total, nwg))
      return fail("slice order", b, nwg);
  std::mt19937_64 rng(7);
  for (int i = 0; i < 2000; ++i) {
    const int64_t x = (int64_t)(rng() % (uint64_t)total);
    const int64_t b = dec_slice_of(x, total, nwg);
    if (!(dec_slice_begin(b, total, nwg) <= x && x < dec_slice_begin(b + 1, total, nwg)))
      return fail("slice_of", x, b);
  }
  // segments
  std::vector<int64_t> span_start(n + 1, 0);
  for (int r = 0; r < n; ++r) span_start[r + 1] = span_start[r] + (int64_t)(kDecSegCost + (ctx[r] + 31) / 32) * hkv;
  std::set<int64_t> partial_slots;
  std::vector<int64_t> pairs_seen((size_t)n * hkv, 0);
  bool merge = false;
  for (int r = 0; r < n; ++r) {
    const int64_t np = (ctx[r] + 31) / 32, span = kDecSegCost + np;
    for (int c = 0; c < hkv; ++c) {
      const int64_t p_first = span_start[r] + c * span + kDecSegCost;  // unit of pair 0
      const int64_t b0 = dec_slice_of(p_first, total, nwg);
      const int64_t b1 = dec_slice_of(p_first + np - 1, total, nwg);
      for (int64_t b = b0; b <= b1; ++b) {
        const int64_t lo = dec_slice_begin(b, total, nwg), hi = dec_slice_begin(b + 1, total, nwg);
        const int64_t a = std::max(lo, p_first), e = std::min(hi, p_first + np);
        if (a >= e) continue;  // (an empty slice between two others)
        pairs_seen[(size_t)r * hkv + c] += e - a;
        const bool whole = a == p_first && e == p_first + np;
        if (!whole) {
          merge = true;
          const int64_t slot = b + (int64_t)r * hkv + c;
          if (slot >= L.slots) return fail("partial slot out of range", slot, L.slots);
          if (!partial_slots.insert(slot).second) return fail("partial slot reused", slot, b);
        }
      }
    }
  }
  for (int r = 0; r < n; ++r)
    for (int c = 0; c < hkv; ++c)
      if (pairs_seen[(size_t)r * hkv + c] != (ctx[r] + 31) / 32) return fail("pairs not covered once", r, c);
  if (merge != decode_needs_merge(ctx.data(), n, hkv, total, nwg))
    return fail("merge decision", merge, nwg);
  // the merge list: exactly the (r, c) with a partial segment, in (r, c)
  // order, with the slices of their first and last pairs
  std::vector<uint32_t> want;
  bool fits = (int64_t)n * hkv <= (1 << kMergeRcBits) && nwg <= (1 << kMergeB0Bits);
  for (int r = 0; r < n && fits; ++r)
    for (int c = 0; c < hkv; ++c) {
      const int64_t np = (ctx[r] + 31) / 32;
      const int64_t first = span_start[r] + c * (kDecSegCost + np) + kDecSegCost;
      const int64_t b0 = dec_slice_of(first, total, nwg), b1 = dec_slice_of(first + np - 1, total, nwg);
      bool split = false;  // from the segment walk: some slice holds only part of (r, c)
      for (int64_t b = b0; b <= b1; ++b)
        if (partial_slots.count(b + (int64_t)r * hkv + c)) split = true;
      if (split != (b0 != b1)) return fail("split pair vs slices", r, c);
      if (!split) continue;
      if (b1 - b0 > 255) fits = false;
      want.push_back((uint32_t)(r * hkv + c) | (uint32_t)b0 << kMergeRcBits |
                     (uint32_t)(b1 - b0) << (kMergeRcBits + kMergeB0Bits));
    }
  std::vector<uint32_t> got(want.size() + 1);
  const int cnt = decode_merge_list(ctx.data(), n, hkv, total, nwg, got.data(), (int)got.size());
  if (!fits) {
    if (cnt != -1) return fail("merge list should not fit", cnt, nwg);
  } else {
    if (cnt != (int)want.size()) return fail("merge list count", cnt, (long)want.size());
    for (size_t i = 0; i < want.size(); ++i)
      if (got[i] != want[i]) return fail("merge list item", (long)i, (long)got[i]);
    if (!want.empty() && decode_merge_list(ctx.data(), n, hkv, total, nwg, got.data(),
                                           (int)want.size() - 1) != -1)
      return fail("merge list past its capacity", (long)want.size(), 0);
  }
  return 0;
}

static int check_prefill_order(int n_items, const MachineShape& m) {
  const int per = pf_per_xcd(n_items, m.xcds);
  const int blocks = per * m.xcds;
  std::vector<int> hits(n_items, 0);
  std::vector<int> last_of_xcd(m.xcds, -1);
  for (int b = 0; b < blocks; ++b) {
    if (!pf_xcd_valid(b, m.xcds, per, n_items)) continue;
    const int it = pf_xcd_item(b, m.xcds, per);
    if (it < 0 || it >= n_items) return fail("item out of range", b, it);
    ++hits[it];
    const int x = b % m.xcds;  // the XCD this workgroup lands on
    if (it / per != x) return fail("item off its XCD slice", b, it);
    if (it <= last_of_xcd[x]) return fail("XCD slice out of order", b, it);
    last_of_xcd[x] = it;
  }
  for (int i = 0; i < n_items; ++i)
    if (hits[i] != 1) return fail("item not taken exactly once", i, hits[i]);
  return 0;
}

static int check_splits(const MachineShape& m) {
  const int slots = kWgPerCu * m.cus;
  // one request: 300-token chunk after 20000 cached tokens, 4 heads (12 items)
  std::vector<int32_t> cu{0, 300}, pre{20000};
  int n = prefill_paged_splits(4, true, cu.data(), pre.data(), 1, 0, m);
  const int items = 3 * 4;
  int want = items > slots / 2 ? 1 : std::min({slots / items, 1 + (20000 + 2 * 128) / 64 / 8, kPfAutoSplits});
  if (want < 1) want = 1;
  if (n != want) return fail("automatic split count", n, want);
  if (prefill_paged_splits(4, false, cu.data(), pre.data(), 1, 0, m) != 1) return fail("unsplittable split", 0, 0);
  if (prefill_paged_splits(4, true, cu.data(), pre.data(), 1, 40, m) != kPfMaxSplits) return fail("split cap", 0, 0);
  // many items: no split
  std::vector<int32_t> cu2{0, 128 * slots}, pre2{0};
  if (prefill_paged_splits(1, true, cu2.data(), pre2.data(), 1, 0, m) != 1) return fail("split of a full call", 0, 0);
  return 0;
}

int main(int argc, char** argv) {
  if (argc != 3) return 2;
  const MachineShape m{std::atoi(argv[1]), std::atoi(argv[2])};
  std::mt19937 rng(20982);
  int cases = 0;
  for (int t = 0; t < 60; ++t) {
    const int n = 1 + (int)(rng() % 300);
    std::vector<int32_t> ctx(n);
    for (auto& c : ctx) c = 1 + (int)(rng() % (t % 3 == 0 ? 16384 : 2000));
    for (int hkv : {1, 4, 8})
      for (int split : {0, 32, 512}) {
        if (check_decode(ctx, hkv, split, 128, m)) return 1;
        ++cases;
      }
  }
  for (int n_items : {1, 7, 8, 9, 255, 256, 257, 1000, 8100}) {
    if (check_prefill_order(n_items, m)) return 1;
    ++cases;
  }
  if (check_splits(m)) return 1;
  std::printf("ok %d\n", cases + 1);
  return 0;
}
