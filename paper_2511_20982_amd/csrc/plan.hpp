// Launch planning of the attention kernels: pure integer arithmetic on the
// host copies of the lengths and the machine shape (CU and XCD counts), with
// no HIP dependency, so the same functions size the launches in the library
// and are checked on the CPU at several machine shapes.  The few formulas the
// kernels evaluate too are constexpr (host and device).
#pragma once
#include <algorithm>
#include <cstddef>
#include <cstdint>

namespace dopd {

// Compute units and XCDs of the device a call runs on.
struct MachineShape {
  int cus;
  int xcds;
};
// Used when no device answers the query (only host-side sizing can run then).
constexpr MachineShape kDefaultMachine{256, 8};

// Four-wave workgroups resident per CU for the decode and prefill kernels
// (both are launched with __launch_bounds__(256, 2)).
constexpr int kWgPerCu = 2;

constexpr size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// ---- decode partition ------------------------------------------------------
// The keys of every (request r, KV head c) are cut into pairs of pages (32
// tokens); (r, c) is a span of kDecSegCost + pairs work units, spans laid out
// r-major then c; workgroup b takes units [b * total / nwg, (b+1) * total / nwg).
constexpr int kDecSegCost = 8;          // work units of a segment start, in pairs
constexpr int kDecMaxSplitTokens = 4096;
constexpr int64_t kDecMinPairsPerWg = 4;  // one pair per wave at least

constexpr int64_t dec_slice_begin(int64_t b, int64_t total, int64_t nwg) {
  return b * total / nwg;
}

inline int64_t decode_total_units(const int32_t* ctx, int32_t n, int hkv) {
  int64_t units = 0;
  for (int32_t r = 0; r < n; ++r) units += (int64_t)(kDecSegCost + (ctx[r] + 31) / 32) * hkv;
  return units;
}

// Resident decode workgroup slots the automatic partition fills: quarter_wgs / 4
// workgroups per CU (8 = two per CU, every slot; fewer leaves slots to the
// prefill items of a fused step).
inline int64_t decode_slots(const MachineShape& m, int quarter_wgs = 4 * kWgPerCu) {
  return std::max<int64_t>(1, (int64_t)std::max(1, m.cus) * std::max(1, quarter_wgs) / 4);
}

// Workgroups of the partition: split_tokens / 32 units each when given, else
// one slice per resident slot (one round).
inline int64_t decode_nwg(int64_t total_units, int32_t split_tokens, const MachineShape& m,
                          int quarter_wgs = 4 * kWgPerCu) {
  if (total_units <= 0) return 0;
  if (split_tokens > 0) {
    const int64_t per = split_tokens / 32;
    return (total_units + per - 1) / per;
  }
  const int64_t slots = decode_slots(m, quarter_wgs);
  return std::max<int64_t>(1, std::min(slots, (total_units + kDecMinPairsPerWg - 1) /
                                                  kDecMinPairsPerWg));
}

// Workspace of the decode: partial slots, at most one per (workgroup, (r, c))
// boundary, indexed workgroup + (r * Hkv + c); [slots][g][d] fp32 partial
// outputs, then [slots][g][2] (m, l), each 256-byte aligned.
struct DecodeLayout {
  int64_t nwg, slots;
  size_t part_o_off, part_ml_off, total;
};

inline DecodeLayout decode_layout(int g, int hkv, int d, const int32_t* ctx, int32_t n,
                                  int32_t split_tokens, const MachineShape& m,
                                  int quarter_wgs = 4 * kWgPerCu) {
  DecodeLayout L{};
  L.nwg = decode_nwg(decode_total_units(ctx, n, hkv), split_tokens, m, quarter_wgs);
  L.slots = L.nwg + (int64_t)n * hkv;
  L.part_o_off = 0;
  L.part_ml_off = align256((size_t)L.slots * g * d * sizeof(float));
  L.total = L.part_ml_off + align256((size_t)L.slots * g * 2 * sizeof(float));
  return L;
}

// The workgroup whose slice holds work unit x (the kernels use the same search).
inline int64_t dec_slice_of(int64_t x, int64_t total, int64_t nwg) {
  int64_t b = x * nwg / total;
  while (b + 1 < nwg && dec_slice_begin(b + 1, total, nwg) <= x) ++b;
  while (b > 0 && dec_slice_begin(b, total, nwg) > x) --b;
  return b;
}

// Does any (r, c) span two slices (then the merge kernel runs)?
inline bool decode_needs_merge(const int32_t* ctx, int32_t n, int hkv, int64_t total,
                               int64_t nwg) {
  int64_t base = 0;
  for (int32_t r = 0; r < n; ++r) {
    const int64_t np = (ctx[r] + 31) / 32, span = kDecSegCost + np;
    for (int c = 0; c < hkv; ++c) {
      const int64_t first = base + c * span + kDecSegCost;  // unit of the first pair
      if (dec_slice_of(first, total, nwg) != dec_slice_of(first + np - 1, total, nwg))
        return true;
    }
    base += span * hkv;
  }
  return false;
}

// The (r, c) whose pairs span several slices (the ones the merge kernel
// combines), listed for the merge kernel's arguments: item = r * Hkv + c
// | b0 << 14 | (b1 - b0) << 24, with b0 and b1 the slices of its first and
// last pair, in (r, c) order.  Returns the count, or -1 when the list would
// not fit that packing (more than 2^14 (r, c), 2^10 workgroups, a span of
// more than 255 slices) or more than max items (the caller then merges with
// the kernel that finds its pairs itself).
constexpr int kMergeRcBits = 14, kMergeB0Bits = 10;

inline int decode_merge_list(const int32_t* ctx, int32_t n, int hkv, int64_t total, int64_t nwg,
                             uint32_t* items, int max) {
  if ((int64_t)n * hkv > (1 << kMergeRcBits) || nwg > (1 << kMergeB0Bits)) return -1;
  int cnt = 0;
  int64_t base = 0;
  for (int32_t r = 0; r < n; ++r) {
    const int64_t np = (ctx[r] + 31) / 32, span = kDecSegCost + np;
    for (int c = 0; c < hkv; ++c) {
      const int64_t first = base + c * span + kDecSegCost;  // unit of the first pair
      const int64_t b0 = dec_slice_of(first, total, nwg), b1 = dec_slice_of(first + np - 1, total, nwg);
      if (b0 == b1) continue;
      if (cnt == max || b1 - b0 > 255) return -1;
      items[cnt++] = (uint32_t)((int64_t)r * hkv + c) | (uint32_t)b0 << kMergeRcBits |
                     (uint32_t)(b1 - b0) << (kMergeRcBits + kMergeB0Bits);
    }
    base += span * hkv;
  }
  return cnt;
}

// ---- prefill work order ----------------------------------------------------
// With the XCD-aware order the work list of n_items items is dealt to the
// XCDs in contiguous slices of per_xcd items; the hardware dispatcher sends
// workgroup b to XCD b % xcds, so workgroup b takes item
// (b % xcds) * per_xcd + b / xcds (none when past the list).
constexpr int pf_per_xcd(int n_items, int xcds) { return (n_items + xcds - 1) / xcds; }
constexpr int pf_xcd_item(int b, int xcds, int per_xcd) {
  return (b % xcds) * per_xcd + b / xcds;
}
constexpr bool pf_xcd_valid(int b, int xcds, int per_xcd, int n_items) {
  return b / xcds < per_xcd && pf_xcd_item(b, xcds, per_xcd) < n_items;
}

// Key splits of the paged prefill: the requested count (at most kPfMaxSplits),
// or automatically, when the call has at most one work item per CU, about
// (resident slots) / items splits (at most kPfAutoSplits), each split of the
// longest item keeping at least 8 key tiles that every row sees.  Each split
// adds T * Hq * d * 8 bytes of fp32 partials written and read back, which costs
// more than it gains once the items fill the CUs.
constexpr int kPfMaxSplits = 16;
constexpr int kPfAutoSplits = 8;
constexpr int kPfTileRows = 128;  // query rows per work item
constexpr int kPfTileKeys = 64;   // keys per tile

inline int prefill_paged_splits(int hq, bool splittable, const int32_t* cu_host,
                                const int32_t* prefix_host, int32_t nreq, int32_t num_splits,
                                const MachineShape& m) {
  if (!splittable) return 1;
  if (num_splits > 0) return std::min(num_splits, kPfMaxSplits);
  const int64_t slots = (int64_t)kWgPerCu * std::max(1, m.cus);
  int64_t items = 0, max_full = 0;
  for (int32_t r = 0; r < nreq; ++r) {
    const int64_t len = cu_host[r + 1] - cu_host[r];
    const int64_t tiles = (len + kPfTileRows - 1) / kPfTileRows;
    items += tiles * hq;
    if (tiles > 0)
      max_full = std::max<int64_t>(max_full,
                                   (prefix_host[r] + (tiles - 1) * kPfTileRows) / kPfTileKeys);
  }
  if (items == 0 || items > slots / 2) return 1;
  int64_t n = slots / items;
  n = std::min<int64_t>(n, 1 + max_full / 8);
  return (int)std::max<int64_t>(1, std::min<int64_t>(n, kPfAutoSplits));
}

inline size_t prefill_paged_ws_bytes(int hq, int d, int64_t T, int nsplit) {
  if (nsplit <= 1) return 0;
  const size_t rows = (size_t)nsplit * T * hq;
  return align256(rows * d * sizeof(float)) + align256(rows * 2 * sizeof(float));
}

}  // namespace dopd
