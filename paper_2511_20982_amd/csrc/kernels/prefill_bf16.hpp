// Variable-length causal prefill attention, bf16 in / fp32 accumulate, gfx950.
//
// Workgroup = 4 waves = one (q tile of 128 rows, request, query head) item;
// each wave owns 32 query rows.  Two workgroups share a CU, so each SIMD runs
// two waves whose MFMA and VALU phases overlap.
//
// Per 64-key tile and wave:
//   S^T[64 tok][32 q] = K[64][d] . Q^T[d][32]       2 x (d/16) v_mfma_f32_32x32x16_bf16
//   O^T[d][32 q]     += V^T[d][64] . P^T[64][32]    (d/32) x 4  v_mfma_f32_32x32x16_bf16
// Computing the transposed products keeps a query row inside one lane pair,
// and the S^T accumulator is directly the P^T B operand of the P.V MFMA (the
// key order of the contraction is matched by the V^T reads).
//
// K and V tiles move from global memory straight into LDS (buffer loads with
// the LDS destination, no registers), double-buffered; K is one tile ahead of
// V so that a step computes S^T of tile j + 1 on the MFMAs while the VALU
// forms P of tile j.  V stays token-major in LDS and the V^T operand is
// gathered with the transposing LDS read.
//
// Softmax: exp2 with the scale folded into one fma; P is rounded to bf16 for
// the P.V product and the row sum l adds the rounded values.  In the steady
// state no row max is taken: p is formed against the running max and only a
// row sum beyond 2^20 (a tile far above it) takes the tile max, rescales O
// and l and forms p again.  Diagonal and ragged tiles take the max and mask
// with a select.
// Work order: with at most 64 requests, each XCD takes a contiguous slice of
// (KV head, request longest first, q tile descending, query head) so the q tiles
// that read the same K/V run together under one L2; otherwise heaviest q
// tiles first.
#pragma once
#include <type_traits>

#include "common.hpp"
#include "../plan.hpp"

namespace dopd {

struct PrefillArgs {
  const uint16_t* q;   // [T][Hq][D]
  const uint16_t* k;   // [T][Hkv][D]
  const uint16_t* v;   // [T][Hkv][D]
  uint16_t* out;       // [T][Hq][D]
  float* lse;          // [T][Hq] or null
  const int32_t* cu;   // [nreq + 1]
  int nreq, hq, hkv, max_tiles;
  int hslots;          // head slots = ceil(hq / kPfHeadsPerWG)
  float scale_log2;
  // XCD-aware order (used when nreq <= kPfMaxOrdered): the work list is
  // (slot block, request by decreasing length, q tile descending, slot of the
  // block); XCD x = workgroup % xcds takes the contiguous slice
  // [x * per_xcd, (x+1) * per_xcd), so the q tiles that share a request's K/V
  // run together on one XCD and share its L2.
  int xcd_order, n_items, per_xcd, tiles_total, xcds;
  int ord[64];         // requests by decreasing length
  // With the XCD order: incl[i] = sum over positions p <= i of the order of
  // (slots per block) x (q tiles of request ord[p]); copies of cu and prefix.
  int incl[64];
  int cu_h[65];
  int prefix_h[64];
  // Chunk prefill over the paged cache (the paged instantiation only): the
  // chunk rows of request r are q[cu[r] .. cu[r+1]), its keys are the cached
  // positions 0 .. prefix[r] + chunk length - 1, read through the page table.
  const uint16_t* k_pool;     // [P][Hkv][16][D]
  const uint16_t* v_pool;     // [P][Hkv][D][16]
  const int32_t* page_table;  // [nreq][pt_stride]
  const int32_t* prefix;      // [nreq]
  int pt_stride;
  // Per-KV-head scales of the cached K and V (null: 1): key = cached value *
  // k_scale[c], value = cached value * v_scale[c] (E4M3 pools, KV8: the pools
  // hold one-byte codes, widened to bf16 exactly as they leave LDS).  The K
  // scale multiplies the softmax scale, the V scale the output.
  const float* k_scale;
  const float* v_scale;
  // Key splits of the paged kernel (nsplit > 1): workgroup b computes split
  // b % nsplit of item b / nsplit, keys of tiles [t_s, t_{s+1}) with
  // t_s = min(s * ntiles / nsplit, nfull) (the last split also takes every
  // tile a row of the item does not see in full), and writes the
  // un-normalised (o, m, l) of its rows to split slot s of part_o / part_ml,
  // [nsplit][T][Hq][D] and [nsplit][T][Hq][2] (m in the exp2 domain); the
  // merge kernel combines them.
  int nsplit;
  float* part_o;
  float* part_ml;
  int part_rows;              // T of the call
};

constexpr int kPfMaxOrdered = 64;

constexpr int kPfBM = kPfTileRows;  // query rows per workgroup (32 per wave)
constexpr int kPfHeadsPerWG = 1;    // heads per workgroup
constexpr int kPfThreads = kPfHeadsPerWG * (kPfBM / 32) * 64;
constexpr int kPfBN = kPfTileKeys;  // keys per tile

// Number of BM-row q tiles of request rr.
__device__ __forceinline__ int pf_tiles(const int32_t* cu, int rr) {
  return (cu[rr + 1] - cu[rr] + kPfBM - 1) / kPfBM;
}

// Maps a workgroup index to (q tile, request, head slot), q tiles in
// decreasing index order (tile i of a request attends to ~ (i+1) key tiles).
__device__ __forceinline__ bool pf_find_item_lpt(const PrefillArgs& a, int b, int& tile,
                                                 int& req, int& slot) {
  const int l = lane_id();
  const bool small = a.nreq <= 64;
  const int nt_l = (small && l < a.nreq) ? pf_tiles(a.cu, l) : 0;
  for (int i = a.max_tiles - 1; i >= 0; --i) {
    for (int r0 = 0; r0 < a.nreq; r0 += 64) {
      const int nt = small ? nt_l : ((r0 + l < a.nreq) ? pf_tiles(a.cu, r0 + l) : 0);
      const unsigned long long hit = __ballot(nt > i);
      const int cnt = __popcll(hit);
      if (b < cnt * a.hslots) {
        const int kth = b / a.hslots;
        // position of the kth set bit
        const int before = __builtin_amdgcn_mbcnt_hi((uint32_t)(hit >> 32),
                                                     __builtin_amdgcn_mbcnt_lo((uint32_t)hit, 0u));
        const unsigned long long sel = __ballot(nt > i && before == kth);
        req = r0 + __ffsll((long long)sel) - 1;
        slot = b % a.hslots;
        tile = i;
        return true;
      }
      b -= cnt * a.hslots;
    }
  }
  return false;
}

// XCD-aware mapping (see PrefillArgs).  Slots are grouped in blocks of the
// slots that read one KV head (GQA) when the group size allows it.
__device__ __forceinline__ bool pf_find_item_xcd(const PrefillArgs& a, int b, int& tile,
                                                 int& req, int& slot) {
  if (!pf_xcd_valid(b, a.xcds, a.per_xcd, a.n_items)) return false;
  const int n = pf_xcd_item(b, a.xcds, a.per_xcd);
  const int g = a.hq / a.hkv;
  const int gs = (g % kPfHeadsPerWG == 0) ? g / kPfHeadsPerWG : 1;  // slots per block
  const int per_blk = gs * a.tiles_total;
  const int blk = n / per_blk;
  const int rem = n - blk * per_blk;
  const int l = lane_id();
  const unsigned long long hit = __ballot(l < a.nreq && rem < a.incl[l]);
  const int k = __builtin_amdgcn_readfirstlane(__ffsll((long long)hit) - 1);
  const int before = k > 0 ? a.incl[k - 1] : 0;
  const int local = rem - before;
  req = __builtin_amdgcn_readfirstlane(a.ord[k]);
  tile = (a.incl[k] - before) / gs - 1 - local / gs;
  slot = blk * gs + local % gs;
  return true;
}

__device__ __forceinline__ bool pf_find_item(const PrefillArgs& a, int b, int& tile, int& req,
                                             int& slot) {
  return a.xcd_order ? pf_find_item_xcd(a, b, tile, req, slot)
                     : pf_find_item_lpt(a, b, tile, req, slot);
}

// LDS of one prefill workgroup: K and V tiles, double-buffered, BN x D bf16
// each, and (dense kernel) a copy of Q operands KS/2 .. KS-1 of every lane,
// [ks - KS/2][thread][8] (16 KiB at d = 128: two workgroups still fit a CU).
// The diagonal steps read those from LDS, so the registers are free there and
// the compiler does not spill the Q operands to scratch (whose reloads would
// wait for the step's tile loads).
template <int D>
constexpr int pf_tile_elems() { return kPfBN * D; }
template <int D, bool PAGED>
constexpr int pf_q_lds_elems() { return PAGED ? 8 : (D / 32) * kPfThreads * 8; }

// One prefill work item (q tile, request, head; with key splits one split of
// it): workgroup `bid` of the prefill's own numbering.  The LDS buffers are
// separate __shared__ arrays of the calling kernel, one per (K/V, buffer):
// with compile-time buffer choices the compiler can tell that LDS reads of one
// buffer never alias the in-flight global->LDS loads into another, and does
// not wait for them.
// PAGED = false: fresh prompts, K/V token-major beside Q (dopd_prefill_attn).
// PAGED = true: chunks attending to the paged cache (dopd_prefill_paged_attn).
template <int D, bool PAGED, bool KV8 = false>
__device__ __forceinline__ void prefill_workgroup(const PrefillArgs& a, int bid, uint16_t* sK0,
                                                  uint16_t* sK1, uint16_t* sV0, uint16_t* sV1,
                                                  uint16_t* sQ) {
  constexpr int BM = kPfBM, BN = kPfBN;
  constexpr int KS = D / 16;     // k-steps of the QK MFMA
  constexpr int ET = D / 32;     // O^T tiles of 32 dims
  constexpr int CPR = D / 8;     // 16-byte chunks per K/V row
  constexpr int KQW = BN * CPR / kPfThreads;   // 16-byte chunks of a K (or V) tile per thread
  static_assert(!KV8 || PAGED, "E4M3 pools are read by the paged kernel only");
  constexpr int NCH8 = D / 16;                 // E4M3: 16-byte chunks per K row
  auto kbuf = [&](int b) { return b ? sK1 : sK0; };
  auto vbuf = [&](int b) { return b ? sV1 : sV0; };

  const int split = PAGED ? bid % a.nsplit : 0;
  int tile, r, h;
  if (!pf_find_item(a, PAGED ? bid / a.nsplit : bid, tile, r, h))
    return;  // uniform across the workgroup
  // The item is wave-uniform; say so, so that what derives from it stays scalar.
  tile = __builtin_amdgcn_readfirstlane(tile);
  r = __builtin_amdgcn_readfirstlane(r);
  h = __builtin_amdgcn_readfirstlane(h);
  {
    const int tid = threadIdx.x, l = lane_id();
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = a.hq / a.hkv, kvh = h / g;
    // With the XCD order the lengths come from the copies in the arguments
    // (scalar loads, read whatever the order: a select between the two
    // sources would become one generic load that waits on memory).
    int seq0 = a.cu_h[min(r, kPfMaxOrdered)];
    int L = a.cu_h[min(r + 1, kPfMaxOrdered)] - seq0;
    int P = PAGED ? a.prefix_h[min(r, kPfMaxOrdered - 1)] : 0;
    if (!a.xcd_order) {
      seq0 = __builtin_amdgcn_readfirstlane(a.cu[r]);
      L = __builtin_amdgcn_readfirstlane(a.cu[r + 1]) - seq0;
      // Cached tokens before the chunk: query row i sits at key position P + i.
      if constexpr (PAGED) P = __builtin_amdgcn_readfirstlane(a.prefix[r]);
    }
    const int q0 = tile * BM;
    const int kv_end = P + min(L, q0 + BM);   // keys of this item: [0, kv_end)
    const int ntiles = (kv_end + BN - 1) / BN;
    // Tiles every row of the item sees in full (positive scales only).
    const int nfull = a.scale_log2 > 0.f ? (P + q0) / BN : 0;
    // Key tiles of this workgroup: [jb, je) (all of them without splits).
    int jb = 0, je = ntiles;
    if constexpr (PAGED) {
      if (a.nsplit > 1) {
        jb = split == 0 ? 0 : min(split * ntiles / a.nsplit, nfull);
        je = split + 1 == a.nsplit ? ntiles : min((split + 1) * ntiles / a.nsplit, nfull);
      }
    }
    const int row_w = q0 + 32 * w;            // first query row of this wave
    const int myq = row_w + (l & 31);         // this lane's query row
    const bool wave_active = row_w < L;
    const int hi = l >> 5;                    // lane half

    // Q^T operand, B of the QK MFMA: lane holds Q[myq][16ks + 8hi + 0..7]
    // (E4M3 pools: Q[myq][32(ks/2) + 16hi + 8(ks%2) + 0..7], the dims one
    // 16-byte read of an E4M3 K row gives a lane over two k-steps; the
    // contraction over d is the same sum in another order).
    // Rows past the chunk read its row 0 (finite values; their results are
    // never stored), so nothing waits for these loads before the tile loads
    // below are issued.
    bf16x8 qop[KS];
    {
      const uint16_t* qp = a.q + ((int64_t)(seq0 + (myq < L ? myq : 0)) * a.hq + h) * D +
                           (KV8 ? 16 : 8) * hi;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        qop[ks] = __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const u32x4*>(qp + (KV8 ? 32 * (ks / 2) + 8 * (ks % 2) : 16 * ks)));
    }

    if constexpr (!PAGED) {  // (this lane's own slots: no barrier needed)
#pragma unroll
      for (int ks = KS / 2; ks < KS; ++ks)
        *reinterpret_cast<bf16x8*>(sQ + ((ks - KS / 2) * kPfThreads + tid) * 8) = qop[ks];
    }
    f32x16 oacc[ET];
#pragma unroll
    for (int et = 0; et < ET; ++et)
#pragma unroll
      for (int x = 0; x < 16; ++x) oacc[et][x] = 0.f;
    float m_run = -INFINITY, l_run = 0.f;

    const int64_t kv_row = (int64_t)a.hkv * D;  // elements between consecutive tokens
    const uint16_t* kg = a.k + (int64_t)seq0 * kv_row + (int64_t)kvh * D;
    const uint16_t* vg = a.v + (int64_t)seq0 * kv_row + (int64_t)kvh * D;

    // LDS tiles, 16-byte chunks.  K: [D/32 chunk groups][BN rows][4 slots],
    // chunk c of row t in group c/4, slot (c%4) ^ ((t/4)%4), so that the 16
    // rows read by 16 lanes at one chunk hit 16 distinct bank groups.  V:
    // [D/32 dim groups][BN tokens][32 dims], token-major.  Wave instruction
    // u of wave w fills LDS chunks [64(4u + w), +64): row 16w + l/4, chunk
    // group u, slot l%4.
    const int k_t = 16 * w + (l >> 2);                            // this lane's row of a tile
    const int k_c = (l & 3) ^ ((k_t >> 2) & 3);                   // K: swizzled slot
    const int v_c = l & 3;                                        // V: plain chunk
    const int row_b = (int)(kv_row * 2);                          // bytes between tokens
    const int lane_k = k_t * row_b + 16 * k_c;
    const int lane_v = k_t * row_b + 16 * v_c;
    // A tile load goes through a buffer descriptor whose base is the tile's
    // first token and whose size covers its valid rows; full tiles use loop
    // invariant lane offsets, ragged tiles clamp to the last valid row.
    auto stage = [&](const uint16_t* g0, uint16_t* lds, int kv0, int lane_full, int chunk) {
      const int rows = min(BN, kv_end - kv0);                   // uniform, >= 1
      const int voff = rows == BN ? lane_full : min(k_t, rows - 1) * row_b + 16 * chunk;
      const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
          (void*)(g0 + (int64_t)kv0 * kv_row), (short)0, (rows - 1) * row_b + 2 * D, 0x00020000);
#pragma unroll
      for (int u = 0; u < KQW; ++u)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            rsrc, (__attribute__((address_space(3))) void*)(lds + (4 * u + w) * 512), 16, voff,
            64 * u, 0, 0);
    };
    // Paged: wave w loads page kv0/16 + w of the tile (clamped to the last
    // page that holds keys), K rows in the order pi (bits 2 and 3 of the slot
    // swapped) so that each lane's P values are 8 consecutive keys per P.V
    // k-step; V^T page blocks keep their dim-major rows: LDS V tile
    // [D/32 dim groups][8 key chunks][32 dims][8 keys], wave w filling chunks
    // 2w, 2w+1 (its page).  Slots past the end of the cache hold anything;
    // they are masked (scores by select, V operand bits by AND).
    const int32_t* pt_row = PAGED ? a.page_table + (int64_t)r * a.pt_stride : nullptr;
    const int last_page = (kv_end - 1) / kPage;
    const int pk_slot = ((l >> 2) & 3) | ((l >> 3) & 4) | ((l >> 1) & 8);  // pi(16w + l/4) % 16
    const int lane_pk = pk_slot * (2 * D) + 16 * k_c;
    const int lane_pv = (l & 31) * (2 * kPage) + 16 * (l >> 5);
    // Page id of this wave's page of tile jt (a vector load; made uniform by
    // the caller once it has landed).
    auto page_of = [&](int jt) { return pt_row[min(jt * (BN / kPage) + w, last_page)]; };
    // Page ids of the next K and V tile loads, and the id loaded a step ahead.
    int pid_k = 0, pid_v = 0, pid_ahead = 0;
    auto stage_page = [&](const uint16_t* pool, uint16_t* lds, int page, int lane_off, int u_stride) {
      const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
          (void*)(pool + ((int64_t)page * a.hkv + kvh) * (kPage * D)), (short)0, 2 * kPage * D,
          0x00020000);
#pragma unroll
      for (int u = 0; u < KQW; ++u)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            rsrc, (__attribute__((address_space(3))) void*)(lds + (4 * u + w) * 512), 16, lane_off,
            u_stride * u, 0, 0);
    };
    // E4M3 pools: wave w copies its page block (16 x D bytes) into bytes
    // [16 D w, 16 D (w + 1)) of the tile buffer, instruction u filling its
    // 16-byte chunks [64u, 64u + 64).  K: chunk q is row s = q / NCH8 (page
    // slot pi(s)), physical chunk q % NCH8 holding logical chunk
    // (q % NCH8) ^ (s % NCH8), so that 16 rows read at one logical chunk hit
    // distinct bank groups.  V: chunk q is dim row q (its 16 keys).
    const int lane_k8 = [&] {
      const int s8 = l / NCH8, pc = l % NCH8;  // chunk q = 64u + l: row s8 + (64 / NCH8) u
      return ((s8 & 3) | ((s8 & 4) << 1) | ((s8 & 8) >> 1)) * D + 16 * (pc ^ (s8 % NCH8));
    }();
    auto stage_page8 = [&](const uint16_t* pool, uint16_t* lds, int page, int lane_off, int u_stride) {
      const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
          (void*)(reinterpret_cast<const uint8_t*>(pool) + ((int64_t)page * a.hkv + kvh) * (kPage * D)),
          (short)0, kPage * D, 0x00020000);
#pragma unroll
      for (int u = 0; u < D / 64; ++u)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            rsrc, (__attribute__((address_space(3))) void*)(lds + (w * kPage * D + 1024 * u) / 2), 16,
            lane_off, u_stride * u, 0, 0);
    };
    // (Paged: the page comes from pid_k / pid_v, not from kv0.)
    auto load_k = [&](int buf, int kv0) {
      if constexpr (KV8) stage_page8(a.k_pool, kbuf(buf), pid_k, lane_k8, 4 * D);  // rows s, s + 8: slots pi(s), pi(s) + 4
      else if constexpr (PAGED) stage_page(a.k_pool, kbuf(buf), pid_k, lane_pk, 64);
      else stage(kg, kbuf(buf), kv0, lane_k, k_c);
    };
    auto load_v = [&](int buf, int kv0) {
      if constexpr (KV8) stage_page8(a.v_pool, vbuf(buf), pid_v, 16 * l, 1024);
      else if constexpr (PAGED) stage_page(a.v_pool, vbuf(buf), pid_v, lane_pv, 32 * 2 * kPage);
      else stage(vg, vbuf(buf), kv0, lane_v, v_c);
    };

    // A operand of the QK MFMA: K[32 tt + l%32][16 ks + 8 hi + 0..7] = chunk
    // 2ks + hi of row 32tt + l%32: group ks/2, slot (2(ks%2) + hi) ^ ((l/4)%4).
    const int kr_m = hi ^ ((l >> 2) & 3);
    const int kr_even = (l & 31) * 32 + 8 * kr_m, kr_odd = (l & 31) * 32 + 8 * (kr_m ^ 2);
    auto kread = [&](int buf, int tt, int ks) {
      const int off = (ks >> 1) * (BN * 32) + tt * 1024 + ((ks & 1) ? kr_odd : kr_even);
      return *reinterpret_cast<const bf16x8*>(kbuf(buf) + off);
    };
    // E4M3: row 32tt + l%32 of the tile (wave page (32tt + l%32)/16), logical
    // chunk 2p + hi -> the k-steps 2p and 2p + 1 of this lane.
    const int kr8 = (l & 31) * D;
    auto kread8 = [&](int buf, int tt, int p, bf16x8& k0, bf16x8& k1) {
      const int row = 32 * tt + (l & 31);
      const u32x4 c = *reinterpret_cast<const u32x4*>(
          reinterpret_cast<const uint8_t*>(kbuf(buf)) + tt * 32 * D + kr8 +
          16 * ((2 * p + hi) ^ (row % NCH8)));
      const u32x2 a0 = bf16x4_from_e4m3x4(c[0]), a1 = bf16x4_from_e4m3x4(c[1]);
      const u32x2 a2 = bf16x4_from_e4m3x4(c[2]), a3 = bf16x4_from_e4m3x4(c[3]);
      k0 = __builtin_bit_cast(bf16x8, u32x4{a0[0], a0[1], a1[0], a1[1]});
      k1 = __builtin_bit_cast(bf16x8, u32x4{a2[0], a2[1], a3[0], a3[1]});
    };
    // K operands of a tile: ka[tt][ks].
    auto kread_all = [&](int buf, bf16x8 (&ka)[2][KS]) {
      if constexpr (KV8) {
#pragma unroll
        for (int tt = 0; tt < 2; ++tt)
#pragma unroll
          for (int p = 0; p < KS / 2; ++p) kread8(buf, tt, p, ka[tt][2 * p], ka[tt][2 * p + 1]);
      } else {
#pragma unroll
        for (int tt = 0; tt < 2; ++tt)
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) ka[tt][ks] = kread(buf, tt, ks);
      }
    };
    // A operand of P.V k-step kk = 2tt + hh: V^T[32 et + l%32][keys 32tt + 16hh
    // + 8m + 4hi + 0..3, m = 0, 1], i.e. k-slot 8hi + jj <-> key
    // 32tt + 16hh + 8(jj/4) + 4hi + jj%4, the order of the S^T accumulator.
    // Two transposing LDS reads (4 keys each) gather it from the token-major
    // tile: within each 16-lane group, lane i receives element i%4 of the
    // 8-byte rows read by lanes 4j + i/4, j = 0..3; so source lane s reads key
    // base + s/4, dims 32et + 16((l/16)%2) + 4(s%4) .. + 3, and lane i ends up
    // with dim 32et + 16((l/16)%2) + i of keys base .. base + 3.
    const int vr_base = 128 * hi + 32 * ((l & 15) >> 2) + 16 * ((l >> 4) & 1) + 4 * (l & 3);
    auto vread = [&](int buf, int kk, int et) {
      bf16x8 res;
      if constexpr (KV8) {  // keys 16kk + 8hi + 0..7 of dim 32et + l%32: 8 bytes of its row
        const u32x2 c = *reinterpret_cast<const u32x2*>(
            reinterpret_cast<const uint8_t*>(vbuf(buf)) + kk * (kPage * D) + (32 * et + (l & 31)) * 16 +
            8 * hi);
        const u32x2 a0 = bf16x4_from_e4m3x4(c[0]), a1 = bf16x4_from_e4m3x4(c[1]);
        res = __builtin_bit_cast(bf16x8, u32x4{a0[0], a0[1], a1[0], a1[1]});
      } else if constexpr (PAGED) {  // keys 16kk + 8hi + 0..7 of dim 32et + l%32: one 16-byte chunk
        res = *reinterpret_cast<const bf16x8*>(vbuf(buf) + ((et * 8 + 2 * kk + hi) * 32 + (l & 31)) * 8);
      } else {
        typedef short s16x4_t __attribute__((ext_vector_type(4)));
        typedef __attribute__((address_space(3))) s16x4_t* lds_s16x4;
        const uint16_t* p = vbuf(buf) + et * (BN * 32) + (16 * kk) * 32 + vr_base;
        const s16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4)(p));
        const s16x4_t hi4 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4)(p + 8 * 32));
        const s16x4_t both[2] = {lo, hi4};
        __builtin_memcpy(&res, both, 16);
      }
      return res;
    };

    // Scores stay raw until the exponent: p = 2^(s*c - m) as one fma, with the
    // running max m kept in the scaled domain.  For c <= 0 the scores are
    // scaled first and c is taken as 1, so the max is always taken on the
    // exponent.
    const float c_in = PAGED && a.k_scale ? a.scale_log2 * a.k_scale[kvh] : a.scale_log2;
    const float v_sc = PAGED && a.v_scale ? a.v_scale[kvh] : 1.f;
    const bool pos_scale = c_in > 0.f;
    const float c_eff = pos_scale ? c_in : 1.f;
    // Lazy rescaling on masked tiles: the running max only moves when a tile
    // raises it by more than kLazy (log2 units).
    constexpr float kLazy = 8.f;
    // Steady-state trigger: a half-row sum beyond 2^kSumLazy (so every p
    // stays far below overflow while it does not fire).
    constexpr float kSumLazy = 20.f;
    // Last key this lane's row may see (causal and end of request).
    const int last_key = min(P + myq, kv_end - 1);

    f32x16 sa[2], sb[2];  // S^T of two consecutive key tiles (current / next)
    bf16x8 pb[4];         // P^T of the current tile: B operands of the four P.V k-steps
    constexpr int kMfma = 0x008, kDsRead = 0x100;  // sched_group_barrier masks

    auto zero2 = [&](f32x16* s) {
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int x = 0; x < 16; ++x) s[tt][x] = 0.f;
    };
    // Max of this lane pair's query row over the tile, in the exp2 domain
    // (maximum, not fmaxf: no NaN quieting of the MFMA results, 3-input ops).
    auto row_max = [&](const f32x16* s) {
      float mx = __builtin_elementwise_maximum(s[0][0], s[1][0]);
#pragma unroll
      for (int x = 1; x < 16; ++x)
        mx = __builtin_elementwise_maximum(mx, __builtin_elementwise_maximum(s[0][x], s[1][x]));
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx),
                                                       false, false);
      return __builtin_elementwise_maximum(__uint_as_float(sw[0]), __uint_as_float(sw[1])) * c_eff;
    };
    auto rescale_to = [&](float m_tile) {
      const float m_new = fmaxf(m_run, m_tile);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int et = 0; et < ET; ++et) oacc[et] *= alpha;
    };
    // pb = 2^(s c - m) rounded to bf16; returns this lane's half-row sum of
    // the rounded values (the weights the P.V product uses), two at a time.
    auto exponent = [&](const f32x16* s) {
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int x = 0; x < 16; ++x)
          pb[2 * tt + (x >> 3)][x & 7] =
              (__bf16)__builtin_amdgcn_exp2f(__builtin_fmaf(s[tt][x], c_eff, -m_run));
      typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
      const bf16x2_t ones = {(__bf16)1.f, (__bf16)1.f};
      float ps0 = 0.f, ps1 = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        ps0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pb[i], pb[i], 0, 1), ones, ps0, false);
        ps1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pb[i], pb[i], 2, 3), ones, ps1, false);
        ps0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pb[i], pb[i], 4, 5), ones, ps0, false);
        ps1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pb[i], pb[i], 6, 7), ones, ps1, false);
      }
      return ps0 + ps1;
    };
    auto qk = [&](int buf, f32x16* s) {
      bf16x8 ka[2][KS];
      kread_all(buf, ka);
      zero2(s);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
#pragma unroll
        for (int tt = 0; tt < 2; ++tt)
          s[tt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[tt][ks], qop[ks], s[tt], 0, 0, 0);
    };
    // S^T for the diagonal steps of the dense kernel: Q operands KS/2 .. from
    // this lane's copy in LDS.
    auto qk_lq = [&](int buf, f32x16* s) {
      bf16x8 ka[2][KS];
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) ka[tt][ks] = kread(buf, tt, ks);
      zero2(s);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x8 qv =
            ks < KS / 2 ? qop[ks]
                        : *reinterpret_cast<const bf16x8*>(sQ + ((ks - KS / 2) * kPfThreads + tid) * 8);
#pragma unroll
        for (int tt = 0; tt < 2; ++tt)
          s[tt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[tt][ks], qv, s[tt], 0, 0, 0);
      }
    };
    // O^T += V^T P^T of the tile.
    auto pv = [&](int buf) {
      bf16x8 va[4][ET];
#pragma unroll
      for (int kk = 0; kk < 4; ++kk)
#pragma unroll
        for (int et = 0; et < ET; ++et) va[kk][et] = vread(buf, kk, et);
#pragma unroll
      for (int kk = 0; kk < 4; ++kk)
#pragma unroll
        for (int et = 0; et < ET; ++et)
          oacc[et] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[kk][et], pb[kk], oacc[et], 0, 0, 0);
      // Interleaving hints for the dense kernel's P.V only (its V operands
      // come from two transposing reads each).  Measured: hints on the QK
      // products cost the dense kernel 2-3 %, and any hints cost the paged
      // kernel 8 % (404 against 148 bytes of spill per lane).
      if constexpr (!PAGED) {
        __builtin_amdgcn_sched_group_barrier(kDsRead, 2 * ET, 0);
#pragma unroll
        for (int kk = 0; kk < 3; ++kk)
#pragma unroll
          for (int et = 0; et < ET; ++et) {
            __builtin_amdgcn_sched_group_barrier(kMfma, 1, 0);
            __builtin_amdgcn_sched_group_barrier(kDsRead, 2, 0);
          }
        __builtin_amdgcn_sched_group_barrier(kMfma, ET, 0);
      }
    };
    auto softmax_masked = [&](f32x16* s, int kv0) {
      if (!pos_scale) {
#pragma unroll
        for (int tt = 0; tt < 2; ++tt) s[tt] *= c_in;
      }
      // Element (tt, x) of this lane is key kv0 + off + (4 or 8) hi: the
      // accumulator row 32tt + 8(x/4) + 4hi + x%4, through pi on the paged path.
      const int lim = last_key - kv0 - (PAGED ? 8 : 4) * hi;
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int x = 0; x < 16; ++x) {
          const int off = PAGED ? 32 * tt + 16 * (x >> 3) + 4 * ((x >> 2) & 1) + (x & 3)
                                : 32 * tt + 8 * (x >> 2) + (x & 3);
          if (off > lim) s[tt][x] = -INFINITY;
        }
      const float m_tile = row_max(s);  // finite: every row sees key 0 in the first tile
      if (__ballot(m_tile > m_run + kLazy)) rescale_to(m_tile);  // wave-uniform
      l_run += exponent(s);
    };
    // Steady-state step, first part: the softmax of tile j on the VALU while
    // the MFMAs compute S^T of tile j + 1 (K buffer kb).
    auto half_qk = [&](f32x16* sc, f32x16* sn, int kb) {
      bf16x8 ka[2][KS];
      kread_all(kb, ka);
      zero2(sn);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
#pragma unroll
        for (int tt = 0; tt < 2; ++tt)
          sn[tt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[tt][ks], qop[ks], sn[tt], 0, 0, 0);
      float psum = exponent(sc);
      if (__ballot(!(psum <= __builtin_exp2f(kSumLazy)))) {  // wave-uniform, rare
        rescale_to(row_max(sc));
        psum = exponent(sc);
      }
      l_run += psum;
    };

    // Paged: the keys of the last tile past the end of the cache come from
    // slots that may hold anything, NaN included (pages past the last one are
    // read as copies of it).  Their P is 0, but 0 * NaN is not, so once the
    // tile's V pages have landed each wave clears those keys in its own page
    // of the V tile; the barrier that closes the step publishes the zeros.
    auto clear_dead_v = [&](int buf, int jt) {
      if constexpr (KV8) {  // this wave's page: [D dim rows][16 key bytes]
        const int nlive = kv_end - jt * BN;
        if (nlive >= 16 * w + 16) return;
        __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this wave's V page has landed
        const int nv = nlive - 16 * w;       // live keys of the page (may be <= 0)
        uint32_t keep[4];
#pragma unroll
        for (int wd = 0; wd < 4; ++wd) {
          const int nb = nv - 4 * wd;  // live bytes of word wd
          keep[wd] = nb >= 4 ? 0xffffffffu : (nb <= 0 ? 0u : (1u << (8 * nb)) - 1u);
        }
#pragma unroll
        for (int i = 0; i < D / 64; ++i) {
          u32x4* p = reinterpret_cast<u32x4*>(reinterpret_cast<uint8_t*>(vbuf(buf)) + w * (kPage * D) +
                                              (l + 64 * i) * 16);
          u32x4 x = *p;
#pragma unroll
          for (int wd = 0; wd < 4; ++wd) x[wd] &= keep[wd];
          *p = x;
        }
      } else if constexpr (PAGED) {
        const int nlive = kv_end - jt * BN;  // live keys of tile jt (uniform, >= 1)
        if (nlive >= 16 * w + 16) return;    // this wave's page is all live
        __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this wave's V page has landed
        const int kc = 2 * w + hi;           // key chunk of this lane: keys 8kc .. 8kc + 7
        const int nv = nlive - 8 * kc;       // live keys among them
        uint32_t keep[4];
#pragma unroll
        for (int wd = 0; wd < 4; ++wd)
          keep[wd] = (2 * wd + 1 < nv) ? 0xffffffffu : (2 * wd < nv ? 0x0000ffffu : 0u);
#pragma unroll
        for (int et = 0; et < ET; ++et) {
          u32x4* p = reinterpret_cast<u32x4*>(vbuf(buf) + ((et * 8 + kc) * 32 + (l & 31)) * 8);
          u32x4 x = *p;
#pragma unroll
          for (int wd = 0; wd < 4; ++wd) x[wd] &= keep[wd];
          *p = x;
        }
      }
    };

    // K tile s sits in K buffer s % 2 and V tile s in V buffer s % 2; K runs
    // one tile ahead of V.  A step j: loads K(j + 2) and V(j + 1) into the
    // free buffers, computes S^T(j + 1) with the softmax of tile j, then
    // O^T += V^T P^T of tile j; one barrier (which also waits for the loads).
    if constexpr (PAGED) {
      if (jb < je) {  // (an empty split loads and computes nothing)
        const int p0 = __builtin_amdgcn_readfirstlane(page_of(jb));
        const int p1 = __builtin_amdgcn_readfirstlane(page_of(jb + 1));
        pid_k = p0;
        load_k(0, 0);
        pid_k = p1;
        if (je > jb + 1) load_k(1, BN);
        pid_v = p0;
        load_v(0, 0);
        clear_dead_v(0, jb);
        // the first step loads K(jb + 2) and V(jb + 1); the id of tile jb + 3 is read ahead
        pid_v = p1;
        pid_k = __builtin_amdgcn_readfirstlane(page_of(jb + 2));
        pid_ahead = page_of(jb + 3);
      }
    } else {
      load_k(0, 0);
      if (ntiles > 1) load_k(1, BN);
      load_v(0, 0);
    }
    __syncthreads();
    if (wave_active && jb < je) qk(0, sa);  // every active row sees key jb * BN
    // The steady-state steps form p against the running max without taking
    // the tile's max, so start it at the first tile's max (unmasked there).
    if (wave_active && jb < nfull && jb < je) m_run = row_max(sa);
    // The first step's prefetch writes K tile 2 into K buffer 0: every wave
    // must have read tile 0 from it first.
    __syncthreads();

    int j = jb;
    const int nfe = min(nfull, je);  // end of the full tiles of this workgroup
    auto prefetch = [&](int jj, auto par) {  // K(jj + 2) -> K buffer par, V(jj + 1) -> V buffer par ^ 1
      if (jj + 2 < je) load_k(par(), (jj + 2) * BN);
      if (jj + 1 < je) load_v(par() ^ 1, (jj + 1) * BN);
      if constexpr (PAGED) {  // next step: K(jj + 3), V(jj + 2); read the id of tile jj + 4
        pid_v = pid_k;
        pid_k = __builtin_amdgcn_readfirstlane(pid_ahead);  // landed at the last barrier
        pid_ahead = page_of(jj + 4);
      }
    };
    auto even = [] { return 0; };
    auto odd = [] { return 1; };
    // The dense kernel raises the wave's priority over its softmax and the
    // next tile's QK products, so its VALU work issues first and the other
    // workgroup's P.V MFMAs fill the slots it leaves (measured 1-2 % faster;
    // the paged kernel measured slower with it).
    auto step_full = [&](f32x16* sc, f32x16* sn, auto par) {
      prefetch(j, par);
      if (wave_active) {
        if constexpr (!PAGED) __builtin_amdgcn_s_setprio(1);
        half_qk(sc, sn, par() ^ 1);
        if constexpr (!PAGED) __builtin_amdgcn_s_setprio(0);
        pv(par());
      }
      if (j + 1 < je) clear_dead_v(par() ^ 1, j + 1);
      __syncthreads();
    };
    for (; j + 1 < nfe; j += 2) {
      step_full(sa, sb, even);
      ++j;
      step_full(sb, sa, odd);
      --j;
    }
    if (j < nfe) {
      step_full(sa, sb, even);
      ++j;
#pragma unroll
      for (int tt = 0; tt < 2; ++tt) sa[tt] = sb[tt];
    }
    // Diagonal and ragged tiles: masked softmax, then S^T of the next tile.
    auto step_tail = [&](auto par) {
      prefetch(j, par);
      if (wave_active && j * BN <= P + row_w + 31) {  // some key of tile j visible to this wave
        softmax_masked(sa, j * BN);
        pv(par());
      }
      if (wave_active && j + 1 < je && (j + 1) * BN <= P + row_w + 31) {
        if constexpr (PAGED) qk(par() ^ 1, sa);
        else qk_lq(par() ^ 1, sa);
      }
      if (j + 1 < je) clear_dead_v(par() ^ 1, j + 1);
      __syncthreads();
    };
    for (; j < je; ++j) {  // tile j sits in buffer (j - jb) % 2
      if ((j - jb) & 1) step_tail(odd);
      else step_tail(even);
    }
    if (!wave_active) return;
    float l_tot = l_run + __shfl_xor(l_run, 32, 64);
    if constexpr (PAGED) {
      if (a.nsplit > 1) {  // partial (o, m, l) of this split; the merge kernel finishes
        if (myq < L) {
          const int64_t row = ((int64_t)split * a.part_rows + seq0 + myq) * a.hq + h;
          float* po = a.part_o + row * D + 4 * hi;
#pragma unroll
          for (int et = 0; et < ET; ++et)
#pragma unroll
            for (int gq = 0; gq < 4; ++gq)
              *reinterpret_cast<f32x4*>(po + 32 * et + 8 * gq) =
                  f32x4{oacc[et][4 * gq], oacc[et][4 * gq + 1], oacc[et][4 * gq + 2],
                        oacc[et][4 * gq + 3]} * v_sc;
          if (hi == 0) *reinterpret_cast<float2*>(a.part_ml + row * 2) = float2{m_run, l_tot};
        }
        return;
      }
    }
    const float inv = v_sc / l_tot;
    // The wave's 32 x D output block goes through LDS (no load is in flight
    // and every wave is past its last tile read: the loop's last barrier), so
    // that 16 lanes store one 256-byte row instead of 32 rows taking 8-byte
    // pieces.  Wave w uses one of the four tile buffers; rows padded by 16
    // bytes.  Lane holds O^T[e = 32et + 8(x/4) + 4hi + x%4][myq].
    constexpr int RS = D + 8;
    uint16_t* so = w == 0 ? sK0 : w == 1 ? sK1 : w == 2 ? sV0 : sV1;
#pragma unroll
    for (int et = 0; et < ET; ++et)
#pragma unroll
      for (int gq = 0; gq < 4; ++gq) {
        u32x2 x;
        x[0] = pack_bf16x2(oacc[et][4 * gq] * inv, oacc[et][4 * gq + 1] * inv);
        x[1] = pack_bf16x2(oacc[et][4 * gq + 2] * inv, oacc[et][4 * gq + 3] * inv);
        *reinterpret_cast<u32x2*>(so + (l & 31) * RS + 32 * et + 8 * gq + 4 * hi) = x;
      }
    // The LDS writes and reads below are this wave's alone (in order within
    // the wave).
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    constexpr int CH = D / 8;  // 16-byte chunks per row
#pragma unroll
    for (int u = 0; u < 32 * CH / 64; ++u) {
      const int i = l + 64 * u;
      const int rr = i / CH, c = i % CH;
      const u32x4 x = *reinterpret_cast<const u32x4*>(so + rr * RS + 8 * c);
      // (streaming store: the output is not read again by this step, and it
      // is written out now rather than evicted during the next kernel)
      if (row_w + rr < L)
        __builtin_nontemporal_store(
            x, reinterpret_cast<u32x4*>(a.out + ((int64_t)(seq0 + row_w + rr) * a.hq + h) * D + 8 * c));
    }
    if (a.lse && hi == 0 && myq < L)
      a.lse[(int64_t)(seq0 + myq) * a.hq + h] = (m_run + __log2f(l_tot)) * kLn2;
  }
}

template <int D, bool PAGED, bool KV8 = false>
__global__ __launch_bounds__(kPfThreads, 2) void prefill_bf16_kernel(PrefillArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t sK0[pf_tile_elems<D>()], sK1[pf_tile_elems<D>()];
  __shared__ __attribute__((aligned(16))) uint16_t sV0[pf_tile_elems<D>()], sV1[pf_tile_elems<D>()];
  __shared__ __attribute__((aligned(16))) uint16_t sQ[pf_q_lds_elems<D, PAGED>()];
  prefill_workgroup<D, PAGED, KV8>(a, (int)blockIdx.x, sK0, sK1, sV0, sV1, sQ);
}

// Combines the key splits of the paged prefill.  Thread = one 4-dim chunk of
// one (row, head): M = max_s m_s, L = sum_s 2^(m_s - M) l_s,
// o = sum_s 2^(m_s - M) o~_s / L, lse = (M + log2 L) ln 2, splits in order.
template <int D>
__global__ __launch_bounds__(256) void prefill_split_merge_kernel(PrefillArgs a) {
  const int64_t rowheads = (int64_t)a.part_rows * a.hq;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t rh = idx / (D / 4);
  const int e0 = 4 * (int)(idx % (D / 4));
  if (rh >= rowheads) return;
  float M = -INFINITY;
  for (int s = 0; s < a.nsplit; ++s) M = fmaxf(M, a.part_ml[(s * rowheads + rh) * 2]);
  float L = 0.f;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int s = 0; s < a.nsplit; ++s) {
    const float2 ml = *reinterpret_cast<const float2*>(a.part_ml + (s * rowheads + rh) * 2);
    const float wgt = __builtin_amdgcn_exp2f(ml.x - M);  // an empty split has m = -inf -> 0
    L += wgt * ml.y;
    acc += *reinterpret_cast<const f32x4*>(a.part_o + (s * rowheads + rh) * D + e0) * wgt;
  }
  const float inv = 1.f / L;
  u32x2 x;
  x[0] = pack_bf16x2(acc[0] * inv, acc[1] * inv);
  x[1] = pack_bf16x2(acc[2] * inv, acc[3] * inv);
  *reinterpret_cast<u32x2*>(a.out + rh * D + e0) = x;
  if (a.lse && e0 == 0) a.lse[rh] = (M + __log2f(L)) * kLn2;
}

}  // namespace dopd
