// Variable-length causal prefill attention, bf16 in / fp32 accumulate, gfx950.
//
// Workgroup = 4 waves = one (q tile of 128 rows, request, query head); each
// wave owns 32 query rows; two workgroups share a CU, so the two waves on a
// SIMD run out of phase.  K/V stages of 64 keys are staged in LDS (K
// token-major, V transposed to dim-major on the way in), double-buffered, and
// shared by the four waves.  Per stage and wave:
//
//   S^T[64 tok][32 q] = K[64][d] . Q^T[d][32]       2 x (d/16) v_mfma_f32_32x32x16_bf16
//   O^T[d][32 q]     += V^T[d][64] . P^T[64][32]    (d/32) x 4  v_mfma_f32_32x32x16_bf16
//
// Computing the transposed products keeps a whole query row inside one lane
// pair, so the online-softmax row max needs one lane swap, and the MFMA output
// of S^T is already the B operand of the P.V MFMA (the token order of the
// contraction is matched on the V^T LDS reads).  LDS operands are read ahead
// of their MFMAs (pinned scheduling groups); rows are padded so that reads and
// writes are free of bank conflicts.  Scores are scaled into the exp2 domain
// inside one fma; only stages on the diagonal or past the end of the request
// are masked, with a select (never a multiply).
// Work order: with at most 64 requests, each XCD takes a contiguous slice of
// (KV head, request longest first, q tile descending) so the q tiles that read
// the same K/V run together under one L2; otherwise heaviest q tiles first.
#pragma once
#include "common.hpp"

namespace dopd {

struct PrefillArgs {
  const uint16_t* q;   // [T][Hq][D]
  const uint16_t* k;   // [T][Hkv][D]
  const uint16_t* v;   // [T][Hkv][D]
  uint16_t* out;       // [T][Hq][D]
  float* lse;          // [T][Hq] or null
  const int32_t* cu;   // [nreq + 1]
  int nreq, hq, hkv, max_tiles;
  float scale_log2;
  // XCD-aware order (used when nreq <= kPfMaxOrdered): the work list is
  // (KV head, request by decreasing length, q tile descending, query head of
  // the group); XCD x = workgroup % 8 takes the contiguous slice
  // [x * per_xcd, (x+1) * per_xcd), so the q tiles that share a request's K/V
  // run together on one XCD and share its L2.
  int xcd_order, n_items, per_xcd, tiles_total;
  uint8_t ord[64];     // requests by decreasing length
};

constexpr int kPfMaxOrdered = 64;
constexpr int kNumXcd = 8;

constexpr int kPfBM = 128;  // query rows per workgroup (32 per wave)
constexpr int kPfThreads = kPfBM / 32 * 64;
constexpr int kPfBN = 64;   // keys per LDS stage (computed as 64-key sub-tiles)

// Number of BM-row q tiles of request rr.
__device__ __forceinline__ int pf_tiles(const int32_t* cu, int rr) {
  return (cu[rr + 1] - cu[rr] + kPfBM - 1) / kPfBM;
}

// Maps a workgroup index to (q tile, request, head), q tiles in decreasing
// index order (tile i of a request attends to ~ (i+1) key tiles).
__device__ __forceinline__ bool pf_find_item_lpt(const PrefillArgs& a, int b, int& tile,
                                                 int& req, int& head) {
  const int l = lane_id();
  const bool small = a.nreq <= 64;
  const int nt_l = (small && l < a.nreq) ? pf_tiles(a.cu, l) : 0;
  for (int i = a.max_tiles - 1; i >= 0; --i) {
    for (int r0 = 0; r0 < a.nreq; r0 += 64) {
      const int nt = small ? nt_l : ((r0 + l < a.nreq) ? pf_tiles(a.cu, r0 + l) : 0);
      const unsigned long long hit = __ballot(nt > i);
      const int cnt = __popcll(hit);
      if (b < cnt * a.hq) {
        const int kth = b / a.hq;
        // position of the kth set bit
        const int before = __builtin_amdgcn_mbcnt_hi((uint32_t)(hit >> 32),
                                                     __builtin_amdgcn_mbcnt_lo((uint32_t)hit, 0u));
        const unsigned long long sel = __ballot(nt > i && before == kth);
        req = r0 + __ffsll((long long)sel) - 1;
        head = b % a.hq;
        tile = i;
        return true;
      }
      b -= cnt * a.hq;
    }
  }
  return false;
}

// XCD-aware mapping (see PrefillArgs).
__device__ __forceinline__ bool pf_find_item_xcd(const PrefillArgs& a, int b, int& tile,
                                                 int& req, int& head) {
  const int x = b % kNumXcd, j = b / kNumXcd;
  const int n = x * a.per_xcd + j;
  if (j >= a.per_xcd || n >= a.n_items) return false;
  const int g = a.hq / a.hkv;
  const int per_kvh = g * a.tiles_total;
  const int kvh = n / per_kvh;
  const int rem = n - kvh * per_kvh;
  const int l = lane_id();
  const int rr = l < a.nreq ? a.ord[l] : 0;
  const int nt = l < a.nreq ? pf_tiles(a.cu, rr) : 0;
  const int cnt = g * nt;
  const int incl = wave_inclusive_scan(cnt);
  const unsigned long long hit = __ballot(rem < incl);
  const int k = __ffsll((long long)hit) - 1;
  const int local = rem - __shfl(incl - cnt, k, 64);
  req = __shfl(rr, k, 64);
  tile = __shfl(nt, k, 64) - 1 - local / g;
  head = kvh * g + local % g;
  return true;
}

__device__ __forceinline__ bool pf_find_item(const PrefillArgs& a, int b, int& tile, int& req,
                                             int& head) {
  return a.xcd_order ? pf_find_item_xcd(a, b, tile, req, head)
                     : pf_find_item_lpt(a, b, tile, req, head);
}

template <int D>
__global__ __launch_bounds__(kPfThreads, 2) void prefill_bf16_kernel(PrefillArgs a) {
  constexpr int BM = kPfBM, BN = kPfBN, SUB = 64;
  constexpr int KP = D + 8;      // padded K row (elements)
  constexpr int VP = BN + 4;     // padded V^T row (elements): 2 dwords of skew per row
  constexpr int KS = D / 16;     // k-steps of the QK MFMA
  constexpr int ET = D / 32;     // O^T tiles of 32 dims
  constexpr int CPR = D / 8;     // 16-byte chunks per K/V row
  constexpr int NTH = kPfThreads;
  constexpr int KCH = BN * CPR / NTH;   // K chunks staged per thread
  constexpr int VTH = (BN / 4) * CPR;   // threads staging V (4 tokens x 8 dims each)
  __shared__ __attribute__((aligned(16))) uint16_t sK[2][BN * KP];
  __shared__ __attribute__((aligned(16))) uint16_t sV[2][D * VP];

  const int tid = threadIdx.x, l = lane_id(), w = tid >> 6;
  int tile, r, h;
  if (!pf_find_item(a, blockIdx.x, tile, r, h)) return;  // uniform across the workgroup
  const int g = a.hq / a.hkv, kvh = h / g;
  const int seq0 = a.cu[r], L = a.cu[r + 1] - seq0;
  const int q0 = tile * BM;
  const int kv_end = min(L, q0 + BM);
  const int ntiles = (kv_end + BN - 1) / BN;
  const int row_w = q0 + 32 * w;            // first query row of this wave
  const int myq = row_w + (l & 31);         // this lane's query row
  const bool wave_active = row_w < L;
  const int hi = l >> 5;                    // lane half

  // Q^T operand, B of the QK MFMA: lane holds Q[myq][16ks + 8hi + 0..7].
  bf16x8 qop[KS];
  {
    const bool ok = myq < L;
    const uint16_t* qp = a.q + ((int64_t)(seq0 + (ok ? myq : 0)) * a.hq + h) * D + 8 * hi;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      u32x4 x = ok ? *reinterpret_cast<const u32x4*>(qp + 16 * ks) : u32x4{0, 0, 0, 0};
      qop[ks] = __builtin_bit_cast(bf16x8, x);
    }
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

  const int v_tg = tid % (BN / 4), v_col = tid / (BN / 4);  // V staging: tokens 4*v_tg.., dims 8*v_col..
  u32x4 rk[KCH], rv[4];                          // global -> LDS staging registers
  // Rows past the end of the request are read from its last token instead
  // (always in bounds and finite); their scores are masked and their P is 0.
  auto gload_k = [&](int kv0) {
#pragma unroll
    for (int u = 0; u < KCH; ++u) {
      const int ch = tid + NTH * u, t = ch / CPR, col = ch % CPR;
      const int tok = min(kv0 + t, kv_end - 1);
      rk[u] = *reinterpret_cast<const u32x4*>(kg + (int64_t)tok * kv_row + 8 * col);
    }
  };
  auto gload_v = [&](int kv0) {
    if (tid < VTH) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int tok = min(kv0 + 4 * v_tg + u, kv_end - 1);
        rv[u] = *reinterpret_cast<const u32x4*>(vg + (int64_t)tok * kv_row + 8 * v_col);
      }
    }
  };
  auto lstore_k = [&](int buf) {
#pragma unroll
    for (int u = 0; u < KCH; ++u) {
      const int ch = tid + NTH * u, t = ch / CPR, col = ch % CPR;
      *reinterpret_cast<u32x4*>(&sK[buf][t * KP + 8 * col]) = rk[u];
    }
  };
  auto lstore_v = [&](int buf) {
    if (tid < VTH) {
      // 4 tokens x 8 dims -> 8 dim rows of 4 tokens: byte permutes pick the
      // low (even dim) or high (odd dim) bf16 of two token words.
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int wd = i >> 1;
        const uint32_t sel = (i & 1) ? 0x07060302u : 0x05040100u;
        u32x2 x;
        x[0] = __builtin_amdgcn_perm(rv[1][wd], rv[0][wd], sel);
        x[1] = __builtin_amdgcn_perm(rv[3][wd], rv[2][wd], sel);
        *reinterpret_cast<u32x2*>(&sV[buf][(8 * v_col + i) * VP + 4 * v_tg]) = x;
      }
    }
  };

  // Scores stay raw until the exponent: p = 2^(s*c - m) as one fma, with the
  // running max m kept in the scaled domain.  For c <= 0 the scores are scaled
  // first and c is taken as 1, so the max is always taken on the exponent.
  const float c_in = a.scale_log2;
  const bool pos_scale = c_in > 0.f;
  const float c_eff = pos_scale ? c_in : 1.f;
  // Lazy rescaling: the running max only moves when a new tile raises it by
  // more than kLazy (log2 units), so P <= 2^kLazy and the O/l rescale is
  // skipped for most tiles.  The result is the same softmax (the final O/l
  // uses the same m throughout).
  constexpr float kLazy = 8.f;
  // Last key this lane's row may see (causal and end of request).
  const int last_key = min(myq, kv_end - 1);

  f32x16 st[2];   // S^T of the 64-key sub-tile being scored
  bf16x8 pb[4];   // its P^T, the B operands of the four P.V k-steps
  constexpr int kDsRead = 0x100, kMfma = 0x008;

  // Operands are read from LDS ahead of the MFMAs that use them (scheduling
  // groups pin the order), so LDS latency overlaps the matrix work.
  auto qk = [&](int buf, int sub) {  // st = S^T of keys [64 sub, 64 sub + 64) of the stage
    bf16x8 ka[2][KS];
#pragma unroll
    for (int tt = 0; tt < 2; ++tt) {
      const uint16_t* kr = &sK[buf][(SUB * sub + 32 * tt + (l & 31)) * KP + 8 * hi];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) ka[tt][ks] = *reinterpret_cast<const bf16x8*>(kr + 16 * ks);
    }
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int x = 0; x < 16; ++x) st[tt][x] = 0.f;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
        st[tt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[tt][ks], qop[ks], st[tt], 0, 0, 0);
    __builtin_amdgcn_sched_group_barrier(kDsRead, 4, 0);
#pragma unroll
    for (int ks = 0; ks < KS - 2; ++ks) {
      __builtin_amdgcn_sched_group_barrier(kMfma, 2, 0);
      __builtin_amdgcn_sched_group_barrier(kDsRead, 2, 0);
    }
    __builtin_amdgcn_sched_group_barrier(kMfma, 4, 0);
  };
  auto pv = [&](int buf, int sub) {  // O^T += V^T P^T of the sub-tile
    // k-step (tt, hh): k-slot 8hi + jj <-> key 32tt + 16hh + 8(jj/4) + 4hi + jj%4
    u32x4 va[4][ET];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const int tcol = SUB * sub + 32 * (kk >> 1) + 16 * (kk & 1) + 4 * hi;
#pragma unroll
      for (int et = 0; et < ET; ++et) {
        const uint16_t* vr = &sV[buf][(32 * et + (l & 31)) * VP + tcol];
        const u32x2 lo = *reinterpret_cast<const u32x2*>(vr);
        const u32x2 hi2 = *reinterpret_cast<const u32x2*>(vr + 8);
        va[kk][et] = u32x4{lo[0], lo[1], hi2[0], hi2[1]};
      }
    }
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
#pragma unroll
      for (int et = 0; et < ET; ++et)
        oacc[et] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, va[kk][et]),
                                                           pb[kk], oacc[et], 0, 0, 0);
    __builtin_amdgcn_sched_group_barrier(kDsRead, ET, 0);
#pragma unroll
    for (int kk = 0; kk < 3; ++kk)
#pragma unroll
      for (int et = 0; et < ET; ++et) {
        __builtin_amdgcn_sched_group_barrier(kMfma, 1, 0);
        __builtin_amdgcn_sched_group_barrier(kDsRead, 1, 0);
      }
    __builtin_amdgcn_sched_group_barrier(kMfma, ET, 0);
  };
  auto softmax = [&](int kv0) {  // st (keys kv0 ..) -> pb, updating m_run, l_run (and O lazily)
    // lane holds S^T[t = kv0 + 32tt + 8(x/4) + 4hi + x%4][q = myq]
    if (!pos_scale) {
#pragma unroll
      for (int tt = 0; tt < 2; ++tt) st[tt] *= c_in;
    }
    if (kv0 + SUB - 1 > row_w || kv0 + SUB > kv_end) {  // diagonal or ragged sub-tile
      const int lim = last_key - kv0 - 4 * hi;  // mask offsets beyond it
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int x = 0; x < 16; ++x)
          if (32 * tt + 8 * (x >> 2) + (x & 3) > lim) st[tt][x] = -INFINITY;
    }
    float mx = fmaxf(st[0][0], st[1][0]);
#pragma unroll
    for (int x = 1; x < 16; ++x) mx = fmaxf(mx, fmaxf(st[0][x], st[1][x]));
    {
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx),
                                                       false, false);
      mx = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));  // max with lane ^ 32
    }
    const float m_tile = mx * c_eff;  // finite: key 0 is seen in the first sub-tile
    if (__ballot(m_tile > m_run + kLazy)) {  // wave-uniform
      const float m_new = fmaxf(m_run, m_tile);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int et = 0; et < ET; ++et) oacc[et] *= alpha;
    }
    float psum = 0.f;
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int x = 0; x < 16; ++x) {
        const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(st[tt][x], c_eff, -m_run));
        psum += p;
        pb[2 * tt + (x >> 3)][x & 7] = (__bf16)p;
      }
    l_run += psum;
  };

  // Stages of 128 keys, double-buffered in LDS; the next stage's global loads
  // are in flight while the current one is computed as two 64-key sub-tiles;
  // one barrier per stage.
  gload_k(0);
  gload_v(0);
  lstore_k(0);
  lstore_v(0);
  __syncthreads();
  for (int j = 0; j < ntiles; ++j) {
    const int cur = j & 1;
    gload_k((j + 1) * BN);  // unconditional: past the end it re-reads the last row
    gload_v((j + 1) * BN);
#pragma unroll
    for (int sub = 0; sub < BN / SUB; ++sub) {
      const int kv0 = j * BN + SUB * sub;
      if (wave_active && kv0 < kv_end && kv0 <= row_w + 31) {  // some key visible to this wave
        qk(cur, sub);
        softmax(kv0);
        pv(cur, sub);
      }
    }
    if (j + 1 < ntiles) {
      lstore_k(cur ^ 1);  // that buffer was last read before the previous barrier
      lstore_v(cur ^ 1);
    }
    __syncthreads();
  }

  if (!wave_active || myq >= L) return;
  float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  const float inv = 1.f / l_tot;
  // lane holds O^T[e = 32et + 8(x/4) + 4hi + x%4][myq]
  uint16_t* op = a.out + ((int64_t)(seq0 + myq) * a.hq + h) * D + 4 * hi;
#pragma unroll
  for (int et = 0; et < ET; ++et)
#pragma unroll
    for (int gq = 0; gq < 4; ++gq) {
      u32x2 x;
      x[0] = pack_bf16x2(oacc[et][4 * gq] * inv, oacc[et][4 * gq + 1] * inv);
      x[1] = pack_bf16x2(oacc[et][4 * gq + 2] * inv, oacc[et][4 * gq + 3] * inv);
      *reinterpret_cast<u32x2*>(op + 32 * et + 8 * gq) = x;
    }
  if (a.lse && hi == 0) a.lse[(int64_t)(seq0 + myq) * a.hq + h] = (m_run + __log2f(l_tot)) * kLn2;
}

}  // namespace dopd
