// Variable-length causal prefill attention, bf16 in / fp32 accumulate, gfx950.
//
// Workgroup = 4 waves = one (q tile of 128 rows, request, query head); each
// wave owns 32 query rows.  K/V tiles of 64 tokens are staged in LDS (K
// token-major, V transposed to dim-major on the way in) and shared by the four
// waves.  Per tile and wave:
//
//   S^T[64 tok][32 q] = K[64][d] . Q^T[d][32]       2 x (d/16) v_mfma_f32_32x32x16_bf16
//   O^T[d][32 q]     += V^T[d][64] . P^T[64][32]    (d/32) x 4  v_mfma_f32_32x32x16_bf16
//
// Computing the transposed products keeps a whole query row inside one lane
// pair, so the online-softmax row max and row sum need a single cross-lane
// step, and the MFMA output of S^T is already the B operand of the P.V MFMA
// (the token order of the contraction is matched on the V^T LDS reads).
// Scores are scaled into the exp2 domain; only tiles on the diagonal or past
// the end of the request are masked, with a select (never a multiply).
// Work items are issued heaviest first (latest q tiles of every request
// first) so long prompts do not leave a tail.
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
};

constexpr int kPfBM = 128;  // query rows per workgroup
constexpr int kPfBN = 64;   // keys per LDS tile

// Number of BM-row q tiles of request rr.
__device__ __forceinline__ int pf_tiles(const int32_t* cu, int rr) {
  return (cu[rr + 1] - cu[rr] + kPfBM - 1) / kPfBM;
}

// Maps a workgroup index to (q tile, request, head), q tiles in decreasing
// index order (tile i of a request attends to ~ (i+1) key tiles).
__device__ __forceinline__ bool pf_find_item(const PrefillArgs& a, int b, int& tile, int& req,
                                             int& head) {
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

template <int D>
__global__ __launch_bounds__(256, 2) void prefill_bf16_kernel(PrefillArgs a) {
  constexpr int BM = kPfBM, BN = kPfBN;
  constexpr int KP = D + 8;      // padded K row (elements)
  constexpr int VP = BN + 8;     // padded V^T row (elements)
  constexpr int KS = D / 16;     // k-steps of the QK MFMA
  constexpr int ET = D / 32;     // O^T tiles of 32 dims
  constexpr int CPR = D / 8;     // 16-byte chunks per K/V row
  constexpr int KCH = BN * CPR / 256;   // K chunks staged per thread
  constexpr int VTH = (BN / 4) * CPR;   // threads staging V (4 tokens x 8 dims each)
  __shared__ __attribute__((aligned(16))) uint16_t sK[BN * KP];
  __shared__ __attribute__((aligned(16))) uint16_t sV[D * VP];

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

  u32x4 kreg[KCH], vreg[4];
  const int v_tg = tid % 16, v_col = tid / 16;  // V staging: tokens 4*v_tg.., dims 8*v_col..
  auto gload = [&](int kv0) {
#pragma unroll
    for (int u = 0; u < KCH; ++u) {
      const int ch = tid + 256 * u, t = ch / CPR, col = ch % CPR, tok = kv0 + t;
      kreg[u] = tok < kv_end ? *reinterpret_cast<const u32x4*>(kg + (int64_t)tok * kv_row + 8 * col)
                             : u32x4{0, 0, 0, 0};
    }
    if (tid < VTH) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int tok = kv0 + 4 * v_tg + u;
        vreg[u] = tok < kv_end
                      ? *reinterpret_cast<const u32x4*>(vg + (int64_t)tok * kv_row + 8 * v_col)
                      : u32x4{0, 0, 0, 0};
      }
    }
  };
  auto lstore = [&]() {
#pragma unroll
    for (int u = 0; u < KCH; ++u) {
      const int ch = tid + 256 * u, t = ch / CPR, col = ch % CPR;
      *reinterpret_cast<u32x4*>(&sK[t * KP + 8 * col]) = kreg[u];
    }
    if (tid < VTH) {
#pragma unroll
      for (int i = 0; i < 8; ++i) {  // dim 8*v_col + i, tokens 4*v_tg .. +3
        const int wd = i >> 1, sh = (i & 1) * 16;
        const uint32_t t0 = (vreg[0][wd] >> sh) & 0xffffu, t1 = (vreg[1][wd] >> sh) & 0xffffu;
        const uint32_t t2 = (vreg[2][wd] >> sh) & 0xffffu, t3 = (vreg[3][wd] >> sh) & 0xffffu;
        u32x2 x;
        x[0] = t0 | (t1 << 16);
        x[1] = t2 | (t3 << 16);
        *reinterpret_cast<u32x2*>(&sV[(8 * v_col + i) * VP + 4 * v_tg]) = x;
      }
    }
  };

  gload(0);
  lstore();
  __syncthreads();

  for (int j = 0; j < ntiles; ++j) {
    const int kv0 = j * BN;
    if (j + 1 < ntiles) gload(kv0 + BN);
    const bool skip = !wave_active || kv0 > row_w + 31;  // whole tile above this wave's rows
    if (!skip) {
      f32x16 st[2];
#pragma unroll
      for (int tt = 0; tt < 2; ++tt) {
#pragma unroll
        for (int x = 0; x < 16; ++x) st[tt][x] = 0.f;
        const uint16_t* kr = &sK[(32 * tt + (l & 31)) * KP + 8 * hi];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const bf16x8 ka = *reinterpret_cast<const bf16x8*>(kr + 16 * ks);
          st[tt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qop[ks], st[tt], 0, 0, 0);
        }
      }
      // lane holds S^T[t = kv0 + 32tt + 8(x/4) + 4hi + x%4][q = myq]
      const bool need_mask = (kv0 + BN - 1 > row_w) || (kv0 + BN > kv_end);
      float mx = -INFINITY;
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int x = 0; x < 16; ++x) {
          float y = st[tt][x] * a.scale_log2;
          if (need_mask) {
            const int t = kv0 + 32 * tt + 8 * (x >> 2) + 4 * hi + (x & 3);
            if (t > myq || t >= kv_end) y = -INFINITY;
          }
          st[tt][x] = y;
          mx = fmaxf(mx, y);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float m_new = fmaxf(m_run, mx);  // finite: key 0 is seen in the first tile
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      float psum = 0.f;
      bf16x8 pb[4];  // B operands of the four P.V k-steps
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int x = 0; x < 16; ++x) {
          const float p = __builtin_amdgcn_exp2f(st[tt][x] - m_new);
          psum += p;
          pb[2 * tt + (x >> 3)][x & 7] = (__bf16)p;
        }
      l_run = l_run * alpha + psum;
      m_run = m_new;
#pragma unroll
      for (int et = 0; et < ET; ++et) oacc[et] *= alpha;
      // k-step (tt, hh): k-slot 8hi + jj <-> token 32tt + 16hh + 8(jj/4) + 4hi + jj%4
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const int tcol = 32 * (kk >> 1) + 16 * (kk & 1) + 4 * hi;
#pragma unroll
        for (int et = 0; et < ET; ++et) {
          const uint16_t* vr = &sV[(32 * et + (l & 31)) * VP + tcol];
          const u32x2 lo = *reinterpret_cast<const u32x2*>(vr);
          const u32x2 hi2 = *reinterpret_cast<const u32x2*>(vr + 8);
          const u32x4 va = {lo[0], lo[1], hi2[0], hi2[1]};
          oacc[et] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, va),
                                                             pb[kk], oacc[et], 0, 0, 0);
        }
      }
    }
    __syncthreads();
    if (j + 1 < ntiles) {
      lstore();
      __syncthreads();
    }
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
