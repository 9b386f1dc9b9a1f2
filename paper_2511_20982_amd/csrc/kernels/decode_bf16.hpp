// Paged single-query decode attention, bf16 in / fp32 accumulate, gfx950.
//
// Work item = one wave = (request r, KV head c, key split s).  The wave walks
// the split's pages two at a time (32 tokens) and computes, for the
// g = Hq/Hkv query heads of the group (padded to 16 MFMA columns):
//
//   S^T[32 tok][16 heads] = K[32 tok][d] . Q^T[d][16]      (v_mfma_f32_16x16x32_bf16)
//   O^T[d][16 heads]     += V^T[d][32 tok] . P^T[32][16]   (v_mfma_f32_16x16x32_bf16)
//
// with an online softmax in the exp2 domain.  K pages are token-major and V
// pages dim-major, so every MFMA operand is a 16-byte load straight from HBM
// (no LDS).  Because a contraction index may be permuted freely as long as
// both operands agree, each lane reads a 64-byte run of one K row, and the
// token order inside a page pair is arranged so that the softmax output of
// the QK MFMA is already the B operand of the PV MFMA.
//
// Splits of one (r, c) write un-normalised partials (m, l, o~) to the
// workspace; the last split to finish (device-scope counter) merges them in
// split order:  M = max m_s,  L = sum e^(m_s-M) l_s,  o = sum e^(m_s-M) o~_s / L.
// That merge is exact in real arithmetic, so the result does not depend on the
// split size beyond rounding.  A request with a single split writes directly.
#pragma once
#include "common.hpp"

namespace dopd {

struct DecodeArgs {
  const uint16_t* q;          // [B][Hq][D]
  const uint16_t* k_pool;     // [P][Hkv][16][D]
  const uint16_t* v_pool;     // [P][Hkv][D][16]
  const int32_t* page_table;  // [B][pt_stride]
  const int32_t* ctx_lens;    // [B]
  uint16_t* out;              // [B][Hq][D]
  float* lse;                 // [B][Hq] or null
  int* counters;              // [B][Hkv], zero on entry and on exit
  float* part_o;              // [items][g][D]
  float* part_ml;             // [items][g][2]
  int pt_stride, nreq, hq, hkv, split;
  float scale_log2;           // softmax_scale * log2(e)
};

template <int D>
__global__ __launch_bounds__(64) void decode_bf16_kernel(DecodeArgs a) {
  constexpr int NQK = D / 32;  // QK MFMAs (k = 32) per 16-token row block
  constexpr int NT = D / 16;   // O^T tiles of 16 dims
  constexpr int SPAN = D / 4;  // contiguous dims of a K row read by one lane
  const int l = lane_id();
  const int hq = a.hq, hkv = a.hkv, g = hq / hkv, split = a.split;

  int r, local;
  auto items = [&](int rr) { return ((a.ctx_lens[rr] + split - 1) / split) * hkv; };
  if (!find_owner(blockIdx.x, a.nreq, items, r, local)) return;
  const int c = local % hkv;
  const int s = local / hkv;
  const int ctx = a.ctx_lens[r];
  const int nsplit = (ctx + split - 1) / split;
  const int t_begin = s * split;
  const int ntok = min(split, ctx - t_begin);

  const int hl = l & 15;  // head within the group (MFMA column)
  const int qg = l >> 4;  // lane group 0..3 (MFMA k-slot group)

  // Q^T operand: lane holds q[r][c*g+hl][SPAN*qg + 8i + j].
  bf16x8 qop[NQK];
  {
    const bool ok = hl < g;
    const uint16_t* qp = a.q + ((int64_t)r * hq + c * g + (ok ? hl : 0)) * D + SPAN * qg;
#pragma unroll
    for (int i = 0; i < NQK; ++i) {
      u32x4 x = ok ? *reinterpret_cast<const u32x4*>(qp + 8 * i) : u32x4{0, 0, 0, 0};
      qop[i] = __builtin_bit_cast(bf16x8, x);
    }
  }

  f32x4 oacc[NT];
#pragma unroll
  for (int n = 0; n < NT; ++n) oacc[n] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;

  // Pair-token of this lane's A-operand row in the two QK MFMAs of a pair.
  const int mrow = l & 15;
  const int tq1 = 8 * (mrow >> 2) + (mrow & 3);  // MFMA #1 rows: 0-3, 8-11, 16-19, 24-27
  const int tq2 = tq1 + 4;                       // MFMA #2 rows: 4-7, 12-15, 20-23, 28-31
  const int64_t kstride_page = (int64_t)hkv * kPage * D;
  const uint16_t* kbase = a.k_pool + (int64_t)c * kPage * D + SPAN * qg;
  const uint16_t* vbase = a.v_pool + (int64_t)c * D * kPage + (int64_t)hl * kPage + 8 * (qg & 1);
  const int32_t* pt = a.page_table + (int64_t)r * a.pt_stride + t_begin / kPage;
  const int npages = (ntok + kPage - 1) / kPage;

  for (int pc = 0; pc < npages; pc += 64) {
    const int pid_l = (pc + l < npages) ? pt[pc + l] : 0;
    const int chunk_pairs = (min(64, npages - pc) + 1) / 2;
    for (int pp = 0; pp < chunk_pairs; ++pp) {
      const int pageA = __shfl(pid_l, 2 * pp, 64);
      const int pageB = __shfl(pid_l, 2 * pp + 1, 64);
      const int tok0 = (pc + 2 * pp) * kPage;  // split-local token of the pair start
      const int valid = min(2 * kPage, ntok - tok0);

      // ---- K operand rows (64-byte runs) for the two QK MFMAs
      u32x4 k1[NQK], k2[NQK];
      {
        const int pa1 = tq1 < kPage ? pageA : pageB, pa2 = tq2 < kPage ? pageA : pageB;
        const uint16_t* p1 = kbase + (int64_t)pa1 * kstride_page + (tq1 & 15) * D;
        const uint16_t* p2 = kbase + (int64_t)pa2 * kstride_page + (tq2 & 15) * D;
        const bool ok1 = tq1 < valid, ok2 = tq2 < valid;
#pragma unroll
        for (int i = 0; i < NQK; ++i) {
          k1[i] = ok1 ? *reinterpret_cast<const u32x4*>(p1 + 8 * i) : u32x4{0, 0, 0, 0};
          k2[i] = ok2 ? *reinterpret_cast<const u32x4*>(p2 + 8 * i) : u32x4{0, 0, 0, 0};
        }
      }
      // ---- V^T operand: row e = 16n + hl, pair tokens 8qg..8qg+7
      u32x4 vv[NT];
      {
        const int pv = qg < 2 ? pageA : pageB;
        const int first = 8 * qg;  // first pair token of this lane's k-slots
        const bool any = first < valid;
        const uint16_t* p = vbase + (int64_t)pv * kstride_page;
#pragma unroll
        for (int n = 0; n < NT; ++n)
          vv[n] = any ? *reinterpret_cast<const u32x4*>(p + (int64_t)(16 * n) * kPage)
                      : u32x4{0, 0, 0, 0};
        if (any && first + 8 > valid) {  // partially valid: zero the dead slots (NaN-safe)
          const int nv = valid - first;  // 1..7 live slots
#pragma unroll
          for (int n = 0; n < NT; ++n)
#pragma unroll
            for (int w = 0; w < 4; ++w) {
              const uint32_t keep = (2 * w + 1 < nv) ? 0xffffffffu : (2 * w < nv ? 0x0000ffffu : 0u);
              vv[n][w] &= keep;
            }
        }
      }

      // ---- S^T = K Q^T
      f32x4 s1 = {0.f, 0.f, 0.f, 0.f}, s2 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int i = 0; i < NQK; ++i) {
        s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, k1[i]), qop[i], s1, 0, 0, 0);
        s2 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, k2[i]), qop[i], s2, 0, 0, 0);
      }
      // lane holds head hl, pair tokens 8qg + 0..3 (s1) and 8qg + 4..7 (s2)
      float x[8];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        x[j] = (8 * qg + j < valid) ? s1[j] * a.scale_log2 : -INFINITY;
        x[4 + j] = (8 * qg + 4 + j < valid) ? s2[j] * a.scale_log2 : -INFINITY;
      }
      float mx = x[0];
#pragma unroll
      for (int j = 1; j < 8; ++j) mx = fmaxf(mx, x[j]);
      mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float m_new = fmaxf(m_run, mx);  // finite: the pair's first token is live
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      float psum = 0.f;
      bf16x8 pb;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float p = __builtin_amdgcn_exp2f(x[j] - m_new);
        psum += p;
        pb[j] = (__bf16)p;
      }
      l_run = l_run * alpha + psum;
      m_run = m_new;
      // ---- O^T += V^T P^T
#pragma unroll
      for (int n = 0; n < NT; ++n) {
        oacc[n] *= alpha;
        oacc[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, vv[n]), pb, oacc[n], 0, 0, 0);
      }
    }
  }

  // Row sum over the four lane groups (each summed its own tokens).
  float l_tot = l_run + __shfl_xor(l_run, 16, 64);
  l_tot += __shfl_xor(l_tot, 32, 64);
  const int head = c * g + hl;

  if (nsplit == 1) {
    if (hl < g) {
      const float inv = 1.f / l_tot;
      uint16_t* op = a.out + ((int64_t)r * hq + head) * D + 4 * qg;
#pragma unroll
      for (int n = 0; n < NT; ++n) {
        u32x2 w;
        w[0] = pack_bf16x2(oacc[n][0] * inv, oacc[n][1] * inv);
        w[1] = pack_bf16x2(oacc[n][2] * inv, oacc[n][3] * inv);
        *reinterpret_cast<u32x2*>(op + 16 * n) = w;
      }
      if (a.lse && qg == 0) a.lse[(int64_t)r * hq + head] = (m_run + __log2f(l_tot)) * kLn2;
    }
    return;
  }

  // ---- split-K: publish the partial, the last split of (r, c) merges.
  const int item = blockIdx.x;
  if (hl < g) {
    float* po = a.part_o + ((int64_t)item * g + hl) * D + 4 * qg;
#pragma unroll
    for (int n = 0; n < NT; ++n) *reinterpret_cast<f32x4*>(po + 16 * n) = oacc[n];
    if (qg == 0) {
      float* pm = a.part_ml + ((int64_t)item * g + hl) * 2;
      pm[0] = m_run;
      pm[1] = l_tot;
    }
  }
  __threadfence();
  int done = 0;
  int* counter = a.counters + (int64_t)r * hkv + c;
  if (l == 0) done = atomicAdd(counter, 1);
  done = __shfl(done, 0, 64);
  if (done != nsplit - 1) return;
  __threadfence();

  const int item0 = blockIdx.x - local + c;  // item of split 0 for this (r, c)
  constexpr int EPL = D / 64;                // output dims per lane
  for (int hh = 0; hh < g; ++hh) {
    // M and L over the splits, lanes stride over splits.
    float mloc = -INFINITY;
    for (int sp = l; sp < nsplit; sp += 64)
      mloc = fmaxf(mloc, a.part_ml[((int64_t)(item0 + sp * hkv) * g + hh) * 2]);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) mloc = fmaxf(mloc, __shfl_xor(mloc, o, 64));
    const float M = mloc;
    float lsum = 0.f;
    for (int sp = l; sp < nsplit; sp += 64) {
      const float* pm = a.part_ml + ((int64_t)(item0 + sp * hkv) * g + hh) * 2;
      lsum += __builtin_amdgcn_exp2f(pm[0] - M) * pm[1];
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) lsum += __shfl_xor(lsum, o, 64);
    float acc[EPL];
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc[e] = 0.f;
    for (int sp = 0; sp < nsplit; ++sp) {
      const int64_t it = item0 + (int64_t)sp * hkv;
      const float wgt = __builtin_amdgcn_exp2f(a.part_ml[(it * g + hh) * 2] - M);
      const float* po = a.part_o + (it * g + hh) * D + EPL * l;
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc[e] += wgt * po[e];
    }
    const float inv = 1.f / lsum;
    uint16_t* op = a.out + ((int64_t)r * hq + c * g + hh) * D + EPL * l;
    if constexpr (EPL == 2) {
      *reinterpret_cast<uint32_t*>(op) = pack_bf16x2(acc[0] * inv, acc[1] * inv);
    } else {
      op[0] = (uint16_t)f32_to_bf16_bits(acc[0] * inv);
    }
    if (a.lse && l == 0) a.lse[(int64_t)r * hq + c * g + hh] = (M + __log2f(lsum)) * kLn2;
  }
  if (l == 0) atomicExch(counter, 0);
}

}  // namespace dopd
