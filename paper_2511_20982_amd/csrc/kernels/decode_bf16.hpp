// Paged single-query decode attention, bf16 in / fp32 accumulate, gfx950.
//
// The key range of every (request r, KV head c) is cut into pairs of pages
// (32 tokens).  Each (r, c) is a span of kDecSegCost + (its pairs) work units
// (the first kDecSegCost units stand for the fixed cost of starting a
// segment: loading q, the page ids and the first pair), and the spans of all
// (r, c), taken r-major then c, form one sequence.  Workgroup b (4 waves)
// takes the contiguous slice [b * total / nwg, (b + 1) * total / nwg) of it,
// so every workgroup gets the same amount of work whatever the context
// lengths (one round over the machine when nwg is the number of resident
// slots).  A slice crosses (r, c) boundaries: the pairs of one (r, c) inside
// it are a segment.  Within a segment the waves take its pairs round-robin; for the
// g = Hq/Hkv query heads of the group (padded to 16 MFMA columns) a wave
// computes per pair
//
//   S^T[32 tok][16 heads] = K[32 tok][d] . Q^T[d][16]      (v_mfma_f32_16x16x32_bf16)
//   O^T[d][16 heads]     += V^T[d][32 tok] . P^T[32][16]   (v_mfma_f32_16x16x32_bf16)
//
// with an online softmax in the exp2 domain.  K pages are token-major and V
// pages dim-major, so every MFMA operand is one 16-byte load straight from HBM
// (no LDS on the streaming path).  A contraction index may be permuted freely
// when both operands agree, so each lane reads a 64-byte run of one K row and
// the token order inside a pair is arranged so that the QK output is already
// the B operand of the PV MFMA.  Loads are unconditional (dead slots are read
// from a live address and masked with selects) and double-buffered in
// registers: the loads of the next pair are in flight while the current pair
// is computed.
//
// The four waves' (m, l, O) are merged through LDS.  A segment that is the
// whole (r, c) writes the output directly; otherwise it writes an
// un-normalised partial to slot b + (r * Hkv + c) of the workspace (distinct
// for distinct segments, since along the sequence b and the (r, c) index both
// only grow), and a second, small kernel merges the partials of every (r, c)
// in slice order:
//   M = max_s m_s,  L = sum_s 2^(m_s-M) l_s,  o = sum_s 2^(m_s-M) o~_s / L.
// That merge is exact in real arithmetic, so the result does not depend on the
// partition beyond rounding.  The kernel boundary orders the partial writes
// before the merge reads; no in-kernel fence or counter is needed (a
// device-scope fence costs a whole-L2 writeback and invalidate on this part).
//
// KV8 = true reads pages of E4M3 codes (one byte per element, same layouts)
// with one scale per KV head: the MFMA operands are the codes widened to
// bf16 (exact), the K scale is folded into the softmax scale and the V scale
// into the output.  Each K lane reads a 32-byte run and each V lane 8 bytes;
// the loaded bytes are converted just before their MFMAs, so the buffers in
// flight stay raw.
#pragma once
#include <type_traits>

#include "common.hpp"
#include "../plan.hpp"

namespace dopd {

struct DecodeArgs {
  const uint16_t* q;          // [B][Hq][D]
  const void* k_pool;         // [P][Hkv][16][D] bf16 or E4M3
  const void* v_pool;         // [P][Hkv][D][16] bf16 or E4M3
  const float* k_scale;       // [Hkv], E4M3 pools only
  const float* v_scale;       // [Hkv], E4M3 pools only
  const int32_t* page_table;  // [B][pt_stride]
  const int32_t* ctx_lens;    // [B]
  uint16_t* out;              // [B][Hq][D]
  float* lse;                 // [B][Hq] or null
  float* part_o;              // [slots][g][D]
  float* part_ml;             // [slots][g][2]
  int pt_stride, nreq, hq, hkv;
  int total_units;            // sum_r (kDecSegCost + ceil(ctx_r / 32)) * Hkv
  int nwg;                    // workgroups of the partition
  float scale_log2;           // softmax_scale * log2(e)
};

constexpr int kDecWaves = 4;
constexpr int kDecChunkPairs = 32 * kDecWaves;  // pairs whose page ids one wave holds at once

// First work unit of workgroup b's slice.
__device__ __forceinline__ int dec_slice_begin(const DecodeArgs& a, int b) {
  return (int)dec_slice_begin((int64_t)b, a.total_units, a.nwg);
}

// The workgroup whose slice holds work unit x (the host planner's search).
__device__ __forceinline__ int dec_slice_of(const DecodeArgs& a, int x) {
  int b = (int)((int64_t)x * a.nwg / a.total_units);
  while (b + 1 < a.nwg && dec_slice_begin(a, b + 1) <= x) ++b;
  while (b > 0 && dec_slice_begin(a, b) > x) --b;
  return b;
}

template <int D, bool KV8>
struct DecodePairBuf {
  u32x4 k1[D / 32], k2[D / 32];  // K rows of the two QK MFMAs
  u32x4 v[D / 16];               // V^T rows, one per 16-dim tile
};
template <int D>
struct DecodePairBuf<D, true> {  // raw E4M3 codes
  u32x4 k1[D / 64], k2[D / 64];
  u32x2 v[D / 16];
};

// bf16 MFMA operand i of a lane's K run (dims 8i .. 8i+7 of the run).
template <bool KV8, class KArr>
__device__ __forceinline__ bf16x8 dec_k_operand(const KArr& k, int i) {
  if constexpr (KV8) {
    const u32x4 w = k[i >> 1];
    const u32x2 lo = bf16x4_from_e4m3x4(w[2 * (i & 1)]), hi = bf16x4_from_e4m3x4(w[2 * (i & 1) + 1]);
    return __builtin_bit_cast(bf16x8, u32x4{lo[0], lo[1], hi[0], hi[1]});
  } else {
    return __builtin_bit_cast(bf16x8, k[i]);
  }
}

// LDS of the wave merge of one decode workgroup: (m, l) of waves 1..3,
// [wave - 1][2][64] floats, and their partial outputs, one block of
// [D / 16][64] f32x4 per wave (8 KiB at d = 128).
template <int D>
constexpr int dec_wave_o_bytes() { return (D / 16) * 64 * 16; }
constexpr int kDecMlBytes = (kDecWaves - 1) * 2 * 64 * 4;

// Workgroup b of the decode partition (its slice of the work units).
// s_ml: kDecMlBytes of LDS; s_o1, s_o2, s_o3: the partial-output blocks of
// waves 1, 2 and 3.
template <int D, bool KV8>
__device__ __forceinline__ void decode_workgroup(const DecodeArgs& a, int b, float* s_ml,
                                                 f32x4* s_o1, f32x4* s_o2, f32x4* s_o3) {
  auto s_o = [&](int i) { return i == 0 ? s_o1 : (i == 1 ? s_o2 : s_o3); };
  using KT = std::conditional_t<KV8, uint8_t, uint16_t>;
  constexpr int NQK = D / 32;  // QK MFMAs (k = 32) per 16-token row block
  constexpr int NT = D / 16;   // O^T tiles of 16 dims
  constexpr int SPAN = D / 4;  // contiguous dims of a K row read by one lane

  const int tid = threadIdx.x, l = lane_id(), w = tid >> 6;
  const int hq = a.hq, hkv = a.hkv, g = hq / hkv;
  if (b >= a.nwg) return;  // uniform
  const int lo = dec_slice_begin(a, b), hi_unit = dec_slice_begin(a, b + 1);
  if (lo >= hi_unit) return;  // uniform

  // (r, unit offset inside r's (c, unit) sequence) of the first unit
  int r, local;
  {
    auto cnt = [&](int rr) { return (kDecSegCost + (a.ctx_lens[rr] + 31) / 32) * hkv; };
    if (!find_owner(lo, a.nreq, cnt, r, local)) return;
  }

  const int hl = l & 15;  // head within the group (MFMA column)
  const int qg = l >> 4;  // lane group 0..3 (MFMA k-slot group)
  const int mrow = l & 15;
  const int tq1 = 8 * (mrow >> 2) + (mrow & 3);  // MFMA #1 rows hold pair tokens 0-3, 8-11, 16-19, 24-27
  const int tq2 = tq1 + 4;                       // MFMA #2 rows hold 4-7, 12-15, 20-23, 28-31
  const int64_t page_elems = (int64_t)hkv * kPage * D;

  int pos = lo;
  while (pos < hi_unit) {  // one (r, c) span per iteration (uniform)
    const int ctx = a.ctx_lens[r];
    const int np = (ctx + 31) / 32;                 // pairs of one (r, c)
    const int span = kDecSegCost + np;              // its work units
    const int c = local / span, u0 = local % span;
    const int u1 = min(span, u0 + (hi_unit - pos));
    const int p0 = max(0, u0 - kDecSegCost), p1 = max(0, u1 - kDecSegCost);  // pairs [p0, p1)
    pos += u1 - u0;
    local += u1 - u0;
    const int rr = r;
    if (local == span * hkv) {
      ++r;
      local = 0;
    }
    if (p0 == p1) continue;  // only start-cost units of this (r, c) fall in the slice
    const int r = rr;  // the segment's request (the loop variable has moved on)

    // Q^T operand: lane holds q[r][c*g+hl][SPAN*qg + 8i + j].
    bf16x8 qop[NQK];
    {
      const bool ok = hl < g;
      const uint16_t* qp = a.q + ((int64_t)r * hq + c * g + (ok ? hl : 0)) * D + SPAN * qg;
#pragma unroll
      for (int i = 0; i < NQK; ++i) {
        u32x4 x = *reinterpret_cast<const u32x4*>(qp + 8 * i);
        if (!ok) x = u32x4{0, 0, 0, 0};
        qop[i] = __builtin_bit_cast(bf16x8, x);
      }
    }

    f32x4 oacc[NT];
#pragma unroll
    for (int n = 0; n < NT; ++n) oacc[n] = f32x4{0.f, 0.f, 0.f, 0.f};
    float m_run = -INFINITY, l_run = 0.f;
    // E4M3 pools: k = code * k_scale[c] scales every score, v = code * v_scale[c] the output.
    const float sl2 = KV8 ? a.scale_log2 * a.k_scale[c] : a.scale_log2;

    const KT* kbase = static_cast<const KT*>(a.k_pool) + (int64_t)c * kPage * D + SPAN * qg;
    const KT* vbase = static_cast<const KT*>(a.v_pool) + (int64_t)c * D * kPage + (int64_t)hl * kPage +
                      8 * (qg & 1);

    // Chunks of up to 128 pairs: lane j of a wave holds the page id of page
    // (j & 1) of the wave's pair j/2 of the chunk.
    for (int cb = p0; cb < p1; cb += kDecChunkPairs) {
      const int t_begin = 32 * cb;
      const int ntok = min(32 * min(p1 - cb, kDecChunkPairs), ctx - t_begin);
      const int npairs = (ntok + 31) / 32;
      const int my_pairs = npairs > w ? (npairs - w + kDecWaves - 1) / kDecWaves : 0;
      const int32_t* pt = a.page_table + (int64_t)r * a.pt_stride + t_begin / kPage;
      const int npages = (ntok + kPage - 1) / kPage;
      int pid = 0;
      {
        const int pg = 2 * (w + kDecWaves * (l >> 1)) + (l & 1);
        if (pg < npages) pid = pt[pg];
      }

    auto load_pair = [&](DecodePairBuf<D, KV8>& buf, int k) {
      const int pair = w + kDecWaves * k;
      const int pageA = __shfl(pid, 2 * k, 64);
      const int pageB = __shfl(pid, 2 * k + 1, 64);
      const int valid = min(32, ntok - 32 * pair);
      // dead tokens read slot 0 of page A (always live) and are masked later
      const int64_t a1 = tq1 < valid ? (int64_t)(tq1 < kPage ? pageA : pageB) * page_elems + (tq1 & 15) * D
                                     : (int64_t)pageA * page_elems;
      const int64_t a2 = tq2 < valid ? (int64_t)(tq2 < kPage ? pageA : pageB) * page_elems + (tq2 & 15) * D
                                     : (int64_t)pageA * page_elems;
      constexpr int KEL = 16 / sizeof(KT);  // elements per 16-byte load
  #pragma unroll
      for (int i = 0; i < SPAN / KEL; ++i) {
        buf.k1[i] = *reinterpret_cast<const u32x4*>(kbase + a1 + KEL * i);
        buf.k2[i] = *reinterpret_cast<const u32x4*>(kbase + a2 + KEL * i);
      }
      const int pv = (qg < 2 || valid <= kPage) ? pageA : pageB;
      const KT* p = vbase + (int64_t)pv * page_elems;
  #pragma unroll
      for (int n = 0; n < NT; ++n) {
        if constexpr (KV8)
          buf.v[n] = *reinterpret_cast<const u32x2*>(p + (int64_t)(16 * n) * kPage);
        else
          buf.v[n] = *reinterpret_cast<const u32x4*>(p + (int64_t)(16 * n) * kPage);
      }
    };

    auto compute_pair = [&](DecodePairBuf<D, KV8>& buf, int k) {
      const int pair = w + kDecWaves * k;
      const int valid = min(32, ntok - 32 * pair);
      f32x4 s1 = {0.f, 0.f, 0.f, 0.f}, s2 = {0.f, 0.f, 0.f, 0.f};
  #pragma unroll
      for (int i = 0; i < NQK; ++i) {
        s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(dec_k_operand<KV8>(buf.k1, i), qop[i], s1, 0, 0, 0);
        s2 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(dec_k_operand<KV8>(buf.k2, i), qop[i], s2, 0, 0, 0);
      }
      // lane holds head hl, pair tokens 8qg + 0..3 (s1) and 8qg + 4..7 (s2)
      float x[8];
  #pragma unroll
      for (int j = 0; j < 4; ++j) {
        x[j] = s1[j] * sl2;
        x[4 + j] = s2[j] * sl2;
      }
      if (valid < 32) {  // last pair of a ragged split: mask dead tokens, zero dead V slots
  #pragma unroll
        for (int j = 0; j < 8; ++j)
          if (8 * qg + j >= valid) x[j] = -INFINITY;
        const int nv = valid - 8 * qg;  // live slots among this lane's 8
  #pragma unroll
        for (int n = 0; n < NT; ++n) {
          if constexpr (KV8) {
  #pragma unroll
            for (int wd = 0; wd < 2; ++wd) {  // one byte per slot
              const int live = min(4, max(0, nv - 4 * wd));
              const uint32_t keep = live >= 4 ? 0xffffffffu : ((1u << (8 * live)) - 1u);
              buf.v[n][wd] &= keep;
            }
          } else {
  #pragma unroll
            for (int wd = 0; wd < 4; ++wd) {
              const uint32_t keep = (2 * wd + 1 < nv) ? 0xffffffffu : (2 * wd < nv ? 0x0000ffffu : 0u);
              buf.v[n][wd] &= keep;
            }
          }
        }
      }
      float mx = fmaxf(fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])),
                       fmaxf(fmaxf(x[4], x[5]), fmaxf(x[6], x[7])));
      mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float m_new = fmaxf(m_run, mx);  // finite: a pair's first token is live
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      float psum = 0.f;
      bf16x8 pb;
  #pragma unroll
      for (int j = 0; j < 8; ++j) {
        // the row sum adds the bf16-rounded weights the P.V product applies
        pb[j] = (__bf16)__builtin_amdgcn_exp2f(x[j] - m_new);
        psum += (float)pb[j];
      }
      l_run = l_run * alpha + psum;
      m_run = m_new;
  #pragma unroll
      for (int n = 0; n < NT; ++n) {
        oacc[n] *= alpha;
        bf16x8 vop;
        if constexpr (KV8) {
          const u32x2 lo = bf16x4_from_e4m3x4(buf.v[n][0]), hi = bf16x4_from_e4m3x4(buf.v[n][1]);
          vop = __builtin_bit_cast(bf16x8, u32x4{lo[0], lo[1], hi[0], hi[1]});
        } else {
          vop = __builtin_bit_cast(bf16x8, buf.v[n]);
        }
        oacc[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vop, pb, oacc[n], 0, 0, 0);
      }
    };

      if (my_pairs > 0) {
        // Prefetch loads are issued unconditionally (past the end they re-read
        // the last pair, an L2 hit) so the compiler can wait for exactly the
        // buffer being computed while the other one is in flight.
        const int last = my_pairs - 1;
        DecodePairBuf<D, KV8> b0, b1;
        load_pair(b0, 0);
        for (int k = 0; k < my_pairs; k += 2) {
          load_pair(b1, min(k + 1, last));
          compute_pair(b0, k);
          load_pair(b0, min(k + 2, last));
          if (k + 1 < my_pairs) compute_pair(b1, k + 1);
        }
      }
    }

    // Row sum over the four lane groups (each summed its own tokens).
    float l_tot = l_run + __shfl_xor(l_run, 16, 64);
    l_tot += __shfl_xor(l_tot, 32, 64);

    // ---- merge the four waves in wave 0 (identical lane layouts)
    if (w > 0) {
      s_ml[(w - 1) * 128 + l] = m_run;
      s_ml[(w - 1) * 128 + 64 + l] = l_tot;
#pragma unroll
      for (int n = 0; n < NT; ++n) s_o(w - 1)[n * 64 + l] = oacc[n];
    }
    __syncthreads();
    if (w == 0) {
      float mw[kDecWaves], lw[kDecWaves];
      mw[0] = m_run;
      lw[0] = l_tot;
      float M = m_run;
#pragma unroll
      for (int i = 1; i < kDecWaves; ++i) {
        mw[i] = s_ml[(i - 1) * 128 + l];
        lw[i] = s_ml[(i - 1) * 128 + 64 + l];
        M = fmaxf(M, mw[i]);
      }
      float sc[kDecWaves], L = 0.f;
#pragma unroll
      for (int i = 0; i < kDecWaves; ++i) {
        sc[i] = __builtin_amdgcn_exp2f(mw[i] - M);  // a wave without pairs has m = -inf -> 0
        L += sc[i] * lw[i];
      }
      const float vsc = KV8 ? a.v_scale[c] : 1.f;
#pragma unroll
      for (int n = 0; n < NT; ++n) {
        f32x4 o = oacc[n] * sc[0];
#pragma unroll
        for (int i = 1; i < kDecWaves; ++i) o += s_o(i - 1)[n * 64 + l] * sc[i];
        oacc[n] = KV8 ? o * vsc : o;
      }
      const int head = c * g + hl;
      if (hl < g) {
        if (p0 == 0 && p1 == np) {  // the whole (r, c): final output
          const float inv = 1.f / L;
          uint16_t* op = a.out + ((int64_t)r * hq + head) * D + 4 * qg;
#pragma unroll
          for (int n = 0; n < NT; ++n) {
            u32x2 wv;
            wv[0] = pack_bf16x2(oacc[n][0] * inv, oacc[n][1] * inv);
            wv[1] = pack_bf16x2(oacc[n][2] * inv, oacc[n][3] * inv);
            *reinterpret_cast<u32x2*>(op + 16 * n) = wv;
          }
          if (a.lse && qg == 0) a.lse[(int64_t)r * hq + head] = (M + __log2f(L)) * kLn2;
        } else {  // a partial for the merge kernel
          const int64_t slot = (int64_t)b + r * hkv + c;
          float* po = a.part_o + (slot * g + hl) * D + 4 * qg;
#pragma unroll
          for (int n = 0; n < NT; ++n) *reinterpret_cast<f32x4*>(po + 16 * n) = oacc[n];
          if (qg == 0) *reinterpret_cast<float2*>(a.part_ml + (slot * g + hl) * 2) = float2{M, L};
        }
      }
    }
    __syncthreads();  // the LDS merge buffers are reused by the next segment
  }
}

template <int D, bool KV8>
__global__ __launch_bounds__(256, 2) void decode_split_kernel(DecodeArgs a) {
  __shared__ __attribute__((aligned(16))) float s_ml[kDecMlBytes / 4];
  __shared__ __attribute__((aligned(16))) f32x4 s_o[kDecWaves - 1][D / 16 * 64];
  decode_workgroup<D, KV8>(a, (int)blockIdx.x, s_ml, s_o[0], s_o[1], s_o[2]);
}

// The merge of the (r, c) whose pairs span more than one slice: the partials
// of (r, c) from slices b0 .. b1 (slot b + r * Hkv + c) are folded in slice
// order into the output; thread = one 4-dim chunk of one query head.
template <int D>
__device__ __forceinline__ void decode_merge_pair(const DecodeArgs& a, int r, int c, int b0, int b1) {
  const int tid = threadIdx.x;
  const int hq = a.hq, hkv = a.hkv, g = hq / hkv;
  const int64_t rc = (int64_t)r * hkv + c;
  const int chunks = g * (D / 4);
  for (int ch = tid; ch < chunks; ch += 256) {
    const int hh = ch / (D / 4), e0 = 4 * (ch % (D / 4));
    float M = -INFINITY, L = 0.f;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    auto fold = [&](float2 ml, f32x4 ov) {  // online log-sum-exp merge, slice order
      const float Mn = fmaxf(M, ml.x);
      const float s_old = __builtin_amdgcn_exp2f(M - Mn), s_new = __builtin_amdgcn_exp2f(ml.x - Mn);
      L = L * s_old + ml.y * s_new;
      acc = acc * s_old + ov * s_new;
      M = Mn;
    };
    int b = b0;
    for (; b + 4 <= b1 + 1; b += 4) {  // four independent loads in flight
      float2 ml[4];
      f32x4 ov[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int64_t sl = b + u + rc;
        ml[u] = *reinterpret_cast<const float2*>(a.part_ml + (sl * g + hh) * 2);
        ov[u] = *reinterpret_cast<const f32x4*>(a.part_o + (sl * g + hh) * D + e0);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) fold(ml[u], ov[u]);
    }
    for (; b <= b1; ++b) {
      const int64_t sl = b + rc;
      fold(*reinterpret_cast<const float2*>(a.part_ml + (sl * g + hh) * 2),
           *reinterpret_cast<const f32x4*>(a.part_o + (sl * g + hh) * D + e0));
    }
    const float inv = 1.f / L;
    uint16_t* op = a.out + ((int64_t)r * hq + c * g + hh) * D + e0;
    u32x2 wv;
    wv[0] = pack_bf16x2(acc[0] * inv, acc[1] * inv);
    wv[1] = pack_bf16x2(acc[2] * inv, acc[3] * inv);
    *reinterpret_cast<u32x2*>(op) = wv;
    if (a.lse && e0 == 0) a.lse[(int64_t)r * hq + c * g + hh] = (M + __log2f(L)) * kLn2;
  }
}

// Workgroup = one (r, c); it finds the slices of its first and last pair
// itself (a scan over the context lengths) and returns when they are one.
template <int D>
__global__ __launch_bounds__(256) void decode_merge_kernel(DecodeArgs a) {
  const int l = lane_id();
  const int hkv = a.hkv;
  const int r = blockIdx.x / hkv, c = blockIdx.x % hkv;
  const int np = (a.ctx_lens[r] + 31) / 32;
  int base = 0;  // first work unit of request r
  for (int r0 = 0; r0 < r; r0 += 64) {
    const int rr = r0 + l;
    const int v = rr < r ? (kDecSegCost + (a.ctx_lens[rr] + 31) / 32) * hkv : 0;
    base += __shfl(wave_inclusive_scan(v), 63, 64);
  }
  const int first = base + c * (kDecSegCost + np) + kDecSegCost;  // unit of the first pair
  const int b0 = dec_slice_of(a, first), b1 = dec_slice_of(a, first + np - 1);
  if (b0 == b1) return;  // one segment: written directly
  decode_merge_pair<D>(a, r, c, b0, b1);
}

// The (r, c) to merge as the host listed them (decode_merge_list): workgroup
// = one list item, whose (r, c) and slices come from the kernel arguments, so
// the merge starts with the loads of the partials.
constexpr int kMergeListMax = 768;
struct DecodeMergeList {
  int n;
  uint32_t item[kMergeListMax];
};

template <int D>
__global__ __launch_bounds__(256) void decode_merge_list_kernel(DecodeArgs a, DecodeMergeList m) {
  const uint32_t it = m.item[blockIdx.x];
  const int rc = (int)(it & ((1u << kMergeRcBits) - 1));
  const int b0 = (int)((it >> kMergeRcBits) & ((1u << kMergeB0Bits) - 1));
  const int b1 = b0 + (int)(it >> (kMergeRcBits + kMergeB0Bits));
  decode_merge_pair<D>(a, rc / a.hkv, rc % a.hkv, b0, b1);
}

}  // namespace dopd
