// Paged KV write of fresh prompts that also emits their handoff buffer.
//
// A prefill-completed request's cache is exactly the K/V rows its prefill
// just produced, so the handoff buffer ((K/V, head, token, dim) order, one
// layer) can be written from the same fresh rows the paged write reads,
// instead of gathering the pages back from the pool afterwards: every K/V byte
// is read once and written twice (pool page and handoff buffer), in one
// launch.  One workgroup per (request, logical page) x KV head; start
// position 0 for every request (fresh prompts).  K rows are copied in 16-byte
// chunks to both destinations; V rows go to the handoff buffer as they are
// (token-major) and to the dim-major pool page through LDS.  Slots of a
// request's last page past its length are never touched.
#pragma once
#include "common.hpp"

namespace dopd {

struct WritePackArgs {
  const uint16_t* k_new;      // [T][Hkv][D] bf16
  const uint16_t* v_new;      // [T][Hkv][D]
  uint16_t* k_pool;           // [P][Hkv][16][D]
  uint16_t* v_pool;           // [P][Hkv][D][16]
  const int32_t* page_table;  // [nreq][pt_stride] (rows of these requests)
  int pt_stride;
  const int32_t* cu;          // [nreq + 1] rows of each request in k_new / v_new
  int nreq, hkv;
  uint16_t* out;              // handoff buffer, or null (paged write only)
  const int64_t* out_off;     // [nreq] element offset of each request's block
  // E4M3 pools (the E4M3 workgroup only): pools and handoff buffer hold one
  // byte per element, the code of sat(x * fp32(1 / scale[h])).
  const float* k_scale;       // [Hkv]
  const float* v_scale;       // [Hkv]
};

// Workgroup (bx, h): logical page bx of the concatenated page lists, KV head h.
// s_v: LDS of 16 * (D + 8) bf16.
template <int D>
__device__ __forceinline__ void kv_write_pack_workgroup(const WritePackArgs& a, int bx, int h,
                                                        uint16_t* s_v) {
  constexpr int kEl = 8;        // bf16 elements per 16-byte chunk
  constexpr int CPR = D / kEl;  // chunks per token row
  constexpr int TP = D + kEl;   // padded LDS row (elements)
  auto pages = [&](int rr) { return (a.cu[rr + 1] - a.cu[rr] + kPage - 1) / kPage; };
  int r, lp;
  if (!find_owner(bx, a.nreq, pages, r, lp)) return;  // uniform
  const int tid = threadIdx.x;
  const int n = a.cu[r + 1] - a.cu[r];
  const int s1 = min(kPage, n - lp * kPage);  // live slots [0, s1) of this page
  const int64_t page = a.page_table[(int64_t)r * a.pt_stride + lp];
  const int64_t row_elems = (int64_t)a.hkv * D;
  const int64_t src0 = (int64_t)(a.cu[r] + lp * kPage) * row_elems + (int64_t)h * D;
  uint16_t* kdst = a.k_pool + (page * a.hkv + h) * kPage * D;
  uint16_t* vdst = a.v_pool + (page * a.hkv + h) * D * kPage;
  uint16_t* pk = nullptr;
  uint16_t* pv = nullptr;
  bool aligned = false;
  if (a.out) {
    const int64_t base = a.out_off[r];
    pk = a.out + base + ((int64_t)h * n + lp * kPage) * D;
    pv = a.out + base + ((int64_t)(a.hkv + h) * n + lp * kPage) * D;
    aligned = (base & (kEl - 1)) == 0;  // the rest of the offset is a multiple of D
  }
  for (int i = tid; i < kPage * CPR; i += 256) {
    const int slot = i / CPR, c = i % CPR;
    if (slot < s1) {
      const int64_t src = src0 + (int64_t)slot * row_elems + kEl * c;
      const u32x4 kx = *reinterpret_cast<const u32x4*>(a.k_new + src);
      const u32x4 vx = *reinterpret_cast<const u32x4*>(a.v_new + src);
      // Streaming stores: neither copy is read again by this step.
      __builtin_nontemporal_store(kx, reinterpret_cast<u32x4*>(kdst + slot * D + kEl * c));
      *reinterpret_cast<u32x4*>(&s_v[slot * TP + kEl * c]) = vx;
      if (aligned) {
        __builtin_nontemporal_store(kx, reinterpret_cast<u32x4*>(pk + slot * D + kEl * c));
        __builtin_nontemporal_store(vx, reinterpret_cast<u32x4*>(pv + slot * D + kEl * c));
      } else if (pk) {
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          pk[slot * D + kEl * c + 2 * w] = (uint16_t)(kx[w] & 0xffffu);
          pk[slot * D + kEl * c + 2 * w + 1] = (uint16_t)(kx[w] >> 16);
          pv[slot * D + kEl * c + 2 * w] = (uint16_t)(vx[w] & 0xffffu);
          pv[slot * D + kEl * c + 2 * w + 1] = (uint16_t)(vx[w] >> 16);
        }
      }
    }
  }
  __syncthreads();
  // V^T: dim row e of the page holds its 16 slots; one 16-byte run per thread.
  constexpr int RUNS = kPage / kEl;  // 16-byte runs per dim row
  for (int i = tid; i < D * RUNS; i += 256) {
    const int e = i / RUNS, run = i % RUNS;
    uint16_t* drow = vdst + e * kPage + run * kEl;
    if (s1 == kPage) {
      u32x4 x;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const int s = run * kEl + 2 * w;
        x[w] = (uint32_t)s_v[s * TP + e] | ((uint32_t)s_v[(s + 1) * TP + e] << 16);
      }
      *reinterpret_cast<u32x4*>(drow) = x;
    } else {
      for (int k = 0; k < kEl; ++k) {
        const int s = run * kEl + k;
        if (s < s1) drow[k] = s_v[s * TP + e];
      }
    }
  }
}

// The same over E4M3 pools: each fresh bf16 element x of KV head h becomes the
// code of sat(x * fp32(1 / scale[h])) (as the E4M3 paged writer computes it),
// written to the pool page and to the handoff buffer.  s_v: LDS of
// 16 * (D + 8) bytes.
template <int D>
__device__ __forceinline__ void kv_write_pack_e4m3_workgroup(const WritePackArgs& a, int bx, int h,
                                                             uint8_t* s_v) {
  constexpr int CPR = D / 8;  // 8-element chunks per token row
  constexpr int TP = D + 8;   // padded LDS row (bytes)
  auto pages = [&](int rr) { return (a.cu[rr + 1] - a.cu[rr] + kPage - 1) / kPage; };
  int r, lp;
  if (!find_owner(bx, a.nreq, pages, r, lp)) return;  // uniform
  const int tid = threadIdx.x;
  const int n = a.cu[r + 1] - a.cu[r];
  const int s1 = min(kPage, n - lp * kPage);  // live slots [0, s1) of this page
  const int64_t page = a.page_table[(int64_t)r * a.pt_stride + lp];
  const int64_t row_elems = (int64_t)a.hkv * D;
  const int64_t src0 = (int64_t)(a.cu[r] + lp * kPage) * row_elems + (int64_t)h * D;
  uint8_t* kdst = reinterpret_cast<uint8_t*>(a.k_pool) + (page * a.hkv + h) * kPage * D;
  uint8_t* vdst = reinterpret_cast<uint8_t*>(a.v_pool) + (page * a.hkv + h) * D * kPage;
  uint8_t* pk = nullptr;
  uint8_t* pv = nullptr;
  bool aligned = false;
  if (a.out) {
    const int64_t base = a.out_off[r];
    uint8_t* out8 = reinterpret_cast<uint8_t*>(a.out);
    pk = out8 + base + ((int64_t)h * n + lp * kPage) * D;
    pv = out8 + base + ((int64_t)(a.hkv + h) * n + lp * kPage) * D;
    aligned = (base & 7) == 0;  // the rest of the offset is a multiple of D
  }
  const float kinv = 1.0f / a.k_scale[h], vinv = 1.0f / a.v_scale[h];
  auto codes8 = [](u32x4 x, float inv) {  // 8 bf16 -> 8 codes
    u32x2 o;
#pragma unroll
    for (int w = 0; w < 2; ++w)
      o[w] = e4m3x4_from_f32(bf16_bits_to_f32(x[2 * w] & 0xffffu) * inv,
                             bf16_bits_to_f32(x[2 * w] >> 16) * inv,
                             bf16_bits_to_f32(x[2 * w + 1] & 0xffffu) * inv,
                             bf16_bits_to_f32(x[2 * w + 1] >> 16) * inv);
    return o;
  };
  for (int i = tid; i < kPage * CPR; i += 256) {
    const int slot = i / CPR, c = i % CPR;
    if (slot < s1) {
      const int64_t src = src0 + (int64_t)slot * row_elems + 8 * c;
      const u32x2 kc = codes8(*reinterpret_cast<const u32x4*>(a.k_new + src), kinv);
      const u32x2 vc = codes8(*reinterpret_cast<const u32x4*>(a.v_new + src), vinv);
      *reinterpret_cast<u32x2*>(kdst + slot * D + 8 * c) = kc;
      *reinterpret_cast<u32x2*>(&s_v[slot * TP + 8 * c]) = vc;
      if (aligned) {
        *reinterpret_cast<u32x2*>(pk + slot * D + 8 * c) = kc;
        *reinterpret_cast<u32x2*>(pv + slot * D + 8 * c) = vc;
      } else if (pk) {
#pragma unroll
        for (int b = 0; b < 8; ++b) {
          pk[slot * D + 8 * c + b] = (uint8_t)(kc[b / 4] >> (8 * (b % 4)));
          pv[slot * D + 8 * c + b] = (uint8_t)(vc[b / 4] >> (8 * (b % 4)));
        }
      }
    }
  }
  __syncthreads();
  // V^T: dim row e of the page holds its 16 slots (16 bytes).
  for (int e = tid; e < D; e += 256) {
    uint8_t* drow = vdst + e * kPage;
    if (s1 == kPage) {
      u32x4 x;
#pragma unroll
      for (int w = 0; w < 4; ++w)
        x[w] = (uint32_t)s_v[(4 * w) * TP + e] | ((uint32_t)s_v[(4 * w + 1) * TP + e] << 8) |
               ((uint32_t)s_v[(4 * w + 2) * TP + e] << 16) |
               ((uint32_t)s_v[(4 * w + 3) * TP + e] << 24);
      *reinterpret_cast<u32x4*>(drow) = x;
    } else {
      for (int s = 0; s < s1; ++s) drow[s] = s_v[s * TP + e];
    }
  }
}

template <int D>
__global__ __launch_bounds__(256) void kv_write_pack_kernel(WritePackArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t s_v[kPage * (D + 8)];
  kv_write_pack_workgroup<D>(a, (int)blockIdx.x / a.hkv, (int)blockIdx.x % a.hkv, s_v);
}

}  // namespace dopd
