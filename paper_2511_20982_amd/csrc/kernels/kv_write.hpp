// Paged KV writer: scatters fresh token-major K/V rows into the page pools.
//   k_pool[page][Hkv][16][d]  (token-major page),  v_pool[page][Hkv][d][16]  (dim-major page)
// One workgroup per (request, touched logical page); pure bit copy.
#pragma once
#include "common.hpp"

namespace dopd {

template <typename T>  // uint16_t (bf16 bits) or uint32_t (fp32 bits)
__global__ __launch_bounds__(256) void kv_write_kernel(
    const T* __restrict__ k_new, const T* __restrict__ v_new, T* __restrict__ k_pool,
    T* __restrict__ v_pool, const int32_t* __restrict__ page_table, int pt_stride,
    const int32_t* __restrict__ cu_new, const int32_t* __restrict__ start_pos, int nreq, int hkv,
    int d) {
  // Touched logical pages of request r: those holding positions [start, start + n).
  auto touched = [&](int rr) {
    const int n = cu_new[rr + 1] - cu_new[rr];
    if (n <= 0) return 0;
    const int s = start_pos[rr];
    return (s + n - 1) / kPage - s / kPage + 1;
  };
  int r, local;
  if (!find_owner(blockIdx.x, nreq, touched, r, local)) return;

  const int n = cu_new[r + 1] - cu_new[r];
  const int start = start_pos[r];
  const int lp = start / kPage + local;                 // logical page
  const int p_lo = max(start, lp * kPage);              // first position written in this page
  const int p_hi = min(start + n, lp * kPage + kPage);  // one past the last
  const int s0 = p_lo - lp * kPage, s1 = p_hi - lp * kPage;
  const int64_t page = page_table[(int64_t)r * pt_stride + lp];
  const int64_t src0 = cu_new[r] + (p_lo - start);      // source row of slot s0
  const int64_t row_elems = (int64_t)hkv * d;

  // K: rows (slot, head) of d elements, copied in 16-byte chunks.
  constexpr int kEl = 16 / sizeof(T);
  const int cpr = d / kEl;
  const int nk = (s1 - s0) * hkv * cpr;
  for (int i = threadIdx.x; i < nk; i += blockDim.x) {
    const int chunk = i % cpr;
    const int rest = i / cpr;
    const int h = rest % hkv;
    const int slot = s0 + rest / hkv;
    const u32x4* src =
        reinterpret_cast<const u32x4*>(k_new + (src0 + slot - s0) * row_elems + (int64_t)h * d) + chunk;
    u32x4* dst = reinterpret_cast<u32x4*>(k_pool + ((page * hkv + h) * kPage + slot) * d) + chunk;
    *dst = *src;
  }

  // V: rows (head, e) of the page's 16 slots.
  const int nv = hkv * d;
  const bool full = (s0 == 0 && s1 == kPage);
  for (int i = threadIdx.x; i < nv; i += blockDim.x) {
    const int e = i % d, h = i / d;
    T* dst = v_pool + ((page * hkv + h) * d + e) * kPage;
    const T* src = v_new + (src0 - s0) * row_elems + (int64_t)h * d + e;   // slot s at + s*row_elems
    if (full) {
      T vals[kPage];
#pragma unroll
      for (int s = 0; s < kPage; ++s) vals[s] = src[s * row_elems];
      u32x4* d4 = reinterpret_cast<u32x4*>(dst);
#pragma unroll
      for (int c = 0; c < kPage / kEl; ++c) {
        u32x4 x;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          if constexpr (sizeof(T) == 2)
            x[w] = (uint32_t)vals[c * kEl + 2 * w] | ((uint32_t)vals[c * kEl + 2 * w + 1] << 16);
          else
            x[w] = vals[c * kEl + w];
        }
        d4[c] = x;
      }
    } else {
      for (int s = s0; s < s1; ++s) dst[s] = src[s * row_elems];
    }
  }
}

}  // namespace dopd
