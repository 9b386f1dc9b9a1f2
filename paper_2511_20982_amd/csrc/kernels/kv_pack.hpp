// Handoff packer: gathers each request's pages into one contiguous buffer in
// (layer, K/V, head, token, dim) order.  One workgroup per (page, handoff,
// layer*2*Hkv + kv*Hkv + head); K pages are copied row for row, V pages are
// transposed from [d][16] to [16][d] through LDS.
#pragma once
#include "common.hpp"

namespace dopd {

template <typename T>  // uint8_t (E4M3 codes), uint16_t (bf16) or uint32_t (fp32) elements
__global__ __launch_bounds__(256) void kv_pack_kernel(
    const T* __restrict__ k_pool, const T* __restrict__ v_pool, int num_pages,
    const int32_t* __restrict__ page_table, int pt_stride, const int32_t* __restrict__ req_ids,
    const int32_t* __restrict__ seq_lens, const int64_t* __restrict__ out_off, int hkv, int d,
    T* __restrict__ out) {
  __shared__ __attribute__((aligned(16))) T sv[128 * kPage];
  const int pg = blockIdx.x, n = blockIdx.y, z = blockIdx.z;
  const int len = seq_lens[n];
  if (pg * kPage >= len) return;  // uniform for the workgroup
  const int layer = z / (2 * hkv);
  const int kv = (z / hkv) % 2;
  const int h = z % hkv;
  const int r = req_ids[n];
  const int64_t page = page_table[(int64_t)r * pt_stride + pg];
  const int nvalid = min(kPage, len - pg * kPage);
  const int64_t lpage = (int64_t)layer * num_pages + page;
  T* dst = out + out_off[n] + ((((int64_t)layer * 2 + kv) * hkv + h) * len + (int64_t)pg * kPage) * d;
  constexpr int kEl = 16 / sizeof(T);
  const bool aligned = ((reinterpret_cast<uintptr_t>(dst) & 15) == 0);
  const int nel = nvalid * d;

  if (kv == 0) {
    const T* src = k_pool + (lpage * hkv + h) * kPage * d;
    if (aligned) {
      const int nch = nel / kEl;
      for (int i = threadIdx.x; i < nch; i += blockDim.x)
        // streaming stores: the packed buffer leaves the caches at once
        // (it goes to another instance), not during the next kernel
        __builtin_nontemporal_store(reinterpret_cast<const u32x4*>(src)[i],
                                    reinterpret_cast<u32x4*>(dst) + i);
    } else {
      for (int i = threadIdx.x; i < nel; i += blockDim.x) dst[i] = src[i];
    }
    return;
  }
  // V: stage the dim-major page block in LDS, then write token rows.
  const T* src = v_pool + (lpage * hkv + h) * d * kPage;
  const int nch = d * kPage / kEl;
  for (int i = threadIdx.x; i < nch; i += blockDim.x)
    reinterpret_cast<u32x4*>(sv)[i] = reinterpret_cast<const u32x4*>(src)[i];
  __syncthreads();
  if (aligned) {
    const int cpr = d / kEl;  // 16-byte chunks per token row
    for (int i = threadIdx.x; i < nvalid * cpr; i += blockDim.x) {
      const int t = i / cpr, e0 = (i % cpr) * kEl;
      u32x4 x;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        if constexpr (sizeof(T) == 1)
          x[w] = (uint32_t)sv[(e0 + 4 * w) * kPage + t] |
                 ((uint32_t)sv[(e0 + 4 * w + 1) * kPage + t] << 8) |
                 ((uint32_t)sv[(e0 + 4 * w + 2) * kPage + t] << 16) |
                 ((uint32_t)sv[(e0 + 4 * w + 3) * kPage + t] << 24);
        else if constexpr (sizeof(T) == 2)
          x[w] = (uint32_t)sv[(e0 + 2 * w) * kPage + t] |
                 ((uint32_t)sv[(e0 + 2 * w + 1) * kPage + t] << 16);
        else
          x[w] = sv[(e0 + w) * kPage + t];
      }
      __builtin_nontemporal_store(x, reinterpret_cast<u32x4*>(dst) + i);
    }
  } else {
    for (int i = threadIdx.x; i < nel; i += blockDim.x) {
      const int t = i / d, e = i % d;
      dst[i] = sv[e * kPage + t];
    }
  }
}

}  // namespace dopd
