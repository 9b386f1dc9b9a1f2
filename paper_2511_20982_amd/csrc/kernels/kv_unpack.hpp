// Handoff unpack on the receiving instance: scatters a packed
// (layer, K/V, head, token, dim) buffer into the local page pools, the inverse
// of kv_pack.  One workgroup per (page, handoff, layer*2*Hkv + kv*Hkv + head);
// K rows are copied as they are, V rows are transposed to the dim-major page
// block through LDS.  Slots past the request's length are never touched.
#pragma once
#include "common.hpp"

namespace dopd {

template <typename T, int D>
__global__ __launch_bounds__(256) void kv_unpack_kernel(
    const T* __restrict__ in, const int64_t* __restrict__ in_off, const int32_t* __restrict__ req_ids,
    const int32_t* __restrict__ seq_lens, T* __restrict__ k_pool, T* __restrict__ v_pool,
    int num_pages, const int32_t* __restrict__ page_table, int pt_stride, int hkv) {
  constexpr int kEl = 16 / sizeof(T);
  constexpr int CPR = D / kEl;   // 16-byte chunks per token row
  constexpr int TP = D + kEl;    // padded LDS row (elements)
  __shared__ __attribute__((aligned(16))) T s_v[kPage * TP];
  const int pg = blockIdx.x, n = blockIdx.y, z = blockIdx.z, tid = threadIdx.x;
  const int len = seq_lens[n];
  if (pg * kPage >= len) return;  // uniform for the workgroup
  const int layer = z / (2 * hkv);
  const int kv = (z / hkv) % 2;
  const int h = z % hkv;
  const int r = req_ids[n];
  const int64_t page = page_table[(int64_t)r * pt_stride + pg];
  const int nvalid = min(kPage, len - pg * kPage);
  const int64_t lpage = (int64_t)layer * num_pages + page;
  const T* src = in + in_off[n] + ((((int64_t)layer * 2 + kv) * hkv + h) * len + (int64_t)pg * kPage) * D;
  const bool aligned = ((reinterpret_cast<uintptr_t>(src) & 15) == 0);

  if (kv == 0) {
    T* dst = k_pool + (lpage * hkv + h) * kPage * D;
    if (aligned) {
      // streaming stores (here and below): the pages leave the caches now,
      // not as write-back during the kernels that follow
      for (int i = tid; i < nvalid * CPR; i += 256)
        __builtin_nontemporal_store(reinterpret_cast<const u32x4*>(src)[i],
                                    reinterpret_cast<u32x4*>(dst) + i);
    } else {
      for (int i = tid; i < nvalid * D; i += 256) dst[i] = src[i];
    }
    return;
  }
  // V: token rows into LDS, then dim rows of the page's slots.
  if (aligned) {
    for (int i = tid; i < nvalid * CPR; i += 256) {
      const int t = i / CPR, c = i % CPR;
      *reinterpret_cast<u32x4*>(&s_v[t * TP + c * kEl]) = reinterpret_cast<const u32x4*>(src)[i];
    }
  } else {
    for (int i = tid; i < nvalid * D; i += 256) s_v[(i / D) * TP + i % D] = src[i];
  }
  __syncthreads();
  T* vdst = v_pool + (lpage * hkv + h) * D * kPage;
  constexpr int RUNS = kPage / kEl;  // 16-byte runs per dim row
  for (int i = tid; i < D * RUNS; i += 256) {
    const int e = i / RUNS, run = i % RUNS;
    T* drow = vdst + e * kPage + run * kEl;
    if (nvalid == kPage) {
      u32x4 x;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        if constexpr (sizeof(T) == 1) {
          const int s = run * kEl + 4 * w;
          x[w] = (uint32_t)s_v[s * TP + e] | ((uint32_t)s_v[(s + 1) * TP + e] << 8) |
                 ((uint32_t)s_v[(s + 2) * TP + e] << 16) | ((uint32_t)s_v[(s + 3) * TP + e] << 24);
        } else if constexpr (sizeof(T) == 2) {
          const int s = run * kEl + 2 * w;
          x[w] = (uint32_t)s_v[s * TP + e] | ((uint32_t)s_v[(s + 1) * TP + e] << 16);
        } else {
          x[w] = s_v[(run * kEl + w) * TP + e];
        }
      }
      __builtin_nontemporal_store(x, reinterpret_cast<u32x4*>(drow));
    } else {
      for (int k = 0; k < kEl; ++k) {
        const int s = run * kEl + k;
        if (s < nvalid) drow[k] = s_v[s * TP + e];
      }
    }
  }
}

}  // namespace dopd
