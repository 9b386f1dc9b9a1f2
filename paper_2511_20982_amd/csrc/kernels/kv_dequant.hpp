// Dequantises the E4M3 cache pages a chunk prefill reads into bf16 pages.
//
// Every E4M3 value is a bf16 value, so the bf16 pages hold the codes' values
// exactly; the per-KV-head scales are not applied here (the prefill folds the
// K scale into its softmax scale and the V scale into its output).  The pages
// of request r (logical pages 0 .. ceil((prefix_r + n_r) / 16) - 1, nothing
// for an empty chunk) are packed in call order, and the page table of the
// packed pages is written beside them.  One workgroup per (packed page, KV
// head); 8 codes -> 8 bf16 per thread and iteration, both page layouts
// element for element.
#pragma once
#include "common.hpp"

namespace dopd {

struct DequantArgs {
  const uint8_t* k_pool;      // [P][Hkv][16][D] E4M3 codes
  const uint8_t* v_pool;      // [P][Hkv][D][16]
  const int32_t* page_table;  // [nreq][pt_stride]
  int pt_stride;
  const int32_t* cu;          // [nreq + 1] chunk rows
  const int32_t* prefix;      // [nreq] cached tokens before the chunk
  int nreq, hkv;
  uint16_t* k_out;            // [pages][Hkv][16][D] bf16
  uint16_t* v_out;            // [pages][Hkv][D][16]
  int32_t* pt_out;            // [nreq][pt_out_stride]: packed page of logical page i
  int pt_out_stride;
};

template <int D>
__global__ __launch_bounds__(256) void kv_dequant_pages_kernel(DequantArgs a) {
  const int j = (int)blockIdx.x / a.hkv, h = (int)blockIdx.x % a.hkv;
  auto pages = [&](int rr) {
    const int n = a.cu[rr + 1] - a.cu[rr];
    return n > 0 ? (a.prefix[rr] + n + kPage - 1) / kPage : 0;
  };
  int r, i;
  if (!find_owner(j, a.nreq, pages, r, i)) return;  // uniform
  const int64_t src = a.page_table[(int64_t)r * a.pt_stride + i];
  if (h == 0 && threadIdx.x == 0) a.pt_out[(int64_t)r * a.pt_out_stride + i] = j;
  constexpr int kElems = kPage * D;  // one page-head block
  const uint8_t* ks = a.k_pool + (src * a.hkv + h) * kElems;
  const uint8_t* vs = a.v_pool + (src * a.hkv + h) * kElems;
  uint16_t* kd = a.k_out + ((int64_t)j * a.hkv + h) * kElems;
  uint16_t* vd = a.v_out + ((int64_t)j * a.hkv + h) * kElems;
  for (int e = 8 * (int)threadIdx.x; e < kElems; e += 8 * 256) {
    const u32x2 kc = *reinterpret_cast<const u32x2*>(ks + e);
    const u32x2 vc = *reinterpret_cast<const u32x2*>(vs + e);
    const u32x2 k0 = bf16x4_from_e4m3x4(kc[0]), k1 = bf16x4_from_e4m3x4(kc[1]);
    const u32x2 v0 = bf16x4_from_e4m3x4(vc[0]), v1 = bf16x4_from_e4m3x4(vc[1]);
    *reinterpret_cast<u32x4*>(kd + e) = u32x4{k0[0], k0[1], k1[0], k1[1]};
    *reinterpret_cast<u32x4*>(vd + e) = u32x4{v0[0], v0[1], v1[0], v1[1]};
  }
}

}  // namespace dopd
