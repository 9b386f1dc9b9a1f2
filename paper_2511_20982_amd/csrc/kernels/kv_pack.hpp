// Handoff packer: gathers each request's pages into one contiguous buffer in
// (layer, K/V, head, token, dim) order.
//
// The work is a list of blocks, one per (handoff n, z, page pg) with
// z = (layer * 2 + kv) * Hkv + head, pages fastest, then z, then handoffs;
// a block is one page of one head: 16 tokens x D elements.  A workgroup
// takes PER consecutive blocks (consecutive pages of one (n, z), so its
// output is one contiguous run).  Every thread first issues all of its
// 16-byte loads for the workgroup's blocks, so each workgroup keeps PER
// blocks in flight (few workgroups, each with many loads: a small pack is
// bounded by how fast workgroups start, not by HBM); the blocks go to LDS
// token-major (V pages transposed from [D][16] on the way in) and leave as
// 16-byte token-row chunks.
#pragma once
#include "common.hpp"

namespace dopd {

template <typename T>
struct PackArgs {
  const T* k_pool;            // [layers][P][Hkv][16][D]
  const T* v_pool;            // [layers][P][Hkv][D][16]
  int num_pages;
  const int32_t* page_table;  // [..][pt_stride]
  int pt_stride;
  const int32_t* req_ids;     // [nhand] page-table rows
  const int32_t* seq_lens;    // [nhand]
  const int64_t* out_off;     // [nhand] element offsets of each handoff's block
  int hkv, nz, nhand;         // nz = layers * 2 * Hkv
  int nblocks;                // nz * sum_n ceil(len_n / 16)
  T* out;
};

// Blocks of one workgroup, kept in LDS: source page block, destination,
// tokens present, K or V.
template <typename T>
struct PackBlock {
  const T* src;
  T* dst;
  int nvalid;  // 0: no block
  int is_v;
};

// Blocks per workgroup: 16 KiB of blocks (4 bf16 pages of a head at D = 128;
// measured against 4, 8, 32 and 64 KiB on the 1- and 28-layer handoffs).
constexpr int kPackBytesPerWg = 16384;
template <typename T, int D>
constexpr int pack_blocks_per_wg() {
  return kPackBytesPerWg >= kPage * D * (int)sizeof(T) ? kPackBytesPerWg / (kPage * D * (int)sizeof(T)) : 1;
}

template <typename T, int D, int PER>
__global__ __launch_bounds__(256) void kv_pack_kernel(PackArgs<T> a) {
  constexpr int C = D * (int)sizeof(T);      // 16-byte chunks per block
  constexpr int NPT = (PER * C + 255) / 256;  // chunks per thread
  constexpr int EL = 16 / (int)sizeof(T);     // elements per chunk
  constexpr int CPR = D / EL;                 // chunks per token row
  __shared__ __attribute__((aligned(16))) T sb[PER * kPage * D];
  __shared__ PackBlock<T> meta[PER];
  const int tid = threadIdx.x;
  const int b0 = (int)blockIdx.x * PER;

  if (tid < 64) {  // wave 0 places the workgroup's blocks
    auto count = [&](int n) { return a.nz * ((a.seq_lens[n] + kPage - 1) / kPage); };
    int n, i;
    const bool found = find_owner(b0, a.nhand, count, n, i);  // uniform; b0 < nblocks
    if (tid < PER) {
      PackBlock<T> m{nullptr, nullptr, 0, 0};
      if (found && b0 + tid < a.nblocks) {
        i += tid;
        int len = a.seq_lens[n];
        int np = (len + kPage - 1) / kPage;
        while (i >= a.nz * np) {  // the block lies in a later handoff
          i -= a.nz * np;
          ++n;
          len = a.seq_lens[n];
          np = (len + kPage - 1) / kPage;
        }
        const int z = i / np, pg = i % np;
        const int layer = z / (2 * a.hkv), kv = (z / a.hkv) % 2, h = z % a.hkv;
        const int64_t page = a.page_table[(int64_t)a.req_ids[n] * a.pt_stride + pg];
        const int64_t blk = (((int64_t)layer * a.num_pages + page) * a.hkv + h) * (kPage * D);
        m.src = (kv ? a.v_pool : a.k_pool) + blk;
        m.dst = a.out + a.out_off[n] + ((int64_t)z * len + (int64_t)pg * kPage) * D;
        m.nvalid = min(kPage, len - pg * kPage);
        m.is_v = kv;
      }
      meta[tid] = m;
    }
  }
  __syncthreads();

  u32x4 x[NPT];
#pragma unroll
  for (int k = 0; k < NPT; ++k) {
    const int c = tid + 256 * k;
    const int j = c / C;  // wave-uniform
    if (c < PER * C && meta[j].nvalid > 0)
      x[k] = reinterpret_cast<const u32x4*>(meta[j].src)[c % C];
  }
  // Into LDS token-major: K chunks as they are, V chunks (EL tokens of one
  // dim) scattered to their token rows.
#pragma unroll
  for (int k = 0; k < NPT; ++k) {
    const int c = tid + 256 * k;
    const int j = c / C, cc = c % C;
    if (c >= PER * C || meta[j].nvalid == 0) continue;
    if (!meta[j].is_v) {
      reinterpret_cast<u32x4*>(sb)[c] = x[k];
    } else {
      const int e = cc * EL / kPage, t0 = cc * EL % kPage;
      const T* xe = reinterpret_cast<const T*>(&x[k]);
      T* s = sb + j * (kPage * D) + e;
#pragma unroll
      for (int u = 0; u < EL; ++u) s[(t0 + u) * D] = xe[u];
    }
  }
  __syncthreads();

#pragma unroll
  for (int k = 0; k < NPT; ++k) {
    const int c = tid + 256 * k;
    const int j = c / C, cc = c % C;
    if (c >= PER * C || cc / CPR >= meta[j].nvalid) continue;  // past the last token
    const u32x4 y = reinterpret_cast<const u32x4*>(sb)[c];
    T* d = meta[j].dst + cc * EL;
    if ((reinterpret_cast<uintptr_t>(d) & 15) == 0) {
      // streaming stores: the packed buffer leaves the caches at once (it
      // goes to another instance), not during the next kernel
      __builtin_nontemporal_store(y, reinterpret_cast<u32x4*>(d));
    } else {
      const T* ye = reinterpret_cast<const T*>(&y);
#pragma unroll
      for (int e = 0; e < EL; ++e) d[e] = ye[e];
    }
  }
}

}  // namespace dopd
