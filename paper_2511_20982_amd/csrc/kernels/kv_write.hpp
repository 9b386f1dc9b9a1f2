// Paged KV writer: scatters fresh token-major K/V rows into the page pools.
//   k_pool[page][Hkv][16][d]  (token-major page),  v_pool[page][Hkv][d][16]  (dim-major page)
// One workgroup per (request, touched logical page) x KV head; pure bit copy.
// K rows are copied in 16-byte chunks; the V block is read as whole token rows
// (16-byte loads), transposed through LDS and written as 16-byte runs of
// slots.  Slots of a page outside the written range are never touched.
#pragma once
#include "common.hpp"

namespace dopd {

constexpr int kKvwThreads = 256;

template <typename T, int D>  // T: uint16_t (bf16 bits) or uint32_t (fp32 bits)
__global__ __launch_bounds__(kKvwThreads) void kv_write_kernel(
    const T* __restrict__ k_new, const T* __restrict__ v_new, T* __restrict__ k_pool,
    T* __restrict__ v_pool, const int32_t* __restrict__ page_table, int pt_stride,
    const int32_t* __restrict__ cu_new, const int32_t* __restrict__ start_pos, int nreq, int hkv) {
  constexpr int kEl = 16 / sizeof(T);  // elements per 16-byte chunk
  constexpr int CPR = D / kEl;         // chunks per token row
  constexpr int TP = D + kEl;          // padded LDS row (elements)
  __shared__ __attribute__((aligned(16))) T s_v[kPage * TP];

  // Touched logical pages of request r: those holding positions [start, start + n).
  auto touched = [&](int rr) {
    const int n = cu_new[rr + 1] - cu_new[rr];
    if (n <= 0) return 0;
    const int s = start_pos[rr];
    return (s + n - 1) / kPage - s / kPage + 1;
  };
  int r, local;
  if (!find_owner(blockIdx.x, nreq, touched, r, local)) return;  // uniform
  const int h = blockIdx.y;
  const int tid = threadIdx.x;

  const int n = cu_new[r + 1] - cu_new[r];
  const int start = start_pos[r];
  const int lp = start / kPage + local;                 // logical page
  const int p_lo = max(start, lp * kPage);              // first position written in this page
  const int p_hi = min(start + n, lp * kPage + kPage);  // one past the last
  const int s0 = p_lo - lp * kPage, s1 = p_hi - lp * kPage;
  const int64_t page = page_table[(int64_t)r * pt_stride + lp];
  const int64_t src0 = cu_new[r] + (p_lo - start);      // source row of slot s0
  const int64_t row_elems = (int64_t)hkv * D;
  T* kdst = k_pool + (page * hkv + h) * kPage * D;
  T* vdst = v_pool + (page * hkv + h) * D * kPage;

  // K: slot-major rows, chunk per thread; V rows staged in LDS.
  for (int i = tid; i < kPage * CPR; i += kKvwThreads) {
    const int slot = i / CPR, c = i % CPR;
    if (slot >= s0 && slot < s1) {
      const int64_t src = (src0 + slot - s0) * row_elems + (int64_t)h * D;  // source row
      // Streaming (nontemporal) store: the rows are not read again soon, and
      // they leave the caches now instead of being written back while the
      // decode that follows streams the pools.
      __builtin_nontemporal_store(reinterpret_cast<const u32x4*>(k_new + src)[c],
                                  reinterpret_cast<u32x4*>(kdst + slot * D) + c);
      *reinterpret_cast<u32x4*>(&s_v[slot * TP + c * kEl]) =
          reinterpret_cast<const u32x4*>(v_new + src)[c];
    }
  }
  __syncthreads();
  // V^T: dim row e holds the page's 16 slots; a thread writes one 16-byte run.
  constexpr int RUNS = kPage / kEl;  // 16-byte runs per dim row
  const bool full = (s0 == 0 && s1 == kPage);
  for (int i = tid; i < D * RUNS; i += kKvwThreads) {
    const int e = i / RUNS, run = i % RUNS;
    T* drow = vdst + e * kPage + run * kEl;
    if (full) {
      u32x4 x;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        if constexpr (sizeof(T) == 2) {
          const int s = run * kEl + 2 * w;
          x[w] = (uint32_t)s_v[s * TP + e] | ((uint32_t)s_v[(s + 1) * TP + e] << 16);
        } else {
          x[w] = s_v[(run * kEl + w) * TP + e];
        }
      }
      *reinterpret_cast<u32x4*>(drow) = x;
    } else {
      for (int k = 0; k < kEl; ++k) {
        const int s = run * kEl + k;
        if (s >= s0 && s < s1) drow[k] = s_v[s * TP + e];
      }
    }
  }
}

// FP8 variant: the same placement, with each bf16 element x of KV head h
// stored as the E4M3 code of sat(x * fp32(1 / scale[h])) (product in fp32,
// rounded to nearest even; codes rounded to nearest even).  Pools hold one
// byte per element.  K rows: 8 elements (16 bytes in, 8 out) per thread; the
// V codes are staged in LDS and written as dim rows of 16 slots (16 bytes).
template <int D>
__global__ __launch_bounds__(kKvwThreads) void kv_write_e4m3_kernel(
    const uint16_t* __restrict__ k_new, const uint16_t* __restrict__ v_new,
    const float* __restrict__ k_scale, const float* __restrict__ v_scale,
    uint8_t* __restrict__ k_pool, uint8_t* __restrict__ v_pool,
    const int32_t* __restrict__ page_table, int pt_stride, const int32_t* __restrict__ cu_new,
    const int32_t* __restrict__ start_pos, int nreq, int hkv) {
  constexpr int CPR = D / 8;  // 8-element chunks per token row
  constexpr int TP = D + 8;   // padded LDS row (bytes)
  __shared__ __attribute__((aligned(16))) uint8_t s_v[kPage * TP];

  auto touched = [&](int rr) {
    const int n = cu_new[rr + 1] - cu_new[rr];
    if (n <= 0) return 0;
    const int s = start_pos[rr];
    return (s + n - 1) / kPage - s / kPage + 1;
  };
  int r, local;
  if (!find_owner(blockIdx.x, nreq, touched, r, local)) return;  // uniform
  const int h = blockIdx.y;
  const int tid = threadIdx.x;

  const int n = cu_new[r + 1] - cu_new[r];
  const int start = start_pos[r];
  const int lp = start / kPage + local;
  const int p_lo = max(start, lp * kPage);
  const int p_hi = min(start + n, lp * kPage + kPage);
  const int s0 = p_lo - lp * kPage, s1 = p_hi - lp * kPage;
  const int64_t page = page_table[(int64_t)r * pt_stride + lp];
  const int64_t src0 = cu_new[r] + (p_lo - start);
  const int64_t row_elems = (int64_t)hkv * D;
  uint8_t* kdst = k_pool + (page * hkv + h) * kPage * D;
  uint8_t* vdst = v_pool + (page * hkv + h) * D * kPage;
  const float kinv = 1.0f / k_scale[h], vinv = 1.0f / v_scale[h];

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
  for (int i = tid; i < kPage * CPR; i += kKvwThreads) {
    const int slot = i / CPR, c = i % CPR;
    if (slot >= s0 && slot < s1) {
      const int64_t src = (src0 + slot - s0) * row_elems + (int64_t)h * D;
      reinterpret_cast<u32x2*>(kdst + slot * D)[c] =
          codes8(reinterpret_cast<const u32x4*>(k_new + src)[c], kinv);
      *reinterpret_cast<u32x2*>(&s_v[slot * TP + c * 8]) =
          codes8(reinterpret_cast<const u32x4*>(v_new + src)[c], vinv);
    }
  }
  __syncthreads();
  // V^T: dim row e holds the page's 16 slots, one 16-byte run.
  const bool full = (s0 == 0 && s1 == kPage);
  for (int e = tid; e < D; e += kKvwThreads) {
    uint8_t* drow = vdst + e * kPage;
    if (full) {
      u32x4 x;
#pragma unroll
      for (int w = 0; w < 4; ++w)
        x[w] = (uint32_t)s_v[(4 * w) * TP + e] | ((uint32_t)s_v[(4 * w + 1) * TP + e] << 8) |
               ((uint32_t)s_v[(4 * w + 2) * TP + e] << 16) |
               ((uint32_t)s_v[(4 * w + 3) * TP + e] << 24);
      *reinterpret_cast<u32x4*>(drow) = x;
    } else {
      for (int s = s0; s < s1; ++s) drow[s] = s_v[s * TP + e];
    }
  }
}

}  // namespace dopd
