// fp32 attention (prefill and decode): one wave per (query row, head), lanes
// split the head dimension, keys are visited in order with an online softmax
// in fp32.  Used for the fp32 parity configuration; the bf16 paths are the
// performance paths.
#pragma once
#include "common.hpp"

namespace dopd {

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

// Attends one query row held as q[e = lane + 64*i] against n keys.
// key(j, i) / val(j, i) return element lane + 64*i of key/value j.
template <int D, class KeyFn, class ValFn>
__device__ __forceinline__ void attend_row_f32(const float (&qv)[D / 64], int n, float scale,
                                               KeyFn key, ValFn val, float (&o)[D / 64],
                                               float& lse_out) {
  float m = -INFINITY, l = 0.f;
#pragma unroll
  for (int i = 0; i < D / 64; ++i) o[i] = 0.f;
  for (int j = 0; j < n; ++j) {
    float part = 0.f;
#pragma unroll
    for (int i = 0; i < D / 64; ++i) part += qv[i] * key(j, i);
    const float s = wave_sum(part) * scale;
    const float m_new = fmaxf(m, s);
    const float alpha = expf(m - m_new);
    const float p = expf(s - m_new);
    l = l * alpha + p;
#pragma unroll
    for (int i = 0; i < D / 64; ++i) o[i] = o[i] * alpha + p * val(j, i);
    m = m_new;
  }
  const float inv = 1.f / l;
#pragma unroll
  for (int i = 0; i < D / 64; ++i) o[i] *= inv;
  lse_out = m + logf(l);
}

// Causal varlen prefill, fp32.  Grid: (T, Hq); block: 64.
template <int D>
__global__ __launch_bounds__(64) void prefill_f32_kernel(
    const float* __restrict__ q, const float* __restrict__ k, const float* __restrict__ v,
    float* __restrict__ out, float* __restrict__ lse, const int32_t* __restrict__ cu, int nreq,
    int hq, int hkv, float scale) {
  const int t = blockIdx.x, h = blockIdx.y, lane = lane_id();
  int lo = 0, hi = nreq;  // request r with cu[r] <= t < cu[r+1]
  while (hi - lo > 1) {
    const int mid = (lo + hi) / 2;
    if (cu[mid] <= t) lo = mid; else hi = mid;
  }
  const int r = lo;
  const int base = cu[r], i = t - base;
  const int c = h / (hq / hkv);
  float qv[D / 64], o[D / 64], ls;
#pragma unroll
  for (int x = 0; x < D / 64; ++x) qv[x] = q[((int64_t)t * hq + h) * D + lane + 64 * x];
  auto key = [&](int j, int x) { return k[((int64_t)(base + j) * hkv + c) * D + lane + 64 * x]; };
  auto val = [&](int j, int x) { return v[((int64_t)(base + j) * hkv + c) * D + lane + 64 * x]; };
  attend_row_f32<D>(qv, i + 1, scale, key, val, o, ls);
#pragma unroll
  for (int x = 0; x < D / 64; ++x) out[((int64_t)t * hq + h) * D + lane + 64 * x] = o[x];
  if (lse && lane == 0) lse[(int64_t)t * hq + h] = ls;
}

// Paged single-query decode, fp32.  Grid: (B, Hq); block: 64.
template <int D>
__global__ __launch_bounds__(64) void decode_f32_kernel(
    const float* __restrict__ q, const float* __restrict__ k_pool,
    const float* __restrict__ v_pool, const int32_t* __restrict__ page_table, int pt_stride,
    const int32_t* __restrict__ ctx_lens, int hq, int hkv, float scale, float* __restrict__ out,
    float* __restrict__ lse) {
  const int r = blockIdx.x, h = blockIdx.y, lane = lane_id();
  const int c = h / (hq / hkv);
  const int n = ctx_lens[r];
  const int32_t* pt = page_table + (int64_t)r * pt_stride;
  float qv[D / 64], o[D / 64], ls;
#pragma unroll
  for (int x = 0; x < D / 64; ++x) qv[x] = q[((int64_t)r * hq + h) * D + lane + 64 * x];
  auto key = [&](int j, int x) {
    const int64_t page = pt[j / kPage];
    return k_pool[((page * hkv + c) * kPage + j % kPage) * D + lane + 64 * x];
  };
  auto val = [&](int j, int x) {
    const int64_t page = pt[j / kPage];
    return v_pool[((page * hkv + c) * D + lane + 64 * x) * kPage + j % kPage];
  };
  attend_row_f32<D>(qv, n, scale, key, val, o, ls);
#pragma unroll
  for (int x = 0; x < D / 64; ++x) out[((int64_t)r * hq + h) * D + lane + 64 * x] = o[x];
  if (lse && lane == 0) lse[(int64_t)r * hq + h] = ls;
}

// Chunk prefill over the paged cache, fp32: chunk token i of request r (query
// row cu[r] + i) attends to cached positions 0 .. prefix[r] + i.  Grid: (T, Hq).
template <int D>
__global__ __launch_bounds__(64) void prefill_paged_f32_kernel(
    const float* __restrict__ q, const float* __restrict__ k_pool,
    const float* __restrict__ v_pool, const int32_t* __restrict__ page_table, int pt_stride,
    const int32_t* __restrict__ cu, const int32_t* __restrict__ prefix, int nreq, int hq,
    int hkv, float scale, float* __restrict__ out, float* __restrict__ lse) {
  const int t = blockIdx.x, h = blockIdx.y, lane = lane_id();
  int lo = 0, hi = nreq;  // request r with cu[r] <= t < cu[r+1]
  while (hi - lo > 1) {
    const int mid = (lo + hi) / 2;
    if (cu[mid] <= t) lo = mid; else hi = mid;
  }
  const int r = lo;
  const int n = prefix[r] + (t - cu[r]) + 1;
  const int c = h / (hq / hkv);
  const int32_t* pt = page_table + (int64_t)r * pt_stride;
  float qv[D / 64], o[D / 64], ls;
#pragma unroll
  for (int x = 0; x < D / 64; ++x) qv[x] = q[((int64_t)t * hq + h) * D + lane + 64 * x];
  auto key = [&](int j, int x) {
    const int64_t page = pt[j / kPage];
    return k_pool[((page * hkv + c) * kPage + j % kPage) * D + lane + 64 * x];
  };
  auto val = [&](int j, int x) {
    const int64_t page = pt[j / kPage];
    return v_pool[((page * hkv + c) * D + lane + 64 * x) * kPage + j % kPage];
  };
  attend_row_f32<D>(qv, n, scale, key, val, o, ls);
#pragma unroll
  for (int x = 0; x < D / 64; ++x) out[((int64_t)t * hq + h) * D + lane + 64 * x] = o[x];
  if (lse && lane == 0) lse[(int64_t)t * hq + h] = ls;
}

}  // namespace dopd
