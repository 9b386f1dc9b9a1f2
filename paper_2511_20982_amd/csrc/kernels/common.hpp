// Shared device helpers for the gfx950 attention kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dopd {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kPage = 16;        // tokens per cache page
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t b) { return __uint_as_float(b << 16); }

// fp32 -> bf16 bits, round to nearest even; NaN stays a quiet NaN.
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0u;
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return f32_to_bf16_bits(lo) | (f32_to_bf16_bits(hi) << 16);
}

// ---- OCP E4M3 (1 sign, 4 exponent bits with bias 7, 3 mantissa bits; no
// infinities; largest finite 448) KV-page codes.
// Saturates to [-448, 448] before the conversion (a NaN stays NaN), so the
// hardware conversion only ever rounds (to nearest even) inside the range.
__device__ __forceinline__ float e4m3_saturate(float y) {
  return y > 448.f ? 448.f : (y < -448.f ? -448.f : y);
}

// Four fp32 values -> four E4M3 codes, byte i holding value i.
__device__ __forceinline__ uint32_t e4m3x4_from_f32(float a, float b, float c, float d) {
  int w = __builtin_amdgcn_cvt_pk_fp8_f32(e4m3_saturate(a), e4m3_saturate(b), 0, false);
  w = __builtin_amdgcn_cvt_pk_fp8_f32(e4m3_saturate(c), e4m3_saturate(d), w, true);
  return (uint32_t)w;
}

// Four E4M3 codes (byte i = element i) -> four bf16 as two packed pairs.
// Exact: every E4M3 value is a bf16 value.
__device__ __forceinline__ u32x2 bf16x4_from_e4m3x4(uint32_t w) {
  const bf16x2 lo = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)w, 1.0f, false);
  const bf16x2 hi = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)w, 1.0f, true);
  return u32x2{__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi)};
}

__device__ __forceinline__ int lane_id() { return __lane_id(); }

// Wave-wide inclusive prefix sum (wave64).
__device__ __forceinline__ int wave_inclusive_scan(int x) {
  const int l = lane_id();
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int y = __shfl_up(x, o, 64);
    if (l >= o) x += y;
  }
  return x;
}

// Locates the owner of global item `idx` when request r owns count(r) items,
// laid out request after request.  Every lane of the wave gets the same answer.
// Returns false when idx is past the last item.
template <class CountFn>
__device__ __forceinline__ bool find_owner(int idx, int nreq, CountFn count, int& owner,
                                           int& local) {
  const int l = lane_id();
  int base = 0;
  for (int r0 = 0; r0 < nreq; r0 += 64) {
    const int r = r0 + l;
    const int c = (r < nreq) ? count(r) : 0;
    const int incl = wave_inclusive_scan(c);
    const int total = __shfl(incl, 63, 64);
    if (idx < base + total) {
      const unsigned long long hit = __ballot(idx - base < incl);
      const int ol = __ffsll((long long)hit) - 1;
      const int excl = __shfl(incl - c, ol, 64);
      owner = r0 + ol;
      local = idx - base - excl;
      return true;
    }
    base += total;
  }
  return false;
}

}  // namespace dopd
