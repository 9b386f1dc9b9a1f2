// One launch for a PD-aggregated step: the decode of a batch of requests and
// the prefill of a batch of fresh prompts on the same instance, with the
// prompts' paged KV write and their handoff buffer, as workgroups of three
// kinds in one grid (POD-style co-scheduling: a memory-bound decode slice and
// a compute-bound prefill item can share a CU).
//
// Block ranges of the grid, in the order the host chose (schedule):
//   [wp_first, + n_wp)  write + pack: (logical page, KV head) of the prompts
//   [pf_first, + n_pf)  prefill items (the XCD-aware order of the prefill
//                       kernel; pf_first is a multiple of the XCD count so a
//                       block's XCD is the one the order assumes)
//   [dec_first, + n_dec) decode slices (the decode partition's workgroups)
// KV8: the decode reads E4M3 pages and the write + pack quantises the fresh
// rows to E4M3 codes with one scale per KV head (the prefill reads the bf16
// fresh rows either way).
// The three kinds touch disjoint memory: the decode reads the pages of the
// decode requests, the write fills the pages of the prompts, the prefill
// reads only the fresh rows.  The decode's split-K partials are merged by the
// decode merge kernel launched after this one on the same stream.
//
// LDS: the prefill's K/V tile buffers (separate arrays, as in the prefill
// kernel); the decode's wave merge and the writer's V staging reuse them.
#pragma once
#include "decode_bf16.hpp"
#include "kv_write_pack.hpp"
#include "prefill_bf16.hpp"

namespace dopd {

struct PdStepArgs {
  DecodeArgs dec;
  PrefillArgs pf;
  WritePackArgs wp;
  int wp_first, n_wp;    // write + pack blocks (n_wp = pages x Hkv)
  int pf_first, n_pf;    // prefill blocks
  int dec_first, n_dec;  // decode blocks (n_dec = dec.nwg)
};

template <int D, bool KV8 = false>
__global__ __launch_bounds__(kPfThreads, 2) void pd_step_kernel(PdStepArgs s) {
  __shared__ __attribute__((aligned(16))) uint16_t sK0[pf_tile_elems<D>()], sK1[pf_tile_elems<D>()];
  __shared__ __attribute__((aligned(16))) uint16_t sV0[pf_tile_elems<D>()], sV1[pf_tile_elems<D>()];
  __shared__ __attribute__((aligned(16))) uint16_t sQ[pf_q_lds_elems<D, false>()];
  static_assert(2 * dec_wave_o_bytes<D>() <= (int)sizeof(sK0) &&
                    dec_wave_o_bytes<D>() <= (int)sizeof(sK1) && kDecMlBytes <= (int)sizeof(sQ),
                "decode merge buffers fit the prefill tiles");
  static_assert(kPage * (D + 8) * 2 <= (int)sizeof(sV0), "writer staging fits a V tile");
  const int b = blockIdx.x;
  if (b >= s.pf_first && b < s.pf_first + s.n_pf) {
    prefill_workgroup<D, false>(s.pf, b - s.pf_first, sK0, sK1, sV0, sV1, sQ);
  } else if (b >= s.dec_first && b < s.dec_first + s.n_dec) {
    constexpr int kWaveElems = dec_wave_o_bytes<D>() / 2;  // bf16 elements of one block
    decode_workgroup<D, KV8>(s.dec, b - s.dec_first, reinterpret_cast<float*>(sQ),
                               reinterpret_cast<f32x4*>(sK0),
                               reinterpret_cast<f32x4*>(sK0 + kWaveElems),
                               reinterpret_cast<f32x4*>(sK1));
  } else if (b >= s.wp_first && b < s.wp_first + s.n_wp) {
    const int j = b - s.wp_first;
    if constexpr (KV8)
      kv_write_pack_e4m3_workgroup<D>(s.wp, j / s.wp.hkv, j % s.wp.hkv, reinterpret_cast<uint8_t*>(sV0));
    else
      kv_write_pack_workgroup<D>(s.wp, j / s.wp.hkv, j % s.wp.hkv, sV0);
  }
}

}  // namespace dopd
