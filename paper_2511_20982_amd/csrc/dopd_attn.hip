// C ABI of the gfx950 attention hot path (declarations and contracts in
// include/dopd_attn.h).  Host side: argument validation before any HIP call,
// launch planning from the host copies of the lengths, launches on the
// caller's stream.  No allocation, no synchronisation, no state.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstring>
#include <mutex>

#include "dopd_attn.h"
#include "kernels/attn_f32.hpp"
#include "kernels/common.hpp"
#include "kernels/decode_bf16.hpp"
#include "kernels/kv_pack.hpp"
#include "kernels/kv_unpack.hpp"
#include "kernels/kv_write.hpp"
#include "kernels/kv_write_pack.hpp"
#include "kernels/pd_step.hpp"
#include "kernels/prefill_bf16.hpp"
#include "plan.hpp"

namespace {

thread_local int32_t g_last_hip_error = 0;

dopd_status hip_status(hipError_t e) {
  if (e == hipSuccess) return DOPD_OK;
  g_last_hip_error = (int32_t)e;
  return DOPD_ERR_HIP;
}

dopd_status launch_status() { return hip_status(hipGetLastError()); }

hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

// Checks the parts of the shape every entry point relies on.
dopd_status check_shape(const dopd_attn_shape* s) {
  if (!s) return DOPD_ERR_NULL_POINTER;
  if (s->num_q_heads <= 0 || s->num_kv_heads <= 0 || s->num_q_heads % s->num_kv_heads != 0)
    return DOPD_ERR_INVALID_SHAPE;
  if (s->head_dim != 64 && s->head_dim != 128) return DOPD_ERR_UNSUPPORTED;
  if (s->page_size != dopd::kPage) return DOPD_ERR_UNSUPPORTED;
  if (s->dtype != DOPD_BF16 && s->dtype != DOPD_FP32 && s->dtype != DOPD_FP8_E4M3)
    return DOPD_ERR_UNSUPPORTED;
  return DOPD_OK;
}

// Entry points whose pools hold bf16 or fp32 only.
dopd_status check_shape_no_fp8(const dopd_attn_shape* s) {
  const dopd_status st = check_shape(s);
  if (st != DOPD_OK) return st;
  return s->dtype == DOPD_FP8_E4M3 ? DOPD_ERR_UNSUPPORTED : DOPD_OK;
}


// ---- machine shape ----------------------------------------------------------
// CU and XCD counts of each device, read once (hipDeviceGetAttribute) the
// first time a call plans a launch on it with that device current.
constexpr int kMaxDevices = 64;
std::once_flag g_machine_once[kMaxDevices];
dopd::MachineShape g_machine[kMaxDevices];

dopd::MachineShape machine_shape() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();  // no device: host-side sizing only
    return dopd::kDefaultMachine;
  }
  std::call_once(g_machine_once[dev], [dev] {
    int cus = 0, xcds = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus <= 0)
      cus = dopd::kDefaultMachine.cus;
    if (hipDeviceGetAttribute(&xcds, hipDeviceAttributeNumberOfXccs, dev) != hipSuccess ||
        xcds <= 0 || cus % xcds != 0)
      xcds = 1;  // unknown: one dispatch order (correct, not XCD-aware)
    (void)hipGetLastError();
    g_machine[dev] = dopd::MachineShape{cus, xcds};
  });
  return g_machine[dev];
}

// ---- static decode scratch (dopd_decode_attn_noalloc) ------------------------
// The split-K partials of dopd_decode_attn_noalloc live in this file-scope
// device array instead of a caller's workspace; every device the library runs
// on holds its own copy until the process ends.  In host code `scratch` is
// only a stand-in for the symbol: the device address comes from
// hipGetSymbolAddress, once per device with that device current.
static __device__ __align__(256) unsigned char scratch[DOPD_DECODE_NOALLOC_SCRATCH_BYTES];

std::once_flag g_scratch_once[kMaxDevices];
void* g_scratch_ptr[kMaxDevices];
hipError_t g_scratch_err[kMaxDevices];

// Device address of the current device's scratch array.
dopd_status scratch_address(void** ptr) {
  int dev = -1;
  const hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_status(e);
  if (dev < 0 || dev >= kMaxDevices) return DOPD_ERR_INVALID_SHAPE;
  std::call_once(g_scratch_once[dev], [dev] {
    g_scratch_err[dev] = hipGetSymbolAddress(&g_scratch_ptr[dev], HIP_SYMBOL(scratch));
  });
  if (g_scratch_err[dev] != hipSuccess) return hip_status(g_scratch_err[dev]);
  *ptr = g_scratch_ptr[dev];
  return DOPD_OK;
}

// ---- decode planning --------------------------------------------------------
constexpr int kMaxGroupBf16 = 16;   // query heads per KV head handled by one decode wave

dopd_status check_decode_host(const dopd_attn_shape* s, const int32_t* ctx_host, int32_t n,
                              int32_t split) {
  dopd_status st = check_shape(s);
  if (st != DOPD_OK) return st;
  if (n < 0) return DOPD_ERR_INVALID_SHAPE;
  if (n > 0 && !ctx_host) return DOPD_ERR_NULL_POINTER;
  for (int32_t r = 0; r < n; ++r)
    if (ctx_host[r] < 1) return DOPD_ERR_INVALID_SHAPE;
  if (split < 0 || (split > 0 && split % 32 != 0) || split > dopd::kDecMaxSplitTokens)
    return DOPD_ERR_INVALID_SHAPE;
  if (s->dtype != DOPD_FP32 && s->num_q_heads / s->num_kv_heads > kMaxGroupBf16)
    return DOPD_ERR_UNSUPPORTED;
  return DOPD_OK;
}

// How the decode's partials are merged: not at all (every (request, KV head)
// is one segment), by the kernel over the listed (r, c) (count > 0), or by
// the kernel that finds them itself (the list does not fit its arguments).
struct DecodeMergePlan {
  bool needed = false;
  int count = 0;
  dopd::DecodeMergeList list;
};

// Decode arguments and workspace layout of the bf16-operand decode (bf16 or
// E4M3 pools) after the host checks; quarter_wgs: resident decode workgroups
// per CU, in quarters, the automatic partition plans for.
template <bool KV8>
dopd_status plan_decode_bf16(const dopd_attn_shape* s, const void* q, const void* k_pool,
                             const void* v_pool, const float* k_scale, const float* v_scale,
                             const int32_t* pt, int32_t pt_stride, const int32_t* ctx,
                             const int32_t* ctx_host, int32_t nreq, int32_t split_tokens,
                             void* out, float* lse, void* workspace, size_t workspace_bytes,
                             int quarter_wgs, dopd::DecodeArgs* a_out,
                             DecodeMergePlan* merge_out) {
  const int hkv = s->num_kv_heads, hq = s->num_q_heads, d = s->head_dim;
  const int64_t total = dopd::decode_total_units(ctx_host, nreq, hkv);
  if (total > INT32_MAX / 2) return DOPD_ERR_INVALID_SHAPE;
  const dopd::DecodeLayout L = dopd::decode_layout(hq / hkv, hkv, d, ctx_host, nreq,
                                                   split_tokens, machine_shape(), quarter_wgs);
  const int64_t nwg = L.nwg;
  if (!workspace) return DOPD_ERR_NULL_POINTER;
  if (workspace_bytes < L.total) return DOPD_ERR_WORKSPACE_TOO_SMALL;
  if ((reinterpret_cast<uintptr_t>(workspace) & 255) != 0) return DOPD_ERR_INVALID_SHAPE;
  char* ws = static_cast<char*>(workspace);
  merge_out->count = dopd::decode_merge_list(ctx_host, nreq, hkv, total, nwg,
                                              merge_out->list.item, dopd::kMergeListMax);
  merge_out->list.n = std::max(0, merge_out->count);
  merge_out->needed = merge_out->count > 0 ||
                      (merge_out->count < 0 && dopd::decode_needs_merge(ctx_host, nreq, hkv, total, nwg));
  dopd::DecodeArgs& a = *a_out;
  a.q = (const uint16_t*)q;
  a.k_pool = k_pool;
  a.v_pool = v_pool;
  a.k_scale = k_scale;
  a.v_scale = v_scale;
  a.page_table = pt;
  a.ctx_lens = ctx;
  a.out = (uint16_t*)out;
  a.lse = lse;
  a.part_o = reinterpret_cast<float*>(ws + L.part_o_off);
  a.part_ml = reinterpret_cast<float*>(ws + L.part_ml_off);
  a.pt_stride = pt_stride;
  a.nreq = nreq;
  a.hq = hq;
  a.hkv = hkv;
  a.total_units = (int)total;
  a.nwg = (int)nwg;
  a.scale_log2 = s->softmax_scale * dopd::kLog2e;
  return DOPD_OK;
}

// The decode's second kernel: merges the (request, KV head) pairs whose keys
// span several slices (nothing to launch when there are none).
dopd_status launch_decode_merge(const dopd::DecodeArgs& a, const DecodeMergePlan& m, int d,
                                hipStream_t strm) {
  if (!m.needed) return DOPD_OK;
  if (m.count > 0) {
    if (d == 64)
      hipLaunchKernelGGL(dopd::decode_merge_list_kernel<64>, dim3((unsigned)m.count), dim3(256), 0,
                         strm, a, m.list);
    else
      hipLaunchKernelGGL(dopd::decode_merge_list_kernel<128>, dim3((unsigned)m.count), dim3(256), 0,
                         strm, a, m.list);
    return launch_status();
  }
  const unsigned items = (unsigned)((int64_t)a.nreq * a.hkv);
  if (d == 64)
    hipLaunchKernelGGL(dopd::decode_merge_kernel<64>, dim3(items), dim3(256), 0, strm, a);
  else
    hipLaunchKernelGGL(dopd::decode_merge_kernel<128>, dim3(items), dim3(256), 0, strm, a);
  return launch_status();
}

// The bf16-operand decode after the host checks: plan the partition, check the
// workspace, launch the split kernel and, when some (request, KV head) spans
// two slices, the merge kernel.
template <bool KV8>
dopd_status launch_decode_bf16(const dopd_attn_shape* s, const void* q, const void* k_pool,
                               const void* v_pool, const float* k_scale, const float* v_scale,
                               const int32_t* pt, int32_t pt_stride, const int32_t* ctx,
                               const int32_t* ctx_host, int32_t nreq, int32_t split_tokens,
                               void* out, float* lse, void* workspace, size_t workspace_bytes,
                               hipStream_t strm) {
  dopd::DecodeArgs a;
  DecodeMergePlan merge;
  const dopd_status pst = plan_decode_bf16<KV8>(s, q, k_pool, v_pool, k_scale, v_scale, pt,
                                                pt_stride, ctx, ctx_host, nreq, split_tokens,
                                                out, lse, workspace, workspace_bytes,
                                                4 * dopd::kWgPerCu, &a, &merge);
  if (pst != DOPD_OK) return pst;
  if (s->head_dim == 64)
    hipLaunchKernelGGL((dopd::decode_split_kernel<64, KV8>), dim3((unsigned)a.nwg), dim3(256), 0, strm, a);
  else
    hipLaunchKernelGGL((dopd::decode_split_kernel<128, KV8>), dim3((unsigned)a.nwg), dim3(256), 0, strm, a);
  const dopd_status st = launch_status();
  if (st != DOPD_OK) return st;
  return launch_decode_merge(a, merge, s->head_dim, strm);
}

}  // namespace

extern "C" {

const char* dopd_status_string(dopd_status status) {
  switch (status) {
    case DOPD_OK: return "ok";
    case DOPD_ERR_NULL_POINTER: return "null pointer argument";
    case DOPD_ERR_INVALID_SHAPE: return "invalid shape, count or length";
    case DOPD_ERR_UNSUPPORTED: return "unsupported dtype, head_dim, page_size or head ratio for this entry point";
    case DOPD_ERR_WORKSPACE_TOO_SMALL: return "workspace too small";
    case DOPD_ERR_HIP: return "HIP launch error";
    default: return "unknown status";
  }
}

int32_t dopd_last_hip_error(void) { return g_last_hip_error; }

dopd_status dopd_validate_page_table_host(const int32_t* pt, int32_t stride, int32_t n,
                                          const int32_t* lens, int32_t num_pages) {
  if (n < 0 || num_pages < 0) return DOPD_ERR_INVALID_SHAPE;
  if (n == 0) return DOPD_OK;
  if (!pt || !lens) return DOPD_ERR_NULL_POINTER;
  for (int32_t r = 0; r < n; ++r) {
    if (lens[r] < 0) return DOPD_ERR_INVALID_SHAPE;
    const int64_t need = ((int64_t)lens[r] + dopd::kPage - 1) / dopd::kPage;
    if (need > stride) return DOPD_ERR_INVALID_SHAPE;
    for (int64_t i = 0; i < need; ++i) {
      const int32_t p = pt[(int64_t)r * stride + i];
      if (p < 0 || p >= num_pages) return DOPD_ERR_INVALID_SHAPE;
    }
  }
  return DOPD_OK;
}

// ---------------------------------------------------------------- prefill
extern "C++" {
namespace {

// Fills the work-order fields of `a` for chunk lengths cu_host (and, on the
// paged path, cached prefixes prefix_host) and returns the prefill's block
// count: items are (q tile, request, head), with at most 64 requests in the
// XCD-aware order (requests ranked by the keys their last row sees, dealt to
// the XCDs in contiguous slices), else heaviest q tile first.
template <bool PAGED>
dopd_status plan_prefill_bf16(dopd::PrefillArgs& a, const int32_t* cu_host,
                              const int32_t* prefix_host, int32_t nreq, int64_t* blocks_out) {
  int max_len = 0;
  int64_t tiles = 0;
  for (int32_t r = 0; r < nreq; ++r) {
    const int len = cu_host[r + 1] - cu_host[r];
    max_len = std::max(max_len, len);
    tiles += (len + dopd::kPfBM - 1) / dopd::kPfBM;
  }
  a.nreq = nreq;
  a.max_tiles = (max_len + dopd::kPfBM - 1) / dopd::kPfBM;
  a.hslots = (a.hq + dopd::kPfHeadsPerWG - 1) / dopd::kPfHeadsPerWG;
  const int64_t items = tiles * a.hslots;
  if (items > INT32_MAX / 2) return DOPD_ERR_INVALID_SHAPE;
  int64_t blocks = items;
  a.xcd_order = 0;
  a.n_items = (int)items;
  a.tiles_total = (int)tiles;
  a.per_xcd = 0;
  a.xcds = 1;
  std::memset(a.ord, 0, sizeof(a.ord));
  if (nreq <= dopd::kPfMaxOrdered) {
    // requests by decreasing key count (stable), dealt to XCDs in contiguous slices
    auto keys = [&](int r) {
      return (int64_t)(cu_host[r + 1] - cu_host[r]) + (PAGED ? prefix_host[r] : 0);
    };
    int order[dopd::kPfMaxOrdered];
    for (int32_t r = 0; r < nreq; ++r) order[r] = r;
    std::stable_sort(order, order + nreq, [&](int x, int y) { return keys(x) > keys(y); });
    for (int32_t r = 0; r < nreq; ++r) a.ord[r] = order[r];
    // slots per block, as the kernel groups them
    const int g = a.hq / a.hkv;
    const int gs = (g % dopd::kPfHeadsPerWG == 0) ? g / dopd::kPfHeadsPerWG : 1;
    int sum = 0;
    for (int32_t i = 0; i < nreq; ++i) {
      const int r = order[i];
      sum += gs * ((cu_host[r + 1] - cu_host[r] + dopd::kPfBM - 1) / dopd::kPfBM);
      a.incl[i] = sum;
    }
    for (int32_t r = 0; r <= nreq; ++r) a.cu_h[r] = cu_host[r];
    for (int32_t r = 0; r < nreq; ++r) a.prefix_h[r] = PAGED ? prefix_host[r] : 0;
    a.xcd_order = 1;
    a.xcds = machine_shape().xcds;
    a.per_xcd = dopd::pf_per_xcd((int)items, a.xcds);
    blocks = (int64_t)a.per_xcd * a.xcds;
  }
  blocks *= a.nsplit;  // (nsplit > 1 only on the paged path)
  if (blocks > INT32_MAX / 2) return DOPD_ERR_INVALID_SHAPE;
  *blocks_out = blocks;
  return DOPD_OK;
}

// Plans and launches the bf16 prefill kernel over chunk lengths cu_host (and,
// on the paged path, the cached prefixes prefix_host).  Work items are
// (q tile, request, head); with at most 64 requests the XCD-aware order is
// used, requests ranked by the keys their last row sees.
template <bool PAGED, bool KV8 = false>
dopd_status launch_prefill_bf16(dopd::PrefillArgs a, int d, const int32_t* cu_host,
                                const int32_t* prefix_host, int32_t nreq, hipStream_t strm) {
  int64_t blocks = 0;
  const dopd_status pst = plan_prefill_bf16<PAGED>(a, cu_host, prefix_host, nreq, &blocks);
  if (pst != DOPD_OK) return pst;
  if (blocks == 0) return DOPD_OK;
  if (d == 64)
    hipLaunchKernelGGL((dopd::prefill_bf16_kernel<64, PAGED, KV8>), dim3((unsigned)blocks),
                       dim3(dopd::kPfThreads), 0, strm, a);
  else
    hipLaunchKernelGGL((dopd::prefill_bf16_kernel<128, PAGED, KV8>), dim3((unsigned)blocks),
                       dim3(dopd::kPfThreads), 0, strm, a);
  const dopd_status st = launch_status();
  if (st != DOPD_OK || a.nsplit == 1) return st;
  const int64_t threads = (int64_t)a.part_rows * a.hq * (d / 4);
  const unsigned merge_blocks = (unsigned)((threads + 255) / 256);
  if (d == 64)
    hipLaunchKernelGGL(dopd::prefill_split_merge_kernel<64>, dim3(merge_blocks), dim3(256), 0, strm, a);
  else
    hipLaunchKernelGGL(dopd::prefill_split_merge_kernel<128>, dim3(merge_blocks), dim3(256), 0, strm, a);
  return launch_status();
}

// Key splits of a paged prefill call on the current device (bf16 with a
// positive scale only: the split bounds assume every row sees its first key).
int paged_splits(const dopd_attn_shape* s, const int32_t* cu_host, const int32_t* prefix_host,
                 int32_t nreq, int32_t num_splits) {
  return dopd::prefill_paged_splits(s->num_q_heads,
                                    s->dtype == DOPD_BF16 && s->softmax_scale > 0.f, cu_host,
                                    prefix_host, nreq, num_splits, machine_shape());
}

dopd::PrefillArgs prefill_args(const dopd_attn_shape* s, const void* q, void* out, float* lse,
                               const int32_t* cu) {
  dopd::PrefillArgs a;
  std::memset(&a, 0, sizeof(a));
  a.q = (const uint16_t*)q;
  a.out = (uint16_t*)out;
  a.lse = lse;
  a.cu = cu;
  a.hq = s->num_q_heads;
  a.hkv = s->num_kv_heads;
  a.scale_log2 = s->softmax_scale * dopd::kLog2e;
  a.nsplit = 1;
  return a;
}

}  // namespace
}  // extern "C++"

size_t dopd_prefill_workspace_size(const dopd_attn_shape* s, const int32_t* cu_host,
                                   int32_t nreq) {
  (void)s;
  (void)cu_host;
  (void)nreq;
  return 0;  // the work list is derived from cu_host and passed by value
}

dopd_status dopd_prefill_attn(const dopd_attn_shape* s, const void* q, const void* k,
                              const void* v, void* out, float* lse, const int32_t* cu,
                              const int32_t* cu_host, int32_t nreq, void* workspace,
                              size_t workspace_bytes, void* stream) {
  (void)workspace_bytes;  // nothing is needed (dopd_prefill_workspace_size is 0)
  dopd_status st = check_shape_no_fp8(s);
  if (st != DOPD_OK) return st;
  if (nreq < 0) return DOPD_ERR_INVALID_SHAPE;
  if ((reinterpret_cast<uintptr_t>(workspace) & 255) != 0) return DOPD_ERR_INVALID_SHAPE;
  if (nreq == 0) return DOPD_OK;
  if (!q || !k || !v || !out || !cu || !cu_host) return DOPD_ERR_NULL_POINTER;
  if (cu_host[0] != 0) return DOPD_ERR_INVALID_SHAPE;
  for (int32_t r = 0; r < nreq; ++r)
    if (cu_host[r + 1] < cu_host[r]) return DOPD_ERR_INVALID_SHAPE;
  const int64_t T = cu_host[nreq];
  if (T == 0) return DOPD_OK;
  const int hq = s->num_q_heads, hkv = s->num_kv_heads, d = s->head_dim;
  hipStream_t strm = as_stream(stream);
  if (s->dtype == DOPD_FP32) {
    dim3 grid((unsigned)T, (unsigned)hq);
    if (d == 64)
      hipLaunchKernelGGL(dopd::prefill_f32_kernel<64>, grid, dim3(64), 0, strm, (const float*)q,
                         (const float*)k, (const float*)v, (float*)out, lse, cu, nreq, hq, hkv,
                         s->softmax_scale);
    else
      hipLaunchKernelGGL(dopd::prefill_f32_kernel<128>, grid, dim3(64), 0, strm, (const float*)q,
                         (const float*)k, (const float*)v, (float*)out, lse, cu, nreq, hq, hkv,
                         s->softmax_scale);
    return launch_status();
  }
  dopd::PrefillArgs a = prefill_args(s, q, out, lse, cu);
  a.k = (const uint16_t*)k;
  a.v = (const uint16_t*)v;
  return launch_prefill_bf16<false>(a, d, cu_host, nullptr, nreq, strm);
}

// dopd_prefill_paged_attn(_split): checks, then the fp32 kernel or the bf16
// kernel with num_splits key splits (1: no workspace needed).
static dopd_status prefill_paged_impl(const dopd_attn_shape* s, const void* q, const void* k_pool,
                               const void* v_pool, int32_t num_pages, const int32_t* page_table,
                               int32_t pt_stride, const int32_t* cu, const int32_t* cu_host,
                               const int32_t* prefix, const int32_t* prefix_host, int32_t nreq,
                               int32_t num_splits, void* out, float* lse, void* workspace,
                               size_t workspace_bytes, void* stream,
                               const float* k_scale = nullptr, const float* v_scale = nullptr,
                               bool kv8 = false) {
  dopd_status st = check_shape_no_fp8(s);
  if (st != DOPD_OK) return st;
  if (nreq < 0 || num_pages < 0 || pt_stride < 0 || num_splits < 0) return DOPD_ERR_INVALID_SHAPE;
  if (nreq == 0) return DOPD_OK;
  if (!q || !k_pool || !v_pool || !page_table || !cu || !cu_host || !prefix || !prefix_host ||
      !out)
    return DOPD_ERR_NULL_POINTER;
  if (cu_host[0] != 0) return DOPD_ERR_INVALID_SHAPE;
  for (int32_t r = 0; r < nreq; ++r) {
    const int64_t n = (int64_t)cu_host[r + 1] - cu_host[r];
    if (n < 0 || prefix_host[r] < 0) return DOPD_ERR_INVALID_SHAPE;
    // every page the request's keys touch must have a page-table column
    if (n > 0 && (prefix_host[r] + n + dopd::kPage - 1) / dopd::kPage > pt_stride)
      return DOPD_ERR_INVALID_SHAPE;
  }
  const int64_t T = cu_host[nreq];
  if (T == 0) return DOPD_OK;
  const int hq = s->num_q_heads, hkv = s->num_kv_heads, d = s->head_dim;
  hipStream_t strm = as_stream(stream);
  if (s->dtype == DOPD_FP32) {
    dim3 grid((unsigned)T, (unsigned)hq);
    if (d == 64)
      hipLaunchKernelGGL(dopd::prefill_paged_f32_kernel<64>, grid, dim3(64), 0, strm,
                         (const float*)q, (const float*)k_pool, (const float*)v_pool, page_table,
                         pt_stride, cu, prefix, nreq, hq, hkv, s->softmax_scale, (float*)out, lse);
    else
      hipLaunchKernelGGL(dopd::prefill_paged_f32_kernel<128>, grid, dim3(64), 0, strm,
                         (const float*)q, (const float*)k_pool, (const float*)v_pool, page_table,
                         pt_stride, cu, prefix, nreq, hq, hkv, s->softmax_scale, (float*)out, lse);
    return launch_status();
  }
  dopd::PrefillArgs a = prefill_args(s, q, out, lse, cu);
  a.k_pool = (const uint16_t*)k_pool;
  a.v_pool = (const uint16_t*)v_pool;
  a.page_table = page_table;
  a.prefix = prefix;
  a.pt_stride = pt_stride;
  a.k_scale = k_scale;
  a.v_scale = v_scale;
  const int nsplit = num_splits == 1 ? 1 : paged_splits(s, cu_host, prefix_host, nreq, num_splits);
  if (nsplit > 1) {
    if (T * hq * (int64_t)nsplit > INT32_MAX / 2) return DOPD_ERR_INVALID_SHAPE;
    if (!workspace) return DOPD_ERR_NULL_POINTER;
    if (workspace_bytes < dopd::prefill_paged_ws_bytes(hq, d, T, nsplit))
      return DOPD_ERR_WORKSPACE_TOO_SMALL;
    if ((reinterpret_cast<uintptr_t>(workspace) & 255) != 0) return DOPD_ERR_INVALID_SHAPE;
    const size_t rows = (size_t)nsplit * T * hq;
    a.nsplit = nsplit;
    a.part_rows = (int)T;
    a.part_o = static_cast<float*>(workspace);
    a.part_ml = reinterpret_cast<float*>(static_cast<char*>(workspace) +
                                         dopd::align256(rows * d * sizeof(float)));
  }
  return kv8 ? launch_prefill_bf16<true, true>(a, d, cu_host, prefix_host, nreq, strm)
             : launch_prefill_bf16<true>(a, d, cu_host, prefix_host, nreq, strm);
}

dopd_status dopd_prefill_paged_attn(const dopd_attn_shape* s, const void* q, const void* k_pool,
                                    const void* v_pool, int32_t num_pages,
                                    const int32_t* page_table, int32_t pt_stride,
                                    const int32_t* cu, const int32_t* cu_host,
                                    const int32_t* prefix, const int32_t* prefix_host,
                                    int32_t nreq, void* out, float* lse, void* stream) {
  return prefill_paged_impl(s, q, k_pool, v_pool, num_pages, page_table, pt_stride, cu, cu_host,
                            prefix, prefix_host, nreq, 1, out, lse, nullptr, 0, stream);
}

size_t dopd_prefill_paged_workspace_size(const dopd_attn_shape* s, const int32_t* cu_host,
                                         const int32_t* prefix_host, int32_t nreq,
                                         int32_t num_splits) {
  if (check_shape_no_fp8(s) != DOPD_OK || nreq < 0 || num_splits < 0) return 0;
  if (nreq == 0) return 256;
  if (!cu_host || !prefix_host || cu_host[0] != 0) return 0;
  for (int32_t r = 0; r < nreq; ++r)
    if (cu_host[r + 1] < cu_host[r] || prefix_host[r] < 0) return 0;
  const int nsplit = num_splits == 1 ? 1 : paged_splits(s, cu_host, prefix_host, nreq, num_splits);
  return std::max<size_t>(256, dopd::prefill_paged_ws_bytes(s->num_q_heads, s->head_dim,
                                                            cu_host[nreq], nsplit));
}

dopd_status dopd_prefill_paged_attn_split(const dopd_attn_shape* s, const void* q,
                                          const void* k_pool, const void* v_pool,
                                          int32_t num_pages, const int32_t* page_table,
                                          int32_t pt_stride, const int32_t* cu,
                                          const int32_t* cu_host, const int32_t* prefix,
                                          const int32_t* prefix_host, int32_t nreq,
                                          int32_t num_splits, void* out, float* lse,
                                          void* workspace, size_t workspace_bytes, void* stream) {
  return prefill_paged_impl(s, q, k_pool, v_pool, num_pages, page_table, pt_stride, cu, cu_host,
                            prefix, prefix_host, nreq, num_splits, out, lse, workspace,
                            workspace_bytes, stream);
}

// ---------------------------------------------------------------- E4M3 chunk prefill
// The paged prefill over E4M3 pools: the same work list and workspace (split
// partials only) as the bf16 pools; the kernel widens the codes as they leave
// LDS.
extern "C++" {
namespace {
dopd_attn_shape as_bf16(const dopd_attn_shape* s) {
  dopd_attn_shape b = *s;
  b.dtype = DOPD_BF16;
  return b;
}
}  // namespace
}  // extern "C++"

size_t dopd_prefill_paged_fp8_workspace_size(const dopd_attn_shape* s, const int32_t* cu_host,
                                             const int32_t* prefix_host, int32_t nreq,
                                             int32_t num_splits) {
  if (check_shape(s) != DOPD_OK || s->dtype != DOPD_FP8_E4M3) return 0;
  const dopd_attn_shape b = as_bf16(s);
  return dopd_prefill_paged_workspace_size(&b, cu_host, prefix_host, nreq, num_splits);
}

dopd_status dopd_prefill_paged_attn_fp8(const dopd_attn_shape* s, const void* q,
                                        const void* k_pool, const void* v_pool,
                                        const float* k_scale, const float* v_scale,
                                        int32_t num_pages, const int32_t* page_table,
                                        int32_t pt_stride, const int32_t* cu,
                                        const int32_t* cu_host, const int32_t* prefix,
                                        const int32_t* prefix_host, int32_t nreq,
                                        int32_t num_splits, void* out, float* lse,
                                        void* workspace, size_t workspace_bytes, void* stream) {
  dopd_status st = check_shape(s);
  if (st != DOPD_OK) return st;
  if (s->dtype != DOPD_FP8_E4M3) return DOPD_ERR_UNSUPPORTED;
  if (nreq > 0 && (!k_scale || !v_scale)) return DOPD_ERR_NULL_POINTER;
  const dopd_attn_shape b = as_bf16(s);
  return prefill_paged_impl(&b, q, k_pool, v_pool, num_pages, page_table, pt_stride, cu, cu_host,
                            prefix, prefix_host, nreq, num_splits, out, lse, workspace,
                            workspace_bytes, stream, k_scale, v_scale, true);
}

// ---------------------------------------------------------------- kv write
dopd_status dopd_kv_write(const dopd_attn_shape* s, const void* k_new, const void* v_new,
                          void* k_pool, void* v_pool, int32_t num_pages, const int32_t* pt,
                          int32_t pt_stride, const int32_t* cu_new, const int32_t* start_pos,
                          int32_t nreq, int32_t total_new, void* stream) {
  dopd_status st = check_shape_no_fp8(s);
  if (st != DOPD_OK) return st;
  if (nreq < 0 || total_new < 0 || num_pages < 0 || pt_stride < 0) return DOPD_ERR_INVALID_SHAPE;
  if (nreq == 0 || total_new == 0) return DOPD_OK;
  if (!k_new || !v_new || !k_pool || !v_pool || !pt || !cu_new || !start_pos)
    return DOPD_ERR_NULL_POINTER;
  // Touched pages per request <= n/16 + 2, so this bounds the item count.
  const int64_t blocks = (int64_t)total_new / dopd::kPage + 2 * (int64_t)nreq + 1;
  if (blocks > INT32_MAX || s->num_kv_heads > 65535) return DOPD_ERR_INVALID_SHAPE;
  hipStream_t strm = as_stream(stream);
  const int hkv = s->num_kv_heads, d = s->head_dim;
  const dim3 grid((unsigned)blocks, (unsigned)hkv), block(dopd::kKvwThreads);
  if (s->dtype == DOPD_BF16) {
    auto* kn = (const uint16_t*)k_new; auto* vn = (const uint16_t*)v_new;
    auto* kp = (uint16_t*)k_pool; auto* vp = (uint16_t*)v_pool;
    if (d == 64)
      hipLaunchKernelGGL((dopd::kv_write_kernel<uint16_t, 64>), grid, block, 0, strm, kn, vn, kp, vp, pt,
                         pt_stride, cu_new, start_pos, nreq, hkv);
    else
      hipLaunchKernelGGL((dopd::kv_write_kernel<uint16_t, 128>), grid, block, 0, strm, kn, vn, kp, vp, pt,
                         pt_stride, cu_new, start_pos, nreq, hkv);
  } else {
    auto* kn = (const uint32_t*)k_new; auto* vn = (const uint32_t*)v_new;
    auto* kp = (uint32_t*)k_pool; auto* vp = (uint32_t*)v_pool;
    if (d == 64)
      hipLaunchKernelGGL((dopd::kv_write_kernel<uint32_t, 64>), grid, block, 0, strm, kn, vn, kp, vp, pt,
                         pt_stride, cu_new, start_pos, nreq, hkv);
    else
      hipLaunchKernelGGL((dopd::kv_write_kernel<uint32_t, 128>), grid, block, 0, strm, kn, vn, kp, vp, pt,
                         pt_stride, cu_new, start_pos, nreq, hkv);
  }
  return launch_status();
}

dopd_status dopd_kv_write_fp8(const dopd_attn_shape* s, const void* k_new, const void* v_new,
                              const float* k_scale, const float* v_scale, void* k_pool,
                              void* v_pool, int32_t num_pages, const int32_t* pt,
                              int32_t pt_stride, const int32_t* cu_new, const int32_t* start_pos,
                              int32_t nreq, int32_t total_new, void* stream) {
  dopd_status st = check_shape(s);
  if (st != DOPD_OK) return st;
  if (s->dtype != DOPD_FP8_E4M3) return DOPD_ERR_UNSUPPORTED;
  if (nreq < 0 || total_new < 0 || num_pages < 0 || pt_stride < 0) return DOPD_ERR_INVALID_SHAPE;
  if (nreq == 0 || total_new == 0) return DOPD_OK;
  if (!k_new || !v_new || !k_scale || !v_scale || !k_pool || !v_pool || !pt || !cu_new ||
      !start_pos)
    return DOPD_ERR_NULL_POINTER;
  const int64_t blocks = (int64_t)total_new / dopd::kPage + 2 * (int64_t)nreq + 1;
  if (blocks > INT32_MAX || s->num_kv_heads > 65535) return DOPD_ERR_INVALID_SHAPE;
  hipStream_t strm = as_stream(stream);
  const int hkv = s->num_kv_heads;
  const dim3 grid((unsigned)blocks, (unsigned)hkv), block(dopd::kKvwThreads);
  auto* kn = (const uint16_t*)k_new;
  auto* vn = (const uint16_t*)v_new;
  auto* kp = (uint8_t*)k_pool;
  auto* vp = (uint8_t*)v_pool;
  if (s->head_dim == 64)
    hipLaunchKernelGGL(dopd::kv_write_e4m3_kernel<64>, grid, block, 0, strm, kn, vn, k_scale,
                       v_scale, kp, vp, pt, pt_stride, cu_new, start_pos, nreq, hkv);
  else
    hipLaunchKernelGGL(dopd::kv_write_e4m3_kernel<128>, grid, block, 0, strm, kn, vn, k_scale,
                       v_scale, kp, vp, pt, pt_stride, cu_new, start_pos, nreq, hkv);
  return launch_status();
}

// ---------------------------------------------------------------- decode
size_t dopd_decode_workspace_size(const dopd_attn_shape* s, const int32_t* ctx_host, int32_t n,
                                  int32_t split_tokens) {
  if (check_decode_host(s, ctx_host, n, split_tokens) != DOPD_OK) return 0;
  if (n == 0 || s->dtype == DOPD_FP32) return 256;
  return dopd::decode_layout(s->num_q_heads / s->num_kv_heads, s->num_kv_heads, s->head_dim,
                             ctx_host, n, split_tokens, machine_shape())
      .total;
}

dopd_status dopd_decode_attn(const dopd_attn_shape* s, const void* q, const void* k_pool,
                             const void* v_pool, int32_t num_pages, const int32_t* pt,
                             int32_t pt_stride, const int32_t* ctx, const int32_t* ctx_host,
                             int32_t nreq, int32_t split_tokens, void* out, float* lse,
                             void* workspace, size_t workspace_bytes, void* stream) {
  dopd_status st = check_decode_host(s, ctx_host, nreq, split_tokens);
  if (st != DOPD_OK) return st;
  if (s->dtype == DOPD_FP8_E4M3) return DOPD_ERR_UNSUPPORTED;  // dopd_decode_attn_fp8
  if (num_pages < 0 || pt_stride < 0) return DOPD_ERR_INVALID_SHAPE;
  if (nreq == 0) return DOPD_OK;
  if (!q || !k_pool || !v_pool || !pt || !ctx || !out) return DOPD_ERR_NULL_POINTER;
  for (int32_t r = 0; r < nreq; ++r)
    if ((int64_t)(ctx_host[r] + dopd::kPage - 1) / dopd::kPage > pt_stride)
      return DOPD_ERR_INVALID_SHAPE;
  const int hq = s->num_q_heads, hkv = s->num_kv_heads, d = s->head_dim;
  hipStream_t strm = as_stream(stream);
  if (s->dtype == DOPD_FP32) {
    dim3 grid((unsigned)nreq, (unsigned)hq);
    if (d == 64)
      hipLaunchKernelGGL(dopd::decode_f32_kernel<64>, grid, dim3(64), 0, strm, (const float*)q,
                         (const float*)k_pool, (const float*)v_pool, pt, pt_stride, ctx, hq, hkv,
                         s->softmax_scale, (float*)out, lse);
    else
      hipLaunchKernelGGL(dopd::decode_f32_kernel<128>, grid, dim3(64), 0, strm, (const float*)q,
                         (const float*)k_pool, (const float*)v_pool, pt, pt_stride, ctx, hq, hkv,
                         s->softmax_scale, (float*)out, lse);
    return launch_status();
  }
  return launch_decode_bf16<false>(s, q, k_pool, v_pool, nullptr, nullptr, pt, pt_stride, ctx,
                                   ctx_host, nreq, split_tokens, out, lse, workspace,
                                   workspace_bytes, strm);
}

dopd_status dopd_decode_attn_fp8(const dopd_attn_shape* s, const void* q, const void* k_pool,
                                 const void* v_pool, const float* k_scale, const float* v_scale,
                                 int32_t num_pages, const int32_t* pt, int32_t pt_stride,
                                 const int32_t* ctx, const int32_t* ctx_host, int32_t nreq,
                                 int32_t split_tokens, void* out, float* lse, void* workspace,
                                 size_t workspace_bytes, void* stream) {
  dopd_status st = check_decode_host(s, ctx_host, nreq, split_tokens);
  if (st != DOPD_OK) return st;
  if (s->dtype != DOPD_FP8_E4M3) return DOPD_ERR_UNSUPPORTED;
  if (num_pages < 0 || pt_stride < 0) return DOPD_ERR_INVALID_SHAPE;
  if (nreq == 0) return DOPD_OK;
  if (!q || !k_pool || !v_pool || !k_scale || !v_scale || !pt || !ctx || !out)
    return DOPD_ERR_NULL_POINTER;
  for (int32_t r = 0; r < nreq; ++r)
    if ((int64_t)(ctx_host[r] + dopd::kPage - 1) / dopd::kPage > pt_stride)
      return DOPD_ERR_INVALID_SHAPE;
  return launch_decode_bf16<true>(s, q, k_pool, v_pool, k_scale, v_scale, pt, pt_stride, ctx,
                                  ctx_host, nreq, split_tokens, out, lse, workspace,
                                  workspace_bytes, as_stream(stream));
}

dopd_status dopd_decode_attn_noalloc(const dopd_attn_shape* s, const void* q,
                                     const void* k_pool, const void* v_pool, int32_t num_pages,
                                     const int32_t* pt, int32_t pt_stride, const int32_t* ctx,
                                     const int32_t* ctx_host, int32_t nreq, int32_t split_tokens,
                                     void* out, float* lse, void* stream) {
  dopd_status st = check_decode_host(s, ctx_host, nreq, split_tokens);
  if (st != DOPD_OK) return st;
  if (s->dtype == DOPD_FP8_E4M3) return DOPD_ERR_UNSUPPORTED;
  if (nreq == 0) return DOPD_OK;
  size_t need = 0;
  if (s->dtype == DOPD_BF16)
    need = dopd::decode_layout(s->num_q_heads / s->num_kv_heads, s->num_kv_heads, s->head_dim,
                               ctx_host, nreq, split_tokens, machine_shape())
               .total;
  if (need > DOPD_DECODE_NOALLOC_SCRATCH_BYTES) return DOPD_ERR_WORKSPACE_TOO_SMALL;
  void* ws = nullptr;
  st = scratch_address(&ws);
  if (st != DOPD_OK) return st;
  return dopd_decode_attn(s, q, k_pool, v_pool, num_pages, pt, pt_stride, ctx, ctx_host, nreq,
                          split_tokens, out, lse, ws, DOPD_DECODE_NOALLOC_SCRATCH_BYTES, stream);
}

// ---------------------------------------------------------------- write + pack
extern "C++" {
namespace {

// Host checks shared by the write+pack and the PD step: bf16 fresh prompts
// with start position 0, each prompt's pages inside the page-table row.
dopd_status check_fresh_prompts(const int32_t* cu_host, int32_t nreq, int32_t pt_stride,
                                int64_t* pages_out) {
  if (cu_host[0] != 0) return DOPD_ERR_INVALID_SHAPE;
  int64_t pages = 0;
  for (int32_t r = 0; r < nreq; ++r) {
    const int64_t n = (int64_t)cu_host[r + 1] - cu_host[r];
    if (n < 0) return DOPD_ERR_INVALID_SHAPE;
    const int64_t np = (n + dopd::kPage - 1) / dopd::kPage;
    if (np > pt_stride) return DOPD_ERR_INVALID_SHAPE;
    pages += np;
  }
  *pages_out = pages;
  return DOPD_OK;
}

dopd::WritePackArgs write_pack_args(const void* k_new, const void* v_new, void* k_pool,
                                    void* v_pool, const int32_t* pt, int32_t pt_stride,
                                    const int32_t* cu, int32_t nreq, int hkv,
                                    const int64_t* out_offsets, void* out) {
  dopd::WritePackArgs w;
  w.k_new = (const uint16_t*)k_new;
  w.v_new = (const uint16_t*)v_new;
  w.k_pool = (uint16_t*)k_pool;
  w.v_pool = (uint16_t*)v_pool;
  w.page_table = pt;
  w.pt_stride = pt_stride;
  w.cu = cu;
  w.nreq = nreq;
  w.hkv = hkv;
  w.out = (uint16_t*)out;
  w.out_off = out_offsets;
  w.k_scale = nullptr;
  w.v_scale = nullptr;
  return w;
}

}  // namespace
}  // extern "C++"

dopd_status dopd_kv_write_pack_for_handoff(const dopd_attn_shape* s, const void* k_new,
                                           const void* v_new, void* k_pool, void* v_pool,
                                           int32_t num_pages, const int32_t* pt,
                                           int32_t pt_stride, const int32_t* cu,
                                           const int32_t* cu_host, int32_t nreq,
                                           const int64_t* out_offsets, void* out, void* stream) {
  dopd_status st = check_shape(s);
  if (st != DOPD_OK) return st;
  if (s->dtype != DOPD_BF16) return DOPD_ERR_UNSUPPORTED;
  if (nreq < 0 || num_pages < 0 || pt_stride < 0) return DOPD_ERR_INVALID_SHAPE;
  if (nreq == 0) return DOPD_OK;
  if (!k_new || !v_new || !k_pool || !v_pool || !pt || !cu || !cu_host)
    return DOPD_ERR_NULL_POINTER;
  if ((out == nullptr) != (out_offsets == nullptr)) return DOPD_ERR_NULL_POINTER;
  int64_t pages = 0;
  st = check_fresh_prompts(cu_host, nreq, pt_stride, &pages);
  if (st != DOPD_OK) return st;
  const int64_t blocks = pages * s->num_kv_heads;
  if (blocks == 0) return DOPD_OK;
  if (blocks > INT32_MAX) return DOPD_ERR_INVALID_SHAPE;
  const dopd::WritePackArgs w = write_pack_args(k_new, v_new, k_pool, v_pool, pt, pt_stride, cu,
                                                nreq, s->num_kv_heads, out_offsets, out);
  hipStream_t strm = as_stream(stream);
  if (s->head_dim == 64)
    hipLaunchKernelGGL(dopd::kv_write_pack_kernel<64>, dim3((unsigned)blocks), dim3(256), 0, strm, w);
  else
    hipLaunchKernelGGL(dopd::kv_write_pack_kernel<128>, dim3((unsigned)blocks), dim3(256), 0, strm, w);
  return launch_status();
}

// ---------------------------------------------------------------- PD step
extern "C++" {
namespace {
constexpr int kPdLastSchedule = DOPD_PD_DECODE_FIRST_WIDE;
constexpr int kPdAutoSchedule = DOPD_PD_PREFILL_FIRST;

// Decode workgroups per CU (in quarters) of a fused-step schedule.
int pd_decode_quarters(int schedule) {
  if (schedule == DOPD_PD_AUTO) schedule = kPdAutoSchedule;
  switch (schedule) {
    case DOPD_PD_DECODE_FIRST: return 4;       // one per CU
    case DOPD_PD_DECODE_FIRST_WIDE: return 6;  // three per two CUs
    default: return 4 * dopd::kWgPerCu;        // every slot
  }
}
}  // namespace
}  // extern "C++"

size_t dopd_pd_step_workspace_size(const dopd_attn_shape* s, const int32_t* ctx_host,
                                   int32_t num_dec, int32_t schedule) {
  if (check_decode_host(s, ctx_host, num_dec, 0) != DOPD_OK) return 0;
  if ((s->dtype != DOPD_BF16 && s->dtype != DOPD_FP8_E4M3) || schedule < DOPD_PD_AUTO ||
      schedule > kPdLastSchedule)
    return 0;
  if (num_dec == 0) return 256;
  return dopd::decode_layout(s->num_q_heads / s->num_kv_heads, s->num_kv_heads, s->head_dim,
                             ctx_host, num_dec, 0, machine_shape(), pd_decode_quarters(schedule))
      .total;
}

// dopd_pd_step(_fp8): bf16 pools, or (kv8) E4M3 pools with per-head scales.
static dopd_status pd_step_impl(const dopd_attn_shape* s, const void* q_dec,
                                const int32_t* dec_page_table, const int32_t* ctx,
                                const int32_t* ctx_host, int32_t num_dec, void* out_dec,
                                float* lse_dec, const void* q, const void* k, const void* v,
                                const int32_t* cu, const int32_t* cu_host, int32_t num_pre,
                                const int32_t* pre_page_table, void* out_pre, float* lse_pre,
                                void* k_pool, void* v_pool, int32_t num_pages, int32_t pt_stride,
                                const int64_t* handoff_offsets, void* handoff_out,
                                int32_t schedule, void* workspace, size_t workspace_bytes,
                                void* stream, bool kv8, const float* k_scale,
                                const float* v_scale) {
  dopd_status st = check_decode_host(s, ctx_host, num_dec, 0);
  if (st != DOPD_OK) return st;
  if (s->dtype != (kv8 ? DOPD_FP8_E4M3 : DOPD_BF16)) return DOPD_ERR_UNSUPPORTED;
  if (schedule < DOPD_PD_AUTO || schedule > kPdLastSchedule || num_pre < 0 ||
      num_pages < 0 || pt_stride < 0)
    return DOPD_ERR_INVALID_SHAPE;
  if (num_dec == 0 && num_pre == 0) return DOPD_OK;
  if (!k_pool || !v_pool) return DOPD_ERR_NULL_POINTER;
  if (num_dec > 0 && (!q_dec || !dec_page_table || !ctx || !out_dec)) return DOPD_ERR_NULL_POINTER;
  if (num_pre > 0 && (!q || !k || !v || !cu || !cu_host || !pre_page_table || !out_pre))
    return DOPD_ERR_NULL_POINTER;
  if ((handoff_out == nullptr) != (handoff_offsets == nullptr)) return DOPD_ERR_NULL_POINTER;
  if (kv8 && (!k_scale || !v_scale)) return DOPD_ERR_NULL_POINTER;
  for (int32_t r = 0; r < num_dec; ++r)
    if ((int64_t)(ctx_host[r] + dopd::kPage - 1) / dopd::kPage > pt_stride)
      return DOPD_ERR_INVALID_SHAPE;
  int64_t pages = 0;
  if (num_pre > 0) {
    st = check_fresh_prompts(cu_host, num_pre, pt_stride, &pages);
    if (st != DOPD_OK) return st;
  }
  if (schedule == DOPD_PD_AUTO) schedule = kPdAutoSchedule;
  const int hkv = s->num_kv_heads, d = s->head_dim;
  dopd::PdStepArgs p;
  std::memset(&p, 0, sizeof(p));
  DecodeMergePlan merge;
  if (num_dec > 0) {
    st = kv8 ? plan_decode_bf16<true>(s, q_dec, k_pool, v_pool, k_scale, v_scale, dec_page_table,
                                      pt_stride, ctx, ctx_host, num_dec, 0, out_dec, lse_dec,
                                      workspace, workspace_bytes, pd_decode_quarters(schedule),
                                      &p.dec, &merge)
             : plan_decode_bf16<false>(s, q_dec, k_pool, v_pool, nullptr, nullptr, dec_page_table,
                                       pt_stride, ctx, ctx_host, num_dec, 0, out_dec, lse_dec,
                                       workspace, workspace_bytes, pd_decode_quarters(schedule),
                                       &p.dec, &merge);
    if (st != DOPD_OK) return st;
    p.n_dec = p.dec.nwg;
  }
  int64_t pf_blocks = 0;
  if (num_pre > 0 && cu_host[num_pre] > 0) {
    dopd_attn_shape sb = *s;  // the prefill reads the bf16 fresh rows
    sb.dtype = DOPD_BF16;
    p.pf = prefill_args(&sb, q, out_pre, lse_pre, cu);
    p.pf.k = (const uint16_t*)k;
    p.pf.v = (const uint16_t*)v;
    st = plan_prefill_bf16<false>(p.pf, cu_host, nullptr, num_pre, &pf_blocks);
    if (st != DOPD_OK) return st;
    p.wp = write_pack_args(k, v, k_pool, v_pool, pre_page_table, pt_stride, cu, num_pre, hkv,
                           handoff_offsets, handoff_out);
    p.wp.k_scale = k_scale;
    p.wp.v_scale = v_scale;
  }
  p.n_pf = (int)pf_blocks;
  if (pages * hkv > INT32_MAX / 4) return DOPD_ERR_INVALID_SHAPE;
  p.n_wp = (int)(pages * hkv);
  // Block ranges; the prefill range starts on a multiple of the XCD count so
  // its XCD-aware order holds (blocks in the gaps exit at once).
  const int64_t xc = std::max(1, p.pf.xcds);
  auto round_up = [&](int64_t x) { return (x + xc - 1) / xc * xc; };
  int64_t total;
  if (schedule == DOPD_PD_PREFILL_FIRST) {
    p.wp_first = 0;
    p.pf_first = (int)round_up(p.n_wp);
    p.dec_first = p.pf_first + p.n_pf;
    total = (int64_t)p.dec_first + p.n_dec;
  } else {
    p.dec_first = 0;
    p.wp_first = p.n_dec;
    p.pf_first = (int)round_up((int64_t)p.n_dec + p.n_wp);
    total = (int64_t)p.pf_first + p.n_pf;
  }
  if (total > INT32_MAX / 2) return DOPD_ERR_INVALID_SHAPE;
  if (total == 0) return DOPD_OK;
  hipStream_t strm = as_stream(stream);
  const dim3 grid((unsigned)total), block(dopd::kPfThreads);
  if (kv8) {
    if (d == 64) hipLaunchKernelGGL((dopd::pd_step_kernel<64, true>), grid, block, 0, strm, p);
    else hipLaunchKernelGGL((dopd::pd_step_kernel<128, true>), grid, block, 0, strm, p);
  } else {
    if (d == 64) hipLaunchKernelGGL((dopd::pd_step_kernel<64, false>), grid, block, 0, strm, p);
    else hipLaunchKernelGGL((dopd::pd_step_kernel<128, false>), grid, block, 0, strm, p);
  }
  st = launch_status();
  if (st != DOPD_OK) return st;
  return launch_decode_merge(p.dec, merge, d, strm);
}

dopd_status dopd_pd_step(const dopd_attn_shape* s, const void* q_dec,
                         const int32_t* dec_page_table, const int32_t* ctx,
                         const int32_t* ctx_host, int32_t num_dec, void* out_dec,
                         float* lse_dec, const void* q, const void* k, const void* v,
                         const int32_t* cu, const int32_t* cu_host, int32_t num_pre,
                         const int32_t* pre_page_table, void* out_pre, float* lse_pre,
                         void* k_pool, void* v_pool, int32_t num_pages, int32_t pt_stride,
                         const int64_t* handoff_offsets, void* handoff_out, int32_t schedule,
                         void* workspace, size_t workspace_bytes, void* stream) {
  return pd_step_impl(s, q_dec, dec_page_table, ctx, ctx_host, num_dec, out_dec, lse_dec, q, k, v,
                      cu, cu_host, num_pre, pre_page_table, out_pre, lse_pre, k_pool, v_pool,
                      num_pages, pt_stride, handoff_offsets, handoff_out, schedule, workspace,
                      workspace_bytes, stream, false, nullptr, nullptr);
}

dopd_status dopd_pd_step_fp8(const dopd_attn_shape* s, const void* q_dec,
                             const int32_t* dec_page_table, const int32_t* ctx,
                             const int32_t* ctx_host, int32_t num_dec, void* out_dec,
                             float* lse_dec, const void* q, const void* k, const void* v,
                             const int32_t* cu, const int32_t* cu_host, int32_t num_pre,
                             const int32_t* pre_page_table, void* out_pre, float* lse_pre,
                             void* k_pool, void* v_pool, const float* k_scale,
                             const float* v_scale, int32_t num_pages, int32_t pt_stride,
                             const int64_t* handoff_offsets, void* handoff_out, int32_t schedule,
                             void* workspace, size_t workspace_bytes, void* stream) {
  return pd_step_impl(s, q_dec, dec_page_table, ctx, ctx_host, num_dec, out_dec, lse_dec, q, k, v,
                      cu, cu_host, num_pre, pre_page_table, out_pre, lse_pre, k_pool, v_pool,
                      num_pages, pt_stride, handoff_offsets, handoff_out, schedule, workspace,
                      workspace_bytes, stream, true, k_scale, v_scale);
}

// ---------------------------------------------------------------- handoff pack
dopd_status dopd_kv_pack_for_handoff(const dopd_attn_shape* s, int32_t num_layers,
                                     const void* k_pool, const void* v_pool, int32_t num_pages,
                                     const int32_t* pt, int32_t pt_stride, const int32_t* req_ids,
                                     const int32_t* seq_lens, const int32_t* seq_lens_host,
                                     const int64_t* out_offsets, int32_t num_handoff, void* out,
                                     void* stream) {
  dopd_status st = check_shape(s);
  if (st != DOPD_OK) return st;
  if (num_layers < 1 || num_pages < 0 || pt_stride < 0 || num_handoff < 0)
    return DOPD_ERR_INVALID_SHAPE;
  if (num_handoff == 0) return DOPD_OK;
  if (!k_pool || !v_pool || !pt || !req_ids || !seq_lens || !seq_lens_host || !out_offsets || !out)
    return DOPD_ERR_NULL_POINTER;
  int max_len = 0;
  for (int32_t n = 0; n < num_handoff; ++n) {
    if (seq_lens_host[n] < 0) return DOPD_ERR_INVALID_SHAPE;
    if ((int64_t)(seq_lens_host[n] + dopd::kPage - 1) / dopd::kPage > pt_stride)
      return DOPD_ERR_INVALID_SHAPE;
    max_len = std::max(max_len, seq_lens_host[n]);
  }
  if (max_len == 0) return DOPD_OK;
  const int64_t zdim = (int64_t)num_layers * 2 * s->num_kv_heads;
  int64_t pages = 0;
  for (int32_t n = 0; n < num_handoff; ++n) pages += (seq_lens_host[n] + dopd::kPage - 1) / dopd::kPage;
  if (zdim * pages > INT32_MAX - 64) return DOPD_ERR_INVALID_SHAPE;
  hipStream_t strm = as_stream(stream);
  auto launch = [&](auto type_tag) {
    using T = decltype(type_tag);
    dopd::PackArgs<T> a;
    a.k_pool = static_cast<const T*>(k_pool);
    a.v_pool = static_cast<const T*>(v_pool);
    a.num_pages = num_pages;
    a.page_table = pt;
    a.pt_stride = pt_stride;
    a.req_ids = req_ids;
    a.seq_lens = seq_lens;
    a.out_off = out_offsets;
    a.hkv = s->num_kv_heads;
    a.nz = (int)zdim;
    a.nhand = num_handoff;
    a.nblocks = (int)(zdim * pages);
    a.out = static_cast<T*>(out);
    if (s->head_dim == 64) {
      constexpr int per = dopd::pack_blocks_per_wg<T, 64>();
      hipLaunchKernelGGL((dopd::kv_pack_kernel<T, 64, per>), dim3((a.nblocks + per - 1) / per),
                         dim3(256), 0, strm, a);
    } else {
      constexpr int per = dopd::pack_blocks_per_wg<T, 128>();
      hipLaunchKernelGGL((dopd::kv_pack_kernel<T, 128, per>), dim3((a.nblocks + per - 1) / per),
                         dim3(256), 0, strm, a);
    }
  };
  if (s->dtype == DOPD_FP8_E4M3)
    launch(uint8_t{});
  else if (s->dtype == DOPD_BF16)
    launch(uint16_t{});
  else
    launch(uint32_t{});
  return launch_status();
}

// ---------------------------------------------------------------- handoff unpack
dopd_status dopd_kv_unpack_from_handoff(const dopd_attn_shape* s, int32_t num_layers,
                                        const void* in, const int64_t* in_offsets,
                                        const int32_t* req_ids, const int32_t* seq_lens,
                                        const int32_t* seq_lens_host, int32_t num_handoff,
                                        void* k_pool, void* v_pool, int32_t num_pages,
                                        const int32_t* pt, int32_t pt_stride, void* stream) {
  dopd_status st = check_shape(s);
  if (st != DOPD_OK) return st;
  if (num_layers < 1 || num_pages < 0 || pt_stride < 0 || num_handoff < 0)
    return DOPD_ERR_INVALID_SHAPE;
  if (num_handoff == 0) return DOPD_OK;
  if (!in || !in_offsets || !req_ids || !seq_lens || !seq_lens_host || !k_pool || !v_pool || !pt)
    return DOPD_ERR_NULL_POINTER;
  int max_len = 0;
  for (int32_t n = 0; n < num_handoff; ++n) {
    if (seq_lens_host[n] < 0) return DOPD_ERR_INVALID_SHAPE;
    if ((int64_t)(seq_lens_host[n] + dopd::kPage - 1) / dopd::kPage > pt_stride)
      return DOPD_ERR_INVALID_SHAPE;
    max_len = std::max(max_len, seq_lens_host[n]);
  }
  if (max_len == 0) return DOPD_OK;
  const int64_t zdim = (int64_t)num_layers * 2 * s->num_kv_heads;
  if (zdim > 65535 || num_handoff > 65535) return DOPD_ERR_INVALID_SHAPE;
  dim3 grid((unsigned)((max_len + dopd::kPage - 1) / dopd::kPage), (unsigned)num_handoff,
            (unsigned)zdim);
  hipStream_t strm = as_stream(stream);
  const int hkv = s->num_kv_heads;
  if (s->dtype == DOPD_FP8_E4M3) {
    auto* src = (const uint8_t*)in;
    auto* kp = (uint8_t*)k_pool; auto* vp = (uint8_t*)v_pool;
    if (s->head_dim == 64)
      hipLaunchKernelGGL((dopd::kv_unpack_kernel<uint8_t, 64>), grid, dim3(256), 0, strm, src,
                         in_offsets, req_ids, seq_lens, kp, vp, num_pages, pt, pt_stride, hkv);
    else
      hipLaunchKernelGGL((dopd::kv_unpack_kernel<uint8_t, 128>), grid, dim3(256), 0, strm, src,
                         in_offsets, req_ids, seq_lens, kp, vp, num_pages, pt, pt_stride, hkv);
  } else if (s->dtype == DOPD_BF16) {
    auto* src = (const uint16_t*)in;
    auto* kp = (uint16_t*)k_pool; auto* vp = (uint16_t*)v_pool;
    if (s->head_dim == 64)
      hipLaunchKernelGGL((dopd::kv_unpack_kernel<uint16_t, 64>), grid, dim3(256), 0, strm, src,
                         in_offsets, req_ids, seq_lens, kp, vp, num_pages, pt, pt_stride, hkv);
    else
      hipLaunchKernelGGL((dopd::kv_unpack_kernel<uint16_t, 128>), grid, dim3(256), 0, strm, src,
                         in_offsets, req_ids, seq_lens, kp, vp, num_pages, pt, pt_stride, hkv);
  } else {
    auto* src = (const uint32_t*)in;
    auto* kp = (uint32_t*)k_pool; auto* vp = (uint32_t*)v_pool;
    if (s->head_dim == 64)
      hipLaunchKernelGGL((dopd::kv_unpack_kernel<uint32_t, 64>), grid, dim3(256), 0, strm, src,
                         in_offsets, req_ids, seq_lens, kp, vp, num_pages, pt, pt_stride, hkv);
    else
      hipLaunchKernelGGL((dopd::kv_unpack_kernel<uint32_t, 128>), grid, dim3(256), 0, strm, src,
                         in_offsets, req_ids, seq_lens, kp, vp, num_pages, pt, pt_stride, hkv);
  }
  return launch_status();
}

}  // extern "C"
