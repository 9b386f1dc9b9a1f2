/*
 * dopd_attn.h -- C ABI of the MI355X (gfx950) attention hot path inside the
 * prefill (P) and decode (D) instances of a prefill/decode-disaggregated LLM
 * server.
 *
 * The operation is attention as defined by Eq. 1 of the paper,
 *     out = softmax(scale * Q K^T) V,
 * with the softmax scale as an argument (Eq. 1 prints no scale; callers
 * normally pass 1/sqrt(head_dim)).  A P-instance runs a variable-length causal
 * prefill over a batch of prompts (the per-request input lengths of the
 * length-aware batching of Sec. IV-C, Alg. 1) and writes K/V into a paged
 * cache (the KV-cache blocks of Sec. I and Sec. V-C); a D-instance runs
 * single-query attention over each request's cached context (decode is
 * memory bound, Sec. IV-B, Eq. 12); a prefill-completed request is handed to
 * a D-instance together with its KV cache (Sec. IV-B, Sec. V-C), for which
 * the packer gathers the request's pages into one contiguous buffer.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Pointers are DEVICE pointers unless the parameter name ends in "_host".
 *   The caller owns every buffer; the library never allocates or frees
 *   device memory and keeps no state between calls (re-entrant).
 * - `stream` is a hipStream_t passed as void* (NULL = default stream).  Every
 *   call only enqueues work on that stream; nothing synchronises.
 * - Element types: DOPD_BF16 (bf16 storage, fp32 accumulation, outputs
 *   rounded to nearest even) or DOPD_FP32 (fp32 throughout).
 *   DOPD_FP8_E4M3 describes a paged cache of OCP E4M3 codes (one byte per
 *   element; 1 sign, 4 exponent bits with bias 7, 3 mantissa bits, no
 *   infinities, largest finite value 448) with one fp32 scale per KV head
 *   for K and one for V: a cached element is code_value * scale[head].  Q,
 *   out and fresh K/V stay bf16.  The paper's models store FP8 (Sec. VI-A);
 *   it gives no scaling rule, so the per-head scale is this library's.  It
 *   halves the bytes decode and handoff move.  Entry points that take it:
 *   dopd_kv_write_fp8, dopd_decode_attn_fp8, dopd_decode_workspace_size,
 *   dopd_prefill_paged_attn_fp8 with its workspace size, dopd_pd_step_fp8
 *   with dopd_pd_step_workspace_size, and the handoff pack/unpack (byte
 *   copies); the others return DOPD_ERR_UNSUPPORTED for it.
 * - Fresh tokens are token-major: Q/out [T][Hq][d], K/V [T][Hkv][d].
 * - GQA: query head h uses KV head h / (Hq / Hkv); Hq % Hkv must be 0.
 * - Paged cache (one pool per layer, page_size = 16 tokens):
 *       k_pool[num_pages][Hkv][16][d]   (token-major inside a page)
 *       v_pool[num_pages][Hkv][d][16]   (dim-major inside a page)
 *   page_table[r * page_table_stride + i] is the physical page of logical
 *   page i (tokens 16i .. 16i+15) of request r.  Device-resident page ids are
 *   trusted on the hot path: entries a call reads must lie in
 *   [0, num_pages).  dopd_validate_page_table_host() checks a host copy.
 * - Errors are returned as dopd_status codes; nothing is thrown across the
 *   ABI.  Host-side argument checks run before any HIP call, so an invalid
 *   call touches no device.  DOPD_ERR_HIP means a HIP launch failed; its code
 *   is available from dopd_last_hip_error() on the calling thread.
 */
#ifndef DOPD_ATTN_H
#define DOPD_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t dopd_status;
enum {
  DOPD_OK = 0,
  DOPD_ERR_NULL_POINTER = 1,       /* a required pointer is NULL                 */
  DOPD_ERR_INVALID_SHAPE = 2,      /* counts, lengths or head ratio out of range */
  DOPD_ERR_UNSUPPORTED = 3,        /* dtype / head_dim / page_size not built     */
  DOPD_ERR_UNSUPPORTED_DTYPE = 3,  /* the same code under its narrower name      */
  DOPD_ERR_WORKSPACE_TOO_SMALL = 4,
  DOPD_ERR_HIP = 5
};

enum { DOPD_BF16 = 0, DOPD_FP32 = 1, DOPD_FP8_E4M3 = 2 };

typedef struct {
  int32_t num_q_heads;   /* Hq                                   */
  int32_t num_kv_heads;  /* Hkv, divides Hq                      */
  int32_t head_dim;      /* d: 64 or 128                         */
  int32_t page_size;     /* tokens per cache page: 16            */
  int32_t dtype;         /* DOPD_BF16, DOPD_FP32, DOPD_FP8_E4M3  */
  float softmax_scale;   /* multiplies Q.K before the softmax    */
} dopd_attn_shape;

/*
 * Variable-length causal prefill attention.
 * Paper: Eq. 1 (attention) over each prompt of a P-instance's batch; the
 * batch of prompts with per-request input lengths is the unit of Alg. 1
 * (Sec. IV-C); prefill is the compute-bound phase (Sec. I, Sec. IV-C) whose
 * cost grows with the square of the input length (Eq. 2).
 * Causal, no prefix: token i of a request attends to tokens 0..i of the same
 * request.
 *   q[T][Hq][d], k/v[T][Hkv][d], out[T][Hq][d]; T = cu_seqlens_host[num_reqs].
 *   cu_seqlens[num_reqs+1]: request r owns rows [cu[r], cu[r+1]); cu[0] = 0,
 *     non-decreasing (an empty request is allowed and produces nothing).
 *   cu_seqlens_host: identical host copy, used to size and order the launch
 *     (longest work first; with at most 64 requests the kernel takes the
 *     lengths from it, passed by value); it must equal the device copy.
 *   lse (nullable): fp32 [T][Hq], natural-log log-sum-exp of each row's
 *     scaled scores.
 *   workspace / workspace_bytes: device memory of at least
 *     dopd_prefill_workspace_size() bytes for the same arguments.  The
 *     present kernels keep no state outside q/k/v/out/lse, so that size is
 *     0 and workspace may be NULL; a non-NULL workspace must be 256-byte
 *     aligned.
 * bf16: Q.K and P.V run on bf16 MFMA with fp32 accumulation, P is rounded to
 * bf16 before the P.V product.  fp32: plain fp32 arithmetic.
 */
dopd_status dopd_prefill_attn(const dopd_attn_shape* shape, const void* q, const void* k,
                              const void* v, void* out, float* lse, const int32_t* cu_seqlens,
                              const int32_t* cu_seqlens_host, int32_t num_reqs, void* workspace,
                              size_t workspace_bytes, void* stream);

/*
 * Workspace bytes dopd_prefill_attn needs for these arguments.
 * Paper: as dopd_prefill_attn (Eq. 1 over the request batch of Alg. 1).
 * Returns 0: the dense prefill needs none (its work list is derived from
 * cu_seqlens_host and passed by value).  Returns 0 on bad input as well;
 * dopd_prefill_attn reports those itself.
 */
size_t dopd_prefill_workspace_size(const dopd_attn_shape* shape, const int32_t* cu_seqlens_host,
                                   int32_t num_reqs);

/*
 * Chunk prefill over the paged cache.
 * Paper: Eq. 1 over the KV-cache blocks (Sec. I, Sec. V-C); chunked prefill
 * (Sec. III-A) and ultra-short prefills run beside decode on a D-instance
 * (PD-aggregation by the Request Scheduler, Sec. V-E).
 * The prefill of a request that already holds cached tokens, i.e. one chunk
 * of a prompt processed in chunks or an ultra-short prefill merged into a
 * D-instance's work next to decode.  Eq. 1 over the cache,
 * causal with the chunk aligned to the end of the cache:
 *   request r has prefix_lens[r] cached tokens and a chunk of
 *   n_r = cu_seqlens[r+1] - cu_seqlens[r] new tokens whose K/V must already
 *   be in the pools at positions prefix_lens[r] .. prefix_lens[r] + n_r - 1
 *   (dopd_kv_write with start_pos = prefix_lens); chunk token i (row
 *   cu_seqlens[r] + i of q/out [T][Hq][d]) attends to cached positions
 *   0 .. prefix_lens[r] + i, read through page_table as in dopd_decode_attn.
 *   cu_seqlens / prefix_lens are device arrays with identical host copies
 *   (used to size and order the launch; with at most 64 requests the kernel
 *   takes the lengths and prefixes from them); lse (nullable) fp32 [T][Hq].
 * A chunk of one token is a decode step with context_lens = prefix_lens + 1;
 * prefix_lens = 0 with the whole prompt written first is dopd_prefill_attn.
 * bf16: the same MFMA path and rounding as dopd_prefill_attn.  Returns
 * DOPD_ERR_INVALID_SHAPE if a request's keys need more than page_table_stride
 * pages.
 */
dopd_status dopd_prefill_paged_attn(const dopd_attn_shape* shape, const void* q,
                                    const void* k_pool, const void* v_pool, int32_t num_pages,
                                    const int32_t* page_table, int32_t page_table_stride,
                                    const int32_t* cu_seqlens, const int32_t* cu_seqlens_host,
                                    const int32_t* prefix_lens, const int32_t* prefix_lens_host,
                                    int32_t num_reqs, void* out, float* lse, void* stream);

/*
 * dopd_prefill_paged_attn with key splits.
 * Paper: as dopd_prefill_paged_attn (Eq. 1 over the cached blocks, Sec. III-A,
 * Sec. V-E); the split and its log-sum-exp merge are an exact rewrite of the
 * softmax of Eq. 1.
 * The cached keys of each work item are split over
 * several workgroups, for calls with few work items (chunks of one or a few
 * long prompts fill only part of the GPU): the keys of each (q tile, request,
 * query head) item are cut into up to 16 contiguous ranges (the ranges that
 * every row of the item sees in full, and a last one with the rest),
 * computed by different workgroups, and a second kernel on the same stream
 * merges their un-normalised partials (o, row max, row sum) exactly by
 * log-sum-exp rescaling.  The same operation as dopd_prefill_paged_attn; the
 * result differs from it by rounding only.
 *   num_splits: 0 = automatic (splits only when the call has at most 256
 *     work items, one per CU: about 512 / items splits, at most 8, each with
 *     at least 8 key tiles that every row of the longest item sees), 1 = no
 *     split, n > 1 = n splits (at most 16).  fp32, and scales <= 0, never
 *     split.  Each split adds T * Hq * d * 8 bytes of partials written and
 *     read back.
 *   workspace: device memory of at least dopd_prefill_paged_workspace_size()
 *     bytes for the same arguments, 256-byte aligned, any contents; it holds
 *     the partials ([splits][T][Hq][d + 2] fp32).  May be null when no split
 *     is made.  Calls that overlap in time must not share it.
 */
dopd_status dopd_prefill_paged_attn_split(const dopd_attn_shape* shape, const void* q,
                                          const void* k_pool, const void* v_pool,
                                          int32_t num_pages, const int32_t* page_table,
                                          int32_t page_table_stride, const int32_t* cu_seqlens,
                                          const int32_t* cu_seqlens_host,
                                          const int32_t* prefix_lens,
                                          const int32_t* prefix_lens_host, int32_t num_reqs,
                                          int32_t num_splits, void* out, float* lse,
                                          void* workspace, size_t workspace_bytes, void* stream);

/* Workspace bytes dopd_prefill_paged_attn_split needs for these arguments on
 * the current device (at least 256; 0 on bad input).
 * Paper: as dopd_prefill_paged_attn_split (Eq. 1, Sec. III-A, Sec. V-E). */
size_t dopd_prefill_paged_workspace_size(const dopd_attn_shape* shape,
                                         const int32_t* cu_seqlens_host,
                                         const int32_t* prefix_lens_host, int32_t num_reqs,
                                         int32_t num_splits);

/*
 * Chunk prefill over E4M3 pools.
 * Paper: the prefill of dopd_prefill_paged_attn (Eq. 1 over a cached prefix,
 * Sec. III-A, Sec. V-E) over FP8 blocks, the models' precision (Sec. VI-A).
 * shape->dtype = DOPD_FP8_E4M3: dopd_prefill_paged_attn's operation with
 * K_j = code * k_scale[c] and V_j = code * v_scale[c] for KV head c (pool
 * layouts as there, one byte per element; k_scale/v_scale fp32 device arrays
 * [Hkv], positive and finite, not checked on the device); q and out bf16,
 * lse as there.  The kernel widens the codes to bf16 (exactly: every E4M3
 * value is a bf16 value) as it reads them from LDS, with the K scale folded
 * into the softmax scale and the V scale into the output, in fp32; half the
 * bytes of bf16 pages per cached token.  num_splits as in
 * dopd_prefill_paged_attn_split.
 *   workspace: device memory of at least
 *     dopd_prefill_paged_fp8_workspace_size() bytes for the same arguments
 *     (the key-split partials, as dopd_prefill_paged_workspace_size gives
 *     for bf16 pools), 256-byte aligned, any contents.  May be null when no
 *     split is made.  Calls that overlap in time must not share it.
 */
dopd_status dopd_prefill_paged_attn_fp8(const dopd_attn_shape* shape, const void* q,
                                        const void* k_pool, const void* v_pool,
                                        const float* k_scale, const float* v_scale,
                                        int32_t num_pages, const int32_t* page_table,
                                        int32_t page_table_stride, const int32_t* cu_seqlens,
                                        const int32_t* cu_seqlens_host,
                                        const int32_t* prefix_lens,
                                        const int32_t* prefix_lens_host, int32_t num_reqs,
                                        int32_t num_splits, void* out, float* lse,
                                        void* workspace, size_t workspace_bytes, void* stream);

/* Workspace bytes dopd_prefill_paged_attn_fp8 needs for these arguments on
 * the current device (at least 256; 0 on bad input or a dtype other than
 * DOPD_FP8_E4M3).
 * Paper: as dopd_prefill_paged_attn_fp8 (Eq. 1, Sec. III-A, Sec. VI-A). */
size_t dopd_prefill_paged_fp8_workspace_size(const dopd_attn_shape* shape,
                                             const int32_t* cu_seqlens_host,
                                             const int32_t* prefix_lens_host, int32_t num_reqs,
                                             int32_t num_splits);

/*
 * Paged KV write.
 * Paper: the KV cache kept per request in fixed-size blocks (Sec. I; block
 * count and fragmentation, Sec. II-C; the blocks the Connector moves,
 * Sec. V-C); KV capacity bounds a D-instance's concurrency (Eq. 11, Eq. 13).
 * Request r appends n_r = cu_new_tokens[r+1] - cu_new_tokens[r]
 * tokens at logical positions start_pos[r] .. start_pos[r] + n_r - 1, taken
 * from rows cu_new_tokens[r] .. of k_new/v_new[total_new_tokens][Hkv][d].
 * Position p goes to page page_table[r*stride + p/16], slot p % 16.  Pure bit
 * copy; every other slot of the pools is left untouched.  Prefill writes use
 * start_pos = 0; a decode step appends at start_pos = context_len - 1.
 *   cu_new_tokens[num_reqs+1], start_pos[num_reqs] are device arrays;
 *   total_new_tokens = cu_new_tokens[num_reqs] (host value, sizes the launch).
 */
dopd_status dopd_kv_write(const dopd_attn_shape* shape, const void* k_new, const void* v_new,
                          void* k_pool, void* v_pool, int32_t num_pages,
                          const int32_t* page_table, int32_t page_table_stride,
                          const int32_t* cu_new_tokens, const int32_t* start_pos,
                          int32_t num_reqs, int32_t total_new_tokens, void* stream);

/*
 * Paged KV write into E4M3 pools.
 * Paper: the KV-cache blocks of Sec. I and Sec. V-C stored in FP8, the
 * precision of the evaluated models (Sec. VI-A); the paper gives no scaling
 * rule, the per-head scale is this library's.
 * shape->dtype = DOPD_FP8_E4M3; the same
 * placement as dopd_kv_write, from bf16 k_new/v_new [total_new_tokens][Hkv][d],
 * with element x of KV head h stored as the code
 *     E4M3_rne(sat(x * fp32(1 / scale[h])))
 * where 1/scale[h] and the product are fp32 operations rounded to nearest
 * even, sat() clamps to [-448, 448] (NaN stays NaN) and E4M3_rne rounds to
 * the nearest code, ties to the even code.  k_scale/v_scale: device fp32
 * [Hkv], positive and finite (not checked on the device).  k_pool/v_pool:
 * one byte per element, same page layouts.  Other slots are untouched.
 */
dopd_status dopd_kv_write_fp8(const dopd_attn_shape* shape, const void* k_new, const void* v_new,
                              const float* k_scale, const float* v_scale, void* k_pool,
                              void* v_pool, int32_t num_pages, const int32_t* page_table,
                              int32_t page_table_stride, const int32_t* cu_new_tokens,
                              const int32_t* start_pos, int32_t num_reqs,
                              int32_t total_new_tokens, void* stream);

/*
 * Paged single-query decode attention.
 * Paper: Eq. 1 for one new token per request over its cached blocks; decode
 * time is dominated by reading the KV cache from HBM (Sec. I, Sec. IV-B,
 * Eq. 12; D-instance model, Sec. IV-D).
 * For request r with context_lens[r]
 * cached tokens (counting the current one, whose K/V must already be in the
 * cache) and every query head h,
 *   out[r][h] = softmax_j(scale * q[r][h] . K_j) V_j,  j < context_lens[r].
 *   q/out [num_reqs][Hq][d]; lse (nullable) fp32 [num_reqs][Hq].
 *   context_lens_host: identical host copy (>= 1 each), used to size the
 *     launch and the key-range split.
 *   split_tokens: size of the key range each workgroup takes, 0 = automatic
 *     (one equal share per resident workgroup), else a positive multiple of
 *     32, at most 4096 (in tokens; a range may span several requests).  The
 *     result does not depend on it beyond rounding.
 *   workspace: device memory of at least dopd_decode_workspace_size() bytes
 *     for the same arguments, 256-byte aligned, any contents; it holds the
 *     split-K partials.  Calls that overlap in time must not share it.
 * bf16 path: the keys of all (request, KV head) pairs are cut into equal
 * shares, one per workgroup, so that long and short contexts balance; each
 * page is read once for all Hq/Hkv query heads of the group (at most 16); a
 * (request, KV head) whose keys fall in several shares is finished by a
 * second kernel that merges the partials exactly (log-sum-exp rescaling), on
 * the same stream.
 */
dopd_status dopd_decode_attn(const dopd_attn_shape* shape, const void* q, const void* k_pool,
                             const void* v_pool, int32_t num_pages, const int32_t* page_table,
                             int32_t page_table_stride, const int32_t* context_lens,
                             const int32_t* context_lens_host, int32_t num_reqs,
                             int32_t split_tokens, void* out, float* lse, void* workspace,
                             size_t workspace_bytes, void* stream);

/*
 * Decode over E4M3 pools.
 * Paper: Eq. 1 as in dopd_decode_attn over FP8 blocks (the models' precision,
 * Sec. VI-A), halving the bytes Eq. 12 charges per cached token.
 * shape->dtype = DOPD_FP8_E4M3: dopd_decode_attn's
 * operation with K_j = code * k_scale[c] and V_j = code * v_scale[c] for KV
 * head c; q and out bf16, lse as there.  The codes are widened to bf16
 * (exactly) for the same MFMA path; the K scale multiplies the softmax scale
 * and the V scale the output, in fp32.  Same partition, workspace
 * (dopd_decode_workspace_size with the same shape) and split_tokens rules;
 * half the bytes of the bf16 cache per token.
 */
dopd_status dopd_decode_attn_fp8(const dopd_attn_shape* shape, const void* q,
                                 const void* k_pool, const void* v_pool, const float* k_scale,
                                 const float* v_scale, int32_t num_pages,
                                 const int32_t* page_table, int32_t page_table_stride,
                                 const int32_t* context_lens, const int32_t* context_lens_host,
                                 int32_t num_reqs, int32_t split_tokens, void* out, float* lse,
                                 void* workspace, size_t workspace_bytes, void* stream);

/* Workspace bytes dopd_decode_attn(_fp8) needs for these arguments on the
 * current device (at least 256; 0 on bad input).
 * Paper: as dopd_decode_attn (Eq. 1, Sec. IV-B, Eq. 12); the split-K partials
 * are an exact rewrite of the softmax of Eq. 1. */
size_t dopd_decode_workspace_size(const dopd_attn_shape* shape,
                                  const int32_t* context_lens_host, int32_t num_reqs,
                                  int32_t split_tokens);

/* Size of the static device scratch of dopd_decode_attn_noalloc (32 MiB). */
#define DOPD_DECODE_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)

/*
 * dopd_decode_attn without a caller workspace, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation.  Same operation, arguments (minus the
 * workspace), kernels and results as dopd_decode_attn (bf16 and fp32 caches;
 * E4M3 returns DOPD_ERR_UNSUPPORTED).  The split-K partials go to a static
 * device array of DOPD_DECODE_NOALLOC_SCRATCH_BYTES (32 MiB) that the library
 * holds on every device it runs on until the process ends; its address is
 * looked up once per device (hipGetSymbolAddress, with that device current).
 * Nothing is allocated or freed by the call.  A call whose partials need
 * more than that (dopd_decode_workspace_size with the same arguments above
 * the limit) returns DOPD_ERR_WORKSPACE_TOO_SMALL before any device work.
 * The array keeps the last call's contents and needs no clearing (every
 * partial is written before it is read).  All calls on one device share it:
 * calls that overlap in time on one device (two streams, two threads) race
 * and must be serialised by the caller.
 */
dopd_status dopd_decode_attn_noalloc(const dopd_attn_shape* shape, const void* q,
                                     const void* k_pool, const void* v_pool, int32_t num_pages,
                                     const int32_t* page_table, int32_t page_table_stride,
                                     const int32_t* context_lens,
                                     const int32_t* context_lens_host, int32_t num_reqs,
                                     int32_t split_tokens, void* out, float* lse, void* stream);

/*
 * Paged KV write of fresh prompts that also emits their handoff buffer.
 * Paper: a prefill-completed request is handed to a D-instance with its KV
 * cache (Sec. IV-B) by the Connector (Sec. V-C); the KV-cache blocks of
 * Sec. I.  A fresh prompt's cache is exactly the K/V rows its prefill
 * produced, so the buffer dopd_kv_pack_for_handoff would gather from the
 * pages afterwards is written from those rows in the same pass as the pages.
 * Request r (rows cu_seqlens[r] .. cu_seqlens[r+1] - 1 of
 * k_new/v_new[T][Hkv][d], bf16) is written at positions 0 .. n_r - 1 of its
 * pages exactly as dopd_kv_write with start_pos = 0, and, when out is not
 * NULL, to
 *   out[out_offsets[r] + ((c*Hkv + h)*n_r + t)*d + e]   (c = 0: K, 1: V),
 * the one-layer (K/V, head, token, dim) block of dopd_kv_pack_for_handoff.
 * out_offsets [num_reqs] (int64 element offsets, device); out and
 * out_offsets are both NULL or both given.  cu_seqlens / cu_seqlens_host as
 * in dopd_prefill_attn.  bf16 only.  Bit copy; other slots untouched.
 */
dopd_status dopd_kv_write_pack_for_handoff(const dopd_attn_shape* shape, const void* k_new,
                                           const void* v_new, void* k_pool, void* v_pool,
                                           int32_t num_pages, const int32_t* page_table,
                                           int32_t page_table_stride, const int32_t* cu_seqlens,
                                           const int32_t* cu_seqlens_host, int32_t num_reqs,
                                           const int64_t* out_offsets, void* out, void* stream);

/* Block order of dopd_pd_step's single launch. */
enum {
  DOPD_PD_AUTO = 0,           /* the library's choice (DOPD_PD_PREFILL_FIRST)          */
  DOPD_PD_PREFILL_FIRST = 1,  /* write/pack and prefill workgroups dispatched first,
                                 then the decode slices (two per CU)                   */
  DOPD_PD_DECODE_FIRST = 2,   /* the decode slices first, one per CU, then the
                                 write/pack and prefill workgroups in the other slot    */
  DOPD_PD_DECODE_FIRST_WIDE = 3 /* the decode slices first, three per two CUs; the
                                 write/pack and prefill workgroups in the slots left    */
};

/*
 * One PD-aggregated step in a single launch: the decode of a batch of
 * requests and the prefill of a batch of fresh prompts on the same instance,
 * with the prompts' paged KV write and (optionally) their handoff buffer.
 * Paper: PD-aggregation, ultra-short requests prefilled on a D-instance next
 * to its decode (Request Scheduler, Sec. V-E); co-scheduling prefill and
 * decode work in one kernel (POD-style, Sec. III-A); Eq. 1 for both.
 * Same results as, in one stream order,
 *   dopd_decode_attn(q_dec, dec_page_table, context_lens ..., out_dec, lse_dec)
 *   dopd_prefill_attn(q, k, v, cu_seqlens ..., out_pre, lse_pre)
 *   dopd_kv_write_pack_for_handoff(k, v, pre_page_table ..., handoff_offsets,
 *                                  handoff_out)
 * (the decode's automatic partition; results equal those calls' up to the
 * rounding of a different split), run as workgroups of three kinds in one
 * grid (plus the decode's merge kernel when a context spans several slices),
 * so that memory-bound decode slices and compute-bound prefill items share
 * the CUs.  The decode requests' pages and the prompts' pages must be
 * disjoint (the decode never reads what the write fills in this step).
 *   dec_page_table / pre_page_table: rows of the decode requests and of the
 *     prompts, both of page_table_stride columns, into the same pools.
 *   schedule: DOPD_PD_* block order.
 *   workspace: dopd_pd_step_workspace_size() bytes (decode partials),
 *     256-byte aligned, any contents.
 * bf16 pools (dopd_pd_step_fp8: E4M3 pools).  Either batch may be empty.
 */
dopd_status dopd_pd_step(const dopd_attn_shape* shape, const void* q_dec,
                         const int32_t* dec_page_table, const int32_t* context_lens,
                         const int32_t* context_lens_host, int32_t num_dec, void* out_dec,
                         float* lse_dec, const void* q, const void* k, const void* v,
                         const int32_t* cu_seqlens, const int32_t* cu_seqlens_host,
                         int32_t num_pre, const int32_t* pre_page_table, void* out_pre,
                         float* lse_pre, void* k_pool, void* v_pool, int32_t num_pages,
                         int32_t page_table_stride, const int64_t* handoff_offsets,
                         void* handoff_out, int32_t schedule, void* workspace,
                         size_t workspace_bytes, void* stream);

/*
 * The same PD-aggregated step over E4M3 pools.
 * Paper: PD-aggregation on a D-instance (Sec. V-E) serving the FP8 models of
 * Sec. VI-A, whose KV blocks are FP8; Eq. 1 for both kinds of work.
 * shape->dtype = DOPD_FP8_E4M3; k_scale/v_scale: fp32 device arrays [Hkv]
 * (positive and finite, not checked on the device).  Same results as, in one
 * stream order,
 *   dopd_decode_attn_fp8(q_dec, k_pool, v_pool, k_scale, v_scale ...)
 *   dopd_prefill_attn(q, k, v ...)   (the fresh rows stay bf16)
 *   the E4M3 paged write of k, v (dopd_kv_write_fp8's codes) and, with
 *   handoff_out, the pack of those codes (dopd_kv_pack_for_handoff over the
 *   E4M3 pools: one byte per element, handoff_offsets in elements = bytes)
 * up to the rounding of a different decode split.  Other arguments, the
 * block orders, the workspace (dopd_pd_step_workspace_size with the E4M3
 * shape) and the disjoint-pages rule as for dopd_pd_step.
 */
dopd_status dopd_pd_step_fp8(const dopd_attn_shape* shape, const void* q_dec,
                             const int32_t* dec_page_table, const int32_t* context_lens,
                             const int32_t* context_lens_host, int32_t num_dec, void* out_dec,
                             float* lse_dec, const void* q, const void* k, const void* v,
                             const int32_t* cu_seqlens, const int32_t* cu_seqlens_host,
                             int32_t num_pre, const int32_t* pre_page_table, void* out_pre,
                             float* lse_pre, void* k_pool, void* v_pool, const float* k_scale,
                             const float* v_scale, int32_t num_pages, int32_t page_table_stride,
                             const int64_t* handoff_offsets, void* handoff_out,
                             int32_t schedule, void* workspace, size_t workspace_bytes,
                             void* stream);

/* Workspace bytes dopd_pd_step (bf16 shape) or dopd_pd_step_fp8 (E4M3 shape)
 * needs for this decode batch and schedule on the current device (at least
 * 256; 0 on bad input).
 * Paper: as dopd_pd_step (Sec. V-E, Sec. III-A; the split-K partials of the
 * decode are an exact rewrite of the softmax of Eq. 1). */
size_t dopd_pd_step_workspace_size(const dopd_attn_shape* shape,
                                   const int32_t* context_lens_host, int32_t num_dec,
                                   int32_t schedule);

/*
 * Handoff pack of prefill-completed requests.
 * Paper: a P-instance hands each prefill-completed request with its KV cache
 * to a D-instance (Sec. IV-B); the Connector's KV transmitter moves the blocks
 * (Sec. V-C), at a cost that grows with block count and fragmentation
 * (Sec. II-C), which one contiguous buffer per request removes.
 * Handoff n
 * (request req_ids[n], seq_lens[n] cached tokens) is written to
 *   out[out_offsets[n] + (((layer*2 + c)*Hkv + h)*len + t)*d + e]
 * with c = 0 for K and 1 for V, i.e. (layer, K/V, head, token, dim) order.
 *   k_pool/v_pool carry a leading layer dimension: [num_layers][num_pages]...
 *   req_ids, seq_lens [num_handoff], out_offsets [num_handoff+1] (int64
 *   element offsets) are device arrays; seq_lens_host is a host copy that
 *   sizes the launch.  Tail slots of a request's last page are not copied.
 */
dopd_status dopd_kv_pack_for_handoff(const dopd_attn_shape* shape, int32_t num_layers,
                                     const void* k_pool, const void* v_pool, int32_t num_pages,
                                     const int32_t* page_table, int32_t page_table_stride,
                                     const int32_t* req_ids, const int32_t* seq_lens,
                                     const int32_t* seq_lens_host, const int64_t* out_offsets,
                                     int32_t num_handoff, void* out, void* stream);

/*
 * Handoff unpack on the receiving (D) instance.
 * Paper: the KV blocks of a prefill-completed request that the Connector
 * delivers to a D-instance (Sec. IV-B, Sec. V-C).
 * The inverse of dopd_kv_pack_for_handoff:
 * element (layer, c, h, t, e) of handoff n, read from
 *   in[in_offsets[n] + (((layer*2 + c)*Hkv + h)*len + t)*d + e],  len = seq_lens[n],
 * is written to slot t % 16 of page page_table[req_ids[n]*stride + t/16] of
 * the local pools (c = 0: k_pool, 1: v_pool; both with a leading layer
 * dimension of num_pages pages).  Tail slots of the last page are not
 * touched.  req_ids, seq_lens [num_handoff], in_offsets [num_handoff] (int64
 * element offsets) are device arrays; seq_lens_host sizes the launch.  Bit copy.
 */
dopd_status dopd_kv_unpack_from_handoff(const dopd_attn_shape* shape, int32_t num_layers,
                                        const void* in, const int64_t* in_offsets,
                                        const int32_t* req_ids, const int32_t* seq_lens,
                                        const int32_t* seq_lens_host, int32_t num_handoff,
                                        void* k_pool, void* v_pool, int32_t num_pages,
                                        const int32_t* page_table, int32_t page_table_stride,
                                        void* stream);

/*
 * Host check of a page table copy.
 * Paper: the per-request KV-cache blocks (Sec. I, Sec. V-C).
 * For each request r, the entries
 * page_table_host[r*stride + i], i < ceil(lens_host[r]/16), must lie in
 * [0, num_pages).  Returns DOPD_OK or DOPD_ERR_INVALID_SHAPE.
 */
dopd_status dopd_validate_page_table_host(const int32_t* page_table_host,
                                          int32_t page_table_stride, int32_t num_reqs,
                                          const int32_t* lens_host, int32_t num_pages);

/* Static description of a status code.
 * Paper: none (error reporting of this library). */
const char* dopd_status_string(dopd_status status);

/* hipError_t of the last DOPD_ERR_HIP on the calling thread (0 if none).
 * Paper: none (error reporting of this library). */
int32_t dopd_last_hip_error(void);

#ifdef __cplusplus
}
#endif
#endif /* DOPD_ATTN_H */
