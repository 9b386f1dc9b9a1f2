"""Seeded synthetic workloads for the prefill/decode attention hot path.

This module only draws data: request lengths, page allocations, Q/K/V values
and poison.  It contains none of the attention arithmetic and none of the
cache index maps beyond "which physical slot is live", so both the fp64
oracle and the HIP path consume exactly the same arrays.

Storage conventions (shared by every consumer):

* bf16 tensors are ``numpy.uint16`` arrays holding bf16 bit patterns;
  fp32 tensors are ``numpy.float32``.
* Fresh tokens (prefill inputs, new decode tokens) are token-major:
  Q ``[T][Hq][d]``, K/V ``[T][Hkv][d]``.
* Paged cache, one pool per layer (the K/V cache blocks of the paper's
  disaggregated design, Sec. I and the Connector of Sec. V-C):
  ``k_pool[page][Hkv][page_size][d]`` (token-major within a page) and
  ``v_pool[page][Hkv][d][page_size]`` (dim-major within a page).
* ``page_table[r][i]`` is the physical page of request ``r``'s logical page
  ``i``; padding is -1.
* Unused pages and unused tail slots hold NaN (bf16 0x7FC0, fp32 quiet NaN).

Length laws (the paper's heavy-tailed input lengths, Sec. IV-A and Eq. 9,
stand-ins for the production traces of the evaluation, Sec. VI-A):
lognormal ``clip(rint(exp(N(ln median, sigma^2))), lo, hi)`` and a bimodal
short/long mix.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

PAGE_SIZE = 16
BF16_NAN = np.uint16(0x7FC0)
SEED_BASE = 20982


# ---------------------------------------------------------------- value helpers
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bf16 (round to nearest, ties to even); returns uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounding = np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    out = ((u + rounding) >> np.uint32(16)).astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        out[nan] = BF16_NAN
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float32."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def normal(rng: np.random.Generator, shape, dtype: str) -> np.ndarray:
    """N(0,1) drawn in fp32, then stored in ``dtype`` ("bf16" bits or "fp32")."""
    x = rng.standard_normal(size=shape, dtype=np.float32)
    return f32_to_bf16_bits(x) if dtype == "bf16" else x


def nan_array(shape, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return np.full(shape, BF16_NAN, dtype=np.uint16)
    return np.full(shape, np.nan, dtype=np.float32)


def lognormal_lengths(rng, n, median, sigma, lo, hi) -> np.ndarray:
    x = np.exp(rng.normal(math.log(median), sigma, size=n))
    return np.clip(np.rint(x), lo, hi).astype(np.int32)


def bimodal_lengths(rng, n, long_frac, short_lo, short_hi, long_lo, long_hi):
    """Exactly round(long_frac*n) long requests at shuffled positions; bounds inclusive."""
    n_long = int(round(long_frac * n))
    is_long = rng.permutation(np.array([True] * n_long + [False] * (n - n_long)))
    short = rng.integers(short_lo, short_hi + 1, size=n)
    long_ = rng.integers(long_lo, long_hi + 1, size=n)
    return np.where(is_long, long_, short).astype(np.int32), is_long


# ---------------------------------------------------------------- page allocation
def allocate_pages(rng, cap_lens, pool_pages=None, slack=1.25):
    """Random physical pages for each request's ``ceil(cap_len/16)`` logical pages.

    Requests take successive entries of one random permutation of the pool, in
    request order.  Returns (page_table[B][stride] int32 with -1 padding,
    num_pages)."""
    cap_lens = np.asarray(cap_lens, dtype=np.int64)
    need = (cap_lens + PAGE_SIZE - 1) // PAGE_SIZE
    total = int(need.sum())
    if pool_pages is None:
        pool_pages = int(math.ceil(slack * total))
    assert pool_pages >= total
    perm = rng.permutation(pool_pages).astype(np.int32)
    stride = max(1, int(need.max()) if len(need) else 1)
    pt = np.full((len(cap_lens), stride), -1, dtype=np.int32)
    pos = 0
    for r, n in enumerate(need):
        pt[r, :n] = perm[pos:pos + n]
        pos += int(n)
    return pt, pool_pages


def empty_pools(num_pages, hkv, d, dtype, num_layers=1):
    """NaN-filled K and V pools in the page layouts described above."""
    kshape = (num_pages, hkv, PAGE_SIZE, d)
    vshape = (num_pages, hkv, d, PAGE_SIZE)
    if num_layers != 1:
        kshape = (num_layers,) + kshape
        vshape = (num_layers,) + vshape
    return nan_array(kshape, dtype), nan_array(vshape, dtype)


def fill_live_slots(rng, k_pool, v_pool, page_table, ctx_lens, dtype):
    """Draw N(0,1) values for every live slot (slot < ctx of its owner).

    Values are drawn page by page in (request, logical page) order, K block
    then V block, so the draw does not depend on where a page sits in the pool.
    Dead tail slots keep their NaN poison."""
    hkv, d = k_pool.shape[1], k_pool.shape[3]
    for r, ctx in enumerate(ctx_lens):
        n_pages = (int(ctx) + PAGE_SIZE - 1) // PAGE_SIZE
        if n_pages == 0:
            continue
        pages = page_table[r, :n_pages]
        kb = normal(rng, (n_pages, hkv, PAGE_SIZE, d), dtype)
        vb = normal(rng, (n_pages, hkv, d, PAGE_SIZE), dtype)
        tail = int(ctx) - PAGE_SIZE * (n_pages - 1)
        if tail < PAGE_SIZE:
            kb[-1, :, tail:, :] = nan_array((), dtype)
            vb[-1, :, :, tail:] = nan_array((), dtype)
        k_pool[pages] = kb
        v_pool[pages] = vb


# ---------------------------------------------------------------- workloads
@dataclass
class Workload:
    """One seeded workload; fields not used by a workload stay None."""
    name: str
    seed: int
    dtype: str
    hq: int
    hkv: int
    d: int
    scale: float
    page_size: int = PAGE_SIZE
    # prefill batch
    prefill_lens: np.ndarray | None = None
    cu_seqlens: np.ndarray | None = None
    q: np.ndarray | None = None
    k: np.ndarray | None = None
    v: np.ndarray | None = None
    prefill_rows: np.ndarray | None = None      # page-table rows of the prefill requests
    # paged cache
    num_pages: int = 0
    k_pool: np.ndarray | None = None
    v_pool: np.ndarray | None = None
    page_table: np.ndarray | None = None
    # decode batch
    context_lens: np.ndarray | None = None
    q_dec: np.ndarray | None = None
    # decode steps after the prefill (the tiny fp32 workload): list of
    # (q[B][Hq][d], k[B][Hkv][d], v[B][Hkv][d])
    steps: list = field(default_factory=list)
    # handoff
    handoff_reqs: np.ndarray | None = None
    handoff_lens: np.ndarray | None = None
    notes: dict = field(default_factory=dict)


def cu_from_lens(lens) -> np.ndarray:
    cu = np.zeros(len(lens) + 1, dtype=np.int32)
    cu[1:] = np.cumsum(np.asarray(lens, dtype=np.int64))
    return cu


def prefill_batch(rng, lens, hq, hkv, d, dtype):
    t = int(np.sum(lens))
    q = normal(rng, (t, hq, d), dtype)
    k = normal(rng, (t, hkv, d), dtype)
    v = normal(rng, (t, hkv, d), dtype)
    return q, k, v


def steep_score_batch(rng, lens, hq, hkv, d, pattern, rise=40.0):
    """bf16 Q/K/V of packed requests whose attention scores (at the softmax
    scale 1/sqrt(d)) climb steeply along each request, far beyond what N(0,1)
    inputs reach: the inputs that drive an online softmax's rescaling.

    Every query row is a shared direction u (entries +-1, so |u|^2 = d) plus
    N(0, 1/4) noise; key t of a request is beta_t * u / sqrt(d) plus N(0, 1/4)
    noise, so its score against any row is about beta_t (in natural-log
    units) plus O(1).  V is N(0,1).  Patterns (t = position in the request):
      "ramp":  beta_t = rise * t / 64 (rise per 64-key tile),
      "jump":  beta_t = 0 for t < 256, then 150 + rise * (t - 256) / 64
               (a step of more than 128 in the log2 domain),
      "spike": beta_t = 0 except one key per request at position 64*5 + 17
               (or the last position of a shorter request) with beta = 450.
    """
    lens = np.asarray(lens, np.int64)
    t = int(lens.sum())
    u = np.where(rng.integers(0, 2, d) == 1, 1.0, -1.0).astype(np.float32)
    q = u[None, None, :] + 0.5 * rng.standard_normal((t, hq, d), dtype=np.float32)
    pos = np.concatenate([np.arange(n) for n in lens]) if t else np.zeros(0, np.int64)
    if pattern == "ramp":
        beta = rise * pos / 64.0
    elif pattern == "jump":
        beta = np.where(pos < 256, 0.0, 150.0 + rise * (pos - 256) / 64.0)
    elif pattern == "spike":
        beta = np.zeros(t)
        starts = np.concatenate([[0], np.cumsum(lens)[:-1]])
        for s0, n in zip(starts, lens):
            if n > 0:
                beta[s0 + min(64 * 5 + 17, n - 1)] = 450.0
    else:
        raise ValueError(pattern)
    k = (beta[:, None, None] / math.sqrt(d)) * u[None, None, :] + \
        0.5 * rng.standard_normal((t, hkv, d), dtype=np.float32)
    v = rng.standard_normal((t, hkv, d), dtype=np.float32)
    return (f32_to_bf16_bits(q.astype(np.float32)), f32_to_bf16_bits(k.astype(np.float32)),
            f32_to_bf16_bits(v))


def tiny_fp32(seed=SEED_BASE + 1, n_steps=8) -> Workload:
    """Tiny fp32 check: 4 requests {17,64,5,120}, 8/2 heads, d 64, 64-page pool,
    prefill then ``n_steps`` decode steps per request."""
    rng = np.random.default_rng(seed)
    lens = np.array([17, 64, 5, 120], dtype=np.int32)
    hq, hkv, d, dt = 8, 2, 64, "fp32"
    page_table, num_pages = allocate_pages(rng, lens + n_steps, pool_pages=64)
    q, k, v = prefill_batch(rng, lens, hq, hkv, d, dt)
    steps = []
    for _ in range(n_steps):
        steps.append((normal(rng, (4, hq, d), dt), normal(rng, (4, hkv, d), dt),
                      normal(rng, (4, hkv, d), dt)))
    k_pool, v_pool = empty_pools(num_pages, hkv, d, dt)
    return Workload("tiny_fp32_prefill_then_decode", seed, dt, hq, hkv, d, 1.0 / math.sqrt(d),
                    prefill_lens=lens, cu_seqlens=cu_from_lens(lens), q=q, k=k, v=v,
                    prefill_rows=np.arange(4, dtype=np.int32), num_pages=num_pages,
                    k_pool=k_pool, v_pool=v_pool, page_table=page_table, steps=steps)


def decode_workload(name, seed, ctx, hq, hkv, d, dtype="bf16") -> Workload:
    rng = np.random.default_rng(seed)
    ctx = np.asarray(ctx, dtype=np.int32)
    page_table, num_pages = allocate_pages(rng, ctx)
    k_pool, v_pool = empty_pools(num_pages, hkv, d, dtype)
    fill_live_slots(rng, k_pool, v_pool, page_table, ctx, dtype)
    q_dec = normal(rng, (len(ctx), hq, d), dtype)
    return Workload(name, seed, dtype, hq, hkv, d, 1.0 / math.sqrt(d), num_pages=num_pages,
                    k_pool=k_pool, v_pool=v_pool, page_table=page_table,
                    context_lens=ctx, q_dec=q_dec)


def decode_mha_7b(seed=SEED_BASE + 2) -> Workload:
    """Decode, MHA layer shaped like a 7B model: B 64, 32 heads, d 128, bf16,
    ctx lognormal(1024, 0.8) clipped to [16, 4096]."""
    rng = np.random.default_rng(seed)
    ctx = lognormal_lengths(rng, 64, 1024, 0.8, 16, 4096)
    w = decode_workload("decode_mha_7b_b64", seed, ctx, 32, 32, 128)
    return w


def varlen_prefill(seed=SEED_BASE + 3) -> Workload:
    """Varlen causal prefill + paged write: 16 prompts lognormal(1500, 1.0)
    clipped to [32, 8192], 32/32 heads, d 128, bf16."""
    rng = np.random.default_rng(seed)
    lens = lognormal_lengths(rng, 16, 1500, 1.0, 32, 8192)
    hq = hkv = 32
    d, dt = 128, "bf16"
    page_table, num_pages = allocate_pages(rng, lens)
    q, k, v = prefill_batch(rng, lens, hq, hkv, d, dt)
    k_pool, v_pool = empty_pools(num_pages, hkv, d, dt)
    return Workload("varlen_prefill_16_prompts", seed, dt, hq, hkv, d, 1.0 / math.sqrt(d),
                    prefill_lens=lens, cu_seqlens=cu_from_lens(lens), q=q, k=k, v=v,
                    prefill_rows=np.arange(16, dtype=np.int32), num_pages=num_pages,
                    k_pool=k_pool, v_pool=v_pool, page_table=page_table)


def decode_gqa_70b(seed=SEED_BASE + 4) -> Workload:
    """High-concurrency GQA decode, 70B-shaped: B 256, 64/8 heads, d 128, bf16;
    51 long contexts U[4096,16384] and 205 short U[100,500] at shuffled positions."""
    rng = np.random.default_rng(seed)
    ctx, is_long = bimodal_lengths(rng, 256, 0.2, 100, 500, 4096, 16384)
    w = decode_workload("decode_gqa_70b_b256", seed, ctx, 64, 8, 128)
    w.notes["n_long"] = int(is_long.sum())
    return w


def mixed_step(seed=SEED_BASE + 5, num_layers=1) -> Workload:
    """Mixed P/D step: 28/4 heads, d 128, bf16; prefill 8x512 writing the shared
    pool, 192 decode requests with ctx lognormal(2048, 0.7) clipped to
    [64, 16384], then the 8 prefilled requests are packed for handoff.

    Page-table rows 0..191 are the decode requests, 192..199 the prefill ones."""
    rng = np.random.default_rng(seed)
    hq, hkv, d, dt = 28, 4, 128, "bf16"
    n_dec, n_pre, pre_len = 192, 8, 512
    ctx = lognormal_lengths(rng, n_dec, 2048, 0.7, 64, 16384)
    pre_lens = np.full(n_pre, pre_len, dtype=np.int32)
    page_table, num_pages = allocate_pages(rng, np.concatenate([ctx, pre_lens]))
    k_pool, v_pool = empty_pools(num_pages, hkv, d, dt)
    fill_live_slots(rng, k_pool, v_pool, page_table[:n_dec], ctx, dt)
    q_dec = normal(rng, (n_dec, hq, d), dt)
    q, k, v = prefill_batch(rng, pre_lens, hq, hkv, d, dt)
    rows = np.arange(n_dec, n_dec + n_pre, dtype=np.int32)
    w = Workload("mixed_step_192_decode_8x512_prefill", seed, dt, hq, hkv, d, 1.0 / math.sqrt(d),
                 prefill_lens=pre_lens, cu_seqlens=cu_from_lens(pre_lens), q=q, k=k, v=v,
                 prefill_rows=rows, num_pages=num_pages, k_pool=k_pool, v_pool=v_pool,
                 page_table=page_table, context_lens=ctx, q_dec=q_dec,
                 handoff_reqs=rows.copy(), handoff_lens=pre_lens.copy())
    w.notes["num_layers"] = num_layers
    return w




def handoff_offsets(handoff_lens, num_layers, hkv, d) -> np.ndarray:
    """Back-to-back element offsets of each request's (layer, K/V, head, token, dim) block."""
    sizes = np.asarray(handoff_lens, dtype=np.int64) * (num_layers * 2 * hkv * d)
    off = np.zeros(len(sizes) + 1, dtype=np.int64)
    off[1:] = np.cumsum(sizes)
    return off
