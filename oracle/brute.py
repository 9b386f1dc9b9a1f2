"""Dense numpy fp64 brute force of Eq. 1 (softmax(sigma*Q K^T + mask) V).

TEST INFRASTRUCTURE ONLY.  Written as whole-matrix algebra, independently of
the loop-form C oracle, so that each pins the other on tiny inputs.  The KV
head of query head h is h // (Hq/Hkv).
"""
from __future__ import annotations

import numpy as np


def widen(a: np.ndarray) -> np.ndarray:
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


def softmax_rows(s: np.ndarray) -> np.ndarray:
    m = np.max(s, axis=-1, keepdims=True)
    p = np.exp(s - m)
    return p / np.sum(p, axis=-1, keepdims=True)


def attention_dense(q, k, v, sigma, causal):
    """q[L][d], k/v[N][d]; causal aligns query i with key i (top-left)."""
    s = sigma * (q @ k.T)
    if causal:
        mask = np.triu(np.ones((q.shape[0], k.shape[0]), dtype=bool), k=1)
        s = np.where(mask, -np.inf, s)
    return softmax_rows(s) @ v


def prefill(q, k, v, cu_seqlens, scale):
    q, k, v = widen(q), widen(k), widen(v)
    sigma = float(np.float32(scale))
    hq, hkv = q.shape[1], k.shape[1]
    g = hq // hkv
    out = np.zeros_like(q)
    for r in range(len(cu_seqlens) - 1):
        a, b = int(cu_seqlens[r]), int(cu_seqlens[r + 1])
        for h in range(hq):
            out[a:b, h] = attention_dense(q[a:b, h], k[a:b, h // g], v[a:b, h // g], sigma, True)
    return out


def gather_context(k_pool, v_pool, page_table, r, ctx, page_size=16):
    """Contiguous K[ctx][Hkv][d], V[ctx][Hkv][d] of request r from the paged pools."""
    j = np.arange(ctx)
    pages = page_table[r, j // page_size]
    slots = j % page_size
    kk = k_pool[pages, :, slots, :]                 # [ctx][Hkv][d]
    vv = v_pool[pages, :, :, slots]                 # [ctx][Hkv][d]
    return kk, vv


def decode(q, k_pool, v_pool, page_table, context_lens, scale):
    qf = widen(q)
    sigma = float(np.float32(scale))
    hq, hkv = q.shape[1], k_pool.shape[1]
    g = hq // hkv
    out = np.zeros_like(qf)
    for r in range(q.shape[0]):
        kk, vv = gather_context(k_pool, v_pool, page_table, r, int(context_lens[r]))
        kk, vv = widen(kk), widen(vv)
        for h in range(hq):
            out[r, h] = attention_dense(qf[r, h][None, :], kk[:, h // g], vv[:, h // g],
                                        sigma, False)[0]
    return out


def prefill_paged(q, k_pool, v_pool, page_table, cu_q, prefix_lens, scale):
    """Chunk prefill over the paged cache as dense masked algebra: request r's
    cached sequence (prefix + chunk, already in the pools) is gathered whole,
    and chunk row i may see key j iff j <= prefix_lens[r] + i (the chunk sits
    at the end of the cache)."""
    qf = widen(q)
    sigma = float(np.float32(scale))
    hq, hkv = q.shape[1], k_pool.shape[1]
    g = hq // hkv
    out = np.zeros_like(qf)
    for r in range(len(cu_q) - 1):
        a, b = int(cu_q[r]), int(cu_q[r + 1])
        n, pre = b - a, int(prefix_lens[r])
        if n == 0:
            continue
        kk, vv = gather_context(k_pool, v_pool, page_table, r, pre + n)
        kk, vv = widen(kk), widen(vv)
        rows = np.arange(n)[:, None] + pre
        cols = np.arange(pre + n)[None, :]
        for h in range(hq):
            s = sigma * (qf[a:b, h] @ kk[:, h // g].T)
            s = np.where(cols > rows, -np.inf, s)
            out[a:b, h] = softmax_rows(s) @ vv[:, h // g]
    return out
