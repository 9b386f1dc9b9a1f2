"""Pins the fp64 oracle to things other than itself (CPU only).

* an independent dense numpy formulation (oracle/brute.py),
* a library routine: torch.nn.functional.scaled_dot_product_attention in
  float64 on the CPU, GQA via repeat_interleave,
* closed forms and invariants of Eq. 1 (softmax rows sum to one, a single
  key returns its value, scale 0 or equal keys give the prefix mean, the
  two-key logistic form, log-sum-exp),
* invariance of decode under a random permutation of physical pages and
  equality of the last prefill row with a decode step on the same cache,
* the write/pack index maps against a plain reshape of their input.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle import brute
from paper_2511_20982_amd import inputs as I

RTOL = 1e-12


def rand_prefill(seed, lens, hq, hkv, d, dtype):
    rng = np.random.default_rng(seed)
    q, k, v = I.prefill_batch(rng, np.asarray(lens), hq, hkv, d, dtype)
    return q, k, v, I.cu_from_lens(lens)


SHAPES = [
    # lens, hq, hkv, d
    ([1], 1, 1, 8),
    ([5, 1, 9], 4, 4, 16),
    ([17, 3], 8, 2, 16),
    ([7, 12], 7, 1, 8),
    ([16, 33, 2], 8, 1, 32),
]


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("lens,hq,hkv,d", SHAPES)
def test_prefill_matches_dense_bruteforce(dtype, lens, hq, hkv, d):
    q, k, v, cu = rand_prefill(11, lens, hq, hkv, d, dtype)
    scale = 1.0 / math.sqrt(d)
    out, _ = oracle.prefill(q, k, v, cu, scale)
    ref = brute.prefill(q, k, v, cu, scale)
    np.testing.assert_allclose(out, ref, rtol=0, atol=RTOL * 10)


@pytest.mark.parametrize("lens,hq,hkv,d", SHAPES)
def test_prefill_matches_torch_sdpa_float64(lens, hq, hkv, d):
    q, k, v, cu = rand_prefill(12, lens, hq, hkv, d, "bf16")
    scale = 0.3
    out, _ = oracle.prefill(q, k, v, cu, scale)
    qf, kf, vf = (torch.from_numpy(brute.widen(x)) for x in (q, k, v))
    g = hq // hkv
    sigma = float(np.float32(scale))
    for r in range(len(lens)):
        a, b = int(cu[r]), int(cu[r + 1])
        qq = qf[a:b].transpose(0, 1)                                  # [Hq][L][d]
        kk = kf[a:b].transpose(0, 1).repeat_interleave(g, dim=0)      # [Hq][L][d]
        vv = vf[a:b].transpose(0, 1).repeat_interleave(g, dim=0)
        ref = torch.nn.functional.scaled_dot_product_attention(
            qq, kk, vv, is_causal=True, scale=sigma).transpose(0, 1).numpy()
        np.testing.assert_allclose(out[a:b], ref, rtol=0, atol=1e-11)


def test_prefill_lse_is_log_sum_exp_of_scores():
    q, k, v, cu = rand_prefill(13, [9, 4], 4, 2, 16, "fp32")
    scale = 0.25
    _, lse = oracle.prefill(q, k, v, cu, scale)
    qf, kf = q.astype(np.float64), k.astype(np.float64)
    sigma = float(np.float32(scale))
    for r in range(2):
        a, b = int(cu[r]), int(cu[r + 1])
        for h in range(4):
            for i in range(b - a):
                sc = [sigma * float(np.dot(qf[a + i, h], kf[a + j, h // 2])) for j in range(i + 1)]
                assert abs(lse[a + i, h] - np.logaddexp.reduce(sc)) < 1e-12


def test_softmax_rows_sum_to_one_and_equal_probabilities():
    # v_j = basis vector e_j: output row i is the probability row itself.
    L, d = 12, 16
    rng = np.random.default_rng(14)
    q = rng.standard_normal((L, 1, d), dtype=np.float32)
    k = rng.standard_normal((L, 1, d), dtype=np.float32)
    v = np.zeros((L, 1, d), np.float32)
    for j in range(L):
        v[j, 0, j] = 1.0
    out, _ = oracle.prefill(q, k, v, I.cu_from_lens([L]), 0.5)
    p = out[:, 0, :L]
    np.testing.assert_allclose(p.sum(axis=1), 1.0, rtol=0, atol=1e-14)
    assert np.all(np.triu(p, k=1) == 0.0)           # causal: nothing above the diagonal
    i = 7
    sc = np.array([0.5 * np.dot(q[i, 0].astype(np.float64), k[j, 0].astype(np.float64))
                   for j in range(i + 1)])
    np.testing.assert_allclose(p[i, :i + 1], np.exp(sc) / np.exp(sc).sum(), rtol=1e-13)


def test_closed_forms():
    rng = np.random.default_rng(15)
    L, d = 10, 8
    q = rng.standard_normal((L, 2, d), dtype=np.float32)
    k = rng.standard_normal((L, 1, d), dtype=np.float32)
    v = rng.standard_normal((L, 1, d), dtype=np.float32)
    cu = I.cu_from_lens([L])
    vf = v[:, 0].astype(np.float64)
    prefix_mean = np.cumsum(vf, axis=0) / np.arange(1, L + 1)[:, None]
    # single key -> its value, exactly
    out, lse = oracle.prefill(q[:1], k[:1], v[:1], I.cu_from_lens([1]), 0.7)
    assert np.array_equal(out[0, 0], vf[0]) and np.array_equal(out[0, 1], vf[0])
    # scale 0 -> prefix mean; lse = ln(i+1)
    out, lse = oracle.prefill(q, k, v, cu, 0.0)
    np.testing.assert_allclose(out[:, 0], prefix_mean, rtol=0, atol=1e-14)
    np.testing.assert_allclose(lse[:, 0], np.log(np.arange(1, L + 1)), rtol=0, atol=1e-14)
    # all keys equal -> prefix mean at any scale
    k_eq = np.repeat(k[:1], L, axis=0)
    out, _ = oracle.prefill(q, k_eq, v, cu, 1.3)
    np.testing.assert_allclose(out[:, 1], prefix_mean, rtol=0, atol=1e-14)
    # two keys, scores 0 and s -> logistic mix (Eq. 1 literally, scale 1)
    q2 = np.zeros((2, 1, 2), np.float32); q2[:, 0, 0] = 1.0
    k2 = np.zeros((2, 1, 2), np.float32); k2[1, 0, 0] = 2.0
    v2 = np.array([[[1.0, -3.0]], [[5.0, 0.5]]], np.float32)
    out, lse = oracle.prefill(q2, k2, v2, I.cu_from_lens([2]), 1.0)
    w1 = math.exp(2.0) / (1.0 + math.exp(2.0))
    v2d = v2.astype(np.float64)
    np.testing.assert_allclose(out[1, 0], (1 - w1) * v2d[0, 0] + w1 * v2d[1, 0], rtol=1e-14)
    assert abs(lse[1, 0] - math.log(1.0 + math.exp(2.0))) < 1e-15
    np.testing.assert_array_equal(out[0, 0], v2[0, 0])


def test_gqa_equals_mha_with_repeated_kv():
    q, k, v, cu = rand_prefill(16, [11, 6], 8, 2, 16, "bf16")
    out_gqa, lse_gqa = oracle.prefill(q, k, v, cu, 0.25)
    k_rep, v_rep = np.repeat(k, 4, axis=1), np.repeat(v, 4, axis=1)
    out_mha, lse_mha = oracle.prefill(q, k_rep, v_rep, cu, 0.25)
    assert np.array_equal(out_gqa, out_mha) and np.array_equal(lse_gqa, lse_mha)


def test_requests_are_independent():
    # Packing requests back to back must not let them see each other.
    q, k, v, cu = rand_prefill(17, [6, 9], 4, 2, 8, "fp32")
    both, _ = oracle.prefill(q, k, v, cu, 0.4)
    second, _ = oracle.prefill(q[6:], k[6:], v[6:], I.cu_from_lens([9]), 0.4)
    assert np.array_equal(both[6:], second)


# ------------------------------------------------------------------ paged path
def _write_prefill_into_pool(w):
    n = len(w.prefill_lens)
    return oracle.kv_write(w.k, w.v, w.k_pool, w.v_pool, w.page_table[w.prefill_rows],
                           w.cu_seqlens, np.zeros(n, np.int32))


def test_decode_matches_dense_bruteforce():
    w = I.decode_workload("t", 5, [1, 15, 16, 17, 40], 8, 2, 32, "bf16")
    out, _ = oracle.decode(w.q_dec, w.k_pool, w.v_pool, w.page_table, w.context_lens, w.scale)
    ref = brute.decode(w.q_dec, w.k_pool, w.v_pool, w.page_table, w.context_lens, w.scale)
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)
    assert np.all(np.isfinite(out))                  # NaN poison in dead slots never read


def test_decode_invariant_under_page_permutation():
    w = I.decode_workload("t", 6, [3, 31, 64, 50], 4, 4, 16, "bf16")
    out1, lse1 = oracle.decode(w.q_dec, w.k_pool, w.v_pool, w.page_table, w.context_lens, w.scale)
    rng = np.random.default_rng(99)
    perm = rng.permutation(w.num_pages)             # new physical location of each page
    k2 = np.empty_like(w.k_pool); v2 = np.empty_like(w.v_pool)
    k2[perm] = w.k_pool; v2[perm] = w.v_pool
    pt2 = np.where(w.page_table >= 0, perm[np.maximum(w.page_table, 0)], -1).astype(np.int32)
    out2, lse2 = oracle.decode(w.q_dec, k2, v2, pt2, w.context_lens, w.scale)
    assert np.array_equal(out1, out2) and np.array_equal(lse1, lse2)


def test_tiny_fp32_last_prefill_row_equals_decode_step():
    w = I.tiny_fp32()
    out_p, lse_p = oracle.prefill(w.q, w.k, w.v, w.cu_seqlens, w.scale)
    kp, vp = _write_prefill_into_pool(w)
    last = w.cu_seqlens[1:] - 1
    out_d, lse_d = oracle.decode(w.q[last], kp, vp, w.page_table, w.prefill_lens, w.scale)
    np.testing.assert_allclose(out_d, out_p[last], rtol=0, atol=1e-13)
    np.testing.assert_allclose(lse_d, lse_p[last], rtol=0, atol=1e-13)


def test_tiny_fp32_decode_steps_equal_prefill_over_extended_sequence():
    # Appending step tokens with kv_write and decoding must equal a prefill over
    # the prompt extended by those tokens (the row of the appended token).
    w = I.tiny_fp32()
    kp, vp = _write_prefill_into_pool(w)
    n = len(w.prefill_lens)
    ones = I.cu_from_lens(np.ones(n, np.int32))
    qs, ks, vs = [], [], []
    for s, (qd, kd, vd) in enumerate(w.steps):
        kp, vp = oracle.kv_write(kd, vd, kp, vp, w.page_table, ones, w.prefill_lens + s)
        out_d, _ = oracle.decode(qd, kp, vp, w.page_table, w.prefill_lens + s + 1, w.scale)
        qs.append(qd); ks.append(kd); vs.append(vd)
    # extended sequences, rebuilt request by request
    lens2 = w.prefill_lens + len(w.steps)
    q2, k2, v2 = [], [], []
    for r in range(n):
        a, b = w.cu_seqlens[r], w.cu_seqlens[r + 1]
        q2.append(np.concatenate([w.q[a:b]] + [x[r:r + 1] for x in qs]))
        k2.append(np.concatenate([w.k[a:b]] + [x[r:r + 1] for x in ks]))
        v2.append(np.concatenate([w.v[a:b]] + [x[r:r + 1] for x in vs]))
    cu2 = I.cu_from_lens(lens2)
    out_p, _ = oracle.prefill(np.concatenate(q2), np.concatenate(k2), np.concatenate(v2), cu2,
                              w.scale)
    np.testing.assert_allclose(out_d, out_p[cu2[1:] - 1], rtol=0, atol=1e-13)


def test_kv_write_then_pack_is_a_transpose_of_the_input():
    rng = np.random.default_rng(21)
    lens = np.array([5, 16, 33], np.int32)
    hkv, d = 3, 8
    pt, num_pages = I.allocate_pages(rng, lens, pool_pages=12)
    kp, vp = I.empty_pools(num_pages, hkv, d, "bf16")
    knew = I.normal(rng, (int(lens.sum()), hkv, d), "bf16")
    vnew = I.normal(rng, (int(lens.sum()), hkv, d), "bf16")
    cu = I.cu_from_lens(lens)
    kp2, vp2 = oracle.kv_write(knew, vnew, kp, vp, pt, cu, np.zeros(3, np.int32))
    off = I.handoff_offsets(lens, 1, hkv, d)
    out = oracle.pack(kp2, vp2, 1, pt, np.arange(3), lens, off)
    for r in range(3):
        a, b = cu[r], cu[r + 1]
        expect = np.stack([knew[a:b].transpose(1, 0, 2), vnew[a:b].transpose(1, 0, 2)])
        assert np.array_equal(out[off[r]:off[r + 1]], expect.reshape(-1))
    # every slot not written keeps its poison; every written slot is finite
    written_k = ~np.isnan(I.bf16_bits_to_f32(kp2))
    assert written_k.sum() == int(lens.sum()) * hkv * d
    assert (~np.isnan(I.bf16_bits_to_f32(vp2))).sum() == int(lens.sum()) * hkv * d


def test_kv_write_slots_follow_the_page_table():
    # Token p of request r lands in page pt[r][p // 16], slot p % 16: K row-major
    # within the page, V with the slot as the fastest dimension.
    hkv, d = 2, 4
    pt = np.array([[3, 0]], np.int32)
    kp, vp = I.empty_pools(4, hkv, d, "fp32")
    knew = np.arange(20 * hkv * d, dtype=np.float32).reshape(20, hkv, d)
    vnew = -knew
    kp2, vp2 = oracle.kv_write(knew, vnew, kp, vp, pt, I.cu_from_lens([20]), np.zeros(1, np.int32))
    assert np.array_equal(kp2[3, 1, 5], knew[5, 1])
    assert np.array_equal(vp2[3, 1, :, 5], vnew[5, 1])
    assert np.array_equal(kp2[0, 0, 3], knew[19, 0])
    assert np.array_equal(vp2[0, 0, :, 3], vnew[19, 0])
    assert np.isnan(kp2[0, 0, 4]).all() and np.isnan(kp2[1]).all() and np.isnan(kp2[2]).all()


def test_pack_multi_layer_order():
    rng = np.random.default_rng(22)
    L, hkv, d, P = 2, 2, 4, 3
    kp = rng.standard_normal((L, P, hkv, 16, d)).astype(np.float32)
    vp = rng.standard_normal((L, P, hkv, d, 16)).astype(np.float32)
    pt = np.array([[2, 0], [1, -1]], np.int32)
    lens = np.array([20, 7], np.int32)
    off = I.handoff_offsets(lens, L, hkv, d)
    out = oracle.pack(kp, vp, L, pt, np.array([0, 1]), lens, off)
    blk = out[off[0]:off[1]].reshape(L, 2, hkv, 20, d)
    assert np.array_equal(blk[1, 0, 1, 17], kp[1, 0, 1, 1])
    assert np.array_equal(blk[1, 1, 0, 3], vp[1, 2, 0, :, 3])
    blk2 = out[off[1]:off[2]].reshape(L, 2, hkv, 7, d)
    assert np.array_equal(blk2[0, 1, 1, 6], vp[0, 1, 1, :, 6])


def test_unpack_inverts_pack_into_another_page_order():
    # P -> D handoff: pack from one pool, unpack into a pool with another page
    # permutation; every written slot matches, every other slot keeps its poison,
    # and decode over both caches is bit-identical.
    rng = np.random.default_rng(23)
    lens = np.array([37, 16, 1], np.int32)
    hkv, d, layers = 2, 8, 2
    pt_a, n_a = I.allocate_pages(rng, lens, pool_pages=9)
    pt_b, n_b = I.allocate_pages(rng, lens, pool_pages=11)
    ka, va = I.empty_pools(n_a, hkv, d, "bf16", num_layers=layers)
    for layer in range(layers):
        I.fill_live_slots(rng, ka[layer], va[layer], pt_a, lens, "bf16")
    off = I.handoff_offsets(lens, layers, hkv, d)
    req = np.arange(3, dtype=np.int32)
    buf = oracle.pack(ka, va, layers, pt_a, req, lens, off)
    kb0, vb0 = I.empty_pools(n_b, hkv, d, "bf16", num_layers=layers)
    kb, vb = oracle.unpack(buf, off, req, lens, kb0, vb0, layers, pt_b)
    assert np.array_equal(oracle.pack(kb, vb, layers, pt_b, req, lens, off), buf)
    live = (~np.isnan(I.bf16_bits_to_f32(kb))).sum()
    assert live == layers * int(lens.sum()) * hkv * d
    q = I.normal(rng, (3, 4, d), "bf16")
    for layer in range(layers):
        oa, la = oracle.decode(q, ka[layer], va[layer], pt_a, lens, 0.35)
        ob, lb = oracle.decode(q, kb[layer], vb[layer], pt_b, lens, 0.35)
        assert np.array_equal(oa, ob) and np.array_equal(la, lb)


# ---- chunk prefill over the paged cache (prefix-aware, chunk at the end) ----
def _paged_case(seed, prefix, chunk, hq, hkv, d, dtype, extra_pages=3):
    """Requests with cached prefixes whose chunks are already written: full
    sequences of prefix+chunk tokens go through the paged write (start 0), and
    the chunk rows of Q are drawn separately."""
    rng = np.random.default_rng(seed)
    prefix, chunk = np.asarray(prefix, np.int32), np.asarray(chunk, np.int32)
    total = prefix + chunk
    pt, num_pages = I.allocate_pages(rng, total, pool_pages=int(np.sum((total + 15) // 16)) + extra_pages)
    k_pool, v_pool = I.empty_pools(num_pages, hkv, d, dtype)
    _, kf, vf = I.prefill_batch(rng, total, hq, hkv, d, dtype)
    k_pool, v_pool = oracle.kv_write(kf, vf, k_pool, v_pool, pt, I.cu_from_lens(total),
                                     np.zeros(len(total), np.int32))
    q = I.normal(rng, (int(chunk.sum()), hq, d), dtype)
    return q, k_pool, v_pool, pt, I.cu_from_lens(chunk), prefix


PAGED = [
    # prefix, chunk, hq, hkv, d
    ([0], [9], 2, 1, 8),
    ([16, 5, 0], [1, 7, 20], 4, 2, 16),
    ([33, 47], [16, 3], 8, 2, 8),
    ([100], [40], 3, 1, 16),
]


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("prefix,chunk,hq,hkv,d", PAGED)
def test_prefill_paged_matches_dense_bruteforce(dtype, prefix, chunk, hq, hkv, d):
    q, kp, vp, pt, cu, pre = _paged_case(21, prefix, chunk, hq, hkv, d, dtype)
    out, _ = oracle.prefill_paged(q, kp, vp, pt, cu, pre, 0.37)
    ref = brute.prefill_paged(q, kp, vp, pt, cu, pre, 0.37)
    assert np.isfinite(out).all() and np.isfinite(ref).all()
    np.testing.assert_allclose(out, ref, rtol=0, atol=RTOL * 10)


@pytest.mark.parametrize("pieces", [[40], [1, 39], [16, 16, 8], [5, 1, 30, 4], [1] * 12 + [28]])
def test_chunked_prefill_equals_one_shot(pieces):
    """A prompt processed chunk by chunk (each chunk written to the cache and
    attended with the earlier chunks as its prefix) gives the one-shot prefill."""
    rng = np.random.default_rng(23)
    hq, hkv, d, L = 4, 2, 16, int(sum(pieces))
    q, k, v = I.prefill_batch(rng, np.array([L]), hq, hkv, d, "bf16")
    ref, ref_lse = oracle.prefill(q, k, v, I.cu_from_lens([L]), 0.25)
    pt, num_pages = I.allocate_pages(rng, np.array([L]), pool_pages=(L + 15) // 16 + 4)
    kp, vp = I.empty_pools(num_pages, hkv, d, "bf16")
    done = 0
    for n in pieces:
        rows = slice(done, done + n)
        kp, vp = oracle.kv_write(k[rows], v[rows], kp, vp, pt, I.cu_from_lens([n]),
                                 np.array([done], np.int32))
        out, lse = oracle.prefill_paged(q[rows], kp, vp, pt, I.cu_from_lens([n]),
                                        np.array([done], np.int32), 0.25)
        np.testing.assert_allclose(out, ref[rows], rtol=0, atol=1e-12)
        np.testing.assert_allclose(lse, ref_lse[rows], rtol=0, atol=1e-12)
        done += n


def test_prefill_paged_chunk_of_one_is_a_decode_step():
    q, kp, vp, pt, cu, pre = _paged_case(24, [30, 0, 17], [1, 1, 1], 4, 1, 16, "bf16")
    out, lse = oracle.prefill_paged(q, kp, vp, pt, cu, pre, 0.3)
    dec, dlse = oracle.decode(q, kp, vp, pt, pre + 1, 0.3)
    assert np.isfinite(out).all()
    np.testing.assert_allclose(out, dec, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, dlse, rtol=0, atol=1e-12)


def test_prefill_paged_invariant_under_page_permutation():
    q, kp, vp, pt, cu, pre = _paged_case(25, [20, 3], [13, 30], 4, 2, 8, "bf16")
    out, _ = oracle.prefill_paged(q, kp, vp, pt, cu, pre, 0.3)
    rng = np.random.default_rng(5)
    perm = rng.permutation(kp.shape[0])          # new page id of old page p: perm[p]
    kp2, vp2 = np.empty_like(kp), np.empty_like(vp)
    kp2[perm], vp2[perm] = kp, vp
    pt2 = np.where(pt >= 0, perm[np.maximum(pt, 0)], -1).astype(np.int32)
    out2, _ = oracle.prefill_paged(q, kp2, vp2, pt2, cu, pre, 0.3)
    assert np.isfinite(out).all() and np.array_equal(out, out2)


def test_prefill_paged_sampled_rows_match_full():
    q, kp, vp, pt, cu, pre = _paged_case(26, [18, 40], [22, 9], 6, 3, 16, "fp32")
    out, lse = oracle.prefill_paged(q, kp, vp, pt, cu, pre, 0.2)
    tok = np.array([0, 5, 21, 22, 30], np.int32)
    head = np.array([0, 5, 3, 1, 2], np.int32)
    o2, l2 = oracle.prefill_paged(q, kp, vp, pt, cu, pre, 0.2, tok=tok, head=head)
    assert np.isfinite(out).all()
    assert np.array_equal(o2, out[tok, head]) and np.array_equal(l2, lse[tok, head])
