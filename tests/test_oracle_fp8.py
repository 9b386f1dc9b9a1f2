"""Pins of the oracle's FP8 (OCP E4M3) KV-page functions.

The code table is pinned against its closed form and against PyTorch's
float8_e4m3fn type (a library routine); the encoder against brute force over
the 253 finite values, the tie-to-even midpoints and saturation; the decode
over E4M3 pools against the dense brute force over the dequantised values, the
fp32 decode over the same values where they are exact in fp32, and the exact
scale identities, for the decode and for the chunk prefill over E4M3 pools
(against the dense brute force over the dequantised values as well).
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import brute
from paper_2511_20982_amd import inputs as I

CODES = np.arange(256)
FINITE = np.array([c for c in range(256) if c & 0x7F != 0x7F])


def _closed_form(c):
    s, e, m = c >> 7, (c >> 3) & 15, c & 7
    if e == 15 and m == 7:
        return float("nan")
    v = (m / 8.0) * 2.0 ** -6 if e == 0 else (1 + m / 8.0) * 2.0 ** (e - 7)
    return -v if s else v


def test_value_table_closed_form_and_torch():
    v = oracle.e4m3_value(CODES)
    ref = np.array([_closed_form(c) for c in CODES])
    assert np.array_equal(np.isnan(v), np.isnan(ref))
    assert np.array_equal(v[FINITE], ref[FINITE])
    t = torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    assert np.array_equal(v[FINITE], t[FINITE]) and np.isnan(t[[0x7F, 0xFF]]).all()
    pos = v[:0x7F]
    assert np.all(np.diff(pos) > 0)                      # codes 0..126 increase
    assert pos[-1] == 448.0 and pos[1] == 2.0 ** -9 and v[8] == 2.0 ** -6
    assert np.signbit(v[0x80]) and v[0x80] == 0.0        # negative zero


def test_encode_round_trip_every_code():
    v = oracle.e4m3_value(FINITE).astype(np.float32)
    assert np.array_equal(oracle.e4m3_encode(v), FINITE.astype(np.uint8))


def _brute_encode(y):
    """Nearest finite value (ties: even code), saturating."""
    vals = oracle.e4m3_value(np.arange(0x7F))                        # 0 .. 448
    out = []
    for x in np.asarray(y, np.float64):
        a = min(abs(x), 448.0)
        dist = np.abs(vals - a)
        best = np.flatnonzero(dist == dist.min())
        c = int(best[0]) if len(best) == 1 else int(best[best % 2 == 0][0])
        out.append(c | (0x80 if np.signbit(x) else 0))
    return np.array(out, np.uint8)


def test_encode_midpoints_tie_to_even():
    v = oracle.e4m3_value(np.arange(0x7F))
    mids = ((v[:-1] + v[1:]) / 2).astype(np.float32)
    assert np.array_equal(mids.astype(np.float64), (v[:-1] + v[1:]) / 2)   # exact in fp32
    got = oracle.e4m3_encode(mids)
    lo = np.arange(0x7E)
    want = np.where(lo % 2 == 0, lo, lo + 1).astype(np.uint8)
    assert np.array_equal(got, want)
    assert np.array_equal(oracle.e4m3_encode(-mids), want | 0x80)
    # One fp32 ulp either side of a midpoint leaves the tie.
    up = np.nextafter(mids, np.float32(np.inf))
    dn = np.nextafter(mids, np.float32(0))
    assert np.array_equal(oracle.e4m3_encode(up), (lo + 1).astype(np.uint8))
    assert np.array_equal(oracle.e4m3_encode(dn), lo.astype(np.uint8))


def test_encode_random_against_brute_force_and_torch():
    rng = np.random.default_rng(8)
    y = np.concatenate([rng.standard_normal(3000) * 3, rng.standard_normal(1000) * 1e-2,
                        rng.uniform(-460, 460, 1000), [0.0, -0.0, 2.0 ** -10, 2.0 ** -9 * 0.5,
                                                       2.0 ** -9 * 1.5]]).astype(np.float32)
    got = oracle.e4m3_encode(y)
    assert np.array_equal(got, _brute_encode(y))
    inr = np.abs(y) < 448
    t = torch.from_numpy(y[inr]).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(got[inr], t)


def test_encode_saturates_and_keeps_nan():
    y = np.array([448, 449, 464, 480, 1e6, np.inf, -448, -500, -np.inf], np.float32)
    assert list(oracle.e4m3_encode(y)) == [0x7E] * 6 + [0xFE] * 3
    n = oracle.e4m3_encode(np.array([np.nan], np.float32))[0]
    assert n & 0x7F == 0x7F


def test_quantize_per_head_scale():
    rng = np.random.default_rng(9)
    x = I.normal(rng, (7, 3, 16), "bf16")
    scale = np.array([0.25, 3.0 / 448, 1.7], np.float32)
    codes = oracle.e4m3_quantize(x, scale)
    xf = I.bf16_bits_to_f32(x)
    inv = np.float32(1) / scale                        # fp32, nearest even
    y = (xf * inv[None, :, None]).astype(np.float32)
    assert np.array_equal(codes.ravel(), _brute_encode(y.ravel()))
    # A power-of-two scale divides exactly.
    assert np.array_equal(codes[:, 0], oracle.e4m3_encode(xf[:, 0] * 4))
    # The smallest scale saturates the tails of N(0,1) at +-448 * scale.
    v = oracle.e4m3_value(codes[:, 1]) * scale[1]
    assert np.max(np.abs(v)) <= 3.0 + 1e-12
    with pytest.raises(ValueError):
        oracle.e4m3_quantize(x, np.array([1.0, 0.0, 1.0], np.float32))


def _fp8_case(rng, ctx, hq, hkv, d, ks, vs):
    """Decode case with E4M3 pools: bf16 cache quantised by the oracle."""
    w = I.decode_workload("t", int(rng.integers(1 << 30)), ctx, hq, hkv, d, "bf16")
    kp = oracle.e4m3_quantize(w.k_pool.transpose(0, 2, 1, 3).reshape(-1, hkv, d), ks)
    kp = kp.reshape(w.k_pool.shape[0], 16, hkv, d).transpose(0, 2, 1, 3).copy()
    vp = oracle.e4m3_quantize(w.v_pool.transpose(0, 3, 1, 2).reshape(-1, hkv, d), vs)
    vp = vp.reshape(w.v_pool.shape[0], 16, hkv, d).transpose(0, 2, 3, 1).copy()
    return w, kp, vp


def test_decode_e4m3_against_brute_force():
    rng = np.random.default_rng(10)
    ks = np.array([6 / 448, 5 / 448], np.float32)
    vs = np.array([4 / 448, 7 / 448], np.float32)
    w, kp, vp = _fp8_case(rng, [1, 15, 16, 17, 40], 8, 2, 16, ks, vs)
    out, lse = oracle.decode_e4m3(w.q_dec, kp, vp, ks, vs, w.page_table, w.context_lens, w.scale)
    kd = oracle.e4m3_value(kp) * ks[None, :, None, None]
    vd = oracle.e4m3_value(vp) * vs[None, :, None, None]
    live = np.isfinite(out)
    assert live.all()
    ref = brute.decode(w.q_dec, kd, vd, w.page_table, w.context_lens, w.scale)
    assert np.max(np.abs(out - ref)) < 1e-12
    # LSE of the dequantised scores.
    qf = brute.widen(w.q_dec)
    for r in range(len(w.context_lens)):
        kk, _ = brute.gather_context(kd, vd, w.page_table, r, int(w.context_lens[r]))
        for h in range(8):
            s = float(np.float32(w.scale)) * (kk[:, h // 4] @ qf[r, h])
            assert abs(lse[r, h] - np.logaddexp.reduce(s)) < 1e-11


def test_decode_e4m3_equals_fp32_decode_of_exact_values():
    # value * scale is exact in fp32 when the scale has few significant bits.
    rng = np.random.default_rng(11)
    ks = np.array([49 / 4096, 3 / 256], np.float32)
    vs = np.array([5 / 512, 1 / 64], np.float32)
    w, kp, vp = _fp8_case(rng, [3, 32, 33, 70], 4, 2, 16, ks, vs)
    kd = (oracle.e4m3_value(kp) * ks[None, :, None, None])
    vd = (oracle.e4m3_value(vp) * vs[None, :, None, None])
    fin = np.isfinite(kd)
    assert np.array_equal(kd[fin].astype(np.float32).astype(np.float64), kd[fin])
    q32 = I.bf16_bits_to_f32(w.q_dec)
    a, la = oracle.decode_e4m3(q32, kp, vp, ks, vs, w.page_table, w.context_lens, w.scale)
    b, lb = oracle.decode(q32, kd.astype(np.float32), vd.astype(np.float32), w.page_table,
                          w.context_lens, w.scale)
    assert np.array_equal(a, b) and np.array_equal(la, lb)


def test_decode_e4m3_scale_identities():
    rng = np.random.default_rng(12)
    ks = np.array([0.01, 0.02], np.float32)
    vs = np.array([0.03, 0.015], np.float32)
    w, kp, vp = _fp8_case(rng, [5, 48, 20], 4, 2, 32, ks, vs)
    base, lse = oracle.decode_e4m3(w.q_dec, kp, vp, ks, vs, w.page_table, w.context_lens, 0.125)
    # Doubling every V scale doubles the output exactly.
    o2, l2 = oracle.decode_e4m3(w.q_dec, kp, vp, ks, vs * 2, w.page_table, w.context_lens, 0.125)
    assert np.array_equal(o2, 2 * base) and np.array_equal(l2, lse)
    # Doubling the K scales is doubling the softmax scale.
    o3, l3 = oracle.decode_e4m3(w.q_dec, kp, vp, ks * 2, vs, w.page_table, w.context_lens, 0.125)
    o4, l4 = oracle.decode_e4m3(w.q_dec, kp, vp, ks, vs, w.page_table, w.context_lens, 0.25)
    assert np.max(np.abs(o3 - o4)) < 1e-13 and np.max(np.abs(l3 - l4)) < 1e-12
    # Context of one: the output is that token's dequantised V.
    ctx1 = np.ones_like(w.context_lens)
    o5, _ = oracle.decode_e4m3(w.q_dec, kp, vp, ks, vs, w.page_table, ctx1, 0.125)
    for r in range(len(ctx1)):
        p = w.page_table[r, 0]
        for h in range(4):
            assert np.array_equal(o5[r, h], oracle.e4m3_value(vp[p, h // 2, :, 0]) * vs[h // 2])


def test_fp8_pages_write_pack_bit_exact():
    # The paged writer and the packer are byte copies: E4M3 codes go through
    # them like any other element type.
    rng = np.random.default_rng(13)
    lens = np.array([5, 16, 33], np.int32)
    hkv, d = 2, 16
    pt, num_pages = I.allocate_pages(rng, lens, pool_pages=10)
    k = rng.integers(0, 256, (int(lens.sum()), hkv, d)).astype(np.uint8)
    v = rng.integers(0, 256, (int(lens.sum()), hkv, d)).astype(np.uint8)
    kp0 = np.full((num_pages, hkv, 16, d), 0x7F, np.uint8)
    vp0 = np.full((num_pages, hkv, d, 16), 0x7F, np.uint8)
    cu = I.cu_from_lens(lens)
    kp, vp = oracle.kv_write(k, v, kp0, vp0, pt, cu, np.zeros(3, np.int32))
    for r in range(3):
        for t in range(lens[r]):
            pg, sl = pt[r, t // 16], t % 16
            assert np.array_equal(kp[pg, :, sl, :], k[cu[r] + t])
            assert np.array_equal(vp[pg, :, :, sl], v[cu[r] + t])
    off = I.handoff_offsets(lens, 1, hkv, d)
    buf = oracle.pack(kp, vp, 1, pt, np.arange(3, dtype=np.int32), lens, off)
    for r in range(3):
        blk = buf[off[r]:off[r + 1]].reshape(2, hkv, lens[r], d)
        assert np.array_equal(blk[0], k[cu[r]:cu[r + 1]].transpose(1, 0, 2))
        assert np.array_equal(blk[1], v[cu[r]:cu[r + 1]].transpose(1, 0, 2))


# ---- chunk prefill over E4M3 pools -------------------------------------------
def _quantize_pools(kp, vp, ks, vs):
    """E4M3 codes of bf16 pools [P][Hkv][16][d] / [P][Hkv][d][16], one scale per
    KV head (poisoned slots stay NaN codes)."""
    p, hkv, _, d = kp.shape
    k8 = oracle.e4m3_quantize(kp.transpose(0, 2, 1, 3).reshape(-1, hkv, d), ks)
    k8 = k8.reshape(p, 16, hkv, d).transpose(0, 2, 1, 3).copy()
    v8 = oracle.e4m3_quantize(vp.transpose(0, 3, 1, 2).reshape(-1, hkv, d), vs)
    v8 = v8.reshape(p, 16, hkv, d).transpose(0, 2, 3, 1).copy()
    return k8, v8


def _paged_fp8_case(seed, prefix, chunk, hq, hkv, d, ks, vs):
    rng = np.random.default_rng(seed)
    prefix, chunk = np.asarray(prefix, np.int32), np.asarray(chunk, np.int32)
    total = prefix + chunk
    pt, num_pages = I.allocate_pages(rng, np.maximum(total, 1))
    kp, vp = I.empty_pools(num_pages, hkv, d, "bf16")
    _, kf, vf = I.prefill_batch(rng, total, hq, hkv, d, "bf16")
    kp, vp = oracle.kv_write(kf, vf, kp, vp, pt, I.cu_from_lens(total),
                             np.zeros(len(total), np.int32))
    k8, v8 = _quantize_pools(kp, vp, ks, vs)
    q = I.normal(rng, (int(chunk.sum()), hq, d), "bf16")
    return q, k8, v8, pt, I.cu_from_lens(chunk), prefix


def _dequant(k8, v8, ks, vs):
    return (oracle.e4m3_value(k8) * ks.astype(np.float64)[None, :, None, None],
            oracle.e4m3_value(v8) * vs.astype(np.float64)[None, :, None, None])


PF_PREFIX = [0, 1, 15, 16, 17, 40, 0, 33]
PF_CHUNK = [3, 1, 16, 2, 20, 9, 0, 1]


def test_prefill_paged_e4m3_against_brute_force():
    ks = np.array([6 / 448, 5 / 448], np.float32)
    vs = np.array([4 / 448, 7 / 448], np.float32)
    q, k8, v8, pt, cu, pre = _paged_fp8_case(14, PF_PREFIX, PF_CHUNK, 8, 2, 16, ks, vs)
    out, lse = oracle.prefill_paged_e4m3(q, k8, v8, ks, vs, pt, cu, pre, 0.25)
    assert np.isfinite(out).all() and np.isfinite(lse).all()
    kd, vd = _dequant(k8, v8, ks, vs)
    ref = brute.prefill_paged(q, kd, vd, pt, cu, pre, 0.25)
    assert np.max(np.abs(out - ref)) < 1e-12
    qf = brute.widen(q)
    for r in range(len(pre)):
        for i in range(cu[r + 1] - cu[r]):
            kk, _ = brute.gather_context(kd, vd, pt, r, int(pre[r]) + i + 1)
            for h in range(8):
                s = 0.25 * (kk[:, h // 4] @ qf[cu[r] + i, h])
                assert abs(lse[cu[r] + i, h] - np.logaddexp.reduce(s)) < 1e-11


def test_prefill_paged_e4m3_equals_fp32_prefill_of_exact_values():
    ks = np.array([49 / 4096, 3 / 256], np.float32)
    vs = np.array([5 / 512, 1 / 64], np.float32)
    q, k8, v8, pt, cu, pre = _paged_fp8_case(15, PF_PREFIX, PF_CHUNK, 4, 2, 16, ks, vs)
    kd, vd = _dequant(k8, v8, ks, vs)
    fin = np.isfinite(kd)
    assert np.array_equal(kd[fin].astype(np.float32).astype(np.float64), kd[fin])
    q32 = I.bf16_bits_to_f32(q)
    a, la = oracle.prefill_paged_e4m3(q32, k8, v8, ks, vs, pt, cu, pre, 0.125)
    b, lb = oracle.prefill_paged(q32, kd.astype(np.float32), vd.astype(np.float32), pt, cu, pre,
                                 0.125)
    assert np.array_equal(a, b) and np.array_equal(la, lb)


def test_prefill_paged_e4m3_chunk_of_one_is_decode():
    ks = np.array([0.01, 0.02], np.float32)
    vs = np.array([0.03, 0.015], np.float32)
    prefix = np.array([30, 0, 17, 64], np.int32)
    q, k8, v8, pt, cu, pre = _paged_fp8_case(16, prefix, [1, 1, 1, 1], 4, 2, 32, ks, vs)
    out, lse = oracle.prefill_paged_e4m3(q, k8, v8, ks, vs, pt, cu, pre, 0.2)
    dec, dlse = oracle.decode_e4m3(q, k8, v8, ks, vs, pt, pre + 1, 0.2)
    assert np.max(np.abs(out - dec)) < 1e-14 and np.max(np.abs(lse - dlse)) < 1e-13


def test_prefill_paged_e4m3_scale_identities():
    ks = np.array([0.01, 0.02], np.float32)
    vs = np.array([0.03, 0.015], np.float32)
    q, k8, v8, pt, cu, pre = _paged_fp8_case(17, PF_PREFIX, PF_CHUNK, 4, 2, 32, ks, vs)
    base, lse = oracle.prefill_paged_e4m3(q, k8, v8, ks, vs, pt, cu, pre, 0.125)
    o2, l2 = oracle.prefill_paged_e4m3(q, k8, v8, ks, vs * 2, pt, cu, pre, 0.125)
    assert np.array_equal(o2, 2 * base) and np.array_equal(l2, lse)
    o3, l3 = oracle.prefill_paged_e4m3(q, k8, v8, ks * 2, vs, pt, cu, pre, 0.125)
    o4, l4 = oracle.prefill_paged_e4m3(q, k8, v8, ks, vs, pt, cu, pre, 0.25)
    assert np.max(np.abs(o3 - o4)) < 1e-13 and np.max(np.abs(l3 - l4)) < 1e-12
    # The first row of a chunk with no prefix sees only its own key: its output
    # is that token's dequantised V.
    for r in np.flatnonzero((pre == 0) & (np.diff(cu) > 0)):
        p = pt[r, 0]
        for h in range(4):
            assert np.array_equal(base[cu[r], h],
                                  oracle.e4m3_value(v8[p, h // 2, :, 0]) * vs[h // 2])


def test_prefill_paged_e4m3_selected_rows_equal_full():
    ks = np.array([0.01, 0.02], np.float32)
    vs = np.array([0.03, 0.015], np.float32)
    q, k8, v8, pt, cu, pre = _paged_fp8_case(18, PF_PREFIX, PF_CHUNK, 4, 2, 16, ks, vs)
    full, flse = oracle.prefill_paged_e4m3(q, k8, v8, ks, vs, pt, cu, pre, 0.3)
    tok = np.array([0, 5, int(cu[-1]) - 1, 20, 3], np.int32)
    head = np.array([3, 0, 1, 2, 3], np.int32)
    out, lse = oracle.prefill_paged_e4m3(q, k8, v8, ks, vs, pt, cu, pre, 0.3, tok, head)
    assert np.array_equal(out, full[tok, head]) and np.array_equal(lse, flse[tok, head])
