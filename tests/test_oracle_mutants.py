"""Plants plausible mistakes in a copy of the oracle's C source (on the CPU)
and checks that the pins catch every one of them.  The real oracle must pass
the same checks.  This measures the strength of the pins, not the GPU path."""
import ctypes
import os
import subprocess

import numpy as np
import pytest
import torch

import oracle
from oracle import brute
from paper_2511_20982_amd import inputs as I

SRC = os.path.join(os.path.dirname(oracle.__file__), "oracle.c")

MUTANTS = {
    "gqa_head_map_modulo": [("c = h / g", "c = h % hkv")],
    "causal_excludes_diagonal": [("k, koff, 1, v, voff, 1, i + 1, sc", "k, koff, 1, v, voff, 1, i, sc")],
    "causal_sees_one_future_key": [("(maxlen + 1));\n    int64_t *koff = (int64_t *)malloc(sizeof(int64_t) * (maxlen + 1));\n    int64_t *voff",
                                    "(maxlen + 2));\n    int64_t *koff = (int64_t *)malloc(sizeof(int64_t) * (maxlen + 2));\n    int64_t *voff"),
                                   ("k, koff, 1, v, voff, 1, i + 1, sc", "k, koff, 1, v, voff, 1, (i + 2 < len ? i + 2 : len), sc")],
    "no_max_subtraction": [("sc[j] = exp(sc[j] - m);", "sc[j] = exp(sc[j]);")],
    "sign_flip_in_exponent": [("sc[j] = exp(sc[j] - m);", "sc[j] = exp(m - sc[j]);")],
    "scale_ignored": [("sc[j] = sigma * s;", "sc[j] = s;")],
    "missing_normalisation": [("out[e] = acc / l;", "out[e] = acc;")],
    "lse_base2": [("*lse = m + log(l);", "*lse = m + log2(l);")],
    "v_page_layout_token_major": [("voff[j] = (page * hkv + c) * (int64_t)d * OR_PAGE + slot; /* element e at +16e */",
                                   "voff[j] = ((page * hkv + c) * OR_PAGE + slot) * d;"),
                                  ("v_pool, voff, OR_PAGE, ctx[r]", "v_pool, voff, 1, ctx[r]")],
    "decode_slot_off_by_one": [("const int slot = j % OR_PAGE;\n        koff[j]", "const int slot = (j + 1) % OR_PAGE;\n        koff[j]")],
    "decode_misses_current_token": [("v_pool, voff, OR_PAGE, ctx[r], sc", "v_pool, voff, OR_PAGE, ctx[r] - 1, sc")],
    "q_reads_kv_head": [("attend_row(dtype, d, sigma, q, row * d", "attend_row(dtype, d, sigma, q, (((int64_t)(base + i)) * hq + c) * d")],
    "write_v_token_major": [("const int64_t vd = ((page * hkv + h) * d + e) * OR_PAGE + slot;",
                             "const int64_t vd = ((page * hkv + h) * OR_PAGE + slot) * d + e;")],
    "write_wrong_source_row": [("const int64_t tok = cu_new[r] + i;", "const int64_t tok = cu_new[r] + (i ? i - 1 : 0);")],
    "pack_kv_swapped": [("if (c == 0) {\n                src", "if (c == 1) {\n                src")],
    "unpack_kv_swapped": [("if (c == 0) {\n                dst", "if (c == 1) {\n                dst")],
    "unpack_slot_off_by_one": [("const int slot = t % OR_PAGE;\n            const int64_t lp = (int64_t)layer * num_pages + page;\n            for (int e = 0; e < d; ++e) {\n              const int64_t src = off[n]",
                                "const int slot = (t + 1) % OR_PAGE;\n            const int64_t lp = (int64_t)layer * num_pages + page;\n            for (int e = 0; e < d; ++e) {\n              const int64_t src = off[n]")],
    "paged_prefill_top_left": [("const int nkeys = prefix_lens[r] + (int)(t - cu_q[r]) + 1;",
                                "const int nkeys = (int)(t - cu_q[r]) + 1;")],
    "paged_prefill_prefix_off_by_one": [("const int nkeys = prefix_lens[r] + (int)(t - cu_q[r]) + 1;",
                                         "const int nkeys = (prefix_lens[r] > 0 ? prefix_lens[r] - 1 : 0) + (int)(t - cu_q[r]) + 1;")],
    "paged_prefill_chunk_row_as_q_row": [("d, sigma, q, (t * hq + h) * d, k_pool",
                                          "d, sigma, q, ((t - cu_q[r]) * hq + h) * d, k_pool")],
    "paged_prefill_v_token_major": [("koff, 1, v_pool, voff, OR_PAGE, nkeys",
                                     "koff, 1, v_pool, koff, 1, nkeys")],
    "paged_e4m3_scales_swapped": [("prefill_paged_impl(qdtype, OR_E4M3, k_scale, v_scale,",
                                   "prefill_paged_impl(qdtype, OR_E4M3, v_scale, k_scale,")],
    "paged_e4m3_v_scale_dropped": [("v_scale ? (double)v_scale[c] : 1.0, d, sigma, q, (t * hq",
                                    "1.0, d, sigma, q, (t * hq")],
    "e4m3_exponent_bias_8": [("ldexp((double)(8 + m), e - 10)", "ldexp((double)(8 + m), e - 11)")],
    "e4m3_encode_ties_away": [("int m = (int)nearbyint(ldexp(a, 3 - E));", "int m = (int)round(ldexp(a, 3 - E));")],
    "e4m3_overflow_to_nan": [("if (a >= 448.0) return s | 0x7E;", "if (a >= 464.0) return s | 0x7F;")],
    "e4m3_subnormal_step": [("return s | (uint8_t)nearbyint(a * 512.0);", "return s | (uint8_t)nearbyint(a * 256.0);")],
    "quantize_multiplies_by_scale": [("out[i] = oracle_e4m3_encode(xf * inv);", "out[i] = oracle_e4m3_encode(xf * scale[h]);")],
    "quantize_first_head_scale": [("const float inv = 1.0f / scale[h];", "const float inv = 1.0f / scale[0];")],
    "decode_e4m3_k_scale_of_head0": [("k_scale ? (double)k_scale[c] : 1.0", "k_scale ? (double)k_scale[0] : 1.0")],
    "decode_e4m3_v_scale_as_k_scale": [("v_scale ? (double)v_scale[c] : 1.0", "v_scale ? (double)k_scale[c] : 1.0")],
    "pack_token_dim_transposed": [("const int64_t dst = off[n] + ((((int64_t)layer * 2 + c) * hkv + h) * len + t) * d + e;",
                                   "const int64_t dst = off[n] + ((((int64_t)layer * 2 + c) * hkv + h) * d + e) * len + t;")],
}


def _build(tmp_path, name, edits):
    src = open(SRC).read()
    for old, new in edits:
        assert old in src, f"mutant {name}: pattern not found: {old!r}"
        src = src.replace(old, new)
    c = tmp_path / f"{name}.c"
    so = tmp_path / f"{name}.so"
    c.write_text(src)
    subprocess.run(["gcc", "-O1", "-fopenmp", "-fPIC", "-shared", "-o", str(so), str(c), "-lm"],
                   check=True)
    return str(so)


def _load(path):
    lib = ctypes.CDLL(path)
    real = oracle._lib()
    for f in ("oracle_prefill", "oracle_prefill_rows", "oracle_decode", "oracle_kv_write",
              "oracle_pack", "oracle_unpack", "oracle_prefill_paged", "oracle_e4m3_value",
              "oracle_e4m3_encode", "oracle_e4m3_quantize", "oracle_decode_e4m3",
              "oracle_prefill_paged_e4m3"):
        getattr(lib, f).argtypes = getattr(real, f).argtypes
        getattr(lib, f).restype = getattr(real, f).restype
    return lib


# ---- the pins, as checks that return True when they hold ---------------------
def _close(a, b, tol):
    return bool(np.all(np.isfinite(a)) and np.max(np.abs(a - b)) <= tol)


def chk_prefill_brute():
    ok = True
    for dt, lens, hq, hkv, d in [("fp32", [5, 1, 9], 8, 2, 16), ("bf16", [17, 3], 4, 4, 8)]:
        rng = np.random.default_rng(3)
        q, k, v = I.prefill_batch(rng, np.array(lens), hq, hkv, d, dt)
        cu = I.cu_from_lens(lens)
        out, _ = oracle.prefill(q, k, v, cu, 0.3)
        ok &= _close(out, brute.prefill(q, k, v, cu, 0.3), 1e-11)
    return ok


def chk_prefill_sdpa():
    rng = np.random.default_rng(4)
    q, k, v = I.prefill_batch(rng, np.array([13]), 4, 2, 8, "fp32")
    out, _ = oracle.prefill(q, k, v, I.cu_from_lens([13]), 0.5)
    t = [torch.from_numpy(x.astype(np.float64)).transpose(0, 1) for x in (q, k, v)]
    ref = torch.nn.functional.scaled_dot_product_attention(
        t[0], t[1].repeat_interleave(2, 0), t[2].repeat_interleave(2, 0), is_causal=True,
        scale=0.5).transpose(0, 1).numpy()
    return _close(out, ref, 1e-11)


def chk_lse():
    rng = np.random.default_rng(5)
    q, k, v = I.prefill_batch(rng, np.array([6]), 2, 1, 8, "fp32")
    _, lse = oracle.prefill(q, k, v, I.cu_from_lens([6]), 0.5)
    ok = True
    for h in range(2):
        for i in range(6):
            sc = [0.5 * float(np.dot(q[i, h].astype(np.float64), k[j, 0].astype(np.float64)))
                  for j in range(i + 1)]
            ok &= abs(lse[i, h] - np.logaddexp.reduce(sc)) < 1e-12
    return bool(ok)


def chk_decode_brute():
    w = I.decode_workload("t", 5, [1, 15, 16, 17, 40], 8, 2, 16, "bf16")
    out, _ = oracle.decode(w.q_dec, w.k_pool, w.v_pool, w.page_table, w.context_lens, w.scale)
    ref = brute.decode(w.q_dec, w.k_pool, w.v_pool, w.page_table, w.context_lens, w.scale)
    return _close(out, ref, 1e-12)


def chk_last_row_equals_decode():
    w = I.tiny_fp32(n_steps=0)
    out_p, lse_p = oracle.prefill(w.q, w.k, w.v, w.cu_seqlens, w.scale)
    kp, vp = oracle.kv_write(w.k, w.v, w.k_pool, w.v_pool, w.page_table, w.cu_seqlens,
                             np.zeros(4, np.int32))
    last = w.cu_seqlens[1:] - 1
    out_d, lse_d = oracle.decode(w.q[last], kp, vp, w.page_table, w.prefill_lens, w.scale)
    return _close(out_d, out_p[last], 1e-12) and _close(lse_d, lse_p[last], 1e-12)


def chk_write_pack_transpose():
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
    ok = True
    for r in range(3):
        a, b = cu[r], cu[r + 1]
        expect = np.stack([knew[a:b].transpose(1, 0, 2), vnew[a:b].transpose(1, 0, 2)])
        ok &= np.array_equal(out[off[r]:off[r + 1]], expect.reshape(-1))
    return bool(ok)


def chk_closed_forms():
    rng = np.random.default_rng(15)
    L, d = 10, 8
    q = rng.standard_normal((L, 1, d), dtype=np.float32)
    v = rng.standard_normal((L, 1, d), dtype=np.float32)
    k = np.repeat(rng.standard_normal((1, 1, d), dtype=np.float32), L, axis=0)
    vf = v[:, 0].astype(np.float64)
    mean = np.cumsum(vf, axis=0) / np.arange(1, L + 1)[:, None]
    out, lse = oracle.prefill(q, k, v, I.cu_from_lens([L]), 0.0)
    return _close(out[:, 0], mean, 1e-13) and _close(lse[:, 0], np.log(np.arange(1, L + 1)), 1e-13)


def chk_unpack_matches_write():
    # unpack of a packed buffer into a fresh pool equals writing the same tokens
    rng = np.random.default_rng(24)
    lens = np.array([21, 3], np.int32)
    hkv, d = 2, 8
    pt, num_pages = I.allocate_pages(rng, lens, pool_pages=5)
    kp, vp = I.empty_pools(num_pages, hkv, d, "bf16")
    knew = I.normal(rng, (int(lens.sum()), hkv, d), "bf16")
    vnew = I.normal(rng, (int(lens.sum()), hkv, d), "bf16")
    cu = I.cu_from_lens(lens)
    kw, vw = oracle.kv_write(knew, vnew, kp, vp, pt, cu, np.zeros(2, np.int32))
    off = I.handoff_offsets(lens, 1, hkv, d)
    buf = np.concatenate([np.stack([knew[cu[r]:cu[r + 1]].transpose(1, 0, 2),
                                    vnew[cu[r]:cu[r + 1]].transpose(1, 0, 2)]).reshape(-1)
                          for r in range(2)])
    ku, vu = oracle.unpack(buf, off, np.arange(2), lens, kp, vp, 1, pt)
    return bool(np.array_equal(ku, kw) and np.array_equal(vu, vw))


def _paged_pool(rng, prefix, chunk, hq, hkv, d, dtype):
    total = np.asarray(prefix, np.int32) + np.asarray(chunk, np.int32)
    pt, num_pages = I.allocate_pages(rng, total, pool_pages=int(np.sum((total + 15) // 16)) + 2)
    kp, vp = I.empty_pools(num_pages, hkv, d, dtype)
    _, kf, vf = I.prefill_batch(rng, total, hq, hkv, d, dtype)
    kp, vp = oracle.kv_write(kf, vf, kp, vp, pt, I.cu_from_lens(total),
                             np.zeros(len(total), np.int32))
    q = I.normal(rng, (int(np.sum(chunk)), hq, d), dtype)
    return q, kp, vp, pt, I.cu_from_lens(chunk), np.asarray(prefix, np.int32)


def chk_paged_prefill_brute():
    rng = np.random.default_rng(31)
    q, kp, vp, pt, cu, pre = _paged_pool(rng, [20, 3, 0], [5, 18, 7], 4, 2, 8, "fp32")
    out, _ = oracle.prefill_paged(q, kp, vp, pt, cu, pre, 0.4)
    return _close(out, brute.prefill_paged(q, kp, vp, pt, cu, pre, 0.4), 1e-11)


def chk_chunked_equals_one_shot():
    rng = np.random.default_rng(32)
    L, hq, hkv, d = 37, 2, 1, 8
    q, k, v = I.prefill_batch(rng, np.array([L]), hq, hkv, d, "bf16")
    ref, _ = oracle.prefill(q, k, v, I.cu_from_lens([L]), 0.3)
    pt, num_pages = I.allocate_pages(rng, np.array([L]), pool_pages=4)
    kp, vp = I.empty_pools(num_pages, hkv, d, "bf16")
    done = 0
    for n in (9, 1, 20, 7):
        rows = slice(done, done + n)
        kp, vp = oracle.kv_write(k[rows], v[rows], kp, vp, pt, I.cu_from_lens([n]),
                                 np.array([done], np.int32))
        out, _ = oracle.prefill_paged(q[rows], kp, vp, pt, I.cu_from_lens([n]),
                                      np.array([done], np.int32), 0.3)
        if not _close(out, ref[rows], 1e-12):
            return False
        done += n
    return True


def chk_e4m3_table():
    v = oracle.e4m3_value(np.arange(256))
    t = torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    fin = ~np.isnan(t)
    return bool(np.array_equal(np.isnan(v), ~fin) and np.array_equal(v[fin], t[fin]))


def chk_e4m3_encode():
    v = torch.arange(127, dtype=torch.uint8).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    mids = ((v[:-1] + v[1:]) / 2).astype(np.float32)
    lo = np.arange(126)
    ok = np.array_equal(oracle.e4m3_encode(mids), np.where(lo % 2 == 0, lo, lo + 1))
    big = np.array([448, 470, 1e9, -1e9], np.float32)
    ok &= list(oracle.e4m3_encode(big)) == [0x7E, 0x7E, 0x7E, 0xFE]
    y = np.random.default_rng(31).standard_normal(2000).astype(np.float32) * 20
    t = torch.from_numpy(y).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    return bool(ok and np.array_equal(oracle.e4m3_encode(y), t))


def chk_e4m3_quantize():
    rng = np.random.default_rng(32)
    x = I.normal(rng, (5, 3, 8), "fp32")
    scale = np.array([0.5, 0.01, 0.07], np.float32)
    y = x * (np.float32(1) / scale)[None, :, None]
    t = torch.from_numpy(np.clip(y, -448, 448).astype(np.float32)).to(
        torch.float8_e4m3fn).view(torch.uint8).numpy()
    return bool(np.array_equal(oracle.e4m3_quantize(x, scale), t))


def chk_decode_e4m3_brute():
    w = I.decode_workload("t", 33, [1, 17, 40], 4, 2, 16, "bf16")
    rng = np.random.default_rng(33)
    kp = rng.integers(0, 0x7F, w.k_pool.shape).astype(np.uint8) | (
        rng.integers(0, 2, w.k_pool.shape).astype(np.uint8) << 7)
    vp = rng.integers(0, 0x7F, w.v_pool.shape).astype(np.uint8)
    ks = np.array([0.01, 0.03], np.float32)
    vs = np.array([0.02, 0.005], np.float32)
    out, _ = oracle.decode_e4m3(w.q_dec, kp, vp, ks, vs, w.page_table, w.context_lens, w.scale)
    tab = torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    kd = tab[kp] * ks.astype(np.float64)[None, :, None, None]
    vd = tab[vp] * vs.astype(np.float64)[None, :, None, None]
    ref = brute.decode(w.q_dec, kd, vd, w.page_table, w.context_lens, w.scale)
    return _close(out, ref, 1e-12)


def chk_paged_prefill_e4m3_brute():
    rng = np.random.default_rng(34)
    prefix, chunk = [18, 0, 3], [4, 9, 14]
    total = np.asarray(prefix) + np.asarray(chunk)
    pt, num_pages = I.allocate_pages(rng, total, pool_pages=int(np.sum((total + 15) // 16)) + 1)
    kp = rng.integers(0, 0x7F, (num_pages, 2, 16, 8)).astype(np.uint8) | (
        rng.integers(0, 2, (num_pages, 2, 16, 8)).astype(np.uint8) << 7)
    vp = rng.integers(0, 0x7F, (num_pages, 2, 8, 16)).astype(np.uint8)
    q = I.normal(rng, (int(np.sum(chunk)), 4, 8), "bf16")
    cu, pre = I.cu_from_lens(chunk), np.asarray(prefix, np.int32)
    ks = np.array([0.02, 0.06], np.float32)
    vs = np.array([0.03, 0.004], np.float32)
    out, _ = oracle.prefill_paged_e4m3(q, kp, vp, ks, vs, pt, cu, pre, 0.3)
    tab = torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    kd = tab[kp] * ks.astype(np.float64)[None, :, None, None]
    vd = tab[vp] * vs.astype(np.float64)[None, :, None, None]
    return _close(out, brute.prefill_paged(q, kd, vd, pt, cu, pre, 0.3), 1e-12)


CHECKS = [chk_e4m3_table, chk_e4m3_encode, chk_e4m3_quantize, chk_decode_e4m3_brute,
          chk_prefill_brute, chk_prefill_sdpa, chk_lse, chk_decode_brute,
          chk_last_row_equals_decode, chk_write_pack_transpose, chk_closed_forms,
          chk_unpack_matches_write, chk_paged_prefill_brute, chk_chunked_equals_one_shot,
          chk_paged_prefill_e4m3_brute]


def _run_checks():
    failed = []
    for chk in CHECKS:
        try:
            good = chk()
        except Exception:
            good = False
        if not good:
            failed.append(chk.__name__)
    return failed


def test_real_oracle_passes_every_check():
    assert _run_checks() == []


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name, tmp_path, monkeypatch):
    lib = _load(_build(tmp_path, name, MUTANTS[name]))
    monkeypatch.setattr(oracle, "_LIB", lib)
    failed = _run_checks()
    assert failed, f"mutant {name} passed every pin"
