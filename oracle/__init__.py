"""fp64 CPU oracle for the attention hot path -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It shares no code with the HIP
library: ``oracle.c`` is plain C built with gcc, and ``brute.py`` is an
independent dense numpy formulation used to pin it on tiny inputs.

Functions take the arrays produced by ``paper_2511_20982_amd.inputs``
(bf16 as uint16 bit patterns, or float32) and return float64 results.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

from . import build as _build

_LIB = None
BF16, FP32 = 0, 1


def _lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        lib = C.CDLL(_build.LIB)
        P = C.c_void_p
        i32 = C.c_int
        lib.oracle_prefill.argtypes = [i32, i32, i32, i32, C.c_float, P, P, P, P, i32, P, P]
        lib.oracle_prefill_rows.argtypes = [i32, i32, i32, i32, C.c_float, P, P, P, P, i32,
                                            P, P, i32, P, P]
        lib.oracle_decode.argtypes = [i32, i32, i32, i32, C.c_float, P, P, P, P, i32, P, i32, P, P]
        lib.oracle_prefill_paged.argtypes = [i32, i32, i32, i32, C.c_float, P, P, P, P, i32, P,
                                             P, i32, P, P, i32, P, P]
        lib.oracle_kv_write.argtypes = [i32, i32, i32, P, P, P, P, P, i32, P, P, i32]
        lib.oracle_pack.argtypes = [i32, i32, i32, i32, P, P, i32, P, i32, P, P, P, i32, P]
        lib.oracle_unpack.argtypes = [i32, i32, i32, i32, P, P, P, P, i32, P, P, i32, P, i32]
        lib.oracle_e4m3_value.argtypes = [C.c_uint8]
        lib.oracle_e4m3_value.restype = C.c_double
        lib.oracle_e4m3_encode.argtypes = [C.c_float]
        lib.oracle_e4m3_encode.restype = C.c_uint8
        lib.oracle_e4m3_quantize.argtypes = [i32, C.c_int64, i32, i32, P, P, P]
        lib.oracle_decode_e4m3.argtypes = [i32, i32, i32, i32, C.c_float, P, P, P, P, P, P, i32,
                                           P, i32, P, P]
        lib.oracle_prefill_paged_e4m3.argtypes = [i32, i32, i32, i32, C.c_float, P, P, P, P, P,
                                                  P, i32, P, P, i32, P, P, i32, P, P]
        for f in (lib.oracle_prefill, lib.oracle_prefill_rows, lib.oracle_decode,
                  lib.oracle_kv_write, lib.oracle_pack, lib.oracle_unpack,
                  lib.oracle_prefill_paged, lib.oracle_e4m3_quantize, lib.oracle_decode_e4m3,
                  lib.oracle_prefill_paged_e4m3):
            f.restype = i32
        _LIB = lib
    return _LIB


def _dt(a: np.ndarray) -> int:
    if a.dtype == np.uint16:
        return BF16
    if a.dtype == np.float32:
        return FP32
    raise TypeError(f"oracle takes bf16 bits (uint16) or float32, got {a.dtype}")


def _p(a):
    return a.ctypes.data_as(C.c_void_p) if a is not None else None


def _c(a, dtype=None):
    return np.ascontiguousarray(a, dtype=dtype)


def prefill(q, k, v, cu_seqlens, scale):
    """Causal varlen prefill; q[T][Hq][d], k/v[T][Hkv][d] -> (out[T][Hq][d], lse[T][Hq])."""
    q, k, v = _c(q), _c(k), _c(v)
    cu = _c(cu_seqlens, np.int32)
    t, hq, d = q.shape
    hkv = k.shape[1]
    out = np.zeros((t, hq, d), np.float64)
    lse = np.zeros((t, hq), np.float64)
    rc = _lib().oracle_prefill(_dt(q), hq, hkv, d, float(scale), _p(q), _p(k), _p(v), _p(cu),
                               len(cu) - 1, _p(out), _p(lse))
    if rc:
        raise ValueError(f"oracle_prefill rc={rc}")
    return out, lse


def prefill_rows(q, k, v, cu_seqlens, scale, tok, head):
    """Prefill output for selected (token, head) rows -> (out[n][d], lse[n])."""
    q, k, v = _c(q), _c(k), _c(v)
    cu = _c(cu_seqlens, np.int32)
    tok, head = _c(tok, np.int32), _c(head, np.int32)
    _, hq, d = q.shape
    hkv = k.shape[1]
    out = np.zeros((len(tok), d), np.float64)
    lse = np.zeros(len(tok), np.float64)
    rc = _lib().oracle_prefill_rows(_dt(q), hq, hkv, d, float(scale), _p(q), _p(k), _p(v),
                                    _p(cu), len(cu) - 1, _p(tok), _p(head), len(tok),
                                    _p(out), _p(lse))
    if rc:
        raise ValueError(f"oracle_prefill_rows rc={rc}")
    return out, lse


def decode(q, k_pool, v_pool, page_table, context_lens, scale):
    """Paged single-query decode; q[B][Hq][d] -> (out[B][Hq][d], lse[B][Hq])."""
    q, k_pool, v_pool = _c(q), _c(k_pool), _c(v_pool)
    pt = _c(page_table, np.int32)
    ctx = _c(context_lens, np.int32)
    b, hq, d = q.shape
    hkv = k_pool.shape[-3]
    out = np.zeros((b, hq, d), np.float64)
    lse = np.zeros((b, hq), np.float64)
    rc = _lib().oracle_decode(_dt(q), hq, hkv, d, float(scale), _p(q), _p(k_pool), _p(v_pool),
                              _p(pt), pt.shape[1], _p(ctx), b, _p(out), _p(lse))
    if rc:
        raise ValueError(f"oracle_decode rc={rc}")
    return out, lse


def prefill_paged(q, k_pool, v_pool, page_table, cu_q, prefix_lens, scale, tok=None, head=None):
    """Chunk prefill over the paged cache (oracle.c: oracle_prefill_paged).

    Request r holds prefix_lens[r] cached tokens plus the chunk rows
    cu_q[r] .. cu_q[r+1]-1 of q[T][Hq][d], whose K/V are already in the pool;
    chunk token i attends to cached positions 0 .. prefix_lens[r] + i.
    Returns (out[T][Hq][d], lse[T][Hq]), or, with tok/head given, the
    (out[n][d], lse[n]) of those (token, head) rows only."""
    q, k_pool, v_pool = _c(q), _c(k_pool), _c(v_pool)
    pt = _c(page_table, np.int32)
    cu = _c(cu_q, np.int32)
    pre = _c(prefix_lens, np.int32)
    t, hq, d = q.shape
    hkv = k_pool.shape[-3]
    if tok is None:
        tk = hd = None
        nrows = 0
        out = np.zeros((t, hq, d), np.float64)
        lse = np.zeros((t, hq), np.float64)
    else:
        tk, hd = _c(tok, np.int32), _c(head, np.int32)
        nrows = len(tk)
        out = np.zeros((nrows, d), np.float64)
        lse = np.zeros((nrows,), np.float64)
    rc = _lib().oracle_prefill_paged(_dt(q), hq, hkv, d, float(scale), _p(q), _p(k_pool),
                                     _p(v_pool), _p(pt), pt.shape[1], _p(cu), _p(pre), len(pre),
                                     _p(tk) if tk is not None else None,
                                     _p(hd) if hd is not None else None, nrows, _p(out),
                                     _p(lse))
    if rc:
        raise ValueError(f"oracle_prefill_paged rc={rc}")
    return out, lse


def kv_write(k_new, v_new, k_pool, v_pool, page_table, cu_new, start_pos):
    """Returns new (k_pool, v_pool) copies with the new tokens written."""
    k_new, v_new = _c(k_new), _c(v_new)
    kp, vp = k_pool.copy(), v_pool.copy()
    pt = _c(page_table, np.int32)
    cu = _c(cu_new, np.int32)
    st = _c(start_pos, np.int32)
    hkv, d = k_new.shape[1], k_new.shape[2]
    _lib().oracle_kv_write(k_new.itemsize, hkv, d, _p(k_new), _p(v_new), _p(kp), _p(vp),
                           _p(pt), pt.shape[1], _p(cu), _p(st), len(cu) - 1)
    return kp, vp


def pack(k_pool, v_pool, num_layers, page_table, req_ids, seq_lens, out_offsets):
    """Handoff buffer in (layer, K/V, head, token, dim) order per request."""
    k_pool, v_pool = _c(k_pool), _c(v_pool)
    pt = _c(page_table, np.int32)
    req, lens = _c(req_ids, np.int32), _c(seq_lens, np.int32)
    off = _c(out_offsets, np.int64)
    d = k_pool.shape[-1]
    hkv = k_pool.shape[-3]
    num_pages = k_pool.shape[-4]
    out = np.zeros(int(off[-1]), dtype=k_pool.dtype)
    _lib().oracle_pack(k_pool.itemsize, hkv, d, num_layers, _p(k_pool), _p(v_pool), num_pages,
                       _p(pt), pt.shape[1], _p(req), _p(lens), _p(off), len(req), _p(out))
    return out


def unpack(buf, in_offsets, req_ids, seq_lens, k_pool, v_pool, num_layers, page_table):
    """Returns new (k_pool, v_pool) copies with the handoff buffer scattered in."""
    buf = _c(buf)
    kp, vp = k_pool.copy(), v_pool.copy()
    pt = _c(page_table, np.int32)
    req, lens = _c(req_ids, np.int32), _c(seq_lens, np.int32)
    off = _c(in_offsets, np.int64)
    d, hkv, num_pages = kp.shape[-1], kp.shape[-3], kp.shape[-4]
    _lib().oracle_unpack(kp.itemsize, hkv, d, num_layers, _p(buf), _p(off), _p(req), _p(lens),
                         len(req), _p(kp), _p(vp), num_pages, _p(pt), pt.shape[1])
    return kp, vp


# ---- FP8 (OCP E4M3) KV pages ------------------------------------------------
def e4m3_value(codes):
    """float64 value of each E4M3 code (oracle.c: oracle_e4m3_value)."""
    table = np.array([_lib().oracle_e4m3_value(c) for c in range(256)], np.float64)
    return table[np.asarray(codes, np.uint8)]


def e4m3_encode(y):
    """Nearest E4M3 code (ties to even, saturating at 448) of each float32 y."""
    y = _c(y, np.float32)
    out = np.zeros(y.shape, np.uint8)
    one = np.ones(1, np.float32)
    rc = _lib().oracle_e4m3_quantize(FP32, y.size, 1, 1, _p(y), _p(one), _p(out))
    if rc:
        raise ValueError(f"oracle_e4m3_quantize rc={rc}")
    return out


def e4m3_quantize(x, scale):
    """Codes of x[T][Hkv][d] (bf16 bits or float32) with one scale per head:
    E4M3_rne(sat(x * fp32(1/scale[h]))), the product in fp32."""
    x = _c(x)
    sc = _c(scale, np.float32)
    t, hkv, d = x.shape
    if sc.shape != (hkv,):
        raise ValueError("one scale per KV head")
    out = np.zeros(x.shape, np.uint8)
    rc = _lib().oracle_e4m3_quantize(_dt(x), t, hkv, d, _p(x), _p(sc), _p(out))
    if rc:
        raise ValueError(f"oracle_e4m3_quantize rc={rc}")
    return out


def decode_e4m3(q, k_pool, v_pool, k_scale, v_scale, page_table, context_lens, scale):
    """Paged decode over E4M3 pools (uint8 codes, bf16/fp32 q) with per-KV-head
    scales -> (out[B][Hq][d], lse[B][Hq])."""
    q = _c(q)
    k_pool, v_pool = _c(k_pool, np.uint8), _c(v_pool, np.uint8)
    ks, vs = _c(k_scale, np.float32), _c(v_scale, np.float32)
    pt = _c(page_table, np.int32)
    ctx = _c(context_lens, np.int32)
    b, hq, d = q.shape
    hkv = k_pool.shape[-3]
    if ks.shape != (hkv,) or vs.shape != (hkv,):
        raise ValueError("one scale per KV head")
    out = np.zeros((b, hq, d), np.float64)
    lse = np.zeros((b, hq), np.float64)
    rc = _lib().oracle_decode_e4m3(_dt(q), hq, hkv, d, float(scale), _p(q), _p(k_pool),
                                   _p(v_pool), _p(ks), _p(vs), _p(pt), pt.shape[1], _p(ctx), b,
                                   _p(out), _p(lse))
    if rc:
        raise ValueError(f"oracle_decode_e4m3 rc={rc}")
    return out, lse


def prefill_paged_e4m3(q, k_pool, v_pool, k_scale, v_scale, page_table, cu_q, prefix_lens, scale,
                       tok=None, head=None):
    """Chunk prefill over E4M3 pools (uint8 codes, same page layouts) with
    per-KV-head scales (key = value(code) * k_scale[c], value = value(code) *
    v_scale[c]); q bf16 bits or fp32 [T][Hq][d] -> (out[T][Hq][d], lse[T][Hq]),
    or, with tok/head given, the (out[n][d], lse[n]) of those rows only."""
    q = _c(q)
    k_pool, v_pool = _c(k_pool, np.uint8), _c(v_pool, np.uint8)
    ks, vs = _c(k_scale, np.float32), _c(v_scale, np.float32)
    pt = _c(page_table, np.int32)
    cu = _c(cu_q, np.int32)
    pre = _c(prefix_lens, np.int32)
    t, hq, d = q.shape
    hkv = k_pool.shape[-3]
    if tok is None:
        tk = hd = None
        nrows = 0
        out = np.zeros((t, hq, d), np.float64)
        lse = np.zeros((t, hq), np.float64)
    else:
        tk, hd = _c(tok, np.int32), _c(head, np.int32)
        nrows = len(tk)
        out = np.zeros((nrows, d), np.float64)
        lse = np.zeros((nrows,), np.float64)
    rc = _lib().oracle_prefill_paged_e4m3(_dt(q), hq, hkv, d, float(scale), _p(q), _p(k_pool),
                                          _p(v_pool), _p(ks), _p(vs), _p(pt), pt.shape[1],
                                          _p(cu), _p(pre), len(cu) - 1,
                                          _p(tk) if tk is not None else None,
                                          _p(hd) if hd is not None else None, nrows, _p(out),
                                          _p(lse))
    if rc:
        raise ValueError(f"oracle_prefill_paged_e4m3 rc={rc}")
    return out, lse
