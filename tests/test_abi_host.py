"""C ABI checks that need no GPU: the library loads, exports every symbol the
header declares, and rejects invalid arguments on the host before any HIP
call (pointers passed here are never dereferenced)."""
import ctypes as C
import os
import re

import numpy as np
import pytest

from paper_2511_20982_amd import attn as A

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dopd_attn.h")
FAKE = 0x1000  # a non-null device address; host validation fails before it is used


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(A.LIB_PATH):
        from paper_2511_20982_amd import build
        build.build()
    return A.lib()


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(dopd_[a-z_0-9]+)\s*\(", src)))


def test_every_declared_symbol_is_exported(lib):
    names = declared_functions()
    assert set(names) == set(A.EXPORTS)
    for n in names:
        assert hasattr(lib, n), n


def declaration_comments():
    """{function name: the comment block right before its declaration}."""
    src = open(HEADER).read()
    out = {}
    for m in re.finditer(r"/\*((?:(?!\*/).)*)\*/\s*(?:dopd_status|size_t|const char\*|int32_t)\s+"
                         r"(dopd_[a-z_0-9]+)\s*\(", src, flags=re.S):
        out[m.group(2)] = m.group(1)
    return out


# Library bookkeeping with no passage of the paper behind it.
NO_PASSAGE = {"dopd_status_string", "dopd_last_hip_error"}
# A variant of an entry point for callers that cannot allocate device memory.
FOR_CALLERS = {"dopd_decode_attn_noalloc"}


def test_every_declaration_cites_its_passage():
    com = declaration_comments()
    assert set(com) == set(declared_functions())
    for name, text in com.items():
        if name in NO_PASSAGE:
            assert "Paper: none" in text, name
        elif name in FOR_CALLERS:  # names the callers it serves instead
            assert "cannot" in text and "allocate" in text, name
        else:
            assert re.search(r"Paper:.*?\b(Sec\.|Eq\.|Alg\.)", text, flags=re.S), \
                f"{name}: its comment block cites no Sec., Eq. or Alg."


def test_status_strings(lib):
    for s in range(6):
        assert A.status_string(s)
    assert A.status_string(99) == "unknown status"
    assert lib.dopd_last_hip_error() == 0


def _shape(hq=8, hkv=2, d=128, dtype="bf16", page=16):
    return A.make_shape(hq, hkv, d, dtype, page_size=page)


def _prefill(lib, shape, cu_host, ptrs=FAKE, nreq=None):
    cu = np.asarray(cu_host, np.int32)
    n = len(cu) - 1 if nreq is None else nreq
    p = C.c_void_p(ptrs) if ptrs else None
    return lib.dopd_prefill_attn(C.byref(shape), p, p, p, p, None, p, A._hptr(cu), n, None, 0,
                                 None)


def test_prefill_host_validation(lib):
    assert _prefill(lib, _shape(hq=6, hkv=4), [0, 4]) == A.DOPD_ERR_INVALID_SHAPE
    assert _prefill(lib, _shape(d=96), [0, 4]) == A.DOPD_ERR_UNSUPPORTED
    assert _prefill(lib, _shape(page=32), [0, 4]) == A.DOPD_ERR_UNSUPPORTED
    assert _prefill(lib, _shape(), [0, 4], ptrs=0) == A.DOPD_ERR_NULL_POINTER
    assert _prefill(lib, _shape(), [0, 4, 2]) == A.DOPD_ERR_INVALID_SHAPE     # negative length
    assert _prefill(lib, _shape(), [1, 4]) == A.DOPD_ERR_INVALID_SHAPE        # cu[0] != 0
    assert _prefill(lib, _shape(), [0], nreq=-1) == A.DOPD_ERR_INVALID_SHAPE
    assert _prefill(lib, _shape(), [0], nreq=0) == A.DOPD_OK                  # empty batch
    assert _prefill(lib, _shape(), [0, 0, 0]) == A.DOPD_OK                    # all-empty requests
    assert lib.dopd_prefill_attn(None, None, None, None, None, None, None, None, 1, None, 0,
                                 None) == A.DOPD_ERR_NULL_POINTER
    # a workspace that is given must be 256-byte aligned; the prefill needs none
    p = C.c_void_p(FAKE)
    cu = np.array([0, 4], np.int32)
    assert lib.dopd_prefill_attn(C.byref(_shape()), p, p, p, p, None, p, A._hptr(cu), 1,
                                 C.c_void_p(FAKE + 8), 64, None) == A.DOPD_ERR_INVALID_SHAPE
    assert A.dopd_prefill_workspace_size(_shape(), cu, 1) == 0


def _decode(lib, shape, ctx, split=0, ws_bytes=1 << 30, pt_stride=1024, ws=FAKE, nreq=None):
    ctx = np.asarray(ctx, np.int32)
    p = C.c_void_p(FAKE)
    n = len(ctx) if nreq is None else nreq
    return lib.dopd_decode_attn(C.byref(shape), p, p, p, 10, p, pt_stride, p, A._hptr(ctx), n,
                                split, p, None, C.c_void_p(ws) if ws else None, ws_bytes, None)


def test_decode_host_validation(lib):
    s = _shape()
    assert _decode(lib, s, [5, 0]) == A.DOPD_ERR_INVALID_SHAPE               # context < 1
    assert _decode(lib, s, [5], split=48) == A.DOPD_ERR_INVALID_SHAPE        # not a multiple of 32
    assert _decode(lib, s, [5], split=-32) == A.DOPD_ERR_INVALID_SHAPE
    assert _decode(lib, s, [5000], pt_stride=4) == A.DOPD_ERR_INVALID_SHAPE  # table too narrow
    assert _decode(lib, _shape(hq=34, hkv=2), [5]) == A.DOPD_ERR_UNSUPPORTED  # group > 16
    need = A.dopd_decode_workspace_size(s, [3000, 17], 2)
    assert need > 0
    assert _decode(lib, s, [3000, 17], ws_bytes=need - 1) == A.DOPD_ERR_WORKSPACE_TOO_SMALL
    assert _decode(lib, s, [3000, 17], ws=0) == A.DOPD_ERR_NULL_POINTER
    assert _decode(lib, s, [3000, 17], ws=FAKE + 16) == A.DOPD_ERR_INVALID_SHAPE   # misaligned
    assert _decode(lib, s, [], nreq=0) == A.DOPD_OK
    assert A.dopd_decode_workspace_size(s, [0], 1) == 0


def test_decode_workspace_grows_with_smaller_splits(lib):
    s = _shape()
    ctx = [16384, 100, 4096]
    big = A.dopd_decode_workspace_size(s, ctx, 3, 64)
    small = A.dopd_decode_workspace_size(s, ctx, 3, 4096)
    assert big > small > 0
    assert big % 256 == 0


def test_kv_write_and_pack_host_validation(lib):
    s = _shape()
    p = C.c_void_p(FAKE)
    w = lib.dopd_kv_write
    assert w(C.byref(s), p, p, p, p, 10, p, 4, p, p, -1, 5, None) == A.DOPD_ERR_INVALID_SHAPE
    assert w(C.byref(s), None, p, p, p, 10, p, 4, p, p, 1, 5, None) == A.DOPD_ERR_NULL_POINTER
    assert w(C.byref(s), p, p, p, p, 10, p, 4, p, p, 1, 0, None) == A.DOPD_OK    # nothing to do
    lens = np.array([40, 600], np.int32)
    pk = lib.dopd_kv_pack_for_handoff
    assert pk(C.byref(s), 0, p, p, 10, p, 64, p, p, A._hptr(lens), p, 2, p, None) == \
        A.DOPD_ERR_INVALID_SHAPE                                               # no layers
    assert pk(C.byref(s), 1, p, p, 10, p, 8, p, p, A._hptr(lens), p, 2, p, None) == \
        A.DOPD_ERR_INVALID_SHAPE                                               # 600 tokens > 8 pages
    assert pk(C.byref(s), 1, p, p, 10, p, 64, p, p, None, p, 2, p, None) == \
        A.DOPD_ERR_NULL_POINTER
    assert pk(C.byref(_shape(dtype="fp32", d=80)), 1, p, p, 10, p, 64, p, p, A._hptr(lens), p,
              2, p, None) == A.DOPD_ERR_UNSUPPORTED


def test_validate_page_table_host(lib):
    pt = np.array([[3, 1, -1], [0, -1, -1]], np.int32)
    assert A.dopd_validate_page_table_host(pt, 3, 2, [20, 16], 4) == A.DOPD_OK
    assert A.dopd_validate_page_table_host(pt, 3, 2, [40, 16], 4) == A.DOPD_ERR_INVALID_SHAPE
    assert A.dopd_validate_page_table_host(pt, 3, 2, [20, 17], 4) == A.DOPD_ERR_INVALID_SHAPE
    assert A.dopd_validate_page_table_host(pt, 3, 2, [20, 16], 3) == A.DOPD_ERR_INVALID_SHAPE
    assert A.dopd_validate_page_table_host(pt, 3, 0, [], 4) == A.DOPD_OK


def test_unpack_host_validation(lib):
    s = _shape()
    p = C.c_void_p(FAKE)
    lens = np.array([40, 600], np.int32)
    up = lib.dopd_kv_unpack_from_handoff
    assert up(C.byref(s), 0, p, p, p, p, A._hptr(lens), 2, p, p, 10, p, 64, None) == \
        A.DOPD_ERR_INVALID_SHAPE                                               # no layers
    assert up(C.byref(s), 1, p, p, p, p, A._hptr(lens), 2, p, p, 10, p, 8, None) == \
        A.DOPD_ERR_INVALID_SHAPE                                               # table too narrow
    assert up(C.byref(s), 1, p, p, p, p, None, 2, p, p, 10, p, 64, None) == A.DOPD_ERR_NULL_POINTER
    assert up(C.byref(s), 1, p, p, p, p, A._hptr(lens), 0, p, p, 10, p, 64, None) == A.DOPD_OK


def test_prefill_paged_host_validation(lib):
    s = _shape()
    p = C.c_void_p(FAKE)
    cu = np.array([0, 40, 41], np.int32)
    pre = np.array([600, 0], np.int32)
    pp = lib.dopd_prefill_paged_attn
    H = A._hptr
    # request 0 needs ceil(640/16) = 40 page-table columns
    assert pp(C.byref(s), p, p, p, 100, p, 39, p, H(cu), p, H(pre), 2, p, None, None) == \
        A.DOPD_ERR_INVALID_SHAPE                                               # table too narrow
    bad_pre = np.array([-1, 0], np.int32)
    assert pp(C.byref(s), p, p, p, 100, p, 64, p, H(cu), p, H(bad_pre), 2, p, None, None) == \
        A.DOPD_ERR_INVALID_SHAPE                                               # negative prefix
    bad_cu = np.array([0, 40, 30], np.int32)
    assert pp(C.byref(s), p, p, p, 100, p, 64, p, H(bad_cu), p, H(pre), 2, p, None, None) == \
        A.DOPD_ERR_INVALID_SHAPE                                               # decreasing cu
    assert pp(C.byref(s), p, p, p, 100, p, 64, p, H(cu), p, None, 2, p, None, None) == \
        A.DOPD_ERR_NULL_POINTER
    assert pp(C.byref(s), p, p, p, 100, p, 64, p, H(cu), p, H(pre), 0, p, None, None) == A.DOPD_OK


def _decode_fp8(lib, shape, ctx, scales=FAKE, ws=FAKE, ws_bytes=1 << 30):
    ctx = np.asarray(ctx, np.int32)
    p = C.c_void_p(FAKE)
    sc = C.c_void_p(scales) if scales else None
    return lib.dopd_decode_attn_fp8(C.byref(shape), p, p, p, sc, sc, 10, p, 1024, p,
                                    A._hptr(ctx), len(ctx), 0, p, None,
                                    C.c_void_p(ws) if ws else None, ws_bytes, None)


def test_fp8_host_validation(lib):
    f8, b16 = _shape(dtype="fp8"), _shape()
    p = C.c_void_p(FAKE)
    # E4M3 pools only through the entry points that take scales, and the byte copies.
    assert _decode(lib, f8, [5]) == A.DOPD_ERR_UNSUPPORTED
    assert _prefill(lib, f8, [0, 4]) == A.DOPD_ERR_UNSUPPORTED
    assert lib.dopd_kv_write(C.byref(f8), p, p, p, p, 10, p, 4, p, p, 1, 5, None) == \
        A.DOPD_ERR_UNSUPPORTED
    assert _decode_fp8(lib, b16, [5]) == A.DOPD_ERR_UNSUPPORTED
    assert _decode_fp8(lib, f8, [5, 0]) == A.DOPD_ERR_INVALID_SHAPE
    assert _decode_fp8(lib, f8, [5], scales=0) == A.DOPD_ERR_NULL_POINTER
    assert _decode_fp8(lib, f8, [5], ws=0) == A.DOPD_ERR_NULL_POINTER
    assert _decode_fp8(lib, f8, [3000, 17], ws_bytes=256) == A.DOPD_ERR_WORKSPACE_TOO_SMALL
    assert _decode_fp8(lib, _shape(hq=34, hkv=2, dtype="fp8"), [5]) == A.DOPD_ERR_UNSUPPORTED
    # Same partition, same workspace as the bf16 cache.
    ctx = [3000, 17, 900]
    assert A.dopd_decode_workspace_size(f8, ctx, 3) == A.dopd_decode_workspace_size(b16, ctx, 3)
    w8 = lib.dopd_kv_write_fp8
    assert w8(C.byref(b16), p, p, p, p, p, p, 10, p, 4, p, p, 1, 5, None) == A.DOPD_ERR_UNSUPPORTED
    assert w8(C.byref(f8), p, p, None, p, p, p, 10, p, 4, p, p, 1, 5, None) == \
        A.DOPD_ERR_NULL_POINTER
    assert w8(C.byref(f8), p, p, p, p, p, p, 10, p, 4, p, p, -1, 5, None) == \
        A.DOPD_ERR_INVALID_SHAPE
    assert w8(C.byref(f8), p, p, p, p, p, p, 10, p, 4, p, p, 1, 0, None) == A.DOPD_OK
    lens = np.array([40, 600], np.int32)
    assert lib.dopd_kv_pack_for_handoff(C.byref(f8), 1, p, p, 10, p, 8, p, p, A._hptr(lens), p, 2,
                                        p, None) == A.DOPD_ERR_INVALID_SHAPE   # 600 > 8 pages


def _align256(n):
    return (n + 255) // 256 * 256


def test_prefill_paged_split_workspace_size(lib):
    s = _shape()  # 8 query heads, d = 128
    cu = np.array([0, 40, 41], np.int32)
    pre = np.array([600, 0], np.int32)
    ws = A.dopd_prefill_paged_workspace_size

    def need(n):  # [n][T][Hq][d] partial outputs, then [n][T][Hq][2] (m, l)
        rows = n * 41 * 8
        return _align256(rows * 128 * 4) + _align256(rows * 2 * 4)
    # 2 q tiles x 8 heads = 16 items: automatic wants ceil(1024 / 16) = 64
    # splits, capped at 1 + (600 // 64) // 8 = 2 by the fully seen key tiles
    assert ws(s, cu, pre, 2, 0) == need(2)
    assert ws(s, cu, pre, 2, 3) == need(3)
    assert ws(s, cu, pre, 2, 40) == need(16)                    # at most 16 splits
    assert ws(s, cu, pre, 2, 1) == 256                          # no split: nothing needed
    assert ws(_shape(dtype="fp32"), cu, pre, 2, 8) == 256       # fp32 never splits
    assert ws(A.make_shape(8, 2, 128, "bf16", 0.0), cu, pre, 2, 8) == 256  # nor scale <= 0
    assert ws(s, cu, pre, 0, 0) == 256
    assert ws(s, cu, pre, 2, -1) == 0
    assert ws(s, np.array([0, 40, 30], np.int32), pre, 2, 0) == 0
    assert ws(s, cu, np.array([-1, 0], np.int32), 2, 0) == 0
    # a call with many work items (600 q tiles x 8 heads) is not split
    big_cu = np.array([0, 600 * 128], np.int32)
    assert ws(s, big_cu, np.array([5000], np.int32), 1, 0) == 256


def test_prefill_paged_split_host_validation(lib):
    s = _shape()
    p = C.c_void_p(FAKE)
    cu = np.array([0, 40, 41], np.int32)
    pre = np.array([600, 0], np.int32)
    H = A._hptr
    need = A.dopd_prefill_paged_workspace_size(s, cu, pre, 2, 4)

    def call(splits, ws, nbytes, stride=64):
        return lib.dopd_prefill_paged_attn_split(
            C.byref(s), p, p, p, 100, p, stride, p, H(cu), p, H(pre), 2, splits, p, None,
            None if ws is None else C.c_void_p(ws), nbytes, None)
    assert call(4, None, need) == A.DOPD_ERR_NULL_POINTER
    assert call(4, FAKE, need - 1) == A.DOPD_ERR_WORKSPACE_TOO_SMALL
    assert call(4, FAKE + 64, need) == A.DOPD_ERR_INVALID_SHAPE   # not 256-byte aligned
    assert call(-1, FAKE, need) == A.DOPD_ERR_INVALID_SHAPE
    assert call(4, FAKE, need, stride=39) == A.DOPD_ERR_INVALID_SHAPE  # table too narrow


def test_prefill_paged_fp8_workspace_size(lib):
    # The E4M3 chunk prefill reads the pools directly: its workspace is the
    # bf16 paged prefill's (the key-split partials), for E4M3 shapes only.
    s8 = _shape(dtype="fp8")  # 8 query heads, 2 KV heads, d = 128
    cu = np.array([0, 40, 41, 41], np.int32)
    pre = np.array([600, 0, 900], np.int32)
    ws = A.dopd_prefill_paged_fp8_workspace_size
    for n in (1, 0, 3, 40):
        assert ws(s8, cu, pre, 3, n) == A.dopd_prefill_paged_workspace_size(_shape(), cu, pre, 3, n)
    assert ws(s8, cu, pre, 3, 3) > 256
    assert ws(_shape(), cu, pre, 3, 0) == 0                     # bf16 pools: not this entry
    assert ws(s8, cu, pre, 0, 0) == 256
    assert ws(s8, cu, pre, 3, -1) == 0
    assert ws(s8, np.array([0, 40, 30, 41], np.int32), pre, 3, 0) == 0
    assert ws(s8, cu, np.array([0, -1, 0], np.int32), 3, 0) == 0


def test_prefill_paged_fp8_host_validation(lib):
    s8 = _shape(dtype="fp8")
    p = C.c_void_p(FAKE)
    cu = np.array([0, 40, 41], np.int32)
    pre = np.array([600, 0], np.int32)
    H = A._hptr
    need = A.dopd_prefill_paged_fp8_workspace_size(s8, cu, pre, 2, 4)

    def call(splits, ws, nbytes, stride=64, shape=s8, scales=p):
        return lib.dopd_prefill_paged_attn_fp8(
            C.byref(shape), p, p, p, scales, scales, 100, p, stride, p, H(cu), p, H(pre), 2,
            splits, p, None, None if ws is None else C.c_void_p(ws), nbytes, None)
    assert call(4, FAKE, need, shape=_shape()) == A.DOPD_ERR_UNSUPPORTED
    assert call(4, FAKE, need, scales=None) == A.DOPD_ERR_NULL_POINTER
    assert call(4, None, need) == A.DOPD_ERR_NULL_POINTER
    assert call(4, FAKE, need - 1) == A.DOPD_ERR_WORKSPACE_TOO_SMALL
    assert call(4, FAKE + 64, need) == A.DOPD_ERR_INVALID_SHAPE   # not 256-byte aligned
    assert call(-1, FAKE, need) == A.DOPD_ERR_INVALID_SHAPE
    assert call(4, FAKE, need, stride=39) == A.DOPD_ERR_INVALID_SHAPE  # table too narrow


def _write_pack(lib, shape, cu, stride=64, out=FAKE, offs=FAKE, nreq=None):
    cu = np.asarray(cu, np.int32)
    p = C.c_void_p(FAKE)
    n = len(cu) - 1 if nreq is None else nreq
    return lib.dopd_kv_write_pack_for_handoff(
        C.byref(shape), p, p, p, p, 100, p, stride, p, A._hptr(cu), n,
        C.c_void_p(offs) if offs else None, C.c_void_p(out) if out else None, None)


def test_write_pack_host_validation(lib):
    s = _shape()
    assert _write_pack(lib, _shape(dtype="fp32"), [0, 4]) == A.DOPD_ERR_UNSUPPORTED
    assert _write_pack(lib, _shape(dtype="fp8"), [0, 4]) == A.DOPD_ERR_UNSUPPORTED
    assert _write_pack(lib, s, [0, 4], out=0) == A.DOPD_ERR_NULL_POINTER      # offsets without buffer
    assert _write_pack(lib, s, [0, 4], offs=0) == A.DOPD_ERR_NULL_POINTER     # buffer without offsets
    assert _write_pack(lib, s, [1, 4]) == A.DOPD_ERR_INVALID_SHAPE           # cu[0] != 0
    assert _write_pack(lib, s, [0, 4, 2]) == A.DOPD_ERR_INVALID_SHAPE        # negative length
    assert _write_pack(lib, s, [0, 100], stride=6) == A.DOPD_ERR_INVALID_SHAPE  # 7 pages > 6 columns
    assert _write_pack(lib, s, [0], nreq=0) == A.DOPD_OK
    assert _write_pack(lib, s, [0, 0, 0]) == A.DOPD_OK                       # nothing to write


def _pd(lib, shape, ctx, cu, schedule=0, stride=1024, ws_bytes=1 << 30, ws=FAKE, h_out=FAKE,
        h_offs=FAKE):
    ctx = np.asarray(ctx, np.int32)
    cu = np.asarray(cu, np.int32)
    p = C.c_void_p(FAKE)
    return lib.dopd_pd_step(
        C.byref(shape), p, p, p, A._hptr(ctx), len(ctx), p, None, p, p, p, p, A._hptr(cu),
        len(cu) - 1, p, p, None, p, p, 100, stride, C.c_void_p(h_offs) if h_offs else None,
        C.c_void_p(h_out) if h_out else None, schedule, C.c_void_p(ws) if ws else None, ws_bytes,
        None)


def test_pd_step_host_validation(lib):
    s = _shape(hq=28, hkv=4)
    assert _pd(lib, _shape(dtype="fp32"), [5], [0, 4]) == A.DOPD_ERR_UNSUPPORTED
    assert _pd(lib, s, [5, 0], [0, 4]) == A.DOPD_ERR_INVALID_SHAPE      # context < 1
    assert _pd(lib, s, [5], [0, 4], schedule=4) == A.DOPD_ERR_INVALID_SHAPE
    assert _pd(lib, s, [5], [2, 4]) == A.DOPD_ERR_INVALID_SHAPE         # cu[0] != 0
    assert _pd(lib, s, [5000], [0, 4], stride=8) == A.DOPD_ERR_INVALID_SHAPE
    assert _pd(lib, s, [5], [0, 400], stride=8) == A.DOPD_ERR_INVALID_SHAPE
    assert _pd(lib, s, [5], [0, 4], h_out=0) == A.DOPD_ERR_NULL_POINTER
    assert _pd(lib, s, [5], [0, 4], ws=0) == A.DOPD_ERR_NULL_POINTER
    assert _pd(lib, s, [5], [0, 4], ws=FAKE + 8) == A.DOPD_ERR_INVALID_SHAPE  # misaligned
    for sched in (A.DOPD_PD_AUTO, A.DOPD_PD_PREFILL_FIRST, A.DOPD_PD_DECODE_FIRST,
                  A.DOPD_PD_DECODE_FIRST_WIDE):
        need = A.dopd_pd_step_workspace_size(s, [3000, 17], 2, sched)
        assert need >= 256 and need % 256 == 0
        assert _pd(lib, s, [3000, 17], [0, 4], schedule=sched, ws_bytes=need - 1) == \
            A.DOPD_ERR_WORKSPACE_TOO_SMALL
    # one decode slice per CU needs no more partial slots than two
    assert A.dopd_pd_step_workspace_size(s, [16384] * 8, 8, A.DOPD_PD_DECODE_FIRST) <= \
        A.dopd_pd_step_workspace_size(s, [16384] * 8, 8, A.DOPD_PD_PREFILL_FIRST)
    assert A.dopd_pd_step_workspace_size(s, [5], 1, 7) == 0
    assert A.dopd_pd_step_workspace_size(s, [16384] * 8, 8, A.DOPD_PD_DECODE_FIRST_WIDE) <= \
        A.dopd_pd_step_workspace_size(s, [16384] * 8, 8, A.DOPD_PD_PREFILL_FIRST)
    # both batches empty: nothing to do
    assert lib.dopd_pd_step(C.byref(s), None, None, None, None, 0, None, None, None, None, None,
                            None, None, 0, None, None, None, None, None, 0, 0, None, None, 0,
                            None, 0, None) == A.DOPD_OK



def _pd8(lib, shape, ctx, cu, scales=FAKE, ws=FAKE, ws_bytes=1 << 30):
    ctx = np.asarray(ctx, np.int32)
    cu = np.asarray(cu, np.int32)
    p = C.c_void_p(FAKE)
    sc = C.c_void_p(scales) if scales else None
    return lib.dopd_pd_step_fp8(
        C.byref(shape), p, p, p, A._hptr(ctx), len(ctx), p, None, p, p, p, p, A._hptr(cu),
        len(cu) - 1, p, p, None, p, p, sc, sc, 100, 1024, p, p, 0,
        C.c_void_p(ws) if ws else None, ws_bytes, None)


def test_pd_step_fp8_host_validation(lib):
    s8 = _shape(hq=28, hkv=4, dtype="fp8")
    assert _pd8(lib, _shape(hq=28, hkv=4), [5], [0, 4]) == A.DOPD_ERR_UNSUPPORTED  # bf16 shape
    assert _pd(lib, s8, [5], [0, 4]) == A.DOPD_ERR_UNSUPPORTED   # E4M3 shape, bf16 entry
    assert _pd8(lib, s8, [5], [0, 4], scales=0) == A.DOPD_ERR_NULL_POINTER
    assert _pd8(lib, s8, [5, 0], [0, 4]) == A.DOPD_ERR_INVALID_SHAPE
    assert _pd8(lib, s8, [5], [0, 4], ws=0) == A.DOPD_ERR_NULL_POINTER
    need = A.dopd_pd_step_workspace_size(s8, [3000, 17], 2, A.DOPD_PD_AUTO)
    assert need == A.dopd_pd_step_workspace_size(_shape(hq=28, hkv=4), [3000, 17], 2,
                                                 A.DOPD_PD_AUTO)
    assert _pd8(lib, s8, [3000, 17], [0, 4], ws_bytes=need - 1) == A.DOPD_ERR_WORKSPACE_TOO_SMALL
