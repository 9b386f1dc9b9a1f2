"""ctypes binding of ``libdopd_attn.so`` (C ABI in ``include/dopd_attn.h``).

Argument marshalling only: every entry point takes torch tensors (device
memory) or numpy arrays (the ``_host`` copies), passes raw pointers to the
library, and raises :class:`DopdError` on a non-OK status.  All compute runs
in the library's HIP kernels on the given (default: current) HIP stream.
The library is loaded on first use; if it has not been built, the call fails
loudly -- there is no fallback path.
"""
from __future__ import annotations

import ctypes as C
import math
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libdopd_attn.so")

DOPD_OK, DOPD_ERR_NULL_POINTER, DOPD_ERR_INVALID_SHAPE = 0, 1, 2
DOPD_ERR_UNSUPPORTED, DOPD_ERR_WORKSPACE_TOO_SMALL, DOPD_ERR_HIP = 3, 4, 5
DOPD_ERR_UNSUPPORTED_DTYPE = DOPD_ERR_UNSUPPORTED
DOPD_BF16, DOPD_FP32, DOPD_FP8_E4M3 = 0, 1, 2
DOPD_PD_AUTO, DOPD_PD_PREFILL_FIRST, DOPD_PD_DECODE_FIRST, DOPD_PD_DECODE_FIRST_WIDE = 0, 1, 2, 3
PAGE_SIZE = 16

EXPORTS = (
    "dopd_prefill_attn", "dopd_prefill_workspace_size", "dopd_prefill_paged_attn", "dopd_prefill_paged_attn_split",
    "dopd_prefill_paged_workspace_size", "dopd_prefill_paged_attn_fp8",
    "dopd_prefill_paged_fp8_workspace_size", "dopd_kv_write", "dopd_kv_write_fp8",
    "dopd_decode_attn", "dopd_decode_attn_fp8", "dopd_decode_workspace_size",
    "dopd_decode_attn_noalloc",
    "dopd_kv_pack_for_handoff", "dopd_kv_unpack_from_handoff", "dopd_validate_page_table_host",
    "dopd_kv_write_pack_for_handoff", "dopd_pd_step", "dopd_pd_step_fp8",
    "dopd_pd_step_workspace_size",
    "dopd_status_string",
    "dopd_last_hip_error",
)


class DopdError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        msg = status_string(status)
        if status == DOPD_ERR_HIP:
            msg += f" (hipError {lib().dopd_last_hip_error()})"
        super().__init__(f"{where}: {msg}")


class Shape(C.Structure):
    _fields_ = [("num_q_heads", C.c_int32), ("num_kv_heads", C.c_int32),
                ("head_dim", C.c_int32), ("page_size", C.c_int32), ("dtype", C.c_int32),
                ("softmax_scale", C.c_float)]


def make_shape(hq: int, hkv: int, d: int, dtype: str = "bf16", scale: float | None = None,
               page_size: int = PAGE_SIZE) -> Shape:
    """Shape descriptor; the softmax scale defaults to 1/sqrt(d).  dtype "fp8"
    means E4M3 KV pages (bf16 q/out/fresh K/V)."""
    dt = {"bf16": DOPD_BF16, "fp32": DOPD_FP32, "fp8": DOPD_FP8_E4M3}[dtype]
    return Shape(hq, hkv, d, page_size, dt, 1.0 / math.sqrt(d) if scale is None else scale)


_LIB = None


def lib():
    global _LIB
    if _LIB is None:
        # PyTorch ships its own HIP runtime under the same soname as the one
        # the library links; importing it first makes the process load one
        # runtime (its), whatever the caller touches first.
        import torch  # noqa: F401
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                               "or python paper_2511_20982_amd/build.py")
        L = C.CDLL(LIB_PATH)
        P, i32, sz = C.c_void_p, C.c_int32, C.c_size_t
        SP = C.POINTER(Shape)
        L.dopd_prefill_attn.argtypes = [SP, P, P, P, P, P, P, P, i32, P, sz, P]
        L.dopd_prefill_workspace_size.argtypes = [SP, P, i32]
        L.dopd_prefill_workspace_size.restype = sz
        L.dopd_prefill_paged_attn.argtypes = [SP, P, P, P, i32, P, i32, P, P, P, P, i32, P, P, P]
        L.dopd_prefill_paged_attn_split.argtypes = [SP, P, P, P, i32, P, i32, P, P, P, P, i32,
                                                    i32, P, P, P, sz, P]
        L.dopd_prefill_paged_workspace_size.argtypes = [SP, P, P, i32, i32]
        L.dopd_prefill_paged_workspace_size.restype = sz
        L.dopd_prefill_paged_attn_fp8.argtypes = [SP, P, P, P, P, P, i32, P, i32, P, P, P, P, i32,
                                                  i32, P, P, P, sz, P]
        L.dopd_prefill_paged_fp8_workspace_size.argtypes = [SP, P, P, i32, i32]
        L.dopd_prefill_paged_fp8_workspace_size.restype = sz
        L.dopd_kv_write.argtypes = [SP, P, P, P, P, i32, P, i32, P, P, i32, i32, P]
        L.dopd_decode_attn.argtypes = [SP, P, P, P, i32, P, i32, P, P, i32, i32, P, P, P, sz, P]
        L.dopd_kv_write_fp8.argtypes = [SP, P, P, P, P, P, P, i32, P, i32, P, P, i32, i32, P]
        L.dopd_decode_attn_fp8.argtypes = [SP, P, P, P, P, P, i32, P, i32, P, P, i32, i32, P, P,
                                           P, sz, P]
        L.dopd_decode_attn_noalloc.argtypes = [SP, P, P, P, i32, P, i32, P, P, i32, i32, P, P, P]
        L.dopd_decode_workspace_size.argtypes = [SP, P, i32, i32]
        L.dopd_decode_workspace_size.restype = sz
        L.dopd_kv_pack_for_handoff.argtypes = [SP, i32, P, P, i32, P, i32, P, P, P, P, i32, P, P]
        L.dopd_kv_unpack_from_handoff.argtypes = [SP, i32, P, P, P, P, P, i32, P, P, i32, P, i32, P]
        L.dopd_validate_page_table_host.argtypes = [P, i32, i32, P, i32]
        L.dopd_kv_write_pack_for_handoff.argtypes = [SP, P, P, P, P, i32, P, i32, P, P, i32, P,
                                                     P, P]
        L.dopd_pd_step.argtypes = [SP, P, P, P, P, i32, P, P, P, P, P, P, P, i32, P, P, P, P, P,
                                   i32, i32, P, P, i32, P, sz, P]
        L.dopd_pd_step_fp8.argtypes = [SP, P, P, P, P, i32, P, P, P, P, P, P, P, i32, P, P, P,
                                       P, P, P, P, i32, i32, P, P, i32, P, sz, P]
        L.dopd_pd_step_workspace_size.argtypes = [SP, P, i32, i32]
        L.dopd_pd_step_workspace_size.restype = sz
        L.dopd_status_string.argtypes = [i32]
        L.dopd_status_string.restype = C.c_char_p
        L.dopd_last_hip_error.restype = i32
        for f in ("dopd_prefill_attn", "dopd_prefill_paged_attn",
                  "dopd_prefill_paged_attn_split", "dopd_prefill_paged_attn_fp8", "dopd_kv_write",
                  "dopd_kv_write_fp8", "dopd_decode_attn", "dopd_decode_attn_fp8",
                  "dopd_decode_attn_noalloc",
                  "dopd_kv_pack_for_handoff", "dopd_kv_unpack_from_handoff",
                  "dopd_validate_page_table_host", "dopd_kv_write_pack_for_handoff",
                  "dopd_pd_step", "dopd_pd_step_fp8"):
            getattr(L, f).restype = i32
        _LIB = L
    return _LIB


def status_string(status: int) -> str:
    return lib().dopd_status_string(status).decode()


# ------------------------------------------------------------------ marshalling
def _dptr(t):
    """Device pointer of a tensor (None -> NULL)."""
    return None if t is None else C.c_void_p(t.data_ptr())


def _hptr(a):
    """Host pointer of a contiguous int32/int64 numpy array (None -> NULL)."""
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def _host_i32(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.int32)


def _stream(stream):
    if stream is None:
        import torch
        stream = torch.cuda.current_stream()
    return C.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _check(status: int, where: str):
    if status != DOPD_OK:
        raise DopdError(status, where)


# ------------------------------------------------------------------ entry points
def dopd_prefill_attn(shape, q, k, v, out, lse, cu_seqlens, cu_seqlens_host, num_reqs,
                      workspace=None, workspace_bytes=None, stream=None):
    cu_h = _host_i32(cu_seqlens_host)
    if workspace_bytes is None:
        workspace_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().dopd_prefill_attn(C.byref(shape), _dptr(q), _dptr(k), _dptr(v), _dptr(out),
                                   _dptr(lse), _dptr(cu_seqlens), _hptr(cu_h), int(num_reqs),
                                   _dptr(workspace), int(workspace_bytes), _stream(stream)),
           "dopd_prefill_attn")


def dopd_prefill_workspace_size(shape, cu_seqlens_host, num_reqs) -> int:
    cu_h = _host_i32(cu_seqlens_host)
    return int(lib().dopd_prefill_workspace_size(C.byref(shape), _hptr(cu_h), int(num_reqs)))


def dopd_prefill_paged_attn(shape, q, k_pool, v_pool, num_pages, page_table, page_table_stride,
                            cu_seqlens, cu_seqlens_host, prefix_lens, prefix_lens_host, num_reqs,
                            out, lse, stream=None):
    cu_h = _host_i32(cu_seqlens_host)
    pre_h = _host_i32(prefix_lens_host)
    _check(lib().dopd_prefill_paged_attn(C.byref(shape), _dptr(q), _dptr(k_pool), _dptr(v_pool),
                                         int(num_pages), _dptr(page_table), int(page_table_stride),
                                         _dptr(cu_seqlens), _hptr(cu_h), _dptr(prefix_lens),
                                         _hptr(pre_h), int(num_reqs), _dptr(out), _dptr(lse),
                                         _stream(stream)), "dopd_prefill_paged_attn")


def dopd_prefill_paged_workspace_size(shape, cu_seqlens_host, prefix_lens_host, num_reqs,
                                      num_splits=0) -> int:
    cu_h = _host_i32(cu_seqlens_host)
    pre_h = _host_i32(prefix_lens_host)
    return int(lib().dopd_prefill_paged_workspace_size(C.byref(shape), _hptr(cu_h), _hptr(pre_h),
                                                       int(num_reqs), int(num_splits)))


def dopd_prefill_paged_attn_split(shape, q, k_pool, v_pool, num_pages, page_table,
                                  page_table_stride, cu_seqlens, cu_seqlens_host, prefix_lens,
                                  prefix_lens_host, num_reqs, num_splits, out, lse, workspace,
                                  workspace_bytes=None, stream=None):
    cu_h = _host_i32(cu_seqlens_host)
    pre_h = _host_i32(prefix_lens_host)
    if workspace_bytes is None:
        workspace_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().dopd_prefill_paged_attn_split(
        C.byref(shape), _dptr(q), _dptr(k_pool), _dptr(v_pool), int(num_pages),
        _dptr(page_table), int(page_table_stride), _dptr(cu_seqlens), _hptr(cu_h),
        _dptr(prefix_lens), _hptr(pre_h), int(num_reqs), int(num_splits), _dptr(out), _dptr(lse),
        _dptr(workspace), int(workspace_bytes), _stream(stream)), "dopd_prefill_paged_attn_split")


def dopd_prefill_paged_fp8_workspace_size(shape, cu_seqlens_host, prefix_lens_host, num_reqs,
                                          num_splits=0) -> int:
    cu_h = _host_i32(cu_seqlens_host)
    pre_h = _host_i32(prefix_lens_host)
    return int(lib().dopd_prefill_paged_fp8_workspace_size(
        C.byref(shape), _hptr(cu_h), _hptr(pre_h), int(num_reqs), int(num_splits)))


def dopd_prefill_paged_attn_fp8(shape, q, k_pool, v_pool, k_scale, v_scale, num_pages,
                                page_table, page_table_stride, cu_seqlens, cu_seqlens_host,
                                prefix_lens, prefix_lens_host, num_reqs, num_splits, out, lse,
                                workspace, workspace_bytes=None, stream=None):
    cu_h = _host_i32(cu_seqlens_host)
    pre_h = _host_i32(prefix_lens_host)
    if workspace_bytes is None:
        workspace_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().dopd_prefill_paged_attn_fp8(
        C.byref(shape), _dptr(q), _dptr(k_pool), _dptr(v_pool), _dptr(k_scale), _dptr(v_scale),
        int(num_pages), _dptr(page_table), int(page_table_stride), _dptr(cu_seqlens),
        _hptr(cu_h), _dptr(prefix_lens), _hptr(pre_h), int(num_reqs), int(num_splits),
        _dptr(out), _dptr(lse), _dptr(workspace), int(workspace_bytes), _stream(stream)),
        "dopd_prefill_paged_attn_fp8")


def dopd_kv_write(shape, k_new, v_new, k_pool, v_pool, num_pages, page_table,
                  page_table_stride, cu_new_tokens, start_pos, num_reqs, total_new_tokens,
                  stream=None):
    _check(lib().dopd_kv_write(C.byref(shape), _dptr(k_new), _dptr(v_new), _dptr(k_pool),
                               _dptr(v_pool), int(num_pages), _dptr(page_table),
                               int(page_table_stride), _dptr(cu_new_tokens), _dptr(start_pos),
                               int(num_reqs), int(total_new_tokens), _stream(stream)),
           "dopd_kv_write")


def dopd_kv_write_fp8(shape, k_new, v_new, k_scale, v_scale, k_pool, v_pool, num_pages,
                      page_table, page_table_stride, cu_new_tokens, start_pos, num_reqs,
                      total_new_tokens, stream=None):
    _check(lib().dopd_kv_write_fp8(C.byref(shape), _dptr(k_new), _dptr(v_new), _dptr(k_scale),
                                   _dptr(v_scale), _dptr(k_pool), _dptr(v_pool), int(num_pages),
                                   _dptr(page_table), int(page_table_stride),
                                   _dptr(cu_new_tokens), _dptr(start_pos), int(num_reqs),
                                   int(total_new_tokens), _stream(stream)), "dopd_kv_write_fp8")


def dopd_decode_workspace_size(shape, context_lens_host, num_reqs, split_tokens=0) -> int:
    ctx = _host_i32(context_lens_host)
    return int(lib().dopd_decode_workspace_size(C.byref(shape), _hptr(ctx), int(num_reqs),
                                                int(split_tokens)))


def dopd_decode_attn(shape, q, k_pool, v_pool, num_pages, page_table, page_table_stride,
                     context_lens, context_lens_host, num_reqs, split_tokens, out, lse,
                     workspace, workspace_bytes=None, stream=None):
    ctx = _host_i32(context_lens_host)
    if workspace_bytes is None:
        workspace_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().dopd_decode_attn(C.byref(shape), _dptr(q), _dptr(k_pool), _dptr(v_pool),
                                  int(num_pages), _dptr(page_table), int(page_table_stride),
                                  _dptr(context_lens), _hptr(ctx), int(num_reqs),
                                  int(split_tokens), _dptr(out), _dptr(lse), _dptr(workspace),
                                  int(workspace_bytes), _stream(stream)), "dopd_decode_attn")


DECODE_NOALLOC_SCRATCH_BYTES = 32 << 20


def dopd_decode_attn_noalloc(shape, q, k_pool, v_pool, num_pages, page_table, page_table_stride,
                             context_lens, context_lens_host, num_reqs, split_tokens, out, lse,
                             stream=None):
    ctx = _host_i32(context_lens_host)
    _check(lib().dopd_decode_attn_noalloc(C.byref(shape), _dptr(q), _dptr(k_pool), _dptr(v_pool),
                                          int(num_pages), _dptr(page_table),
                                          int(page_table_stride), _dptr(context_lens),
                                          _hptr(ctx), int(num_reqs), int(split_tokens),
                                          _dptr(out), _dptr(lse), _stream(stream)),
           "dopd_decode_attn_noalloc")


def dopd_decode_attn_fp8(shape, q, k_pool, v_pool, k_scale, v_scale, num_pages, page_table,
                         page_table_stride, context_lens, context_lens_host, num_reqs,
                         split_tokens, out, lse, workspace, workspace_bytes=None, stream=None):
    ctx = _host_i32(context_lens_host)
    if workspace_bytes is None:
        workspace_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().dopd_decode_attn_fp8(C.byref(shape), _dptr(q), _dptr(k_pool), _dptr(v_pool),
                                      _dptr(k_scale), _dptr(v_scale), int(num_pages),
                                      _dptr(page_table), int(page_table_stride),
                                      _dptr(context_lens), _hptr(ctx), int(num_reqs),
                                      int(split_tokens), _dptr(out), _dptr(lse),
                                      _dptr(workspace), int(workspace_bytes), _stream(stream)),
           "dopd_decode_attn_fp8")


def dopd_kv_pack_for_handoff(shape, num_layers, k_pool, v_pool, num_pages, page_table,
                             page_table_stride, req_ids, seq_lens, seq_lens_host, out_offsets,
                             num_handoff, out, stream=None):
    lens_h = _host_i32(seq_lens_host)
    _check(lib().dopd_kv_pack_for_handoff(C.byref(shape), int(num_layers), _dptr(k_pool),
                                          _dptr(v_pool), int(num_pages), _dptr(page_table),
                                          int(page_table_stride), _dptr(req_ids),
                                          _dptr(seq_lens), _hptr(lens_h), _dptr(out_offsets),
                                          int(num_handoff), _dptr(out), _stream(stream)),
           "dopd_kv_pack_for_handoff")


def dopd_kv_unpack_from_handoff(shape, num_layers, buf, in_offsets, req_ids, seq_lens,
                                seq_lens_host, num_handoff, k_pool, v_pool, num_pages, page_table,
                                page_table_stride, stream=None):
    lens_h = _host_i32(seq_lens_host)
    _check(lib().dopd_kv_unpack_from_handoff(C.byref(shape), int(num_layers), _dptr(buf),
                                             _dptr(in_offsets), _dptr(req_ids), _dptr(seq_lens),
                                             _hptr(lens_h), int(num_handoff), _dptr(k_pool),
                                             _dptr(v_pool), int(num_pages), _dptr(page_table),
                                             int(page_table_stride), _stream(stream)),
           "dopd_kv_unpack_from_handoff")


def dopd_kv_write_pack_for_handoff(shape, k_new, v_new, k_pool, v_pool, num_pages, page_table,
                                   page_table_stride, cu_seqlens, cu_seqlens_host, num_reqs,
                                   out_offsets, out, stream=None):
    cu_h = _host_i32(cu_seqlens_host)
    _check(lib().dopd_kv_write_pack_for_handoff(
        C.byref(shape), _dptr(k_new), _dptr(v_new), _dptr(k_pool), _dptr(v_pool), int(num_pages),
        _dptr(page_table), int(page_table_stride), _dptr(cu_seqlens), _hptr(cu_h),
        int(num_reqs), _dptr(out_offsets), _dptr(out), _stream(stream)),
        "dopd_kv_write_pack_for_handoff")


def dopd_pd_step_workspace_size(shape, context_lens_host, num_dec, schedule=DOPD_PD_AUTO) -> int:
    ctx = _host_i32(context_lens_host)
    return int(lib().dopd_pd_step_workspace_size(C.byref(shape), _hptr(ctx), int(num_dec),
                                                 int(schedule)))


def dopd_pd_step(shape, q_dec, dec_page_table, context_lens, context_lens_host, num_dec, out_dec,
                 lse_dec, q, k, v, cu_seqlens, cu_seqlens_host, num_pre, pre_page_table,
                 out_pre, lse_pre, k_pool, v_pool, num_pages, page_table_stride,
                 handoff_offsets, handoff_out, schedule, workspace, workspace_bytes=None,
                 stream=None):
    ctx = _host_i32(context_lens_host)
    cu_h = _host_i32(cu_seqlens_host)
    if workspace_bytes is None:
        workspace_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().dopd_pd_step(
        C.byref(shape), _dptr(q_dec), _dptr(dec_page_table), _dptr(context_lens), _hptr(ctx),
        int(num_dec), _dptr(out_dec), _dptr(lse_dec), _dptr(q), _dptr(k), _dptr(v),
        _dptr(cu_seqlens), _hptr(cu_h), int(num_pre), _dptr(pre_page_table), _dptr(out_pre),
        _dptr(lse_pre), _dptr(k_pool), _dptr(v_pool), int(num_pages), int(page_table_stride),
        _dptr(handoff_offsets), _dptr(handoff_out), int(schedule), _dptr(workspace),
        int(workspace_bytes), _stream(stream)), "dopd_pd_step")


def dopd_pd_step_fp8(shape, q_dec, dec_page_table, context_lens, context_lens_host, num_dec,
                     out_dec, lse_dec, q, k, v, cu_seqlens, cu_seqlens_host, num_pre,
                     pre_page_table, out_pre, lse_pre, k_pool, v_pool, k_scale, v_scale,
                     num_pages, page_table_stride, handoff_offsets, handoff_out, schedule,
                     workspace, workspace_bytes=None, stream=None):
    ctx = _host_i32(context_lens_host)
    cu_h = _host_i32(cu_seqlens_host)
    if workspace_bytes is None:
        workspace_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().dopd_pd_step_fp8(
        C.byref(shape), _dptr(q_dec), _dptr(dec_page_table), _dptr(context_lens), _hptr(ctx),
        int(num_dec), _dptr(out_dec), _dptr(lse_dec), _dptr(q), _dptr(k), _dptr(v),
        _dptr(cu_seqlens), _hptr(cu_h), int(num_pre), _dptr(pre_page_table), _dptr(out_pre),
        _dptr(lse_pre), _dptr(k_pool), _dptr(v_pool), _dptr(k_scale), _dptr(v_scale),
        int(num_pages), int(page_table_stride), _dptr(handoff_offsets), _dptr(handoff_out),
        int(schedule), _dptr(workspace), int(workspace_bytes), _stream(stream)),
        "dopd_pd_step_fp8")


def pd_step_workspace(shape, context_lens_host, num_dec, schedule=DOPD_PD_AUTO, device="cuda"):
    """A 256-byte aligned workspace for dopd_pd_step."""
    import torch
    n = dopd_pd_step_workspace_size(shape, context_lens_host, num_dec, schedule)
    if n == 0:
        raise DopdError(DOPD_ERR_INVALID_SHAPE, "dopd_pd_step_workspace_size")
    ws = torch.empty(n + 256, dtype=torch.uint8, device=device)
    off = (-ws.data_ptr()) % 256
    return ws[off:off + n]


def dopd_validate_page_table_host(page_table_host, page_table_stride, num_reqs, lens_host,
                                  num_pages) -> int:
    pt = _host_i32(page_table_host)
    lens = _host_i32(lens_host)
    return int(lib().dopd_validate_page_table_host(_hptr(pt), int(page_table_stride),
                                                   int(num_reqs), _hptr(lens), int(num_pages)))


# ------------------------------------------------------------------ device buffers
def decode_workspace(shape, context_lens_host, num_reqs, split_tokens=0, device="cuda"):
    """A zeroed, 256-byte aligned workspace for dopd_decode_attn."""
    import torch
    n = dopd_decode_workspace_size(shape, context_lens_host, num_reqs, split_tokens)
    if n == 0:
        raise DopdError(DOPD_ERR_INVALID_SHAPE, "dopd_decode_workspace_size")
    ws = torch.zeros(n + 256, dtype=torch.uint8, device=device)
    off = (-ws.data_ptr()) % 256
    return ws[off:off + n]


def prefill_paged_workspace(shape, cu_seqlens_host, prefix_lens_host, num_reqs, num_splits=0,
                            device="cuda"):
    """A 256-byte aligned workspace for dopd_prefill_paged_attn_split."""
    import torch
    n = dopd_prefill_paged_workspace_size(shape, cu_seqlens_host, prefix_lens_host, num_reqs,
                                          num_splits)
    if n == 0:
        raise DopdError(DOPD_ERR_INVALID_SHAPE, "dopd_prefill_paged_workspace_size")
    ws = torch.empty(n + 256, dtype=torch.uint8, device=device)
    off = (-ws.data_ptr()) % 256
    return ws[off:off + n]


def prefill_paged_fp8_workspace(shape, cu_seqlens_host, prefix_lens_host, num_reqs,
                                num_splits=0, device="cuda"):
    """A 256-byte aligned workspace for dopd_prefill_paged_attn_fp8."""
    import torch
    n = dopd_prefill_paged_fp8_workspace_size(shape, cu_seqlens_host, prefix_lens_host, num_reqs,
                                              num_splits)
    if n == 0:
        raise DopdError(DOPD_ERR_INVALID_SHAPE, "dopd_prefill_paged_fp8_workspace_size")
    ws = torch.empty(n + 256, dtype=torch.uint8, device=device)
    off = (-ws.data_ptr()) % 256
    return ws[off:off + n]


def to_device(a: np.ndarray, device="cuda"):
    """numpy array -> device tensor; uint16 arrays are bf16 bit patterns."""
    import torch
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(a).to(device)


def to_host(t) -> np.ndarray:
    """Device tensor -> numpy; bf16 comes back as uint16 bit patterns."""
    import torch
    t = t.detach().to("cpu").contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()
