"""Helpers for the GPU parity tests: run the HIP path through the C ABI on a
seeded workload and compare with the fp64 oracle."""
from __future__ import annotations

import numpy as np
import torch

from paper_2511_20982_amd import attn as A
from paper_2511_20982_amd import inputs as I

DEV = "cuda"
CANARY = 0x5A5A  # guard-band pattern (uint16 words)

# Parity bar: max |gpu - oracle| <= ATOL, and per (request, head) block
# max |gpu - oracle| / rms(oracle) <= NORM_TOL (the absolute bar alone is about
# one standard deviation of the output on long rows).
ATOL = {"bf16": 2e-2, "fp32": 1e-5}
NORM_TOL = {"bf16": 5e-2, "fp32": 1e-4}


def widen(x: np.ndarray) -> np.ndarray:
    if x.dtype == np.uint16:
        return I.bf16_bits_to_f32(x).astype(np.float64)
    return x.astype(np.float64)


def guarded(shape, dtype: torch.dtype, margin: int = 4096):
    """Tensor of `shape` inside a buffer whose margins hold a canary pattern."""
    n = int(np.prod(shape))
    esz = torch.tensor([], dtype=dtype).element_size()
    words = (n * esz + 1) // 2 + margin  # margin bytes on either side
    buf = torch.full((words,), CANARY, dtype=torch.int16, device=DEV)
    body = buf.view(torch.uint8)[margin: margin + n * esz].view(dtype).view(*shape)
    return body, buf, margin


def canary_intact(buf, margin, nbytes) -> bool:
    h = buf.cpu().numpy().view(np.uint8)
    lo = h[:margin]
    hi = h[margin + nbytes: margin + nbytes + margin - 1]
    return bool(np.all(lo == 0x5A) and np.all(hi == 0x5A))


def assert_attention_close(gpu: np.ndarray, ref: np.ndarray, dtype: str, what: str = ""):
    """gpu, ref: [..., d] arrays (gpu already widened to float64)."""
    assert gpu.shape == ref.shape, (gpu.shape, ref.shape)
    assert np.all(np.isfinite(gpu)), f"{what}: non-finite output"
    err = np.abs(gpu - ref)
    max_abs = float(err.max()) if err.size else 0.0
    assert max_abs <= ATOL[dtype], f"{what}: max abs err {max_abs:.3e} > {ATOL[dtype]}"
    if err.size:
        rms = np.sqrt(np.mean(ref ** 2, axis=-1))
        norm = err.max(axis=-1) / np.maximum(rms, 1e-30)
        worst = float(norm.max())
        assert worst <= NORM_TOL[dtype], f"{what}: normalised err {worst:.3e} > {NORM_TOL[dtype]}"
    return max_abs


def shape_of(w, scale=None) -> A.Shape:
    return A.make_shape(w.hq, w.hkv, w.d, w.dtype, w.scale if scale is None else scale)


# ------------------------------------------------------------------ runners
def gpu_prefill(shape, q, k, v, cu, with_lse=True, stream=None):
    qd, kd, vd = A.to_device(q), A.to_device(k), A.to_device(v)
    out, obuf, margin = guarded(qd.shape, qd.dtype)
    lse = torch.full((q.shape[0], q.shape[1]), float("nan"), device=DEV) if with_lse else None
    A.dopd_prefill_attn(shape, qd, kd, vd, out, lse, A.to_device(cu), cu, len(cu) - 1,
                        stream=stream)
    torch.cuda.synchronize()
    assert canary_intact(obuf, margin, out.numel() * out.element_size()), "prefill wrote out of bounds"
    return widen(A.to_host(out)), (lse.cpu().numpy().astype(np.float64) if with_lse else None)


def gpu_prefill_paged(shape, q, k_pool, v_pool, page_table, cu, prefix, with_lse=True,
                      pools_dev=None, splits=None):
    """dopd_prefill_paged_attn, or with splits = n the split entry point with n
    (0: automatic) key splits and a NaN-filled workspace whose guard bytes
    are checked afterwards."""
    if pools_dev is None:
        pools_dev = (A.to_device(k_pool), A.to_device(v_pool))
    kp, vp = pools_dev
    qd = A.to_device(q)
    out, obuf, margin = guarded(qd.shape, qd.dtype)
    lse = torch.full((q.shape[0], q.shape[1]), float("nan"), device=DEV) if with_lse else None
    prefix = np.asarray(prefix, np.int32)
    args = (shape, qd, kp, vp, kp.shape[0], A.to_device(page_table), page_table.shape[1],
            A.to_device(cu), cu, A.to_device(prefix), prefix, len(cu) - 1)
    if splits is None:
        A.dopd_prefill_paged_attn(*args, out, lse)
    else:
        n = A.dopd_prefill_paged_workspace_size(shape, cu, prefix, len(cu) - 1, splits)
        assert n >= 256 and n % 256 == 0
        wbuf = torch.full((n + 4096 + 256,), 0xFF, dtype=torch.uint8, device=DEV)
        off = (-wbuf.data_ptr()) % 256
        ws = wbuf[off:off + n]
        A.dopd_prefill_paged_attn_split(*args, splits, out, lse, ws, n)
        torch.cuda.synchronize()
        assert bool((wbuf[off + n:] == 0xFF).all()), "paged prefill split wrote past its workspace"
    torch.cuda.synchronize()
    assert canary_intact(obuf, margin, out.numel() * out.element_size()), \
        "paged prefill wrote out of bounds"
    return widen(A.to_host(out)), (lse.cpu().numpy().astype(np.float64) if with_lse else None)


def gpu_kv_write(shape, k_new, v_new, k_pool, v_pool, page_table, cu_new, start_pos):
    kp, vp = A.to_device(k_pool), A.to_device(v_pool)
    A.dopd_kv_write(shape, A.to_device(k_new), A.to_device(v_new), kp, vp, k_pool.shape[0],
                    A.to_device(page_table), page_table.shape[1], A.to_device(cu_new),
                    A.to_device(start_pos), len(cu_new) - 1, int(cu_new[-1]))
    torch.cuda.synchronize()
    return A.to_host(kp), A.to_host(vp)


def gpu_decode(shape, q, k_pool, v_pool, page_table, ctx, split=0, with_lse=True, pools_dev=None,
               return_ws=False):
    if pools_dev is None:
        pools_dev = (A.to_device(k_pool), A.to_device(v_pool))
    kp, vp = pools_dev
    qd = A.to_device(q)
    out, obuf, margin = guarded(qd.shape, qd.dtype)
    lse = torch.full((q.shape[0], q.shape[1]), float("nan"), device=DEV) if with_lse else None
    ws = A.decode_workspace(shape, ctx, len(ctx), split)
    A.dopd_decode_attn(shape, qd, kp, vp, kp.shape[0], A.to_device(page_table),
                       page_table.shape[1], A.to_device(ctx), ctx, len(ctx), split, out, lse, ws)
    torch.cuda.synchronize()
    assert canary_intact(obuf, margin, out.numel() * out.element_size()), "decode wrote out of bounds"
    res = (widen(A.to_host(out)), lse.cpu().numpy().astype(np.float64) if with_lse else None)
    if return_ws:
        return res + (ws,)
    return res


def gpu_pack(shape, k_pool, v_pool, num_layers, page_table, req_ids, seq_lens, offsets):
    total = int(offsets[-1])
    dt = {np.dtype(np.uint16): torch.bfloat16, np.dtype(np.float32): torch.float32,
          np.dtype(np.uint8): torch.uint8}[k_pool.dtype]
    out, obuf, margin = guarded((total,), dt)
    kp, vp = A.to_device(k_pool), A.to_device(v_pool)
    num_pages = k_pool.shape[-4]
    A.dopd_kv_pack_for_handoff(shape, num_layers, kp, vp, num_pages, A.to_device(page_table),
                               page_table.shape[1], A.to_device(req_ids), A.to_device(seq_lens),
                               seq_lens, A.to_device(offsets), len(req_ids), out)
    torch.cuda.synchronize()
    assert canary_intact(obuf, margin, out.numel() * out.element_size()), "pack wrote out of bounds"
    return A.to_host(out)


# ------------------------------------------------------------------ E4M3 KV pages
def quantize_pools(k_pool, v_pool, k_scale, v_scale):
    """bf16 pools -> E4M3 code pools (uint8, same layouts), by the oracle's
    quantiser: the inputs of the fp8 decode tests."""
    import oracle
    p, hkv, _, d = k_pool.shape
    kq = oracle.e4m3_quantize(k_pool.transpose(0, 2, 1, 3).reshape(-1, hkv, d), k_scale)
    vq = oracle.e4m3_quantize(v_pool.transpose(0, 3, 1, 2).reshape(-1, hkv, d), v_scale)
    kq = kq.reshape(p, 16, hkv, d).transpose(0, 2, 1, 3).copy()
    vq = vq.reshape(p, 16, hkv, d).transpose(0, 2, 3, 1).copy()
    return kq, vq


def gpu_kv_write_fp8(shape, k_new, v_new, k_scale, v_scale, k_pool, v_pool, page_table, cu_new,
                     start_pos):
    kp, vp = A.to_device(k_pool), A.to_device(v_pool)
    A.dopd_kv_write_fp8(shape, A.to_device(k_new), A.to_device(v_new), A.to_device(k_scale),
                        A.to_device(v_scale), kp, vp, k_pool.shape[0], A.to_device(page_table),
                        page_table.shape[1], A.to_device(cu_new), A.to_device(start_pos),
                        len(cu_new) - 1, int(cu_new[-1]))
    torch.cuda.synchronize()
    return A.to_host(kp), A.to_host(vp)


def gpu_decode_fp8(shape, q, k_pool, v_pool, k_scale, v_scale, page_table, ctx, split=0,
                   with_lse=True, pools_dev=None):
    if pools_dev is None:
        pools_dev = (A.to_device(k_pool), A.to_device(v_pool))
    kp, vp = pools_dev
    qd = A.to_device(q)
    out, obuf, margin = guarded(qd.shape, qd.dtype)
    lse = torch.full((q.shape[0], q.shape[1]), float("nan"), device=DEV) if with_lse else None
    ws = A.decode_workspace(shape, ctx, len(ctx), split)
    A.dopd_decode_attn_fp8(shape, qd, kp, vp, A.to_device(np.asarray(k_scale, np.float32)),
                           A.to_device(np.asarray(v_scale, np.float32)), kp.shape[0],
                           A.to_device(page_table), page_table.shape[1], A.to_device(ctx), ctx,
                           len(ctx), split, out, lse, ws)
    torch.cuda.synchronize()
    assert canary_intact(obuf, margin, out.numel() * out.element_size()), \
        "fp8 decode wrote out of bounds"
    return widen(A.to_host(out)), (lse.cpu().numpy().astype(np.float64) if with_lse else None)


def gpu_prefill_paged_fp8(shape, q, k_pool, v_pool, k_scale, v_scale, page_table, cu, prefix,
                          splits=0, pools_dev=None):
    """dopd_prefill_paged_attn_fp8 with a 0xFF-filled workspace whose guard
    bytes are checked afterwards."""
    if pools_dev is None:
        pools_dev = (A.to_device(k_pool), A.to_device(v_pool))
    kp, vp = pools_dev
    qd = A.to_device(q)
    out, obuf, margin = guarded(qd.shape, qd.dtype)
    lse = torch.full((q.shape[0], q.shape[1]), float("nan"), device=DEV)
    prefix = np.asarray(prefix, np.int32)
    n = A.dopd_prefill_paged_fp8_workspace_size(shape, cu, prefix, len(cu) - 1, splits)
    assert n >= 256 and n % 256 == 0
    wbuf = torch.full((n + 4096 + 256,), 0xFF, dtype=torch.uint8, device=DEV)
    off = (-wbuf.data_ptr()) % 256
    ws = wbuf[off:off + n]
    A.dopd_prefill_paged_attn_fp8(shape, qd, kp, vp, A.to_device(np.asarray(k_scale, np.float32)),
                                  A.to_device(np.asarray(v_scale, np.float32)), kp.shape[0],
                                  A.to_device(page_table), page_table.shape[1], A.to_device(cu),
                                  cu, A.to_device(prefix), prefix, len(cu) - 1, splits, out, lse,
                                  ws, n)
    torch.cuda.synchronize()
    assert bool((wbuf[off + n:] == 0xFF).all()), "fp8 paged prefill wrote past its workspace"
    assert canary_intact(obuf, margin, out.numel() * out.element_size()), \
        "fp8 paged prefill wrote out of bounds"
    return widen(A.to_host(out)), lse.cpu().numpy().astype(np.float64)


def gpu_unpack(shape, buf, offs, req, lens, k_pool, v_pool, layers, pt):
    kp, vp = A.to_device(k_pool), A.to_device(v_pool)
    num_pages = k_pool.shape[-4]
    A.dopd_kv_unpack_from_handoff(shape, layers, A.to_device(buf), A.to_device(offs),
                                  A.to_device(req), A.to_device(lens), lens, len(req), kp, vp,
                                  num_pages, A.to_device(pt), pt.shape[1])
    torch.cuda.synchronize()
    return A.to_host(kp), A.to_host(vp)
