"""GPU: the five seeded workloads at full size, in the launch configuration the
benchmark times, against the fp64 oracle on every output."""
import numpy as np
import pytest
import torch

import oracle
from paper_2511_20982_amd import attn as A
from paper_2511_20982_amd import inputs as I

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu(require_gpu):
    pass


from tests import gpu_util as G  # noqa: E402


def test_tiny_fp32_prefill_then_eight_decode_steps():
    w = I.tiny_fp32()
    sh = G.shape_of(w)
    n = len(w.prefill_lens)
    # prefill on the GPU vs the oracle
    ref_p, ref_lse = oracle.prefill(w.q, w.k, w.v, w.cu_seqlens, w.scale)
    out_p, lse_p = G.gpu_prefill(sh, w.q, w.k, w.v, w.cu_seqlens)
    G.assert_attention_close(out_p, ref_p, "fp32", "tiny fp32 prefill")
    assert np.max(np.abs(lse_p - ref_lse)) < 1e-5
    # the paged cache lives on the GPU for the whole sequence
    kp, vp = A.to_device(w.k_pool), A.to_device(w.v_pool)
    pt = A.to_device(w.page_table)
    A.dopd_kv_write(sh, A.to_device(w.k), A.to_device(w.v), kp, vp, w.num_pages, pt,
                    w.page_table.shape[1], A.to_device(w.cu_seqlens),
                    torch.zeros(n, dtype=torch.int32, device="cuda"), n, int(w.cu_seqlens[-1]))
    ref_kp, ref_vp = oracle.kv_write(w.k, w.v, w.k_pool, w.v_pool, w.page_table, w.cu_seqlens,
                                     np.zeros(n, np.int32))
    ones = I.cu_from_lens(np.ones(n, np.int32))
    for s, (qd, kd, vd) in enumerate(w.steps):
        start = (w.prefill_lens + s).astype(np.int32)
        A.dopd_kv_write(sh, A.to_device(kd), A.to_device(vd), kp, vp, w.num_pages, pt,
                        w.page_table.shape[1], A.to_device(ones), A.to_device(start), n, n)
        ref_kp, ref_vp = oracle.kv_write(kd, vd, ref_kp, ref_vp, w.page_table, ones, start)
        ctx = (w.prefill_lens + s + 1).astype(np.int32)
        out_d, lse_d = G.gpu_decode(sh, qd, None, None, w.page_table, ctx, pools_dev=(kp, vp))
        ref_d, ref_lse_d = oracle.decode(qd, ref_kp, ref_vp, w.page_table, ctx, w.scale)
        G.assert_attention_close(out_d, ref_d, "fp32", f"tiny fp32 decode step {s}")
        assert np.max(np.abs(lse_d - ref_lse_d)) < 1e-5
    torch.cuda.synchronize()
    assert np.array_equal(A.to_host(kp).view(np.uint32), ref_kp.view(np.uint32))
    assert np.array_equal(A.to_host(vp).view(np.uint32), ref_vp.view(np.uint32))


@pytest.mark.parametrize("make", [I.decode_mha_7b, I.decode_gqa_70b], ids=["mha_7b", "gqa_70b"])
def test_full_size_decode(make):
    w = make()
    ref, ref_lse = oracle.decode(w.q_dec, w.k_pool, w.v_pool, w.page_table, w.context_lens, w.scale)
    out, lse = G.gpu_decode(G.shape_of(w), w.q_dec, w.k_pool, w.v_pool, w.page_table, w.context_lens)
    G.assert_attention_close(out, ref, "bf16", f"{w.name} decode")
    assert np.max(np.abs(lse - ref_lse)) < 2e-2


def test_full_size_varlen_prefill_and_write():
    """Every (row, head) output and lse of the varlen prefill batch (16 prompts,
    32 heads, d 128) against the oracle, and the paged write of the whole batch
    bit-exact."""
    w = I.varlen_prefill()
    sh = G.shape_of(w)
    out, lse = G.gpu_prefill(sh, w.q, w.k, w.v, w.cu_seqlens)
    ref, ref_lse = oracle.prefill(w.q, w.k, w.v, w.cu_seqlens, w.scale)
    G.assert_attention_close(out, ref, "bf16", "varlen prefill, all rows")
    assert np.max(np.abs(lse - ref_lse)) < 2e-2
    del out, ref
    # paged write of the whole batch, bit-exact
    n = len(w.prefill_lens)
    gk, gv = G.gpu_kv_write(sh, w.k, w.v, w.k_pool, w.v_pool, w.page_table, w.cu_seqlens,
                            np.zeros(n, np.int32))
    ref_k, ref_v = oracle.kv_write(w.k, w.v, w.k_pool, w.v_pool, w.page_table, w.cu_seqlens,
                                   np.zeros(n, np.int32))
    assert np.array_equal(gk, ref_k) and np.array_equal(gv, ref_v)


def test_full_size_mixed_step_one_stream_decode_first():
    """The mixed step exactly as the benchmark times it: one stream, the decode
    batch first, then prefill, paged write and pack.  Every decode and prefill
    output against the oracle (absolute and per-(row, head) normalised
    error), the write and the pack bit-exact."""
    w = I.mixed_step()
    sh = G.shape_of(w)
    s = torch.cuda.current_stream()
    kp, vp = A.to_device(w.k_pool), A.to_device(w.v_pool)
    pt = A.to_device(w.page_table)
    stride = w.page_table.shape[1]
    q, k, v = A.to_device(w.q), A.to_device(w.k), A.to_device(w.v)
    cu = A.to_device(w.cu_seqlens)
    out_p = torch.empty_like(q)
    n_pre, n_dec = len(w.prefill_lens), len(w.context_lens)
    q_dec = A.to_device(w.q_dec)
    out_d = torch.empty_like(q_dec)
    ws = A.decode_workspace(sh, w.context_lens, n_dec)
    offs = I.handoff_offsets(w.handoff_lens, 1, w.hkv, w.d)
    out_h = torch.empty(int(offs[-1]), dtype=torch.bfloat16, device="cuda")
    ctx_d, start_d = A.to_device(w.context_lens), torch.zeros(n_pre, dtype=torch.int32, device="cuda")
    hreq, hlen, offs_d = A.to_device(w.handoff_reqs), A.to_device(w.handoff_lens), A.to_device(offs)
    torch.cuda.synchronize()
    A.dopd_decode_attn(sh, q_dec, kp, vp, w.num_pages, pt, stride, ctx_d, w.context_lens, n_dec,
                       0, out_d, None, ws, stream=s)
    A.dopd_prefill_attn(sh, q, k, v, out_p, None, cu, w.cu_seqlens, n_pre, stream=s)
    A.dopd_kv_write(sh, k, v, kp, vp, w.num_pages, pt[n_dec:], stride, cu, start_d, n_pre,
                    int(w.cu_seqlens[-1]), s)
    A.dopd_kv_pack_for_handoff(sh, 1, kp, vp, w.num_pages, pt, stride, hreq, hlen,
                               w.handoff_lens, offs_d, n_pre, out_h, s)
    torch.cuda.synchronize()
    ref_d, _ = oracle.decode(w.q_dec, w.k_pool, w.v_pool, w.page_table, w.context_lens, w.scale)
    G.assert_attention_close(G.widen(A.to_host(out_d)), ref_d, "bf16", "mixed step decode (timed order)")
    ref_p, _ = oracle.prefill(w.q, w.k, w.v, w.cu_seqlens, w.scale)
    G.assert_attention_close(G.widen(A.to_host(out_p)), ref_p, "bf16", "mixed step prefill (timed order)")
    ref_kp, ref_vp = oracle.kv_write(w.k, w.v, w.k_pool, w.v_pool, w.page_table[n_dec:],
                                     w.cu_seqlens, np.zeros(n_pre, np.int32))
    assert np.array_equal(A.to_host(kp), ref_kp) and np.array_equal(A.to_host(vp), ref_vp)
    ref_h = oracle.pack(ref_kp, ref_vp, 1, w.page_table, w.handoff_reqs, w.handoff_lens, offs)
    assert np.array_equal(A.to_host(out_h), ref_h)


def test_full_size_mixed_step_two_streams():
    """The mixed step's two-stream form (the benchmark's --streams 2): prefill,
    write and pack on one stream, the decode on another, against the oracle."""
    w = I.mixed_step()
    sh = G.shape_of(w)
    sA = torch.cuda.current_stream()
    sB = torch.cuda.Stream()
    kp, vp = A.to_device(w.k_pool), A.to_device(w.v_pool)
    pt = A.to_device(w.page_table)
    q, k, v = A.to_device(w.q), A.to_device(w.k), A.to_device(w.v)
    cu = A.to_device(w.cu_seqlens)
    out_p = torch.empty_like(q)
    n_pre, n_dec = len(w.prefill_lens), len(w.context_lens)
    q_dec = A.to_device(w.q_dec)
    out_d = torch.empty_like(q_dec)
    ws = A.decode_workspace(sh, w.context_lens, n_dec)
    offs = I.handoff_offsets(w.handoff_lens, 1, w.hkv, w.d)
    out_h = torch.empty(int(offs[-1]), dtype=torch.bfloat16, device="cuda")
    # every device input exists before the streams fork (copies run on stream A)
    ctx_d, start_d = A.to_device(w.context_lens), torch.zeros(n_pre, dtype=torch.int32, device="cuda")
    hreq, hlen, offs_d = A.to_device(w.handoff_reqs), A.to_device(w.handoff_lens), A.to_device(offs)
    torch.cuda.synchronize()
    sB.wait_stream(sA)
    A.dopd_prefill_attn(sh, q, k, v, out_p, None, cu, w.cu_seqlens, n_pre, stream=sA)
    A.dopd_decode_attn(sh, q_dec, kp, vp, w.num_pages, pt, w.page_table.shape[1], ctx_d,
                       w.context_lens, n_dec, 0, out_d, None, ws, stream=sB)
    A.dopd_kv_write(sh, k, v, kp, vp, w.num_pages, pt[n_dec:], w.page_table.shape[1], cu,
                    start_d, n_pre, int(w.cu_seqlens[-1]), sA)
    A.dopd_kv_pack_for_handoff(sh, 1, kp, vp, w.num_pages, pt, w.page_table.shape[1], hreq,
                               hlen, w.handoff_lens, offs_d, n_pre, out_h, sA)
    torch.cuda.synchronize()
    ref_d, _ = oracle.decode(w.q_dec, w.k_pool, w.v_pool, w.page_table, w.context_lens, w.scale)
    G.assert_attention_close(G.widen(A.to_host(out_d)), ref_d, "bf16", "mixed step decode")
    ref_p, _ = oracle.prefill(w.q, w.k, w.v, w.cu_seqlens, w.scale)
    G.assert_attention_close(G.widen(A.to_host(out_p)), ref_p, "bf16", "mixed step prefill")
    ref_kp, ref_vp = oracle.kv_write(w.k, w.v, w.k_pool, w.v_pool, w.page_table[n_dec:],
                                     w.cu_seqlens, np.zeros(n_pre, np.int32))
    ref_h = oracle.pack(ref_kp, ref_vp, 1, w.page_table, w.handoff_reqs, w.handoff_lens, offs)
    assert np.array_equal(A.to_host(out_h), ref_h)
    assert np.array_equal(A.to_host(kp), ref_kp) and np.array_equal(A.to_host(vp), ref_vp)


def test_pack_28_layers_mixed_step_shape():
    """The supplementary 28-layer handoff of the mixed step, bit-exact."""
    rng = np.random.default_rng(5)
    layers, hkv, d = 28, 4, 128
    lens = np.full(8, 512, np.int32)
    pt, num_pages = I.allocate_pages(rng, lens)
    kp = I.normal(rng, (layers, num_pages, hkv, 16, d), "bf16")
    vp = I.normal(rng, (layers, num_pages, hkv, d, 16), "bf16")
    offs = I.handoff_offsets(lens, layers, hkv, d)
    req = np.arange(8, dtype=np.int32)
    out = G.gpu_pack(A.make_shape(28, hkv, d), kp, vp, layers, pt, req, lens, offs)
    ref = oracle.pack(kp, vp, layers, pt, req, lens, offs)
    assert np.array_equal(out, ref)
