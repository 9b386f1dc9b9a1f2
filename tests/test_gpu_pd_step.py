"""GPU: the paged write that also emits the handoff buffer, and the single-
launch PD-aggregated step (decode + prefill + write + pack), against the
fp64 oracle and against the separate entry points."""
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

SCHEDULES = [A.DOPD_PD_AUTO, A.DOPD_PD_PREFILL_FIRST, A.DOPD_PD_DECODE_FIRST,
             A.DOPD_PD_DECODE_FIRST_WIDE]


def _handoff_ref(k, v, kp, vp, pt, cu, lens, offs, hkv, d):
    """Pools after the oracle's write at start 0, and the oracle's pack of
    those requests from them (one layer)."""
    n = len(lens)
    rk, rv = oracle.kv_write(k, v, kp, vp, pt, cu, np.zeros(n, np.int32))
    ref_h = oracle.pack(rk, rv, 1, pt, np.arange(n, dtype=np.int32), lens, offs)
    return rk, rv, ref_h


@pytest.mark.parametrize("shift", [0, 3])
@pytest.mark.parametrize("d", [128, 64])
def test_write_pack_matches_write_then_pack(d, shift):
    """Bit-exact against oracle.kv_write followed by oracle.pack; with shift 3
    the request blocks start at element offsets that are not 16-byte aligned."""
    rng = np.random.default_rng(500 + d + shift)
    lens = np.array([1, 15, 16, 17, 300, 0, 129, 512], np.int32)
    hq, hkv = 8, 2
    _, k, v = I.prefill_batch(rng, lens, hq, hkv, d, "bf16")
    pt, num_pages = I.allocate_pages(rng, np.maximum(lens, 1))
    kp, vp = I.empty_pools(num_pages, hkv, d, "bf16")
    cu = I.cu_from_lens(lens)
    offs = I.handoff_offsets(lens, 1, hkv, d) + shift
    rk, rv, ref_h = _handoff_ref(k, v, kp, vp, pt, cu, lens, offs, hkv, d)
    sh = A.make_shape(hq, hkv, d)
    kpd, vpd = A.to_device(kp), A.to_device(vp)
    total = int(offs[-1])
    out, obuf, margin = G.guarded((total,), torch.bfloat16)
    A.dopd_kv_write_pack_for_handoff(sh, A.to_device(k), A.to_device(v), kpd, vpd, num_pages,
                                     A.to_device(pt), pt.shape[1], A.to_device(cu), cu,
                                     len(lens), A.to_device(offs), out)
    torch.cuda.synchronize()
    assert G.canary_intact(obuf, margin, total * 2), "write+pack wrote outside the buffer"
    assert np.array_equal(A.to_host(kpd), rk) and np.array_equal(A.to_host(vpd), rv)
    got = A.to_host(out)
    assert np.array_equal(got[shift:], ref_h[shift:])
    # without a handoff buffer it is the plain paged write
    kpd2, vpd2 = A.to_device(kp), A.to_device(vp)
    A.dopd_kv_write_pack_for_handoff(sh, A.to_device(k), A.to_device(v), kpd2, vpd2, num_pages,
                                     A.to_device(pt), pt.shape[1], A.to_device(cu), cu,
                                     len(lens), None, None)
    torch.cuda.synchronize()
    assert np.array_equal(A.to_host(kpd2), rk) and np.array_equal(A.to_host(vpd2), rv)


def _run_pd_step(w, sh, schedule, with_lse=True, handoff=True):
    n_pre, n_dec = len(w.prefill_lens), len(w.context_lens)
    stride = w.page_table.shape[1]
    kp, vp = A.to_device(w.k_pool), A.to_device(w.v_pool)
    pt = A.to_device(w.page_table)
    dec_pt, pre_pt = pt[:n_dec], pt[n_dec:]
    q, k, v = A.to_device(w.q), A.to_device(w.k), A.to_device(w.v)
    out_p = torch.empty_like(q)
    q_dec = A.to_device(w.q_dec)
    out_d = torch.empty_like(q_dec)
    lse_d = torch.full((n_dec, w.hq), float("nan"), device="cuda") if with_lse else None
    lse_p = torch.full((q.shape[0], w.hq), float("nan"), device="cuda") if with_lse else None
    offs = I.handoff_offsets(w.prefill_lens, 1, w.hkv, w.d)
    out_h = torch.zeros(int(offs[-1]), dtype=torch.bfloat16, device="cuda") if handoff else None
    ws = A.pd_step_workspace(sh, w.context_lens, n_dec, schedule)
    A.dopd_pd_step(sh, q_dec, dec_pt, A.to_device(w.context_lens), w.context_lens, n_dec, out_d,
                   lse_d, q, k, v, A.to_device(w.cu_seqlens), w.cu_seqlens, n_pre, pre_pt, out_p,
                   lse_p, kp, vp, w.num_pages, stride, A.to_device(offs) if handoff else None,
                   out_h, schedule, ws)
    torch.cuda.synchronize()
    return dict(out_d=out_d, out_p=out_p, lse_d=lse_d, lse_p=lse_p, kp=kp, vp=vp, out_h=out_h,
                offs=offs)


@pytest.mark.parametrize("schedule", SCHEDULES)
def test_pd_step_mixed_step_full_size(schedule):
    """The mixed step (192 decode requests, 8 x 512 prompts, 28/4 heads, d 128)
    in one launch: every decode and prefill output against the oracle, the
    paged write and the handoff buffer bit-exact, and the prefill bit-identical
    to dopd_prefill_attn (same kernel body and work order)."""
    w = I.mixed_step()
    sh = G.shape_of(w)
    n_pre, n_dec = len(w.prefill_lens), len(w.context_lens)
    r = _run_pd_step(w, sh, schedule)
    ref_d, ref_lse_d = oracle.decode(w.q_dec, w.k_pool, w.v_pool, w.page_table[:n_dec],
                                     w.context_lens, w.scale)
    G.assert_attention_close(G.widen(A.to_host(r["out_d"])), ref_d, "bf16", "pd step decode")
    assert np.max(np.abs(r["lse_d"].cpu().numpy() - ref_lse_d)) < 2e-2
    ref_p, ref_lse_p = oracle.prefill(w.q, w.k, w.v, w.cu_seqlens, w.scale)
    got_p = G.widen(A.to_host(r["out_p"]))
    G.assert_attention_close(got_p, ref_p, "bf16", "pd step prefill")
    assert np.max(np.abs(r["lse_p"].cpu().numpy() - ref_lse_p)) < 2e-2
    one, _ = G.gpu_prefill(sh, w.q, w.k, w.v, w.cu_seqlens, with_lse=False)
    assert np.array_equal(got_p, one)
    rk, rv, ref_h = _handoff_ref(w.k, w.v, w.k_pool, w.v_pool, w.page_table[n_dec:],
                                 w.cu_seqlens, w.prefill_lens, r["offs"], w.hkv, w.d)
    assert np.array_equal(A.to_host(r["kp"]), rk) and np.array_equal(A.to_host(r["vp"]), rv)
    assert np.array_equal(A.to_host(r["out_h"]), ref_h)


def test_pd_step_prefill_first_decode_equals_decode_entry():
    """With two decode slices per CU the step's decode partition is the one
    dopd_decode_attn uses: bit-identical outputs."""
    w = I.mixed_step()
    sh = G.shape_of(w)
    n_dec = len(w.context_lens)
    r = _run_pd_step(w, sh, A.DOPD_PD_PREFILL_FIRST, with_lse=False, handoff=False)
    dec, _ = G.gpu_decode(sh, w.q_dec, w.k_pool, w.v_pool, w.page_table[:n_dec], w.context_lens,
                          with_lse=False)
    assert np.array_equal(G.widen(A.to_host(r["out_d"])), dec)


def _small_case(seed, dec_ctx, pre_lens, hq, hkv, d):
    rng = np.random.default_rng(seed)
    dec_ctx, pre_lens = np.asarray(dec_ctx, np.int32), np.asarray(pre_lens, np.int32)
    n_dec = len(dec_ctx)
    caps = np.concatenate([dec_ctx, np.maximum(pre_lens, 1)])
    pt, num_pages = I.allocate_pages(rng, caps)
    kp, vp = I.empty_pools(num_pages, hkv, d, "bf16")
    if n_dec:
        I.fill_live_slots(rng, kp, vp, pt[:n_dec], dec_ctx, "bf16")
    q_dec = I.normal(rng, (n_dec, hq, d), "bf16")
    q, k, v = I.prefill_batch(rng, pre_lens, hq, hkv, d, "bf16")

    class W:
        pass
    w = W()
    w.hq, w.hkv, w.d, w.scale = hq, hkv, d, 1.0 / np.sqrt(d)
    w.context_lens, w.prefill_lens, w.cu_seqlens = dec_ctx, pre_lens, I.cu_from_lens(pre_lens)
    w.page_table, w.num_pages, w.k_pool, w.v_pool = pt, num_pages, kp, vp
    w.q_dec, w.q, w.k, w.v = q_dec, q, k, v
    return w


@pytest.mark.parametrize("schedule", SCHEDULES[1:])
@pytest.mark.parametrize("hq,hkv,d", [(28, 4, 128), (8, 8, 64), (7, 1, 128)])
def test_pd_step_ragged(hq, hkv, d, schedule):
    """Ragged decode contexts and prompt lengths (empty prompts included)."""
    w = _small_case(510 + hq + d, [1, 31, 33, 700, 2049, 5000, 16], [1, 0, 17, 128, 129, 300],
                    hq, hkv, d)
    sh = A.make_shape(hq, hkv, d)
    n_dec = len(w.context_lens)
    r = _run_pd_step(w, sh, schedule)
    ref_d, ref_lse_d = oracle.decode(w.q_dec, w.k_pool, w.v_pool, w.page_table[:n_dec],
                                     w.context_lens, w.scale)
    G.assert_attention_close(G.widen(A.to_host(r["out_d"])), ref_d, "bf16", "ragged pd decode")
    assert np.max(np.abs(r["lse_d"].cpu().numpy() - ref_lse_d)) < 2e-2
    ref_p, ref_lse_p = oracle.prefill(w.q, w.k, w.v, w.cu_seqlens, w.scale)
    G.assert_attention_close(G.widen(A.to_host(r["out_p"])), ref_p, "bf16", "ragged pd prefill")
    assert np.max(np.abs(r["lse_p"].cpu().numpy() - ref_lse_p)) < 2e-2
    rk, rv, ref_h = _handoff_ref(w.k, w.v, w.k_pool, w.v_pool, w.page_table[n_dec:],
                                 w.cu_seqlens, w.prefill_lens, r["offs"], hkv, d)
    assert np.array_equal(A.to_host(r["kp"]), rk) and np.array_equal(A.to_host(r["vp"]), rv)
    assert np.array_equal(A.to_host(r["out_h"]), ref_h)


@pytest.mark.parametrize("which", ["no_decode", "no_prefill"])
def test_pd_step_one_batch_empty(which):
    dec = [] if which == "no_decode" else [5, 900, 3000]
    pre = [] if which == "no_prefill" else [64, 200]
    w = _small_case(520, dec, pre, 28, 4, 128)
    sh = A.make_shape(28, 4, 128)
    r = _run_pd_step(w, sh, A.DOPD_PD_AUTO, handoff=bool(pre))
    if dec:
        ref_d, _ = oracle.decode(w.q_dec, w.k_pool, w.v_pool, w.page_table[:len(dec)],
                                 w.context_lens, w.scale)
        G.assert_attention_close(G.widen(A.to_host(r["out_d"])), ref_d, "bf16", "decode only")
        assert np.array_equal(A.to_host(r["kp"]), w.k_pool)  # nothing written
    if pre:
        ref_p, _ = oracle.prefill(w.q, w.k, w.v, w.cu_seqlens, w.scale)
        G.assert_attention_close(G.widen(A.to_host(r["out_p"])), ref_p, "bf16", "prefill only")


def test_pd_step_repeat_runs_bit_identical():
    w = I.mixed_step()
    sh = G.shape_of(w)
    for schedule in SCHEDULES[1:]:
        a = _run_pd_step(w, sh, schedule)
        b = _run_pd_step(w, sh, schedule)
        for key in ("out_d", "out_p", "lse_d", "lse_p", "kp", "vp", "out_h"):
            # bitwise (the pools hold NaN poison in dead slots)
            x, y = A.to_host(a[key]), A.to_host(b[key])
            assert np.array_equal(x.view(np.uint8), y.view(np.uint8)), (schedule, key)
