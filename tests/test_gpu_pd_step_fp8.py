"""GPU: the single-launch PD-aggregated step over E4M3 pools
(dopd_pd_step_fp8) against the fp64 oracle: the decode over the same codes
and scales, the bf16 prefill of the fresh prompts, the prompts' E4M3 codes in
the pools and in the handoff buffer bit-exact against the oracle's quantiser,
paged write and pack."""
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


def _scales(hkv, seed):
    rng = np.random.default_rng(seed)
    return (rng.uniform(4.0, 7.0, hkv) / 448).astype(np.float32), \
        (rng.uniform(4.0, 7.0, hkv) / 448).astype(np.float32)


def _case(seed, dec_ctx, pre_lens, hq, hkv, d):
    """E4M3 pools holding the decode requests' cache (quantised by the
    oracle; every other slot a NaN code), bf16 q_dec and fresh prompts."""
    rng = np.random.default_rng(seed)
    dec_ctx, pre_lens = np.asarray(dec_ctx, np.int32), np.asarray(pre_lens, np.int32)
    n_dec = len(dec_ctx)
    pt, num_pages = I.allocate_pages(rng, np.concatenate([dec_ctx, np.maximum(pre_lens, 1)]))
    kp, vp = I.empty_pools(num_pages, hkv, d, "bf16")
    if n_dec:
        I.fill_live_slots(rng, kp, vp, pt[:n_dec], dec_ctx, "bf16")
    ks, vs = _scales(hkv, seed)
    k8, v8 = G.quantize_pools(kp, vp, ks, vs)
    q_dec = I.normal(rng, (n_dec, hq, d), "bf16")
    q, k, v = I.prefill_batch(rng, pre_lens, hq, hkv, d, "bf16")
    return dict(dec_ctx=dec_ctx, pre_lens=pre_lens, pt=pt, num_pages=num_pages, k8=k8, v8=v8,
                ks=ks, vs=vs, q_dec=q_dec, q=q, k=k, v=v, cu=I.cu_from_lens(pre_lens))


def _run(c, hq, hkv, d, schedule, shift=0):
    n_dec, n_pre = len(c["dec_ctx"]), len(c["pre_lens"])
    sh = A.make_shape(hq, hkv, d, "fp8")
    stride = c["pt"].shape[1]
    kp, vp = A.to_device(c["k8"]), A.to_device(c["v8"])
    pt = A.to_device(c["pt"])
    q, k, v = A.to_device(c["q"]), A.to_device(c["k"]), A.to_device(c["v"])
    out_p = torch.empty_like(q)
    q_dec = A.to_device(c["q_dec"])
    out_d = torch.empty_like(q_dec)
    lse_d = torch.full((n_dec, hq), float("nan"), device="cuda")
    lse_p = torch.full((q.shape[0], hq), float("nan"), device="cuda")
    offs = I.handoff_offsets(c["pre_lens"], 1, hkv, d) + shift
    total = int(offs[-1])
    out_h, obuf, margin = G.guarded((total,), torch.uint8)
    ws = A.pd_step_workspace(sh, c["dec_ctx"], n_dec, schedule)
    A.dopd_pd_step_fp8(sh, q_dec, pt[:n_dec], A.to_device(c["dec_ctx"]), c["dec_ctx"], n_dec,
                       out_d, lse_d, q, k, v, A.to_device(c["cu"]), c["cu"], n_pre, pt[n_dec:],
                       out_p, lse_p, kp, vp, A.to_device(c["ks"]), A.to_device(c["vs"]),
                       c["num_pages"], stride, A.to_device(offs), out_h, schedule, ws)
    torch.cuda.synchronize()
    assert G.canary_intact(obuf, margin, total), "handoff codes written outside the buffer"
    return dict(out_d=out_d, out_p=out_p, lse_d=lse_d, lse_p=lse_p, kp=kp, vp=vp, out_h=out_h,
                offs=offs)


def _check(c, r, hq, hkv, d, shift=0):
    n_dec, n_pre = len(c["dec_ctx"]), len(c["pre_lens"])
    scale = 1.0 / np.sqrt(d)
    if n_dec:
        ref_d, ref_lse_d = oracle.decode_e4m3(c["q_dec"], c["k8"], c["v8"], c["ks"], c["vs"],
                                              c["pt"][:n_dec], c["dec_ctx"], scale)
        G.assert_attention_close(G.widen(A.to_host(r["out_d"])), ref_d, "bf16",
                                 "E4M3 pd step decode")
        assert np.max(np.abs(r["lse_d"].cpu().numpy() - ref_lse_d)) < 2e-2
    if n_pre:
        ref_p, ref_lse_p = oracle.prefill(c["q"], c["k"], c["v"], c["cu"], scale)
        G.assert_attention_close(G.widen(A.to_host(r["out_p"])), ref_p, "bf16",
                                 "E4M3 pd step prefill")
        assert np.max(np.abs(r["lse_p"].cpu().numpy() - ref_lse_p)) < 2e-2
    rk, rv = oracle.kv_write(oracle.e4m3_quantize(c["k"], c["ks"]),
                             oracle.e4m3_quantize(c["v"], c["vs"]), c["k8"], c["v8"],
                             c["pt"][n_dec:], c["cu"], np.zeros(n_pre, np.int32))
    assert np.array_equal(A.to_host(r["kp"]), rk) and np.array_equal(A.to_host(r["vp"]), rv)
    if n_pre:
        ref_h = oracle.pack(rk, rv, 1, c["pt"][n_dec:], np.arange(n_pre, dtype=np.int32),
                            c["pre_lens"], r["offs"])
        assert np.array_equal(A.to_host(r["out_h"])[shift:], ref_h[shift:])


@pytest.mark.parametrize("schedule", [A.DOPD_PD_AUTO, A.DOPD_PD_DECODE_FIRST])
def test_pd_step_fp8_mixed_step_shape(schedule):
    """The mixed step's shapes (192 decode requests with contexts
    lognormal(2048, 0.7), 8 x 512 prompts, 28/4 heads, d 128) over E4M3 pools."""
    w = I.mixed_step()
    n_dec = len(w.context_lens)
    c = _case(530, w.context_lens, w.prefill_lens, w.hq, w.hkv, w.d)
    r = _run(c, w.hq, w.hkv, w.d, schedule)
    _check(c, r, w.hq, w.hkv, w.d)
    assert n_dec == 192


@pytest.mark.parametrize("shift", [0, 3])
@pytest.mark.parametrize("hq,hkv,d", [(28, 4, 128), (8, 8, 64), (7, 1, 128)])
def test_pd_step_fp8_ragged(hq, hkv, d, shift):
    """Ragged contexts and prompts (an empty prompt among them); with shift 3
    the handoff blocks start at byte offsets that are not 8-byte aligned."""
    c = _case(531 + hq + d + shift, [1, 31, 33, 700, 2049, 5000, 16], [1, 0, 17, 128, 129, 300],
              hq, hkv, d)
    r = _run(c, hq, hkv, d, A.DOPD_PD_PREFILL_FIRST, shift)
    _check(c, r, hq, hkv, d, shift)


def test_pd_step_fp8_decode_equals_fp8_decode_entry():
    """With two decode slices per CU the step's decode is dopd_decode_attn_fp8's
    partition: bit-identical outputs."""
    c = _case(540, [3, 900, 4100, 64, 17], [50, 200], 16, 2, 128)
    r = _run(c, 16, 2, 128, A.DOPD_PD_PREFILL_FIRST)
    sh = A.make_shape(16, 2, 128, "fp8")
    dec, _ = G.gpu_decode_fp8(sh, c["q_dec"], c["k8"], c["v8"], c["ks"], c["vs"],
                              c["pt"][:5], c["dec_ctx"], with_lse=False)
    assert np.array_equal(G.widen(A.to_host(r["out_d"])), dec)
