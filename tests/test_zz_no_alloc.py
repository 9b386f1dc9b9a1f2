"""dopd_decode_attn_noalloc: the decode with its split-K partials in the
library's static device scratch, against dopd_decode_attn with a caller
workspace (same kernels: bit-identical) and the fp64 oracle, on two calls in
a row, the second with a smaller batch; and the host-side rejection of a call
whose partials exceed the scratch."""
import ctypes as C

import numpy as np
import pytest

import oracle
from paper_2511_20982_amd import attn as A
from paper_2511_20982_amd import inputs as I


def _case(seed, ctx, hq, hkv, d=128):
    rng = np.random.default_rng(seed)
    ctx = np.asarray(ctx, np.int32)
    w = I.decode_workload("noalloc", seed, ctx, hq, hkv, d)
    return w


def test_noalloc_rejects_partials_beyond_the_scratch():
    # 2000 requests x 8 KV heads x 16 query heads each: more than 32 MiB of partials
    sh = A.make_shape(128, 8, 128)
    ctx = np.full(2000, 4000, np.int32)
    need = A.dopd_decode_workspace_size(sh, ctx, len(ctx))
    assert need > A.DECODE_NOALLOC_SCRATCH_BYTES
    fake = C.c_void_p(0x1000)
    st = A.lib().dopd_decode_attn_noalloc(C.byref(sh), fake, fake, fake, 10, fake, 1024, fake,
                                          A._hptr(ctx), len(ctx), 0, fake, None, None)
    assert st == A.DOPD_ERR_WORKSPACE_TOO_SMALL


@pytest.mark.gpu
def test_noalloc_matches_workspace_entry_two_calls(require_gpu):
    import torch
    from tests import gpu_util as G

    cases = [
        # first: a large GQA batch with long contexts (several slices per request)
        _case(401, np.concatenate([np.full(40, 9000), np.arange(1, 200) * 7]), 64, 8),
        # then: a smaller batch, fewer heads, shorter contexts
        _case(402, [1, 33, 700, 2049, 5000], 28, 4),
    ]
    for i, w in enumerate(cases):
        sh = G.shape_of(w)
        kp, vp = A.to_device(w.k_pool), A.to_device(w.v_pool)
        pt = A.to_device(w.page_table)
        ctx_d = A.to_device(w.context_lens)
        qd = A.to_device(w.q_dec)
        n = len(w.context_lens)
        assert A.dopd_decode_workspace_size(sh, w.context_lens, n) <= A.DECODE_NOALLOC_SCRATCH_BYTES
        out_na, obuf, margin = G.guarded(qd.shape, qd.dtype)
        lse_na = torch.full((n, w.hq), float("nan"), device="cuda")
        A.dopd_decode_attn_noalloc(sh, qd, kp, vp, w.num_pages, pt, w.page_table.shape[1], ctx_d,
                                   w.context_lens, n, 0, out_na, lse_na)
        torch.cuda.synchronize()
        assert G.canary_intact(obuf, margin, out_na.numel() * out_na.element_size())
        out_ws, lse_ws = G.gpu_decode(sh, w.q_dec, None, None, w.page_table, w.context_lens,
                                      pools_dev=(kp, vp))
        got = G.widen(A.to_host(out_na))
        assert np.array_equal(got, out_ws), f"call {i}: differs from the workspace entry point"
        assert np.array_equal(lse_na.cpu().numpy().astype(np.float64), lse_ws)
        ref, ref_lse = oracle.decode(w.q_dec, w.k_pool, w.v_pool, w.page_table, w.context_lens,
                                     w.scale)
        G.assert_attention_close(got, ref, "bf16", f"noalloc decode call {i}")
        assert np.max(np.abs(lse_ws - ref_lse)) < 2e-2
