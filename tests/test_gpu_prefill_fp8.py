"""GPU: chunk prefill over E4M3 pools (dopd_prefill_paged_attn_fp8) against
the oracle's chunk prefill over the same codes and scales: ragged chunks and
prefixes, GQA, both head sizes, key splits, a chunk of one token against the
fp8 decode, page-permutation invariance and calls with nothing to do."""
import numpy as np
import pytest

import oracle
from paper_2511_20982_amd import inputs as I

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu(require_gpu):
    pass


from tests import gpu_util as G  # noqa: E402

PREFIX = [0, 1, 15, 16, 17, 63, 64, 65, 200, 777, 0, 40, 129]
CHUNK = [9, 1, 16, 30, 64, 65, 128, 129, 1, 300, 0, 200, 77]


def _scales(hkv, seed):
    rng = np.random.default_rng(seed)
    return (rng.uniform(4.0, 7.0, hkv) / 448).astype(np.float32), \
        (rng.uniform(4.0, 7.0, hkv) / 448).astype(np.float32)


def fp8_case(seed, prefix, chunk, hq, hkv, d):
    """E4M3 pools holding prefix + chunk tokens of each request (NaN codes in
    every other slot), per-head scales, and the chunk rows of Q."""
    rng = np.random.default_rng(seed)
    prefix, chunk = np.asarray(prefix, np.int32), np.asarray(chunk, np.int32)
    total = prefix + chunk
    pt, num_pages = I.allocate_pages(rng, np.maximum(total, 1))
    kp, vp = I.empty_pools(num_pages, hkv, d, "bf16")
    _, kf, vf = I.prefill_batch(rng, total, hq, hkv, d, "bf16")
    kp, vp = oracle.kv_write(kf, vf, kp, vp, pt, I.cu_from_lens(total),
                             np.zeros(len(total), np.int32))
    ks, vs = _scales(hkv, seed)
    k8, v8 = G.quantize_pools(kp, vp, ks, vs)
    q = I.normal(rng, (int(chunk.sum()), hq, d), "bf16")
    return q, k8, v8, ks, vs, pt, I.cu_from_lens(chunk), prefix


@pytest.mark.parametrize("splits", [1, 0])
@pytest.mark.parametrize("hq,hkv", [(8, 8), (8, 2), (28, 4), (7, 1)])
@pytest.mark.parametrize("d", [128, 64])
def test_prefill_paged_fp8_matches_oracle(hq, hkv, d, splits):
    q, k8, v8, ks, vs, pt, cu, pre = fp8_case(90 + hq + d, PREFIX, CHUNK, hq, hkv, d)
    scale = 1.0 / np.sqrt(d)
    ref, ref_lse = oracle.prefill_paged_e4m3(q, k8, v8, ks, vs, pt, cu, pre, scale)
    sh = G.A.make_shape(hq, hkv, d, "fp8")
    out, lse = G.gpu_prefill_paged_fp8(sh, q, k8, v8, ks, vs, pt, cu, pre, splits=splits)
    G.assert_attention_close(out, ref, "bf16", f"fp8 chunk prefill hq={hq} hkv={hkv} d={d}")
    assert np.max(np.abs(lse - ref_lse)) < 2e-2


@pytest.mark.parametrize("splits", [4, 16])
@pytest.mark.parametrize("d", [128, 64])
def test_prefill_paged_fp8_key_splits(splits, d):
    # Long prefixes beside short ones, so that the split ranges are uneven.
    q, k8, v8, ks, vs, pt, cu, pre = fp8_case(95 + d, [3000, 40, 1500, 0], [200, 33, 64, 130],
                                              8, 2, d)
    ref, ref_lse = oracle.prefill_paged_e4m3(q, k8, v8, ks, vs, pt, cu, pre, 1 / np.sqrt(d))
    sh = G.A.make_shape(8, 2, d, "fp8")
    out, lse = G.gpu_prefill_paged_fp8(sh, q, k8, v8, ks, vs, pt, cu, pre, splits=splits)
    G.assert_attention_close(out, ref, "bf16", f"fp8 chunk prefill splits={splits}")
    assert np.max(np.abs(lse - ref_lse)) < 2e-2


def test_prefill_paged_fp8_many_requests():
    # More than 64 requests: the heaviest-q-tile-first work order.
    rng = np.random.default_rng(96)
    prefix = rng.integers(0, 300, 70).astype(np.int32)
    chunk = rng.integers(0, 90, 70).astype(np.int32)
    q, k8, v8, ks, vs, pt, cu, pre = fp8_case(96, prefix, chunk, 8, 2, 128)
    ref, ref_lse = oracle.prefill_paged_e4m3(q, k8, v8, ks, vs, pt, cu, pre, 1 / np.sqrt(128))
    sh = G.A.make_shape(8, 2, 128, "fp8")
    for splits in (1, 0):
        out, lse = G.gpu_prefill_paged_fp8(sh, q, k8, v8, ks, vs, pt, cu, pre, splits=splits)
        G.assert_attention_close(out, ref, "bf16", f"fp8 chunk prefill, 70 requests, splits={splits}")
        assert np.max(np.abs(lse - ref_lse)) < 2e-2


def test_prefill_paged_fp8_chunk_of_one_matches_fp8_decode():
    q, k8, v8, ks, vs, pt, cu, pre = fp8_case(97, [30, 0, 17, 2047], [1, 1, 1, 1], 28, 4, 128)
    sh = G.A.make_shape(28, 4, 128, "fp8")
    out, lse = G.gpu_prefill_paged_fp8(sh, q, k8, v8, ks, vs, pt, cu, pre)
    ctx = (pre + 1).astype(np.int32)
    dec, _ = G.gpu_decode_fp8(sh, q, k8, v8, ks, vs, pt, ctx)
    ref, ref_lse = oracle.decode_e4m3(q, k8, v8, ks, vs, pt, ctx, 1 / np.sqrt(128))
    G.assert_attention_close(out, ref, "bf16", "fp8 chunk of one vs oracle decode")
    G.assert_attention_close(out, dec, "bf16", "fp8 chunk of one vs GPU fp8 decode")
    assert np.max(np.abs(lse - ref_lse)) < 2e-2


def test_prefill_paged_fp8_page_permutation_and_scale_variants():
    q, k8, v8, ks, vs, pt, cu, pre = fp8_case(98, [500, 3, 0, 64], [70, 200, 33, 1], 16, 4, 128)
    sh = G.A.make_shape(16, 4, 128, "fp8")
    out1, lse1 = G.gpu_prefill_paged_fp8(sh, q, k8, v8, ks, vs, pt, cu, pre)
    num_pages = k8.shape[0]
    perm = np.random.default_rng(9).permutation(num_pages)
    k2, v2 = np.empty_like(k8), np.empty_like(v8)
    k2[perm], v2[perm] = k8, v8
    pt2 = np.where(pt >= 0, perm[np.maximum(pt, 0)], -1).astype(np.int32)
    out2, lse2 = G.gpu_prefill_paged_fp8(sh, q, k2, v2, ks, vs, pt2, cu, pre)
    assert np.array_equal(out1, out2) and np.array_equal(lse1, lse2)
    for scale in (0.0, 1.0):
        ref, _ = oracle.prefill_paged_e4m3(q, k8, v8, ks, vs, pt, cu, pre, scale)
        out, _ = G.gpu_prefill_paged_fp8(G.A.make_shape(16, 4, 128, "fp8", scale), q, k8, v8,
                                         ks, vs, pt, cu, pre)
        G.assert_attention_close(out, ref, "bf16", f"fp8 chunk prefill scale={scale}")


def test_prefill_paged_fp8_nothing_to_do():
    # Every chunk empty: no kernel runs, the output is untouched, and no
    # workspace is needed; zero requests likewise.
    import torch
    A = G.A
    sh = A.make_shape(8, 2, 64, "fp8")
    kp = torch.zeros((4, 2, 16, 64), dtype=torch.uint8, device=G.DEV)
    vp = torch.zeros((4, 2, 64, 16), dtype=torch.uint8, device=G.DEV)
    sc = torch.ones(2, dtype=torch.float32, device=G.DEV)
    pt = np.array([[0, 1], [2, 3]], np.int32)
    cu = np.zeros(3, np.int32)
    pre = np.array([20, 5], np.int32)
    out = torch.full((1, 8, 64), 7.0, dtype=torch.bfloat16, device=G.DEV)
    assert A.dopd_prefill_paged_fp8_workspace_size(sh, cu, pre, 2, 0) == 256
    A.dopd_prefill_paged_attn_fp8(sh, out, kp, vp, sc, sc, 4, A.to_device(pt), 2,
                                  A.to_device(cu), cu, A.to_device(pre), pre, 2, 0, out, None,
                                  None, 0)
    A.dopd_prefill_paged_attn_fp8(sh, out, kp, vp, sc, sc, 4, A.to_device(pt), 2,
                                  A.to_device(cu), cu, A.to_device(pre), pre, 0, 0, out, None,
                                  None, 0)
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())
