"""GPU: chunk prefill over the paged cache (prefix-aware, chunk aligned to the
end of the cache) against the fp64 oracle, chunked == one-shot, a chunk of
one token == a decode step, and page-permutation invariance."""
import numpy as np
import pytest

import oracle
from paper_2511_20982_amd import inputs as I

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu(require_gpu):
    pass


from tests import gpu_util as G  # noqa: E402


def paged_case(seed, prefix, chunk, hq, hkv, d, dtype):
    """Pools holding prefix + chunk tokens of each request (NaN elsewhere,
    tail slots included), and the chunk rows of Q."""
    rng = np.random.default_rng(seed)
    prefix, chunk = np.asarray(prefix, np.int32), np.asarray(chunk, np.int32)
    total = prefix + chunk
    pt, num_pages = I.allocate_pages(rng, np.maximum(total, 1))
    kp, vp = I.empty_pools(num_pages, hkv, d, dtype)
    _, kf, vf = I.prefill_batch(rng, total, hq, hkv, d, dtype)
    kp, vp = oracle.kv_write(kf, vf, kp, vp, pt, I.cu_from_lens(total),
                             np.zeros(len(total), np.int32))
    q = I.normal(rng, (int(chunk.sum()), hq, d), dtype)
    return q, kp, vp, pt, I.cu_from_lens(chunk), prefix


PREFIX = [0, 1, 15, 16, 17, 63, 64, 65, 200, 777, 0, 40, 129]
CHUNK = [9, 1, 16, 30, 64, 65, 128, 129, 1, 300, 0, 200, 77]


@pytest.mark.parametrize("hq,hkv", [(8, 8), (8, 2), (28, 4), (7, 1)])
@pytest.mark.parametrize("d", [128, 64])
def test_prefill_paged_bf16_matches_oracle(hq, hkv, d):
    q, kp, vp, pt, cu, pre = paged_case(80 + hq + d, PREFIX, CHUNK, hq, hkv, d, "bf16")
    scale = 1.0 / np.sqrt(d)
    ref, ref_lse = oracle.prefill_paged(q, kp, vp, pt, cu, pre, scale)
    out, lse = G.gpu_prefill_paged(G.A.make_shape(hq, hkv, d, "bf16"), q, kp, vp, pt, cu, pre)
    G.assert_attention_close(out, ref, "bf16", f"paged prefill hq={hq} hkv={hkv} d={d}")
    assert np.max(np.abs(lse - ref_lse)) < 2e-2


@pytest.mark.parametrize("d", [64, 128])
def test_prefill_paged_fp32_matches_oracle(d):
    q, kp, vp, pt, cu, pre = paged_case(81, [0, 20, 33], [17, 1, 40], 8, 2, d, "fp32")
    ref, ref_lse = oracle.prefill_paged(q, kp, vp, pt, cu, pre, 1 / np.sqrt(d))
    out, lse = G.gpu_prefill_paged(G.A.make_shape(8, 2, d, "fp32"), q, kp, vp, pt, cu, pre)
    G.assert_attention_close(out, ref, "fp32", "paged prefill fp32")
    assert np.max(np.abs(lse - ref_lse)) < 1e-5


def test_prefill_paged_scale_variants():
    q, kp, vp, pt, cu, pre = paged_case(82, [70, 5], [90, 33], 4, 2, 64, "bf16")
    for scale in (0.0, 1.0, -0.2):
        ref, _ = oracle.prefill_paged(q, kp, vp, pt, cu, pre, scale)
        out, _ = G.gpu_prefill_paged(G.A.make_shape(4, 2, 64, "bf16", scale), q, kp, vp, pt, cu,
                                     pre, with_lse=False)
        G.assert_attention_close(out, ref, "bf16", f"paged scale={scale}")


def test_prefill_paged_long_prefix_all_rows():
    q, kp, vp, pt, cu, pre = paged_case(83, [3000, 1], [700, 500], 4, 2, 128, "bf16")
    out, lse = G.gpu_prefill_paged(G.A.make_shape(4, 2, 128), q, kp, vp, pt, cu, pre)
    ref, ref_lse = oracle.prefill_paged(q, kp, vp, pt, cu, pre, 1 / np.sqrt(128))
    G.assert_attention_close(out, ref, "bf16", "long prefix, all rows")
    assert np.max(np.abs(lse - ref_lse)) < 2e-2


@pytest.mark.parametrize("splits", [None, 4])
@pytest.mark.parametrize("pieces", [[300], [1, 299], [64, 64, 64, 108], [5, 130, 1, 164]])
def test_chunked_prefill_equals_one_shot_on_gpu(pieces, splits):
    """The prompt written and attended chunk by chunk on the GPU (dopd_kv_write
    at start_pos = cached tokens, then dopd_prefill_paged_attn, or the split
    entry point with 4 key splits) agrees with the one-shot dopd_prefill_attn
    and with the oracle."""
    rng = np.random.default_rng(84)
    hq, hkv, d, L = 8, 2, 128, int(sum(pieces))
    q, k, v = I.prefill_batch(rng, np.array([L]), hq, hkv, d, "bf16")
    sh = G.A.make_shape(hq, hkv, d)
    ref, _ = oracle.prefill(q, k, v, I.cu_from_lens([L]), 1 / np.sqrt(d))
    one_shot, _ = G.gpu_prefill(sh, q, k, v, I.cu_from_lens([L]))
    pt, num_pages = I.allocate_pages(rng, np.array([L]))
    kp, vp = I.empty_pools(num_pages, hkv, d, "bf16")
    kpd, vpd = G.A.to_device(kp), G.A.to_device(vp)
    done, outs = 0, []
    for n in pieces:
        rows = slice(done, done + n)
        G.A.dopd_kv_write(sh, G.A.to_device(k[rows]), G.A.to_device(v[rows]), kpd, vpd, num_pages,
                          G.A.to_device(pt), pt.shape[1], G.A.to_device(I.cu_from_lens([n])),
                          G.A.to_device(np.array([done], np.int32)), 1, n)
        out, _ = G.gpu_prefill_paged(sh, q[rows], None, None, pt, I.cu_from_lens([n]),
                                     np.array([done], np.int32), pools_dev=(kpd, vpd),
                                     splits=splits)
        outs.append(out)
        done += n
    chunked = np.concatenate(outs)
    G.assert_attention_close(chunked, ref, "bf16", f"chunked {pieces} vs oracle")
    G.assert_attention_close(chunked, one_shot, "bf16", f"chunked {pieces} vs one-shot")


def test_prefill_paged_chunk_of_one_matches_decode():
    q, kp, vp, pt, cu, pre = paged_case(85, [30, 0, 17, 2047], [1, 1, 1, 1], 28, 4, 128, "bf16")
    sh = G.A.make_shape(28, 4, 128)
    out, lse = G.gpu_prefill_paged(sh, q, kp, vp, pt, cu, pre)
    dec, dlse = G.gpu_decode(sh, q, kp, vp, pt, (pre + 1).astype(np.int32))
    ref, ref_lse = oracle.decode(q, kp, vp, pt, pre + 1, 1 / np.sqrt(128))
    G.assert_attention_close(out, ref, "bf16", "chunk of one vs oracle decode")
    G.assert_attention_close(out, dec, "bf16", "chunk of one vs GPU decode")
    assert np.max(np.abs(lse - ref_lse)) < 2e-2


def test_prefill_paged_invariant_under_page_permutation():
    q, kp, vp, pt, cu, pre = paged_case(86, [100, 7], [150, 60], 8, 2, 128, "bf16")
    sh = G.A.make_shape(8, 2, 128)
    out1, lse1 = G.gpu_prefill_paged(sh, q, kp, vp, pt, cu, pre)
    perm = np.random.default_rng(7).permutation(kp.shape[0])
    kp2, vp2 = np.empty_like(kp), np.empty_like(vp)
    kp2[perm], vp2[perm] = kp, vp
    pt2 = np.where(pt >= 0, perm[np.maximum(pt, 0)], -1).astype(np.int32)
    out2, lse2 = G.gpu_prefill_paged(sh, q, kp2, vp2, pt2, cu, pre)
    assert np.array_equal(out1, out2) and np.array_equal(lse1, lse2)


def test_prefill_paged_many_requests():
    # 80 chunks (more than the length-ordered work list holds), random
    # prefixes and chunk lengths, some empty chunks.
    rng = np.random.default_rng(88)
    prefix = rng.integers(0, 500, 80)
    chunk = rng.integers(0, 200, 80)
    chunk[[0, 41]] = 0
    q, kp, vp, pt, cu, pre = paged_case(89, prefix, chunk, 8, 2, 128, "bf16")
    ref, ref_lse = oracle.prefill_paged(q, kp, vp, pt, cu, pre, 1 / np.sqrt(128))
    out, lse = G.gpu_prefill_paged(G.A.make_shape(8, 2, 128, "bf16"), q, kp, vp, pt, cu, pre)
    G.assert_attention_close(out, ref, "bf16", "paged prefill 80 requests")
    assert np.max(np.abs(lse - ref_lse)) < 2e-2


def test_prefill_paged_64_requests():
    # Exactly 64 chunks (the largest batch whose lengths and prefixes the
    # kernel takes from its arguments), random prefixes, some empty chunks.
    rng = np.random.default_rng(90)
    prefix = rng.integers(0, 700, 64)
    chunk = rng.integers(0, 260, 64)
    chunk[[2, 63]] = 0
    prefix[5] = 0
    q, kp, vp, pt, cu, pre = paged_case(91, prefix, chunk, 8, 2, 128, "bf16")
    ref, ref_lse = oracle.prefill_paged(q, kp, vp, pt, cu, pre, 1 / np.sqrt(128))
    out, lse = G.gpu_prefill_paged(G.A.make_shape(8, 2, 128, "bf16"), q, kp, vp, pt, cu, pre)
    G.assert_attention_close(out, ref, "bf16", "paged prefill 64 requests")
    assert np.max(np.abs(lse - ref_lse)) < 2e-2


def test_prefill_paged_20k_prefix_all_rows():
    # A chunk of 300 tokens after 20000 cached ones (1255 pages of keys per
    # row at the end) beside a fresh 64-token chunk; every row and head.
    q, kp, vp, pt, cu, pre = paged_case(92, [20000, 0], [300, 64], 4, 1, 128, "bf16")
    out, lse = G.gpu_prefill_paged(G.A.make_shape(4, 1, 128), q, kp, vp, pt, cu, pre)
    ref, ref_lse = oracle.prefill_paged(q, kp, vp, pt, cu, pre, 1 / np.sqrt(128))
    G.assert_attention_close(out, ref, "bf16", "20k prefix, all rows")
    assert np.max(np.abs(lse - ref_lse)) < 2e-2


# Key splits (dopd_prefill_paged_attn_split): long prefixes beside short
# ones, ragged chunks; with 16 splits the short items get empty middle splits.
SPLIT_PREFIX = [3000, 1, 777, 129, 40]
SPLIT_CHUNK = [130, 65, 1, 200, 300]


@pytest.mark.parametrize("splits", [0, 2, 3, 8, 16])
@pytest.mark.parametrize("d", [128, 64])
def test_prefill_paged_split_matches_oracle(splits, d):
    q, kp, vp, pt, cu, pre = paged_case(93 + d, SPLIT_PREFIX, SPLIT_CHUNK, 8, 2, d, "bf16")
    sh = G.A.make_shape(8, 2, d)
    ref, ref_lse = oracle.prefill_paged(q, kp, vp, pt, cu, pre, 1 / np.sqrt(d))
    out, lse = G.gpu_prefill_paged(sh, q, kp, vp, pt, cu, pre, splits=splits)
    G.assert_attention_close(out, ref, "bf16", f"paged prefill splits={splits} d={d}")
    assert np.max(np.abs(lse - ref_lse)) < 2e-2
    one, one_lse = G.gpu_prefill_paged(sh, q, kp, vp, pt, cu, pre)
    G.assert_attention_close(out, one, "bf16", f"splits={splits} vs unsplit")
    assert np.max(np.abs(lse - one_lse)) < 2e-2


def test_prefill_paged_split_one_is_the_unsplit_kernel():
    q, kp, vp, pt, cu, pre = paged_case(95, SPLIT_PREFIX, SPLIT_CHUNK, 8, 2, 128, "bf16")
    sh = G.A.make_shape(8, 2, 128)
    out1, lse1 = G.gpu_prefill_paged(sh, q, kp, vp, pt, cu, pre, splits=1)
    out2, lse2 = G.gpu_prefill_paged(sh, q, kp, vp, pt, cu, pre)
    assert np.array_equal(out1, out2) and np.array_equal(lse1, lse2)


def test_prefill_paged_split_scale_variants_do_not_split():
    q, kp, vp, pt, cu, pre = paged_case(96, [700, 5], [90, 33], 4, 2, 64, "bf16")
    for scale in (0.0, -0.2):
        sh = G.A.make_shape(4, 2, 64, "bf16", scale)
        assert G.A.dopd_prefill_paged_workspace_size(sh, cu, pre, 2, 8) == 256
        ref, _ = oracle.prefill_paged(q, kp, vp, pt, cu, pre, scale)
        out, _ = G.gpu_prefill_paged(sh, q, kp, vp, pt, cu, pre, with_lse=False, splits=8)
        G.assert_attention_close(out, ref, "bf16", f"split call, scale={scale}")


def test_prefill_paged_split_20k_prefix_all_rows():
    # The automatic split count on one 300-token chunk after 20000 cached
    # tokens (12 items: splits), every row and head.
    q, kp, vp, pt, cu, pre = paged_case(97, [20000], [300], 4, 1, 128, "bf16")
    sh = G.A.make_shape(4, 1, 128)
    assert G.A.dopd_prefill_paged_workspace_size(sh, cu, pre, 1, 0) > 256
    out, lse = G.gpu_prefill_paged(sh, q, kp, vp, pt, cu, pre, splits=0)
    ref, ref_lse = oracle.prefill_paged(q, kp, vp, pt, cu, pre, 1 / np.sqrt(128))
    G.assert_attention_close(out, ref, "bf16", "split 20k prefix, all rows")
    assert np.max(np.abs(lse - ref_lse)) < 2e-2


def test_prefill_paged_split_gqa_without_lse():
    # 28 query heads over 4 KV heads, 4 key splits, no lse output (the form
    # the chunked bench calls), against the oracle.
    q, kp, vp, pt, cu, pre = paged_case(98, [1500, 64, 0], [200, 37, 90], 28, 4, 128, "bf16")
    sh = G.A.make_shape(28, 4, 128)
    ref, _ = oracle.prefill_paged(q, kp, vp, pt, cu, pre, 1 / np.sqrt(128))
    out, _ = G.gpu_prefill_paged(sh, q, kp, vp, pt, cu, pre, with_lse=False, splits=4)
    G.assert_attention_close(out, ref, "bf16", "split GQA 28/4 without lse")
