"""GPU: paged split-K decode against the fp64 oracle, plus the invariants the
oracle satisfies exactly (page permutation, split size, determinism)."""
import numpy as np
import pytest

import oracle
from paper_2511_20982_amd import inputs as I

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu(require_gpu):
    pass


from tests import gpu_util as G  # noqa: E402

EDGE_CTX = [1, 2, 15, 16, 17, 31, 32, 33, 47, 64, 100, 511, 512, 513, 1000, 2049]


@pytest.mark.parametrize("hq,hkv", [(8, 8), (8, 2), (28, 4), (64, 8), (16, 1), (7, 7)])
@pytest.mark.parametrize("d", [128, 64])
def test_decode_bf16_matches_oracle(hq, hkv, d):
    w = I.decode_workload("t", 40 + hq + d, EDGE_CTX, hq, hkv, d, "bf16")
    ref, ref_lse = oracle.decode(w.q_dec, w.k_pool, w.v_pool, w.page_table, w.context_lens, w.scale)
    out, lse = G.gpu_decode(G.shape_of(w), w.q_dec, w.k_pool, w.v_pool, w.page_table, w.context_lens)
    G.assert_attention_close(out, ref, "bf16", f"decode hq={hq} hkv={hkv} d={d}")
    assert np.max(np.abs(lse - ref_lse)) < 2e-2


@pytest.mark.parametrize("split", [32, 64, 256, 4096])
def test_decode_split_size_independent(split):
    w = I.decode_workload("t", 51, [1, 40, 300, 5000, 16384], 16, 2, 128, "bf16")
    ref, _ = oracle.decode(w.q_dec, w.k_pool, w.v_pool, w.page_table, w.context_lens, w.scale)
    out, _ = G.gpu_decode(G.shape_of(w), w.q_dec, w.k_pool, w.v_pool, w.page_table,
                          w.context_lens, split=split)
    G.assert_attention_close(out, ref, "bf16", f"split={split}")


def test_decode_deterministic_and_page_permutation_bit_identical():
    w = I.decode_workload("t", 52, [3, 700, 4100, 33], 32, 4, 128, "bf16")
    sh = G.shape_of(w)
    out1, lse1 = G.gpu_decode(sh, w.q_dec, w.k_pool, w.v_pool, w.page_table, w.context_lens, split=256)
    out2, lse2 = G.gpu_decode(sh, w.q_dec, w.k_pool, w.v_pool, w.page_table, w.context_lens, split=256)
    assert np.array_equal(out1, out2) and np.array_equal(lse1, lse2)
    perm = np.random.default_rng(7).permutation(w.num_pages)
    k2, v2 = np.empty_like(w.k_pool), np.empty_like(w.v_pool)
    k2[perm], v2[perm] = w.k_pool, w.v_pool
    pt2 = np.where(w.page_table >= 0, perm[np.maximum(w.page_table, 0)], -1).astype(np.int32)
    out3, lse3 = G.gpu_decode(sh, w.q_dec, k2, v2, pt2, w.context_lens, split=256)
    assert np.array_equal(out1, out3) and np.array_equal(lse1, lse3)


def test_decode_without_lse_and_scale_variants():
    w = I.decode_workload("t", 53, [20, 200], 8, 2, 64, "bf16")
    for scale in (0.0, 1.0, 0.3):
        ref, _ = oracle.decode(w.q_dec, w.k_pool, w.v_pool, w.page_table, w.context_lens, scale)
        out, _ = G.gpu_decode(G.shape_of(w, scale), w.q_dec, w.k_pool, w.v_pool, w.page_table,
                              w.context_lens, with_lse=False)
        G.assert_attention_close(out, ref, "bf16", f"scale={scale}")


@pytest.mark.parametrize("d", [64, 128])
def test_decode_fp32_matches_oracle(d):
    w = I.decode_workload("t", 54, [1, 16, 17, 130, 300], 8, 2, d, "fp32")
    ref, ref_lse = oracle.decode(w.q_dec, w.k_pool, w.v_pool, w.page_table, w.context_lens, w.scale)
    out, lse = G.gpu_decode(G.shape_of(w), w.q_dec, w.k_pool, w.v_pool, w.page_table, w.context_lens)
    G.assert_attention_close(out, ref, "fp32", "decode fp32")
    assert np.max(np.abs(lse - ref_lse)) < 1e-5


@pytest.mark.parametrize("split", [0, 64])
def test_decode_bf16_thousand_requests(split):
    # Many more requests than the 64 lanes that look up a slice's first
    # request at once, and than workgroups: slices span dozens of short
    # requests; contexts 1..200 with a few long ones.
    rng = np.random.default_rng(57)
    ctx = rng.integers(1, 201, 1000)
    ctx[[10, 500, 999]] = [3000, 1, 4097]
    w = I.decode_workload("t", 58, ctx, 32, 4, 128, "bf16")
    ref, ref_lse = oracle.decode(w.q_dec, w.k_pool, w.v_pool, w.page_table, w.context_lens, w.scale)
    out, lse = G.gpu_decode(G.shape_of(w), w.q_dec, w.k_pool, w.v_pool, w.page_table,
                            w.context_lens, split=split)
    G.assert_attention_close(out, ref, "bf16", f"decode 1000 requests split={split}")
    assert np.max(np.abs(lse - ref_lse)) < 2e-2
