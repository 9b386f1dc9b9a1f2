"""GPU: varlen causal prefill against the fp64 oracle."""
import numpy as np
import pytest

import oracle
from paper_2511_20982_amd import inputs as I

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu(require_gpu):
    pass


from tests import gpu_util as G  # noqa: E402

RAGGED = [1, 15, 16, 17, 63, 64, 65, 127, 128, 129, 300, 0, 5]


@pytest.mark.parametrize("hq,hkv", [(8, 8), (8, 2), (28, 4), (7, 1)])
@pytest.mark.parametrize("d", [128, 64])
def test_prefill_bf16_matches_oracle(hq, hkv, d):
    rng = np.random.default_rng(60 + hq + d)
    lens = np.array(RAGGED, np.int32)
    q, k, v = I.prefill_batch(rng, lens, hq, hkv, d, "bf16")
    cu = I.cu_from_lens(lens)
    scale = 1.0 / np.sqrt(d)
    ref, ref_lse = oracle.prefill(q, k, v, cu, scale)
    out, lse = G.gpu_prefill(G.A.make_shape(hq, hkv, d, "bf16"), q, k, v, cu)
    G.assert_attention_close(out, ref, "bf16", f"prefill hq={hq} hkv={hkv} d={d}")
    assert np.max(np.abs(lse - ref_lse)) < 2e-2


def test_prefill_bf16_long_prompt_all_rows():
    rng = np.random.default_rng(61)
    lens = np.array([2000, 3, 900], np.int32)
    hq, hkv, d = 4, 2, 128
    q, k, v = I.prefill_batch(rng, lens, hq, hkv, d, "bf16")
    cu = I.cu_from_lens(lens)
    out, lse = G.gpu_prefill(G.A.make_shape(hq, hkv, d), q, k, v, cu)
    ref, ref_lse = oracle.prefill(q, k, v, cu, 1 / np.sqrt(d))
    G.assert_attention_close(out, ref, "bf16", "long prompt, all rows")
    assert np.max(np.abs(lse - ref_lse)) < 2e-2


def test_prefill_bf16_32k_prompt_all_rows():
    # One 32768-token prompt (256 q tiles, 512 key tiles per row at the end)
    # beside two short ones; every row and head against the oracle.
    rng = np.random.default_rng(66)
    lens = np.array([32768, 5, 130], np.int32)
    hq, hkv, d = 4, 1, 128
    q, k, v = I.prefill_batch(rng, lens, hq, hkv, d, "bf16")
    cu = I.cu_from_lens(lens)
    out, lse = G.gpu_prefill(G.A.make_shape(hq, hkv, d), q, k, v, cu)
    ref, ref_lse = oracle.prefill(q, k, v, cu, 1 / np.sqrt(d))
    G.assert_attention_close(out, ref, "bf16", "32k prompt, all rows")
    assert np.max(np.abs(lse - ref_lse)) < 2e-2


def test_prefill_bf16_scale_variants_and_determinism():
    rng = np.random.default_rng(62)
    lens = np.array([70, 129], np.int32)
    q, k, v = I.prefill_batch(rng, lens, 8, 2, 64, "bf16")
    cu = I.cu_from_lens(lens)
    for scale in (0.0, 1.0):
        ref, _ = oracle.prefill(q, k, v, cu, scale)
        out, _ = G.gpu_prefill(G.A.make_shape(8, 2, 64, "bf16", scale), q, k, v, cu, with_lse=False)
        G.assert_attention_close(out, ref, "bf16", f"scale={scale}")
    sh = G.A.make_shape(8, 2, 64, "bf16")
    a1, l1 = G.gpu_prefill(sh, q, k, v, cu)
    a2, l2 = G.gpu_prefill(sh, q, k, v, cu)
    assert np.array_equal(a1, a2) and np.array_equal(l1, l2)


@pytest.mark.parametrize("d", [64, 128])
def test_prefill_fp32_matches_oracle(d):
    rng = np.random.default_rng(63)
    lens = np.array([17, 64, 5, 120, 1], np.int32)
    q, k, v = I.prefill_batch(rng, lens, 8, 2, d, "fp32")
    cu = I.cu_from_lens(lens)
    ref, ref_lse = oracle.prefill(q, k, v, cu, 1 / np.sqrt(d))
    out, lse = G.gpu_prefill(G.A.make_shape(8, 2, d, "fp32"), q, k, v, cu)
    G.assert_attention_close(out, ref, "fp32", "prefill fp32")
    assert np.max(np.abs(lse - ref_lse)) < 1e-5


@pytest.mark.parametrize("d", [128, 64])
def test_prefill_bf16_many_requests(d):
    # More requests than the length-ordered work list holds (64): the work is
    # dealt heaviest q tile first instead.  Lengths 0..300, some empty.
    rng = np.random.default_rng(70 + d)
    lens = rng.integers(0, 301, 100).astype(np.int32)
    lens[[3, 50, 99]] = 0
    q, k, v = I.prefill_batch(rng, lens, 8, 2, d, "bf16")
    cu = I.cu_from_lens(lens)
    ref, ref_lse = oracle.prefill(q, k, v, cu, 1.0 / np.sqrt(d))
    out, lse = G.gpu_prefill(G.A.make_shape(8, 2, d, "bf16"), q, k, v, cu)
    G.assert_attention_close(out, ref, "bf16", f"prefill 100 requests d={d}")
    assert np.max(np.abs(lse - ref_lse)) < 2e-2


@pytest.mark.parametrize("hq,hkv", [(8, 2), (7, 7)])
def test_prefill_bf16_64_requests(hq, hkv):
    # Exactly 64 requests: the largest batch whose work order, lengths and
    # per-request prefix sums the kernel takes from its arguments.  Lengths
    # 0..400 (some empty, some one tile, some ragged), unsorted.
    rng = np.random.default_rng(75 + hq)
    lens = rng.integers(0, 401, 64).astype(np.int32)
    lens[[0, 17, 63]] = 0
    lens[[5, 6]] = [128, 1]
    q, k, v = I.prefill_batch(rng, lens, hq, hkv, 128, "bf16")
    cu = I.cu_from_lens(lens)
    ref, ref_lse = oracle.prefill(q, k, v, cu, 1.0 / np.sqrt(128))
    out, lse = G.gpu_prefill(G.A.make_shape(hq, hkv, 128, "bf16"), q, k, v, cu)
    G.assert_attention_close(out, ref, "bf16", f"prefill 64 requests {hq}/{hkv}")
    assert np.max(np.abs(lse - ref_lse)) < 2e-2
