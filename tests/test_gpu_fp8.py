"""GPU: E4M3 KV pages.  The writer's codes are bit-exact against the oracle's
quantiser (ties, saturation, subnormals included) and leave every other slot
untouched; the decode over E4M3 pools matches the oracle's decode over the
same codes within the bf16 bar; pack/unpack move the codes bit-exactly."""
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


def _scales(hkv, seed):
    rng = np.random.default_rng(seed)
    return (rng.uniform(4.0, 7.0, hkv) / 448).astype(np.float32), \
        (rng.uniform(4.0, 7.0, hkv) / 448).astype(np.float32)


def _byte_pools(rng, num_pages, hkv, d):
    """Pools of random bytes: slots the writer must not touch keep them."""
    return (rng.integers(0, 256, (num_pages, hkv, 16, d)).astype(np.uint8),
            rng.integers(0, 256, (num_pages, hkv, d, 16)).astype(np.uint8))


def _ref_write(knew, vnew, ks, vs, kp, vp, pt, cu, start):
    return oracle.kv_write(oracle.e4m3_quantize(knew, ks), oracle.e4m3_quantize(vnew, vs), kp, vp,
                           pt, cu, start)


@pytest.mark.parametrize("d", [128, 64])
def test_kv_write_fp8_prefill_pages_bit_exact(d):
    rng = np.random.default_rng(61)
    lens = np.array([1, 15, 16, 17, 33, 100, 0, 64], np.int32)
    hkv = 4
    pt, num_pages = I.allocate_pages(rng, lens, pool_pages=80)
    kp, vp = _byte_pools(rng, num_pages, hkv, d)
    t = int(lens.sum())
    knew, vnew = I.normal(rng, (t, hkv, d), "bf16"), I.normal(rng, (t, hkv, d), "bf16")
    # Heads: a power-of-two scale (many exact ties), a tiny one (saturation at
    # +-448), a large one (subnormal codes) and an arbitrary one.
    ks = np.array([0.25, 1.5 / 448, 64.0, 0.0137], np.float32)
    vs = np.array([0.0137, 0.25, 1.5 / 448, 64.0], np.float32)
    cu = I.cu_from_lens(lens)
    start = np.zeros(len(lens), np.int32)
    ref_k, ref_v = _ref_write(knew, vnew, ks, vs, kp, vp, pt, cu, start)
    shape = G.A.make_shape(8, hkv, d, "fp8")
    gk, gv = G.gpu_kv_write_fp8(shape, knew, vnew, ks, vs, kp, vp, pt, cu, start)
    assert np.array_equal(gk, ref_k)
    assert np.array_equal(gv, ref_v)
    # The case does exercise saturation and subnormals.
    codes = oracle.e4m3_quantize(knew, ks)
    assert np.any(codes[:, 1] & 0x7F == 0x7E) and np.any((codes[:, 2] & 0x78) == 0)


def test_kv_write_fp8_appends_at_arbitrary_positions():
    rng = np.random.default_rng(62)
    hkv, d = 2, 128
    cap = np.array([40, 40, 40, 40, 40], np.int32)
    pt, num_pages = I.allocate_pages(rng, cap, pool_pages=20)
    kp, vp = _byte_pools(rng, num_pages, hkv, d)
    n_new = np.array([1, 5, 20, 0, 16], np.int32)
    start = np.array([0, 13, 7, 3, 16], np.int32)
    t = int(n_new.sum())
    knew, vnew = I.normal(rng, (t, hkv, d), "bf16"), I.normal(rng, (t, hkv, d), "bf16")
    ks, vs = _scales(hkv, 3)
    cu = I.cu_from_lens(n_new)
    ref_k, ref_v = _ref_write(knew, vnew, ks, vs, kp, vp, pt, cu, start)
    gk, gv = G.gpu_kv_write_fp8(G.A.make_shape(4, hkv, d, "fp8"), knew, vnew, ks, vs, kp, vp, pt,
                                cu, start)
    assert np.array_equal(gk, ref_k) and np.array_equal(gv, ref_v)


@pytest.mark.parametrize("hq,hkv", [(8, 8), (8, 2), (28, 4), (64, 8), (16, 1), (7, 7)])
@pytest.mark.parametrize("d", [128, 64])
def test_decode_fp8_matches_oracle(hq, hkv, d):
    w = I.decode_workload("t", 70 + hq + d, EDGE_CTX, hq, hkv, d, "bf16")
    ks, vs = _scales(hkv, hq + d)
    kq, vq = G.quantize_pools(w.k_pool, w.v_pool, ks, vs)
    ref, ref_lse = oracle.decode_e4m3(w.q_dec, kq, vq, ks, vs, w.page_table, w.context_lens,
                                      w.scale)
    shape = G.A.make_shape(hq, hkv, d, "fp8", w.scale)
    out, lse = G.gpu_decode_fp8(shape, w.q_dec, kq, vq, ks, vs, w.page_table, w.context_lens)
    G.assert_attention_close(out, ref, "bf16", f"fp8 decode hq={hq} hkv={hkv} d={d}")
    assert np.max(np.abs(lse - ref_lse)) < 2e-2


@pytest.mark.parametrize("split", [32, 256, 4096])
def test_decode_fp8_split_size_independent(split):
    w = I.decode_workload("t", 81, [1, 40, 300, 5000, 16384], 16, 2, 128, "bf16")
    ks, vs = _scales(2, 5)
    kq, vq = G.quantize_pools(w.k_pool, w.v_pool, ks, vs)
    ref, _ = oracle.decode_e4m3(w.q_dec, kq, vq, ks, vs, w.page_table, w.context_lens, w.scale)
    out, _ = G.gpu_decode_fp8(G.A.make_shape(16, 2, 128, "fp8"), w.q_dec, kq, vq, ks, vs,
                              w.page_table, w.context_lens, split=split)
    G.assert_attention_close(out, ref, "bf16", f"fp8 split={split}")


def test_decode_fp8_page_permutation_bit_identical_and_scale_variants():
    w = I.decode_workload("t", 82, [3, 700, 4100, 33], 32, 4, 128, "bf16")
    ks, vs = _scales(4, 6)
    kq, vq = G.quantize_pools(w.k_pool, w.v_pool, ks, vs)
    sh = G.A.make_shape(32, 4, 128, "fp8")
    out1, lse1 = G.gpu_decode_fp8(sh, w.q_dec, kq, vq, ks, vs, w.page_table, w.context_lens)
    perm = np.random.default_rng(8).permutation(w.num_pages)
    k2, v2 = np.empty_like(kq), np.empty_like(vq)
    k2[perm], v2[perm] = kq, vq
    pt2 = np.where(w.page_table >= 0, perm[np.maximum(w.page_table, 0)], -1).astype(np.int32)
    out2, lse2 = G.gpu_decode_fp8(sh, w.q_dec, k2, v2, ks, vs, pt2, w.context_lens)
    assert np.array_equal(out1, out2) and np.array_equal(lse1, lse2)
    for scale in (0.0, 1.0):
        ref, _ = oracle.decode_e4m3(w.q_dec, kq, vq, ks, vs, w.page_table, w.context_lens, scale)
        out, _ = G.gpu_decode_fp8(G.A.make_shape(32, 4, 128, "fp8", scale), w.q_dec, kq, vq, ks,
                                  vs, w.page_table, w.context_lens, with_lse=False)
        G.assert_attention_close(out, ref, "bf16", f"fp8 scale={scale}")


def test_write_then_decode_fp8_on_the_gpu():
    # The fp8 cache written by the GPU writer, read by the GPU decode, against
    # the oracle's quantiser and decode.
    rng = np.random.default_rng(63)
    ctx = np.array([1, 17, 64, 300, 1029], np.int32)
    hq, hkv, d = 28, 4, 128
    pt, num_pages = I.allocate_pages(rng, ctx)
    t = int(ctx.sum())
    knew, vnew = I.normal(rng, (t, hkv, d), "bf16"), I.normal(rng, (t, hkv, d), "bf16")
    q = I.normal(rng, (len(ctx), hq, d), "bf16")
    ks, vs = _scales(hkv, 9)
    kp0 = np.full((num_pages, hkv, 16, d), 0x7F, np.uint8)   # NaN codes in dead slots
    vp0 = np.full((num_pages, hkv, d, 16), 0x7F, np.uint8)
    cu = I.cu_from_lens(ctx)
    start = np.zeros(len(ctx), np.int32)
    shape = G.A.make_shape(hq, hkv, d, "fp8")
    gk, gv = G.gpu_kv_write_fp8(shape, knew, vnew, ks, vs, kp0, vp0, pt, cu, start)
    rk, rv = _ref_write(knew, vnew, ks, vs, kp0, vp0, pt, cu, start)
    assert np.array_equal(gk, rk) and np.array_equal(gv, rv)
    ref, _ = oracle.decode_e4m3(q, rk, rv, ks, vs, pt, ctx, shape.softmax_scale)
    out, _ = G.gpu_decode_fp8(shape, q, gk, gv, ks, vs, pt, ctx)
    G.assert_attention_close(out, ref, "bf16", "fp8 write then decode")


@pytest.mark.parametrize("d,layers", [(128, 1), (64, 3)])
def test_pack_unpack_fp8_bit_exact(d, layers):
    rng = np.random.default_rng(64)
    lens = np.array([1, 16, 17, 250, 0, 33], np.int32)
    hkv = 4
    pt, num_pages = I.allocate_pages(rng, lens, pool_pages=60)
    kp = rng.integers(0, 256, (layers, num_pages, hkv, 16, d)).astype(np.uint8)
    vp = rng.integers(0, 256, (layers, num_pages, hkv, d, 16)).astype(np.uint8)
    req = np.array([3, 0, 5, 1], np.int32)
    hl = lens[req]
    off = I.handoff_offsets(hl, layers, hkv, d)
    ref = oracle.pack(kp, vp, layers, pt, req, hl, off)
    shape = G.A.make_shape(8, hkv, d, "fp8")
    got = G.gpu_pack(shape, kp, vp, layers, pt, req, hl, off)
    assert np.array_equal(got, ref)
    # unpack into fresh pools of another page order equals the oracle's scatter
    pt2, _ = I.allocate_pages(rng, lens, pool_pages=num_pages)
    k0 = rng.integers(0, 256, kp.shape).astype(np.uint8)
    v0 = rng.integers(0, 256, vp.shape).astype(np.uint8)
    rk, rv = oracle.unpack(ref, off, req, hl, k0, v0, layers, pt2)
    gk, gv = G.gpu_unpack(shape, got, off, req, hl, k0, v0, layers, pt2)
    assert np.array_equal(gk, rk) and np.array_equal(gv, rv)


def test_decode_fp8_full_size_gqa_70b_shape():
    # The 70B-shaped GQA decode (B 256, 64/8 heads, bimodal contexts) over an
    # E4M3 cache, whole batch against the oracle.
    w = I.decode_gqa_70b()
    ks, vs = _scales(w.hkv, 10)
    kq, vq = G.quantize_pools(w.k_pool, w.v_pool, ks, vs)
    ref, _ = oracle.decode_e4m3(w.q_dec, kq, vq, ks, vs, w.page_table, w.context_lens, w.scale)
    out, _ = G.gpu_decode_fp8(G.A.make_shape(w.hq, w.hkv, w.d, "fp8", w.scale), w.q_dec, kq, vq,
                              ks, vs, w.page_table, w.context_lens)
    G.assert_attention_close(out, ref, "bf16", "fp8 decode GQA 70B shape")
