"""GPU: paged KV write and handoff pack are bit-exact against the oracle's
index maps, leave every other slot untouched, and stay inside their outputs."""
import numpy as np
import pytest

import oracle
from paper_2511_20982_amd import inputs as I

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu(require_gpu):
    pass


from tests import gpu_util as G  # noqa: E402


@pytest.mark.parametrize("dtype,d", [("bf16", 128), ("bf16", 64), ("fp32", 64), ("fp32", 128)])
def test_kv_write_prefill_pages_bit_exact(dtype, d):
    rng = np.random.default_rng(31)
    lens = np.array([1, 15, 16, 17, 33, 100, 0, 64], np.int32)
    hkv = 4
    pt, num_pages = I.allocate_pages(rng, lens, pool_pages=80)
    kp, vp = I.empty_pools(num_pages, hkv, d, dtype)
    t = int(lens.sum())
    knew, vnew = I.normal(rng, (t, hkv, d), dtype), I.normal(rng, (t, hkv, d), dtype)
    cu = I.cu_from_lens(lens)
    start = np.zeros(len(lens), np.int32)
    ref_k, ref_v = oracle.kv_write(knew, vnew, kp, vp, pt, cu, start)
    shape = G.A.make_shape(8, hkv, d, dtype)
    gk, gv = G.gpu_kv_write(shape, knew, vnew, kp, vp, pt, cu, start)
    assert np.array_equal(gk.view(np.uint8), ref_k.view(np.uint8))
    assert np.array_equal(gv.view(np.uint8), ref_v.view(np.uint8))


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_kv_write_appends_at_arbitrary_positions(dtype):
    # Decode-style appends (1 token) and chunk appends that straddle pages.
    rng = np.random.default_rng(32)
    hkv, d = 2, 64
    cap = np.array([40, 40, 40, 40, 40], np.int32)
    pt, num_pages = I.allocate_pages(rng, cap, pool_pages=20)
    kp, vp = I.empty_pools(num_pages, hkv, d, dtype)
    # pre-fill some content so that untouched slots are not all poison
    kp[:], vp[:] = I.normal(rng, kp.shape, dtype), I.normal(rng, vp.shape, dtype)
    n_new = np.array([1, 5, 20, 0, 16], np.int32)
    start = np.array([0, 13, 7, 3, 16], np.int32)
    t = int(n_new.sum())
    knew, vnew = I.normal(rng, (t, hkv, d), dtype), I.normal(rng, (t, hkv, d), dtype)
    cu = I.cu_from_lens(n_new)
    ref_k, ref_v = oracle.kv_write(knew, vnew, kp, vp, pt, cu, start)
    shape = G.A.make_shape(4, hkv, d, dtype)
    gk, gv = G.gpu_kv_write(shape, knew, vnew, kp, vp, pt, cu, start)
    assert np.array_equal(gk.view(np.uint8), ref_k.view(np.uint8))
    assert np.array_equal(gv.view(np.uint8), ref_v.view(np.uint8))


@pytest.mark.parametrize("dtype,d,layers", [("bf16", 128, 1), ("bf16", 64, 3), ("fp32", 64, 2)])
def test_pack_bit_exact(dtype, d, layers):
    rng = np.random.default_rng(33)
    hkv = 4
    lens = np.array([512, 1, 17, 31, 0, 48], np.int32)
    pt, num_pages = I.allocate_pages(rng, lens, pool_pages=60)
    kp = I.normal(rng, (layers, num_pages, hkv, 16, d), dtype)
    vp = I.normal(rng, (layers, num_pages, hkv, d, 16), dtype)
    req = np.array([0, 2, 1, 5, 3, 4], np.int32)
    seq = lens[req]
    off = I.handoff_offsets(seq, layers, hkv, d)
    ref = oracle.pack(kp, vp, layers, pt, req, seq, off)
    shape = G.A.make_shape(8, hkv, d, dtype)
    out = G.gpu_pack(shape, kp, vp, layers, pt, req, seq, off)
    assert np.array_equal(out.view(np.uint8), ref.view(np.uint8))


def test_pack_unaligned_offsets():
    # Offsets that are not 16-byte aligned take the element-wise path.
    rng = np.random.default_rng(34)
    hkv, d = 2, 64
    lens = np.array([20, 9], np.int32)
    pt, num_pages = I.allocate_pages(rng, lens, pool_pages=4)
    kp = I.normal(rng, (num_pages, hkv, 16, d), "bf16")
    vp = I.normal(rng, (num_pages, hkv, d, 16), "bf16")
    off = I.handoff_offsets(lens, 1, hkv, d) + 3          # shifted by 3 elements
    ref = oracle.pack(kp, vp, 1, pt, np.arange(2), lens, off)
    out = G.gpu_pack(G.A.make_shape(2, hkv, d), kp, vp, 1, pt, np.arange(2, dtype=np.int32), lens, off)
    assert np.array_equal(out[3:], ref[3:])        # elements before off[0] are not written


@pytest.mark.parametrize("dtype,d", [("bf16", 128), ("fp32", 64)])
def test_pack_many_handoffs(dtype, d):
    # More handoffs than one wave scans at once (the block list is found by
    # 64-wide scans), empty handoffs among them, and workgroups whose blocks
    # straddle handoffs.
    rng = np.random.default_rng(39)
    hkv, layers = 2, 2
    lens = rng.integers(0, 70, 150).astype(np.int32)
    lens[[0, 64, 65, 149]] = 0
    lens[[3, 100]] = [16, 129]
    pt, num_pages = I.allocate_pages(rng, np.maximum(lens, 1))
    kp = I.normal(rng, (layers, num_pages, hkv, 16, d), dtype)
    vp = I.normal(rng, (layers, num_pages, hkv, d, 16), dtype)
    req = rng.permutation(len(lens)).astype(np.int32)
    seq = lens[req]
    off = I.handoff_offsets(seq, layers, hkv, d)
    ref = oracle.pack(kp, vp, layers, pt, req, seq, off)
    out = G.gpu_pack(G.A.make_shape(4, hkv, d, dtype), kp, vp, layers, pt, req, seq, off)
    assert np.array_equal(out.view(np.uint8), ref.view(np.uint8))


def test_write_then_pack_round_trip_is_a_transpose():
    rng = np.random.default_rng(35)
    hkv, d = 4, 128
    lens = np.array([512, 77, 16], np.int32)
    pt, num_pages = I.allocate_pages(rng, lens)
    kp, vp = I.empty_pools(num_pages, hkv, d, "bf16")
    t = int(lens.sum())
    knew, vnew = I.normal(rng, (t, hkv, d), "bf16"), I.normal(rng, (t, hkv, d), "bf16")
    cu = I.cu_from_lens(lens)
    shape = G.A.make_shape(28, hkv, d)
    gk, gv = G.gpu_kv_write(shape, knew, vnew, kp, vp, pt, cu, np.zeros(3, np.int32))
    off = I.handoff_offsets(lens, 1, hkv, d)
    out = G.gpu_pack(shape, gk, gv, 1, pt, np.arange(3, dtype=np.int32), lens, off)
    for r in range(3):
        a, b = cu[r], cu[r + 1]
        expect = np.stack([knew[a:b].transpose(1, 0, 2), vnew[a:b].transpose(1, 0, 2)])
        assert np.array_equal(out[off[r]:off[r + 1]], expect.reshape(-1))


@pytest.mark.parametrize("dtype,d,layers", [("bf16", 128, 2), ("bf16", 64, 1), ("fp32", 64, 3),
                                            ("fp32", 128, 1)])
def test_unpack_bit_exact(dtype, d, layers):
    rng = np.random.default_rng(36)
    hkv = 4
    lens = np.array([512, 1, 17, 31, 0, 48], np.int32)
    pt, num_pages = I.allocate_pages(rng, lens, pool_pages=60)
    kp, vp = I.empty_pools(num_pages, hkv, d, dtype, num_layers=layers)
    kp[:], vp[:] = I.normal(rng, kp.shape, dtype), I.normal(rng, vp.shape, dtype)  # old contents
    req = np.array([0, 2, 1, 5, 3, 4], np.int32)
    seq = lens[req]
    offs = I.handoff_offsets(seq, layers, hkv, d)
    buf = I.normal(rng, (int(offs[-1]),), dtype)
    ref_k, ref_v = oracle.unpack(buf, offs, req, seq, kp, vp, layers, pt)
    gk, gv = G.gpu_unpack(G.A.make_shape(8, hkv, d, dtype), buf, offs, req, seq, kp, vp, layers, pt)
    assert np.array_equal(gk.view(np.uint8), ref_k.view(np.uint8))
    assert np.array_equal(gv.view(np.uint8), ref_v.view(np.uint8))


def test_unpack_unaligned_offsets():
    rng = np.random.default_rng(37)
    hkv, d = 2, 64
    lens = np.array([20, 9], np.int32)
    pt, num_pages = I.allocate_pages(rng, lens, pool_pages=4)
    kp, vp = I.empty_pools(num_pages, hkv, d, "bf16")
    offs = I.handoff_offsets(lens, 1, hkv, d) + 3
    buf = I.normal(rng, (int(offs[-1]),), "bf16")
    req = np.arange(2, dtype=np.int32)
    ref_k, ref_v = oracle.unpack(buf, offs, req, lens, kp, vp, 1, pt)
    gk, gv = G.gpu_unpack(G.A.make_shape(2, hkv, d), buf, offs, req, lens, kp, vp, 1, pt)
    assert np.array_equal(gk, ref_k) and np.array_equal(gv, ref_v)


def test_handoff_round_trip_decode_bit_identical():
    """P -> D on one GPU: pack from pool A, unpack into a pool B with another page
    order; decode on both caches gives bit-identical outputs."""
    rng = np.random.default_rng(38)
    hq, hkv, d = 28, 4, 128
    lens = np.array([512, 700, 33, 1], np.int32)
    pt_a, n_a = I.allocate_pages(rng, lens)
    pt_b, n_b = I.allocate_pages(rng, lens, pool_pages=n_a + 7)
    ka, va = I.empty_pools(n_a, hkv, d, "bf16")
    I.fill_live_slots(rng, ka, va, pt_a, lens, "bf16")
    kb, vb = I.empty_pools(n_b, hkv, d, "bf16")
    req = np.arange(4, dtype=np.int32)
    offs = I.handoff_offsets(lens, 1, hkv, d)
    sh = G.A.make_shape(hq, hkv, d)
    buf = G.gpu_pack(sh, ka, va, 1, pt_a, req, lens, offs)
    gk, gv = G.gpu_unpack(sh, buf, offs, req, lens, kb, vb, 1, pt_b)
    ref_k, ref_v = oracle.unpack(buf, offs, req, lens, kb, vb, 1, pt_b)
    assert np.array_equal(gk, ref_k) and np.array_equal(gv, ref_v)
    q = I.normal(rng, (4, hq, d), "bf16")
    out_a, lse_a = G.gpu_decode(sh, q, ka, va, pt_a, lens, split=256)
    out_b, lse_b = G.gpu_decode(sh, q, gk, gv, pt_b, lens, split=256)
    assert np.array_equal(out_a, out_b) and np.array_equal(lse_a, lse_b)
