"""Seeded workload generator: determinism, length laws, page tables, poison."""
import numpy as np

from paper_2511_20982_amd import inputs as I


def test_bf16_rounding_is_nearest_even():
    x = np.array([1.0, 1.0 + 2**-8, 1.0 + 3 * 2**-9, -2.5, np.inf, 0.0], np.float32)
    b = I.f32_to_bf16_bits(x)
    back = I.bf16_bits_to_f32(b)
    assert back[0] == 1.0
    assert back[1] == 1.0                      # tie -> even mantissa
    assert back[2] == 1.0 + 2**-7              # above half -> up
    assert back[3] == -2.5 and np.isinf(back[4]) and back[5] == 0.0
    assert I.f32_to_bf16_bits(np.array([np.nan], np.float32))[0] == 0x7FC0


def test_tiny_fp32_shape_and_pages():
    w = I.tiny_fp32()
    assert list(w.prefill_lens) == [17, 64, 5, 120] and w.q.shape == (206, 8, 64)
    assert w.num_pages == 64
    used = w.page_table[w.page_table >= 0]
    assert len(used) == 16 and len(set(used.tolist())) == 16
    assert np.all(np.isnan(w.k_pool)) and len(w.steps) == 8


def test_generator_is_deterministic():
    a, b = I.tiny_fp32(), I.tiny_fp32()
    assert np.array_equal(a.q, b.q) and np.array_equal(a.page_table, b.page_table)
    assert np.array_equal(a.steps[3][0], b.steps[3][0])


def test_decode_pool_poison_and_live_slots():
    w = I.decode_workload("t", 1, [1, 16, 17, 33], 4, 2, 8, "bf16")
    kf = I.bf16_bits_to_f32(w.k_pool)
    live = (~np.isnan(kf)).all(axis=(1, 3)).sum()   # live (page, slot) pairs
    assert live == 1 + 16 + 17 + 33
    assert (w.page_table[0, 1:] == -1).all()


def test_length_laws():
    rng = np.random.default_rng(0)
    x = I.lognormal_lengths(rng, 200000, 1024, 0.8, 16, 4096)
    assert x.min() >= 16 and x.max() <= 4096
    assert abs(np.median(x) - 1024) < 15
    frac_cap = (x == 4096).mean()
    assert 0.03 < frac_cap < 0.055                 # ~4.2% clipped at the cap
    ctx, is_long = I.bimodal_lengths(np.random.default_rng(1), 256, 0.2, 100, 500, 4096, 16384)
    assert is_long.sum() == 51
    assert ctx[is_long].min() >= 4096 and ctx[~is_long].max() <= 500


def test_handoff_offsets_back_to_back():
    off = I.handoff_offsets([3, 5], 2, 4, 8)
    assert list(off) == [0, 3 * 2 * 2 * 4 * 8, 8 * 2 * 2 * 4 * 8]
