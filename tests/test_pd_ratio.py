"""Host-side scheduler: P/D ratio (Eq. 11-14, Alg. 2) and the length-aware
prefill batcher (Alg. 1, Eq. 10, 16-18).

The paper prints the ratios it deployed but not the inputs that produced
them, so the module's outputs are parity unpinned against the paper.  These
tests pin what the mathematics fixes: the balance of Eq. 14 holds for what
the calculator returns, Kingman's formula is exact for M/G/1 queues
(Pollaczek-Khinchine) and close to a simulated queue, the greedy knapsack is
optimal for equal weights (checked by brute force), the interpolator
reproduces bilinear functions, and the batcher emits every request exactly
once within its length and waiting bounds.
"""
import itertools

import numpy as np
import pytest

from paper_2511_20982_amd import pd_ratio as pr


def _rel(a, b):
    return abs(a - b) / max(abs(a), abs(b), 1e-300)


# ------------------------------------------------------------------ Eq. 11-14
def test_eq14_balance_holds_for_the_ratio():
    rng = np.random.default_rng(11)
    for _ in range(200):
        cc_d, t_p, t_d = rng.uniform(1, 500), rng.uniform(1e-3, 5), rng.uniform(1e-3, 0.2)
        osl, n_d = rng.uniform(16, 4096), int(rng.integers(1, 64))
        n_p = pr.pd_ratio(cc_d, t_p, t_d, osl) * n_d
        # n_p P-instances keep n_p * t_d * osl / t_p requests in flight on the
        # D side: exactly what n_d D-instances at cc_d hold.
        assert _rel(n_p * t_d * osl / t_p, n_d * cc_d) < 1e-12


def test_eq14_rates_match():
    # Same balance read as rates: P finishes n_p / t_p requests per second,
    # D finishes n_d * cc_d / (t_d * osl).
    n_p = pr.pd_ratio(cc_d=96, t_p=0.4, t_d=0.03, osl=512) * 5
    assert _rel(n_p / 0.4, 5 * 96 / (0.03 * 512)) < 1e-12


def test_eq13_memory_and_bandwidth_regimes():
    m_tok = pr.kv_bytes_per_token(80, 8, 128, 1)        # 80 layers, 8 KV heads, fp8
    assert m_tok == 2 * 80 * 8 * 128
    isl, osl = 2048, 512
    # Memory bound: tiny memory, huge bandwidth.
    v_mem = pr.kv_memory(m_gpu=80e9, m_prime=10e9, tp=1, m_model=60e9)
    assert v_mem == 10e9
    v_bw = pr.kv_bandwidth_volume(t_d_slo=0.1, alpha=0.6, tp=1, bw=8e12)
    assert _rel(v_bw, 0.1 * 0.6 * 8e12) < 1e-15
    cc = pr.max_concurrency(v_mem, v_bw, isl, osl, m_tok)
    assert _rel(cc * (isl + osl / 2) * m_tok, min(v_mem, v_bw)) < 1e-12
    assert v_mem < v_bw and _rel(cc, v_mem / ((isl + osl / 2) * m_tok)) < 1e-12
    # Bandwidth bound: the cc requests' KV is read once in exactly t_d_slo.
    v_mem2 = pr.kv_memory(288e9, 8e9, 4, 70e9)
    assert v_mem2 == 280e9 * 4 - 70e9
    cc2 = pr.max_concurrency(v_mem2, v_bw, isl, osl, m_tok)
    assert v_bw < v_mem2
    t_read = cc2 * (isl + osl / 2) * m_tok / (0.6 * 8e12)
    assert _rel(t_read, 0.1) < 1e-12
    # Doubling TP doubles the bandwidth-bound concurrency.
    v_bw4 = pr.kv_bandwidth_volume(0.1, 0.6, 2, 8e12)
    assert _rel(pr.max_concurrency(v_mem2, v_bw4, isl, osl, m_tok), 2 * cc2) < 1e-12


def test_eq13_mean_resident_tokens():
    # A request holds isl + k tokens at decode step k = 0..osl-1; averaged
    # over its life that is isl + (osl-1)/2, the isl + osl/2 of Eq. 13 up to
    # the half token a step.
    isl, osl = 700, 300
    mean = np.mean([isl + k for k in range(osl)])
    assert mean == isl + (osl - 1) / 2
    assert abs(mean - (isl + osl / 2)) <= 0.5


def test_dinstance_headroom_and_alpha_from_bench():
    line = {"roofline": {"bound": "hbm", "frac": 0.6, "achieved": 4800, "peak": 8000}}
    alpha = pr.alpha_from_bench(line)
    assert alpha == 0.6
    d = pr.DInstance(m_gpu=288e9, m_prime=8e9, m_model=70e9, bw=8e12, alpha=alpha)
    m_tok = pr.kv_bytes_per_token(80, 8, 128, 2)
    cc = d.concurrency(2048, 512, m_tok, 0.05)
    v_mem = pr.kv_memory(288e9, 8e9, 1, 70e9)               # 210 GB
    v_bw = pr.kv_bandwidth_volume(0.05, alpha, 1, 8e12)     # 240 GB
    assert _rel(cc, 0.9 * min(v_mem, v_bw) / ((2048 + 256) * m_tok)) < 1e-12
    cc_bw = d.concurrency(2048, 512, m_tok, 0.02)           # 96 GB read per TPOT
    assert _rel(cc_bw, 0.9 * 0.02 * alpha * 8e12 / ((2048 + 256) * m_tok)) < 1e-12
    with pytest.raises(ValueError):
        pr.alpha_from_bench({"roofline": {"bound": "mfma", "frac": 0.3}})


# ------------------------------------------------------------------ interpolator
def _tables(f_ttft, f_tpot, isl, batch, seq):
    return pr.Interpolator(isl, [f_ttft(x) for x in isl], batch, seq,
                           [[f_tpot(b, s) for s in seq] for b in batch])


def test_interpolator_reproduces_bilinear():
    f_ttft = lambda x: 0.01 + 2e-5 * x
    f_tpot = lambda b, s: 0.02 + 1e-4 * b + 3e-6 * s + 2e-8 * b * s
    it = _tables(f_ttft, f_tpot, [128, 512, 2048, 8192], [1, 8, 64, 256], [256, 1024, 4096])
    rng = np.random.default_rng(3)
    for _ in range(100):
        x, b, s = rng.uniform(128, 8192), rng.uniform(1, 256), rng.uniform(256, 4096)
        assert _rel(it.ttft(x), f_ttft(x)) < 1e-12
        assert _rel(it.tpot(b, s), f_tpot(b, s)) < 1e-12
    # Grid points exactly; outside the grid clamps to the edge.
    assert it.ttft(512) == f_ttft(512)
    assert it.ttft(10) == f_ttft(128) and it.ttft(1e6) == f_ttft(8192)
    assert it.tpot(0.5, 10) == f_tpot(1, 256)
    assert it.tpot(1e4, 1e5) == f_tpot(256, 4096)


def test_interpolator_validation_and_tables():
    with pytest.raises(ValueError):
        pr.Interpolator([1, 1], [0, 0], [1], [1], [[0]])
    with pytest.raises(ValueError):
        pr.Interpolator([1, 2], [0, 0], [1, 2], [1], [[0]])
    it = pr.Interpolator.from_tables({"ttft": {"isl": [100], "s": [0.5]},
                                      "tpot": {"batch": [4], "seq": [64], "s": [[0.01]]}})
    assert it.ttft(1e5) == 0.5 and it.tpot(1, 1) == 0.01


# ------------------------------------------------------------------ Alg. 2
def test_ratio_step_satisfies_eq14():
    f_ttft = lambda x: 0.02 + 4e-5 * x
    f_tpot = lambda b, s: 0.015 + 2e-4 * b + 1e-6 * s
    it = _tables(f_ttft, f_tpot, [64, 1024, 16384], [1, 32, 512], [128, 8192])
    rng = np.random.default_rng(14)
    for _ in range(200):
        i_next, o_next = rng.uniform(64, 16384), rng.uniform(16, 2048)
        r_next, cc_max = rng.uniform(1, 5000), rng.uniform(8, 512)
        d = pr.ratio_step(it, i_next, o_next, r_next, cc_max)
        # D side: enough instances, each within the cap.
        assert d.n_d * cc_max >= r_next and r_next / d.n_d <= cc_max * (1 + 1e-12)
        assert d.n_d == 1 or (d.n_d - 1) * cc_max < r_next
        # Lookups at the forecast point and the per-instance batch.
        assert d.ttft == it.ttft(i_next)
        assert d.tpot == it.tpot(r_next / d.n_d, (i_next + o_next) / 2)
        # Eq. 14 with cc_d = r_next / n_d, t_p = ttft, t_d = tpot, osl = o_next.
        lhs = d.n_p_exact * d.tpot * o_next / d.ttft
        assert _rel(lhs, d.n_d * (r_next / d.n_d)) < 1e-12
        assert _rel(d.r_opt, pr.pd_ratio(r_next / d.n_d, d.ttft, d.tpot, o_next)) < 1e-12
        # Rounded up, by less than one instance.
        assert d.n_p >= 1 and d.n_p >= d.n_p_exact * (1 - 1e-12) and d.n_p - 1 < max(d.n_p_exact, 1)


def test_ratio_step_single_d_instance_matches_printed_ratio():
    # With one D-instance the printed R_opt = r_next * ttft / (o_next * tpot)
    # and the Eq. 14 reading coincide.
    it = pr.Interpolator([100, 1000], [0.05, 0.2], [1, 100], [10, 1000], [[0.01, 0.02], [0.03, 0.05]])
    d = pr.ratio_step(it, 550, 200, 40, 64)
    assert d.n_d == 1
    printed = 40 / ((200 * d.tpot) / d.ttft)
    assert _rel(d.r_opt, printed) < 1e-12
    with pytest.raises(ValueError):
        pr.ratio_step(it, 0, 200, 40, 64)


# ------------------------------------------------------------------ Eq. 10, 16, 17
def test_kingman_is_pollaczek_khinchine_for_poisson_arrivals():
    # M/G/1: W_q = lambda E[S^2] / (2 (1 - rho)) = rho (1 + cs2) / (2 (1 - rho)) E[S].
    for rho in (0.1, 0.5, 0.9):
        for cs2 in (0.0, 0.5, 1.0, 3.0):
            es = 0.25
            lam = rho / es
            es2 = (1 + cs2) * es * es
            pk = lam * es2 / (2 * (1 - rho))
            assert _rel(pr.kingman_wait(rho, 1.0, cs2, es), pk) < 1e-12
    # M/M/1: rho / (mu - lambda).
    assert _rel(pr.kingman_wait(0.8, 1, 1, 1 / 5.0), 0.8 / (5.0 - 4.0)) < 1e-12
    with pytest.raises(ValueError):
        pr.kingman_wait(1.0, 1, 1, 1)


def test_kingman_against_simulated_queue():
    # Lindley's recursion W_{n+1} = max(0, W_n + S_n - A_{n+1}) for a G/G/1 queue with gamma inter-arrivals (ca2 = 0.5) and gamma service
    # (cs2 = 0.25) at rho = 0.9: Kingman is a heavy-traffic approximation,
    # within 10 % here.
    rng = np.random.default_rng(10)
    n, rho, es = 400_000, 0.9, 1.0
    ca2, cs2 = 0.5, 0.25
    a = rng.gamma(1 / ca2, ca2 * es / rho, n)
    s = rng.gamma(1 / cs2, cs2 * es, n)
    w, tot = 0.0, 0.0
    for k in range(n - 1):
        w = max(0.0, w + s[k] - a[k + 1])
        tot += w
    sim = tot / (n - 1)
    assert abs(sim - pr.kingman_wait(rho, ca2, cs2, es)) / sim < 0.10


def test_batch_timeout_eq17():
    wq = pr.kingman_wait(0.6, 2.0, 0.5, 0.3)
    assert _rel(pr.batch_timeout(2.0, 0.3, 2.0, 0.5, safety=0.5), 0.5 * wq) < 1e-12
    with pytest.raises(ValueError):
        pr.batch_timeout(2.0, 0.3, 1, 1, safety=0.0)
    with pytest.raises(ValueError):
        pr.batch_timeout(4.0, 0.3, 1, 1)


# ------------------------------------------------------------------ Eq. 18
def _brute_knapsack(w, v, cap):
    best = 0.0
    for m in itertools.product((0, 1), repeat=len(w)):
        if sum(wi * x for wi, x in zip(w, m)) <= cap:
            best = max(best, sum(vi * x for vi, x in zip(v, m)))
    return best


def test_greedy_knapsack_optimal_for_equal_weights():
    rng = np.random.default_rng(18)
    for _ in range(50):
        n = int(rng.integers(1, 11))
        w = [37.0] * n
        v = list(rng.uniform(0, 10, n))
        cap = float(rng.integers(0, 12)) * 37.0
        pick = pr.greedy_knapsack(w, v, cap)
        assert abs(sum(v[i] for i in pick) - _brute_knapsack(w, v, cap)) < 1e-9


def test_greedy_knapsack_feasible_and_ordered():
    rng = np.random.default_rng(19)
    for _ in range(100):
        n = int(rng.integers(1, 10))
        w = list(rng.integers(1, 100, n).astype(float))
        v = list(rng.uniform(0, 5, n))
        cap = float(rng.integers(0, 300))
        pick = pr.greedy_knapsack(w, v, cap)
        assert len(set(pick)) == len(pick)
        assert sum(w[i] for i in pick) <= cap
        ratios = [v[i] / w[i] for i in pick]
        assert ratios == sorted(ratios, reverse=True)
        assert sum(v[i] for i in pick) <= _brute_knapsack(w, v, cap) + 1e-9
        # Maximal: nothing left out still fits.
        rest = cap - sum(w[i] for i in pick)
        assert all(w[i] > rest for i in range(n) if i not in pick)
    # Equal value per token: arrival order, skipping what no longer fits.
    assert pr.greedy_knapsack([5, 9, 3, 4], [5, 9, 3, 4], 12) == [0, 2, 3]


# ------------------------------------------------------------------ Alg. 1
def _simulate(i_next, timeout, lengths, arrivals, value=None):
    b = pr.PrefillBatcher(i_next, timeout, value=value)
    released = []      # (time, batch)
    for rid, (n, t) in enumerate(zip(lengths, arrivals)):
        # Poll at every deadline that falls before this arrival.
        while b.next_deadline() is not None and b.next_deadline() <= t:
            dl = b.next_deadline()
            released += [(dl, x) for x in b.poll(dl)]
        released += [(t, x) for x in b.push(rid, int(n), t)]
    released += [(arrivals[-1], x) for x in b.drain()]
    return released


def test_batcher_emits_each_request_once_within_bounds():
    rng = np.random.default_rng(1)
    n = 3000
    lengths = np.minimum((rng.pareto(1.5, n) + 1) * 64, 32768).astype(int)
    arrivals = np.cumsum(rng.exponential(0.01, n))
    i_next, timeout = 1024, 0.05
    rel = _simulate(i_next, timeout, lengths, arrivals)
    seen = [rid for _, x in rel for rid, _ in x]
    assert sorted(seen) == list(range(n))
    for t, x in rel:
        assert len(x) >= 1
        ids = [r for r, _ in x]
        if len(x) == 1 and lengths[ids[0]] >= i_next:
            assert t == arrivals[ids[0]]                 # long: at once, alone
            continue
        assert all(lengths[r] < i_next for r in ids)     # shorts never mix with longs
        assert sum(lengths[r] for r in ids) <= max(i_next, 1)
        assert all(t - arrivals[r] <= timeout + 1e-12 for r in ids)
        assert all(t >= arrivals[r] for r in ids)


def test_batcher_knapsack_and_timeout_paths():
    b = pr.PrefillBatcher(i_next=100, timeout=1.0)
    assert b.push("a", 60, 0.0) == []
    # a + b reach 100: the knapsack packs both into W_batch = 100.
    assert b.push("b", 40, 0.1) == [[("a", 60), ("b", 40)]]
    assert b.push("c", 70, 0.2) == []
    # c + d = 120 >= 100: greedy by arrival order takes c, skips d (does not
    # fit), and d keeps waiting.
    assert b.push("d", 50, 0.3) == [[("c", 70)]]
    assert b.push("long", 500, 0.4) == [[("long", 500)]]
    assert b.next_deadline() == 1.3
    assert b.poll(1.29) == []
    assert b.poll(1.3) == [[("d", 50)]]
    assert b.drain() == []
    # Value per token decides the pick once the total reaches W_batch.
    b = pr.PrefillBatcher(100, 1.0, value=lambda rid, n: {"x": 1.0, "y": 90.0, "z": 1.0}[rid])
    b.push("x", 50, 0.0)
    b.push("y", 45, 0.0)
    # y (2.0 per token) then z (0.033) fit in 100; x (0.02) does not and waits.
    assert b.push("z", 30, 0.0) == [[("y", 45), ("z", 30)]]
    assert b.drain() == [[("x", 50)]]
    with pytest.raises(ValueError):
        b.push("bad", 0, 0.0)


def test_cu_seqlens():
    assert pr.cu_seqlens([("a", 3), ("b", 5), ("c", 1)]) == [0, 3, 8, 9]
    assert pr.cu_seqlens([]) == [0]
