"""Host-side P/D-ratio calculator and length-aware prefill batcher (CPU).

The scheduler that consumes the attention path's timings: it turns profiled
prefill/decode latencies and the measured decode bandwidth fraction into the
number of prefill (P) and decode (D) instances, and forms the varlen prefill
batches (the cu_seqlens the prefill kernel takes).

* Eq. 11-14 (Sec. IV-B): KV memory left on a D-instance, the KV volume it can
  read within one TPOT SLO, its maximum concurrency, and the P/D ratio that
  balances P production against D consumption.
* The TTFT / TPOT interpolator over profiled tables (Sec. V-D, PD Manager)
  and the ratio step of the dynamic adjustment (Alg. 2).
* The length-aware prefill batcher (Alg. 1, Sec. IV-C) with the greedy
  value-per-token choice for the knapsack of Eq. 18, and the timeout bound of
  Eq. 17 from Kingman's approximation (Eq. 10).

Readings where the paper is loose:
* The ratio step of Alg. 2 divides the total forecast request count by
  o_next * tpot / ttft and then multiplies by n_d again, while Eq. 14 uses the
  concurrency of ONE D-instance.  Taken per Eq. 14 with each of the n_d
  D-instances carrying r_next / n_d requests: n_p = r_next * ttft / (o_next *
  tpot), R_opt = n_p / n_d.  n_p is rounded up (the paper gives no rule).
* The TPOT profile is per D-instance, so it is looked up at the batch one
  D-instance carries, r_next / n_d (the printed step passes r_next: the same
  when n_d = 1).
* The headroom factor applies to cc_d (the paper writes an undefined cc_g).
* alpha of Eq. 12 is the achievable fraction of HBM bandwidth; the decode
  kernel's measured fraction of peak is that number for this GPU.  The alpha
  of Eq. 17 is a different one: a safety factor in (0, 1].
* batchEnough: the collected short requests total at least i_next tokens.
  The batch then run is the greedy knapsack choice with W_batch = i_next; the
  rest stay queued.  On a timeout the collected total is below i_next, so
  everything collected runs.
"""
from __future__ import annotations

import bisect
import math
from dataclasses import dataclass, field
from typing import Callable


# ------------------------------------------------------------------ Eq. 11-14
def kv_memory(m_gpu: float, m_prime: float, tp: int, m_model: float) -> float:
    """Eq. 11: KV-cache bytes a D-instance of tensor-parallel size tp can hold
    (m_prime = activations and other per-GPU memory, m_model = weights)."""
    return (m_gpu - m_prime) * tp - m_model


def kv_bandwidth_volume(t_d_slo: float, alpha: float, tp: int, bw: float) -> float:
    """Eq. 12: KV bytes a D-instance can read from HBM within one TPOT SLO
    t_d_slo (s); alpha = achievable fraction of the per-GPU bandwidth bw (B/s)."""
    return t_d_slo * alpha * tp * bw


def max_concurrency(v_mem: float, v_bw: float, isl: float, osl: float, m_token: float) -> float:
    """Eq. 13: requests a D-instance sustains; on average a request holds
    isl + osl/2 tokens of m_token bytes each."""
    return min(v_mem, v_bw) / ((isl + osl / 2.0) * m_token)


def pd_ratio(cc_d: float, t_p: float, t_d: float, osl: float) -> float:
    """Eq. 14 solved for n_p / n_d.  One P-instance finishes a request every
    t_p, a request stays t_d * osl on its D-instance, so one P-instance keeps
    t_d * osl / t_p requests in flight there; n_d instances hold n_d * cc_d."""
    return cc_d * t_p / (t_d * osl)


def kv_bytes_per_token(num_layers: int, num_kv_heads: int, head_dim: int,
                       bytes_per_el: float) -> float:
    """M_token of Eq. 13: K and V of every layer for one token."""
    return 2.0 * num_layers * num_kv_heads * head_dim * bytes_per_el


@dataclass
class DInstance:
    """What Eq. 11-13 need about one D-instance (bytes, bytes/s)."""
    m_gpu: float
    m_prime: float
    m_model: float
    bw: float
    alpha: float
    tp: int = 1
    headroom: float = 0.9

    def concurrency(self, isl: float, osl: float, m_token: float, t_d_slo: float) -> float:
        """cc_d of Eq. 13 scaled by the burst headroom."""
        v_mem = kv_memory(self.m_gpu, self.m_prime, self.tp, self.m_model)
        v_bw = kv_bandwidth_volume(t_d_slo, self.alpha, self.tp, self.bw)
        return self.headroom * max(0.0, max_concurrency(v_mem, v_bw, isl, osl, m_token))


def alpha_from_bench(bench_line: dict) -> float:
    """alpha of Eq. 12 from a bench.py JSON line whose dominant kernel is the
    HBM-bound decode."""
    roof = bench_line["roofline"]
    if roof.get("bound") != "hbm":
        raise ValueError("the bench line's dominant kernel is not HBM-bound")
    return float(roof["frac"])


# ------------------------------------------------------------------ interpolator
class Interpolator:
    """TTFT(isl) and TPOT(batch, seq) over profiled tables: piecewise linear in
    isl, bilinear in (batch, seq), clamped to the tables' range."""

    def __init__(self, ttft_isl, ttft_s, tpot_batch, tpot_seq, tpot_s):
        self.ttft_isl, self.ttft_s = [float(x) for x in ttft_isl], [float(x) for x in ttft_s]
        self.tpot_batch = [float(x) for x in tpot_batch]
        self.tpot_seq = [float(x) for x in tpot_seq]
        self.tpot_s = [[float(x) for x in row] for row in tpot_s]   # [batch][seq]
        if not self.ttft_isl or len(self.ttft_isl) != len(self.ttft_s):
            raise ValueError("ttft table and its grid differ in length")
        if not self.tpot_batch or not self.tpot_seq:
            raise ValueError("empty tpot grid")
        for xs in (self.ttft_isl, self.tpot_batch, self.tpot_seq):
            if any(b <= a for a, b in zip(xs, xs[1:])):
                raise ValueError("grid points must increase")
        if len(self.tpot_s) != len(self.tpot_batch) or any(
                len(row) != len(self.tpot_seq) for row in self.tpot_s):
            raise ValueError("tpot table shape does not match its grid")

    @classmethod
    def from_tables(cls, tables: dict) -> "Interpolator":
        """From {"ttft": {"isl": [...], "s": [...]},
                 "tpot": {"batch": [...], "seq": [...], "s": [[...], ...]}}."""
        t, d = tables["ttft"], tables["tpot"]
        return cls(t["isl"], t["s"], d["batch"], d["seq"], d["s"])

    @staticmethod
    def _bracket(xs, x):
        if len(xs) == 1:
            return 0, 0, 0.0
        x = min(max(x, xs[0]), xs[-1])
        j = min(bisect.bisect_right(xs, x) - 1, len(xs) - 2)
        return j, j + 1, (x - xs[j]) / (xs[j + 1] - xs[j])

    def ttft(self, isl: float) -> float:
        a, b, t = self._bracket(self.ttft_isl, isl)
        return self.ttft_s[a] * (1 - t) + self.ttft_s[b] * t

    def tpot(self, batch: float, seq: float) -> float:
        i0, i1, u = self._bracket(self.tpot_batch, batch)
        j0, j1, v = self._bracket(self.tpot_seq, seq)
        f = self.tpot_s
        return ((1 - u) * (1 - v) * f[i0][j0] + (1 - u) * v * f[i0][j1]
                + u * (1 - v) * f[i1][j0] + u * v * f[i1][j1])


# ------------------------------------------------------------------ Alg. 2
@dataclass
class RatioDecision:
    n_p: int
    n_d: int
    n_p_exact: float     # before rounding up
    r_opt: float         # n_p_exact / n_d
    ttft: float
    tpot: float


def ratio_step(interp: Interpolator, i_next: float, o_next: float, r_next: float,
               cc_max: float) -> RatioDecision:
    """The ratio step of Alg. 2 for forecast input length i_next, output
    length o_next and r_next requests in flight: n_d = ceil(r_next / cc_max)
    D-instances, TTFT at i_next, TPOT at the batch each D-instance carries and
    the mean length (i_next + o_next)/2, and n_p from the balance of Eq. 14."""
    if not (i_next > 0 and o_next > 0 and r_next > 0 and cc_max > 0):
        raise ValueError("forecasts and the concurrency cap must be positive")
    n_d = max(1, math.ceil(r_next / cc_max))
    ttft = interp.ttft(i_next)
    tpot = interp.tpot(r_next / n_d, (i_next + o_next) / 2.0)
    n_p_exact = n_d * pd_ratio(r_next / n_d, ttft, tpot, o_next)
    n_p = max(1, math.ceil(n_p_exact * (1 - 1e-12)))
    return RatioDecision(n_p, n_d, n_p_exact, n_p_exact / n_d, ttft, tpot)


# ------------------------------------------------------------------ Alg. 1
def kingman_wait(rho: float, ca2: float, cs2: float, mean_service: float) -> float:
    """Eq. 10: mean waiting time of a G/G/1 queue in heavy traffic, with load
    rho, squared coefficients of variation ca2 (inter-arrival) and cs2
    (service), and mean service time."""
    if not 0.0 <= rho < 1.0:
        raise ValueError("load must be in [0, 1)")
    return rho / (1.0 - rho) * (ca2 + cs2) / 2.0 * mean_service


def batch_timeout(arrival_rate: float, mean_service: float, ca2: float, cs2: float,
                  safety: float = 1.0) -> float:
    """Eq. 16-17: rho = lambda * E[S]; the smallest timeout with
    T_timeout >= safety * W_q."""
    if not 0.0 < safety <= 1.0:
        raise ValueError("safety factor must be in (0, 1]")
    return safety * kingman_wait(arrival_rate * mean_service, ca2, cs2, mean_service)


def greedy_knapsack(weights, values, capacity: float):
    """Eq. 18 by the greedy rule: candidates in decreasing value per token
    (ties: lower index first), each taken if it still fits.  Returns the
    chosen indices in the order taken."""
    order = sorted(range(len(weights)),
                   key=lambda i: (-values[i] / weights[i] if weights[i] > 0 else -math.inf, i))
    chosen, used = [], 0.0
    for i in order:
        if used + weights[i] <= capacity:
            chosen.append(i)
            used += weights[i]
    return chosen


@dataclass
class PrefillBatcher:
    """Alg. 1.  A request at least i_next tokens long runs alone at once.
    Shorter ones are collected; when they total i_next or more, the greedy
    knapsack (W_batch = i_next) picks the batch to run and the rest wait;
    when the oldest collected request has waited timeout seconds, everything
    collected runs; an empty queue runs what is collected.  The caller owns
    the clock.  A batch is a list of (request id, length); value(id, length)
    gives v_i (default: the length, i.e. arrival order)."""
    i_next: float
    timeout: float
    value: Callable | None = None
    pending: list = field(default_factory=list)    # (id, length, arrival)

    def _value(self, rid, n):
        return float(n) if self.value is None else float(self.value(rid, n))

    def _take(self, idx):
        idx = set(idx)
        out = [(r, n) for k, (r, n, _) in enumerate(self.pending) if k in idx]
        self.pending = [p for k, p in enumerate(self.pending) if k not in idx]
        return out

    def poll(self, now: float):
        """Batches due at time now."""
        out = []
        while self.pending and sum(n for _, n, _ in self.pending) >= self.i_next:
            w = [n for _, n, _ in self.pending]
            v = [self._value(r, n) for r, n, _ in self.pending]
            pick = greedy_knapsack(w, v, self.i_next)
            if not pick:
                break
            out.append(self._take(pick))
        if self.pending and now >= self.next_deadline():
            out.append(self._take(range(len(self.pending))))
        return out

    def push(self, req_id, length: int, now: float):
        """A request arrives at time now; returns the batches it releases."""
        if length <= 0:
            raise ValueError("request length must be positive")
        out = self.poll(now)
        if length >= self.i_next:
            out.append([(req_id, length)])
            return out
        self.pending.append((req_id, length, now))
        out.extend(self.poll(now))
        return out

    def next_deadline(self):
        """Time at which the oldest collected request times out (None if none)."""
        return min(t for _, _, t in self.pending) + self.timeout if self.pending else None

    def drain(self):
        """Queue empty: run what is collected."""
        return [self._take(range(len(self.pending)))] if self.pending else []


def cu_seqlens(batch) -> list:
    """Prefix sums of a batch's lengths: the varlen layout the prefill takes."""
    cu = [0]
    for _, n in batch:
        cu.append(cu[-1] + int(n))
    return cu
