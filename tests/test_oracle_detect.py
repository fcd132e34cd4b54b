"""Pins of the oracle's monitor (Sec. 5.2: Eq. (5), (6), (8), (9); App. B.2).

Hand-worked golden cases, closed forms for filled periodic windows, brute force on tiny alphabets
(periodicity checked directly from its definition, not by the oracle's trailing scan), and
hand-derived timelines for warmup, cooldown, the K-of-3 vote and the debounce.
"""
import os

import numpy as np
import pytest

import oracle
from conftest import read_golden

P0 = oracle.paper_params()


def _ints(s):
    return [int(x) for x in s.split()]


def test_golden_lz(golden_dir):
    for toks, cost in read_golden(os.path.join(golden_dir, "lz_cost.txt")):
        y = _ints(toks)
        assert oracle.lz_cost(y, 0, len(y)) == int(cost), toks


def test_golden_novelty(golden_dir):
    for toks, span, nov, r in read_golden(os.path.join(golden_dir, "novelty.txt")):
        y = _ints(toks)
        assert oracle.novelty(y, 0, len(y), 4, int(span)) == (int(nov), int(r)), toks


def test_golden_tail(golden_dir):
    for toks, H, copies, min_len, pstar, span in read_golden(
            os.path.join(golden_dir, "tail_align.txt")):
        y = _ints(toks)
        P, T = oracle.tail_best(y, 0, len(y), 256, int(H), int(copies), int(min_len))
        assert P == int(pstar), toks
        assert (len(y) - T if P else -1) == int(span), toks


def _fresh(n, start=1000):
    return list(range(start, start + n))


@pytest.mark.parametrize("P", [1, 2, 3, 4, 7, 12, 28, 29, 51, 52, 100, 256])
def test_closed_forms_filled_periodic_window(P):
    """A window of m = 256 tokens filled by a primitive period-P loop: TTR = P/m, LZ cost = P + 2
    (P literals, then one overlapping match to the end), so CR = (P+2)/m."""
    m = 256
    unit = _fresh(P)
    y = [unit[i % P] for i in range(m)]
    assert oracle.distinct(y, 0, m) == P
    assert oracle.lz_cost(y, 0, m) == (P + 2 if m - P >= 3 else m)
    # vote thresholds of Eq. (8): TTR < 0.2 iff P <= 51; CR < 0.12 iff P + 2 < 30.72
    assert (5 * oracle.distinct(y, 0, m) < m) == (P <= 51)
    assert (25 * oracle.lz_cost(y, 0, m) < 3 * m) == (P <= 28)


def test_all_distinct_window():
    y = _fresh(256)
    assert oracle.distinct(y, 0, 256) == 256
    assert oracle.lz_cost(y, 0, 256) == 256
    nov, r = oracle.novelty(y, 0, 256, 4, 64)
    assert (nov, r) == (64, 64)


def test_loop_has_no_novelty():
    unit = _fresh(9)
    y = _fresh(50, 5000) + [unit[i % 9] for i in range(200)]
    nov, r = oracle.novelty(y, len(y) - 256 if len(y) > 256 else 0, len(y), 4, 64)
    assert r == 64 and nov == 0


def test_window_respects_lo():
    # Tokens before lo must be invisible to every windowed indicator.
    y = [1, 2, 3, 4] * 10 + _fresh(20)
    assert oracle.distinct(y, 40, 60) == 20
    assert oracle.lz_cost(y, 40, 60) == 20


def _brute_lz(y, lo, hi):
    cost, i = 0, lo
    while i < hi:
        best = 0
        for p in range(lo, i):
            k = 0
            while i + k < hi and y[p + k] == y[i + k]:
                k += 1
            best = max(best, k)
        if best >= 3:
            cost, i = cost + 2, i + best
        else:
            cost, i = cost + 1, i + 1
    return cost


def _has_period(y, lo, hi, P):
    """Direct definition: y[lo..hi) has period P iff y[i] == y[i+P] whenever both lie inside."""
    return all(y[i] == y[i + P] for i in range(lo, hi - P))


@pytest.mark.parametrize("alpha", [2, 3])
def test_tail_align_brute_force(alpha):
    rng = np.random.default_rng(alpha)
    for trial in range(300):
        n = int(rng.integers(1, 65))
        y = list(rng.integers(0, alpha, n))
        t0 = int(rng.integers(0, 3)) if n > 3 else 0
        H = int(rng.integers(4, 70))
        L = oracle.tail_align(y, t0, n, 64, H)
        for P in range(1, 65):
            # the longest suffix inside [t0, n) and at most H long that has period P
            T = max(T for T in range(0, min(H, n - t0) + 1) if _has_period(y, n - T, n, P))
            assert L[P] == max(0, T - P), (y, t0, H, P)


def test_lz_brute_force_small_alphabet():
    rng = np.random.default_rng(5)
    for trial in range(200):
        n = int(rng.integers(1, 48))
        y = list(rng.integers(0, 3, n))
        lo = int(rng.integers(0, n))
        assert oracle.lz_cost(y, lo, n) == _brute_lz(y, lo, n)


@pytest.mark.parametrize("P", list(range(1, 257)))
def test_planted_loop_found_at_its_span(P):
    """A planted primitive period-P loop starting at s0 (y[s0-1] differs from the loop's token at
    s0-1+P) is reported with P* = P and span [s0, n-1] once it has >= 3 copies and >= 32 tokens,
    as long as it fits the horizon."""
    s0 = 300
    length = max(3 * P, 32) + 5
    if length > 1024:
        length = 1024
    unit = _fresh(P, 7000)
    y = _fresh(s0, 1) + [unit[i % P] for i in range(length)]
    n = len(y)
    Pst, T = oracle.tail_best(y, 0, n, 256, 1024, 3, 32)
    assert Pst == P
    assert n - T == s0


def test_period_inside_longer_tail_capped_at_horizon():
    unit = _fresh(12, 7000)
    y = _fresh(10) + [unit[i % 12] for i in range(3000)]
    P, T = oracle.tail_best(y, 0, len(y), 256, 1024, 3, 32)
    assert (P, T) == (12, 1024)        # every multiple of 12 ties at T = H; the smallest wins


def test_nested_loop_outer_period_wins():
    motif = _fresh(16, 7000)
    unit = motif * 12 + _fresh(8, 9000)
    y = _fresh(100) + unit * 4
    P, T = oracle.tail_best(y, 0, len(y), 256, 1024, 3, 32)
    assert P == 200 and T == 800


# ------------------------------------------------------------------------------------------------
# Timelines of Eq. (9): warmup, cooldown, escalation, K-of-3 vote, debounce.
# ------------------------------------------------------------------------------------------------
def _run(y, confs, params, t0=0):
    det = oracle.Detector(params)
    return [det.step(y, t0, n, c) for n, c in zip(range(1, len(y) + 1), confs)]


def test_always_on_timeline_warmup_cooldown_levels():
    y = _fresh(200)
    decs = _run(y, [0.0] * 200, oracle.paper_params(mode=1))
    trig = [d["n"] for d in decs if d["trigger"]]
    assert trig == [64, 96, 128, 160, 192]
    assert [d["level"] for d in decs if d["trigger"]] == [0, 1, 2, 3, 3]
    assert [d["n_int"] for d in decs if d["trigger"]] == [1, 2, 3, 4, 5]


def test_period4_loop_timeline():
    """The whole stream is a period-4 loop. By hand: TTR votes from m = 21 (5*4 < m), CR votes
    from m = 51 (25*6 < 3m); TailRep qualifies from n = 32 and debounces at n = 35; the novelty
    rate falls below 0.02 at n = 70 (one of the four first rotations left among the last 64
    positions: 1/64) so Stall holds from n = 73. Warmup is 64,
    so the first trigger is at n = 64, then every 32 tokens with l = 0, 1, 2, 3, 3."""
    unit = _fresh(4)
    y = [unit[i % 4] for i in range(200)]
    decs = _run(y, [0.0] * 200, P0)
    by_n = {d["n"]: d for d in decs}
    assert by_n[20]["votes"] & 1 == 0 and by_n[21]["votes"] & 1 == 1
    assert by_n[50]["votes"] & 2 == 0 and by_n[51]["votes"] & 2 == 2
    assert by_n[31]["period"] == 0 and by_n[32]["period"] == 4
    assert by_n[34]["tailrep_gate"] == 0 and by_n[35]["tailrep_gate"] == 1
    assert by_n[72]["stall_gate"] == 0 and by_n[73]["stall_gate"] == 1
    assert by_n[69]["novel"] == 2 and by_n[70]["novel"] == 1 and by_n[71]["novel"] == 0
    assert [d["n"] for d in decs if d["trigger"]] == [64, 96, 128, 160, 192]
    assert [d["level"] for d in decs if d["trigger"]] == [0, 1, 2, 3, 3]
    assert by_n[64]["span_lo"] == 0


def test_confidence_vote_is_needed_for_a_mid_period_loop():
    """Period 40 fills the window: TTR votes (200 < 256) but CR does not (25*42 > 768), so Warn
    needs the confidence streak: strictly above 0.9 on >= 6 consecutive steps."""
    unit = _fresh(40)
    y = _fresh(50, 5000) + [unit[i % 40] for i in range(400)]
    n_all = len(y)
    confs = [0.5] * n_all
    for n in range(400, 406):
        confs[n - 1] = 0.95
    confs[420 - 1] = 0.9          # not strictly above the threshold: streak resets
    decs = _run(y, confs, P0)
    by_n = {d["n"]: d for d in decs}
    # conf > 0.9 at n = 400..405: the streak reaches 6 at n = 405
    assert by_n[404]["votes"] == 0b001 and by_n[404]["trigger"] == 0
    assert by_n[405]["votes"] == 0b101 and by_n[405]["warn"] == 1
    assert by_n[405]["trigger"] == 1
    assert by_n[406]["votes"] == 0b001 and by_n[420]["votes"] == 0b001


def test_p1_only_mode():
    y = _fresh(300)
    confs = [0.95 if 100 <= n < 140 else 0.1 for n in range(1, 301)]
    decs = _run(y, confs, oracle.paper_params(mode=2))
    assert [d["n"] for d in decs if d["trigger"]] == [105, 137]


def test_ttr_threshold_is_strict():
    # m = 255 tokens with exactly 51 distinct: 51/255 = 0.2 is not below 0.2.
    base = _fresh(51)
    y = [base[i % 51] for i in range(255)]
    det = oracle.Detector(P0)
    d = det.step(y, 0, 255, 0.0)
    assert d["distinct"] == 51 and d["votes"] & 1 == 0
    y2 = [base[i % 50] for i in range(255)]
    d2 = oracle.Detector(P0).step(y2, 0, 255, 0.0)
    assert d2["distinct"] == 50 and d2["votes"] & 1 == 1


def test_warmup_counts_from_t0():
    unit = _fresh(4)
    y = _fresh(500, 3000) + [unit[i % 4] for i in range(200)]
    det = oracle.Detector(P0)
    trig = []
    for n in range(501, 701):
        d = det.step(y, 500, n, 0.0)
        if d["trigger"]:
            trig.append(n - 500)
    assert trig and trig[0] == 64


def test_cr_interval_holds_value():
    unit = _fresh(4)
    y = _fresh(100, 3000) + [unit[i % 4] for i in range(200)]
    det = oracle.Detector(oracle.paper_params(cr_interval=8))
    costs = [det.step(y, 0, n, 0.0)["lz_cost"] for n in range(1, 301)]
    for n in range(1, 301):
        if n % 8 and n > 1:
            assert costs[n - 1] == costs[n - 2]
    assert costs[-1] == oracle.lz_cost(y, 296 - 256, 296)   # last recompute at n = 296
