"""Pins of the oracle's keep set (Eq. (10), Eq. (11), Sec. 5.3) and of its guarded trajectory.

The keep set is checked against a hand-worked fixture, against closed-form contiguous slot ranges
(a different formulation from the oracle's set-membership construction), and against the
invariants of Sec. 5.3: |I_keep| <= B, ascending subsequence, anchors kept, I_bad dropped, the
recent budget R >> l. The trajectory is checked for len <= budget, sorted positions, the H2O
increment of G per step, and the planted span.
"""
import os

import numpy as np
import pytest

import oracle
from conftest import read_golden
from oracle.trajectory import SequenceOracle, prefill_positions


def test_golden_keep_set(golden_dir):
    p = oracle.paper_params(n_anchor=4)
    pos = np.arange(100)
    for span, level, kept in read_golden(os.path.join(golden_dir, "keep_set.txt")):
        got = oracle.keep_set(p, pos, 64, int(span), int(level))
        assert got.tolist() == [int(x) for x in kept.split()]


def _closed_form(pos, budget, span_lo, level, n_anchor=32, recent_div=4, sparse_div=2):
    """Contiguous-range form of the keep set over position-sorted slots."""
    pos = np.asarray(pos)
    L = len(pos)
    t = int(pos[-1])
    R = budget // recent_div
    S = budget // sparse_div - n_anchor
    na = int(np.searchsorted(pos, n_anchor))                    # slots [0, na): anchors
    rc = max(na, int(np.searchsorted(pos, t - R + 1)))          # slots [rc, L): recent window
    bl = L if span_lo < 0 else max(rc, int(np.searchsorted(pos, span_lo)))  # [bl, L): bad
    nr = min(R >> level, bl - rc)
    M = rc - na
    sparse = list(range(na, rc)) if M <= S else [na + (k * M) // S for k in range(S)]
    return list(range(na)) + sparse + list(range(bl - nr, bl))


def test_keep_set_matches_closed_form_and_invariants():
    rng = np.random.default_rng(0)
    p = oracle.paper_params()
    for trial in range(400):
        budget = int(rng.choice([128, 256, 512, 1024, 2048]))
        L = int(rng.integers(1, budget + 1))
        span = int(rng.integers(0, 5 * budget))
        pos = np.sort(rng.choice(span + L + 40, L, replace=False)).astype(np.int32)
        t = int(pos[-1])
        R = budget // 4
        span_lo = -1 if rng.random() < 0.3 else int(rng.integers(max(0, t - 2 * R), t + 1))
        level = int(rng.integers(0, 4))
        keep = oracle.keep_set(p, pos, budget, span_lo, level)
        assert keep.tolist() == _closed_form(pos, budget, span_lo, level)
        assert len(keep) <= budget and len(keep) <= 32 + (budget // 2 - 32) + R
        assert np.all(np.diff(keep) > 0) and (len(keep) == 0 or (keep[0] >= 0 and keep[-1] < L))
        kept_pos = set(pos[keep].tolist())
        assert set(pos[pos < 32].tolist()) <= kept_pos                  # anchors survive
        if span_lo >= 0:
            bad = pos[(pos >= max(span_lo, t - R + 1)) & (pos >= 32)]
            assert not (set(bad.tolist()) & kept_pos)                   # I_bad is dropped
        rec = [j for j in keep if pos[j] >= max(32, t - R + 1)]
        cand = [j for j in range(L) if pos[j] >= max(32, t - R + 1)
                and (span_lo < 0 or pos[j] < span_lo)]
        assert len(rec) == min(R >> level, len(cand))
        assert rec == cand[len(cand) - len(rec):]                       # the most recent ones


def test_prefill_keep_three_quarters():
    p = oracle.paper_params()
    for ctx, budget in [(256, 256), (4096, 1024), (8192, 2048), (32768, 4096)]:
        pos = prefill_positions(p, ctx, budget)
        assert len(pos) == 3 * budget // 4
        assert pos[:32].tolist() == list(range(32))
        assert pos[-(budget // 4):].tolist() == list(range(ctx - budget // 4, ctx))
    assert prefill_positions(p, 300, 512).tolist() == list(range(300))


def test_tiny_trajectory_invariants_and_planted_span():
    from paper_2604_10044_amd.synth import tiny
    wl = tiny()
    so = SequenceOracle(wl, 0)
    assert so.len == 192
    G = wl.group
    prev = so.acc[:, :, :so.len].sum(axis=2)
    for s in range(wl.steps):
        before_len = so.len
        dec = so.step(s)
        if dec["new_len"] < 0:
            np.testing.assert_allclose(so.acc[:, :, :so.len].sum(axis=2) - prev, G, rtol=1e-12)
        assert so.len <= wl.budget[0]
        assert np.all(np.diff(so.pos) > 0)
        prev = so.acc[:, :, :so.len].sum(axis=2)
        if s >= 3:
            assert dec["period"] == 12 and dec["span_lo"] == 160
    assert all(d["trigger"] == 0 for d in so.history)


def test_small_window_trajectory_triggers_and_compacts():
    """With W = 64 a period-4 loop fills the window, TTR (4/64) and CR (6/64) vote and the tail
    repeats, so the guard triggers (every cooldown, escalating l); each keep set drops the loop's
    part of the recent window."""
    from paper_2604_10044_amd.synth import tiny
    wl = tiny(steps=48, period=4)
    p = oracle.paper_params(W=64)
    so = SequenceOracle(wl, 0, params=p)
    trig = []
    for s in range(wl.steps):
        d = so.step(s)
        if d["trigger"]:
            trig.append(d)
            t = wl.ctx[0] + s
            R = wl.budget[0] // 4
            assert not np.any((so.pos >= max(d["span_lo"], t - R + 1)))
            assert so.len == d["new_len"] <= 32 + 96 + (R >> d["level"])
    # The monitor starts at the first decode step (n = 257), so both persistence gates need four
    # steps (n = 260) before the first trigger; the next one follows after the 32-step cooldown.
    assert [d["n"] for d in trig] == [260, 292]
    assert [d["level"] for d in trig] == [0, 1]


# ---------------------------------------------------------------------------------------------
# Baseline keep policies (Sec. 6.1: H2O, StreamingLLM), as read for a cache at its budget.

def test_golden_keep_baseline(golden_dir):
    for policy, n_anchor, pos, score, kept in read_golden(os.path.join(golden_dir,
                                                                        "keep_baseline.txt")):
        p = oracle.paper_params(policy=int(policy), n_anchor=int(n_anchor))
        got = oracle.keep_set_baseline(p, [int(x) for x in pos.split()], 16,
                                       np.array([float(x) for x in score.split()], np.float32))
        assert got.tolist() == [int(x) for x in kept.split()], (policy, n_anchor)


def _h2o_invariants(keep, score, L, budget):
    K = budget // 2 + budget // 4
    R = min(budget // 4, L)
    older = L - R
    keep = np.asarray(keep)
    assert len(keep) == min(L, K)
    assert np.all(np.diff(keep) > 0)
    assert set(range(older, L)) <= set(keep.tolist())             # the recent window is kept
    kept_old = keep[keep < older]
    dropped = np.setdiff1d(np.arange(older), kept_old)
    if len(kept_old) and len(dropped):
        # no dropped slot outranks a kept one: higher score, or equal score and later slot
        ks, ds = score[kept_old], score[dropped]
        assert ks.min() >= ds.max()
        tie = ks.min() == ds.max()
        if tie:
            v = ks.min()
            assert kept_old[score[kept_old] == v].min() > dropped[score[dropped] == v].max()


def test_h2o_keep_invariants_random():
    rng = np.random.default_rng(3)
    for _ in range(300):
        budget = int(rng.choice([16, 64, 128, 512]))
        L = int(rng.integers(1, budget + 1))
        pos = np.sort(rng.choice(4 * budget, L, replace=False)).astype(np.int32)
        # few distinct values so ties across the threshold are common
        score = rng.integers(0, int(rng.choice([2, 5, 1000])), L).astype(np.float32) * 0.25
        keep = oracle.keep_set_baseline(oracle.paper_params(policy=1), pos, budget, score)
        _h2o_invariants(keep, score, L, budget)


def test_h2o_special_cases():
    p = oracle.paper_params(policy=1)
    for budget in (16, 64, 256):
        L = budget
        K = budget // 2 + budget // 4
        pos = np.arange(L, dtype=np.int32)
        # equal scores: a sliding window of the last K slots
        assert oracle.keep_set_baseline(p, pos, budget, np.ones(L, np.float32)).tolist() == \
            list(range(L - K, L))
        # scores falling with the slot: the oldest K - R slots plus the recent window
        R = budget // 4
        dec = np.arange(L, 0, -1).astype(np.float32)
        assert oracle.keep_set_baseline(p, pos, budget, dec).tolist() == \
            list(range(K - R)) + list(range(L - R, L))
        # fewer live slots than K: everything is kept
        assert oracle.keep_set_baseline(p, pos[:K], budget, dec[:K]).tolist() == list(range(K))


def test_streaming_closed_form_random():
    rng = np.random.default_rng(4)
    for _ in range(300):
        budget = int(rng.choice([64, 128, 512, 2048]))
        n_anchor = int(rng.integers(0, 40))
        L = int(rng.integers(1, budget + 1))
        pos = np.sort(rng.choice(3 * budget, L, replace=False)).astype(np.int32)
        keep = oracle.keep_set_baseline(oracle.paper_params(policy=2, n_anchor=n_anchor), pos,
                                        budget)
        K = budget // 2 + budget // 4
        A = int(np.searchsorted(pos, n_anchor))
        w = max(0, K - A)
        ref = list(range(A)) + list(range(max(A, L - w), L))
        assert keep.tolist() == ref


def test_h2o_score_order_and_exact_sums():
    # integer-valued floats: the float32 sum is the exact integer sum
    acc = np.arange(2 * 3 * 5, dtype=np.float32).reshape(2, 3, 5)
    np.testing.assert_array_equal(oracle.h2o_score(acc), acc.sum(axis=(0, 1)))
    # one non-zero entry per slot: the score is that entry, bit for bit
    acc = np.zeros((4, 2, 3), np.float32)
    acc[2, 1] = [0.1, 1e-30, 7.25]
    np.testing.assert_array_equal(oracle.h2o_score(acc), acc[2, 1])
    # the order of additions is layer by layer, head by head: 1e8 + 1 rounds back to 1e8, so the
    # ascending order gives 0 where any order that adds 1 last gives 1
    acc = np.zeros((3, 1, 1), np.float32)
    acc[:, 0, 0] = [1e8, 1.0, -1e8]
    assert oracle.h2o_score(acc)[0] == 0.0
    acc[:, 0, 0] = [1e8, -1e8, 1.0]
    assert oracle.h2o_score(acc)[0] == 1.0


def test_keep_set_cap_leaves_room_for_the_append():
    """The keep set never exceeds budget - 1 slots for any parameters (the next append must fit).
    When the anchors, the recent budget R >> l and the sparse budget do not fit, they are cut in
    that order of priority: no recent slot is dropped for a sparse one, no anchor for either, and
    the anchors kept are the earliest. Where they fit, the set is the closed form above."""
    rng = np.random.default_rng(11)
    for trial in range(1500):
        budget = int(rng.integers(1, 90))
        na = int(rng.choice([0, 4, 32, 64]))
        rd, sd = int(rng.choice([1, 2, 4])), int(rng.choice([1, 2, 3]))
        p = oracle.paper_params(n_anchor=na, recent_div=rd, sparse_div=sd)
        L = int(rng.integers(1, budget + 2))
        pos = np.sort(rng.choice(int(rng.integers(L, 3 * L + 80)), L, replace=False)).astype(np.int32)
        t = int(pos[-1])
        R = budget // rd
        span_lo = -1 if rng.random() < 0.4 else int(rng.integers(max(0, t - 2 * R), t + 1))
        level = int(rng.integers(0, 4))
        keep = oracle.keep_set(p, pos, budget, span_lo, level)
        cap = max(0, budget - 1)
        assert len(keep) <= cap, (trial, len(keep), budget)
        assert np.all(np.diff(keep) > 0)
        anchors = [j for j in range(L) if pos[j] < na]
        recent = [j for j in range(L) if pos[j] >= na and pos[j] >= t - R + 1
                  and (span_lo < 0 or pos[j] < span_lo)]
        middle = [j for j in range(L) if pos[j] >= na and pos[j] < t - R + 1]
        k_a = [j for j in keep if j in set(anchors)]
        k_r = [j for j in keep if j in set(recent)]
        k_m = [j for j in keep if j in set(middle)]
        assert len(k_a) + len(k_r) + len(k_m) == len(keep)       # nothing else (I_bad dropped)
        assert k_a == anchors[:len(k_a)]                         # the earliest anchors
        assert k_r == recent[len(recent) - len(k_r):]            # the most recent clean slots
        if len(k_a) < len(anchors):
            assert not k_r and not k_m, trial                    # anchors come first
        if len(k_r) < min(R >> level, len(recent)):
            assert not k_m, trial                                # then the recent window
        S = budget // sd - na
        if na + max(0, S) + (R >> level) <= cap and rd == 4 and sd == 2:
            assert keep.tolist() == _closed_form(pos, budget, span_lo, level, n_anchor=na), trial


def test_baseline_keep_cap_leaves_room_for_the_append():
    """H2O and StreamingLLM keep at most budget - 1 slots for any divisors: their size
    B/sparse_div + B/recent_div is capped, the most recent slots (H2O) and the earliest anchors
    (StreamingLLM) first."""
    rng = np.random.default_rng(12)
    for trial in range(600):
        budget = int(rng.integers(1, 70))
        rd, sd = int(rng.choice([1, 2, 4])), int(rng.choice([1, 2, 3]))
        na = int(rng.choice([0, 8, 40]))
        L = int(rng.integers(1, budget + 2))
        pos = np.sort(rng.choice(3 * L + 50, L, replace=False)).astype(np.int32)
        K = min(budget // sd + budget // rd, max(0, budget - 1))
        for policy in (1, 2):
            p = oracle.paper_params(policy=policy, recent_div=rd, sparse_div=sd, n_anchor=na)
            score = rng.integers(0, 5, L).astype(np.float32)
            keep = oracle.keep_set_baseline(p, pos, budget, score)
            assert len(keep) <= max(0, budget - 1) and len(keep) == min(K, L), (trial, policy)
            if policy == 1:
                r = min(budget // rd, L, K)
                assert set(range(L - r, L)) <= set(keep.tolist())
            else:
                A = int(np.searchsorted(pos, na))
                a = min(A, K)
                assert keep.tolist()[:a] == list(range(a))
                assert keep.tolist()[a:] == list(range(L - (len(keep) - a), L))
