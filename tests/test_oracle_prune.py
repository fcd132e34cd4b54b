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
