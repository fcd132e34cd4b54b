"""End-to-end parity of the guarded decode loop (GPU GuardedDecoder vs the oracle's
SequenceOracle): per step, every decision field, the cache length and positions; the confidence
within 2e-4; at the end the compacted K/V caches bit for bit and acc within 1e-4 relative.

Float decides an integer only through conf > 0.9 and, under the H2O policy, through the ranking
of the accumulated scores; every oracle conf is checked to sit more than 0.018 away from the
threshold, and every H2O selection to separate the last kept from the first evicted score by at
least 1e-4 relative (the GPU's errors are ~1e-6), so no decision rests on a tie.
"""
import os

import numpy as np
import pytest
import torch

import oracle
from oracle.trajectory import SequenceOracle

pytestmark = pytest.mark.gpu
THREADS = min(16, os.cpu_count() or 1)
# Every followed sequence keeps its oracle confidence this far from the 0.9 threshold at every step
# (the margin rule of tests/golden/conf_margins.py, checked there on the CPU): far above the 2e-4
# confidence tolerance, so the float comparison takes the same decision on both paths.
MARGIN = 0.018
# Relative gap between the last kept and the first evicted H2O score that a selection must clear
# (the scores are float32 sums that the two paths form in the same order).
H2O_MARGIN = 1e-4


def _compare_traj(wl, b_list, steps=None, params=None, check_every=1):
    from paper_2604_10044_amd import lg
    from paper_2604_10044_amd.decoder import GuardedDecoder
    steps = wl.steps if steps is None else steps
    p = oracle.paper_params() if params is None else params
    dec = GuardedDecoder(wl, params=p)
    dec.prefill()
    dec.load_steps(steps)
    ors = {b: SequenceOracle(wl, b, params=p, threads=THREADS) for b in b_list}
    for b in b_list:
        np.testing.assert_array_equal(dec.prefill_positions[b], ors[b].pos)
    trig = 0
    events = []
    for s in range(steps):
        for l in range(dec.L):
            dec.attend_layer(s, l)
        conf_gpu = dec.conf.cpu().numpy()
        dec.detect_prune(s)   # detector and keep set in one launch
        d_gpu = dec.decisions()
        len_gpu = dec.len.cpu().numpy()
        for b in b_list:
            ref = ors[b].step(s)
            assert abs(ref["conf"] - float(np.float32(0.9))) > MARGIN, ("conf on the threshold", b, s)
            if "h2o_margin" in ref:
                assert ref["h2o_margin"] > H2O_MARGIN, ("H2O selection on a near-tie", b, s)
                events.append(s)
            assert abs(conf_gpu[b] - ref["conf"]) <= 2e-4, (b, s, conf_gpu[b], ref["conf"])
            got = d_gpu[b]
            diff = {f: (got[f], ref[f]) for f in lg.DECISION_FIELDS if got[f] != ref[f]}
            assert not diff, (b, s, diff)
            assert len_gpu[b] == ors[b].len, (b, s)
            trig += ref["trigger"]
        if s % check_every == 0 or s == steps - 1:
            pos_gpu = dec.pos.cpu().numpy()
            for b in b_list:
                np.testing.assert_array_equal(pos_gpu[b, :ors[b].len], ors[b].pos)
    # caches after the whole run
    for b in b_list:
        n = ors[b].len
        for l in range(dec.L):
            Kg = dec.K[l][b, :, :n].float().cpu().numpy()
            Vg = dec.V[l][b, :, :n].float().cpu().numpy()
            np.testing.assert_array_equal(Kg, ors[b].K[l, :, :n])
            np.testing.assert_array_equal(Vg, ors[b].V[l, :, :n])
            ag = dec.acc[l][b, :, :n].cpu().numpy()
            ar = ors[b].acc[l, :, :n]
            assert np.all(np.abs(ag - ar) <= 1e-4 * np.maximum(1, np.abs(ar))), (b, l)
    return trig, ors, events


def test_tiny_trajectory():
    from paper_2604_10044_amd.synth import tiny
    trig, ors, _ = _compare_traj(tiny(), [0])
    h = ors[0].history
    assert trig == 0 and all(d["period"] == 12 and d["span_lo"] == 160 for d in h[3:])


def test_tiny_small_window_triggers():
    from paper_2604_10044_amd.synth import tiny
    trig, _, _ = _compare_traj(tiny(steps=80, period=4), [0], params=oracle.paper_params(W=64))
    assert trig >= 2


def test_qwen15b_trajectory():
    from paper_2604_10044_amd.synth import qwen15b
    _compare_traj(qwen15b(steps=256), [0], check_every=8)


def test_llama7b_bench_config_sampled_sequences():
    """The benchmark configuration (batch 32 on the GPU); the oracle follows two looping and two
    i.i.d. sequences through all 128 steps."""
    from paper_2604_10044_amd.synth import llama7b
    _compare_traj(llama7b(), [0, 1, 2, 3], check_every=16)


@pytest.mark.parametrize("policy", [oracle.POLICY_H2O, oracle.POLICY_STREAMING])
def test_baseline_policy_trajectory(policy):
    """The H2O and StreamingLLM baselines (Sec. 6.1) on the 1.5B-shaped sequence (4 layers): the
    prefill leaves 768 slots, so the cache reaches its 1024 budget at steps 255 and 511 and the
    policy's keep set (ranked by the accumulated scores for H2O) prunes it. Seed 6 is one whose
    two H2O selections clear the tie margin (the oracle's gaps are 9e-4 and 3e-4 relative)."""
    from paper_2604_10044_amd.synth import qwen15b
    p = oracle.paper_params(policy=policy)
    _, ors, events = _compare_traj(qwen15b(steps=520, n_layers=4, seed=6), [0], params=p,
                                   check_every=8)
    assert [s for s, d in enumerate(ors[0].history) if d["new_len"] >= 0] == [255, 511]
    if policy == oracle.POLICY_H2O:
        assert events == [255, 511]


@pytest.mark.parametrize("mode", [1, 2])
def test_ablation_mode_trajectory(mode):
    """The Table 3 ablations through the whole loop on the 1.5B-shaped sequence (4 layers, 160
    steps): always-on pruning (mode 1) triggers whenever warmup and cooldown allow; the
    confidence-only rule (mode 2) triggers on the streak alone (a streak of 1 here: the synthetic
    confidence never stays above 0.9 for 6 steps; seed 6 keeps every confidence >= 0.095 from the
    threshold). Both trigger every ~33 steps, so the level escalates to its cap and the recent
    budget shrinks with it. Decisions, lengths, positions and the final caches match the oracle
    step by step."""
    from paper_2604_10044_amd.synth import qwen15b
    if mode == 1:
        p, wl = oracle.paper_params(mode=1), qwen15b(steps=160, n_layers=4)
    else:
        p, wl = oracle.paper_params(mode=2, streak_min=1), qwen15b(steps=160, n_layers=4, seed=6)
    trig, ors, _ = _compare_traj(wl, [0], params=p, check_every=4)
    levels = [d["level"] for d in ors[0].history if d["trigger"]]
    assert trig >= 3 and max(levels) == p["level_max"], levels


def test_8b_long_context_trajectory_sampled():
    """8B-shaped long context (batch 8, 32/8 heads, budget 4096) with 4 of its layers: the nested
    period-16-in-200 loop triggers from step 250 on with escalating levels; sequences 0 and 5
    are followed by the oracle for 300 steps."""
    from paper_2604_10044_amd.synth import llama8b_long
    trig, ors, _ = _compare_traj(llama8b_long(steps=300, n_layers=4), [0, 5], check_every=16)
    assert trig >= 4
    assert any(d["level"] >= 1 for d in ors[0].history)


def test_ragged_trajectory_sampled():
    """Ragged stress (batch 64, budgets 512/2048/8192 in one cap-8192 cache) with 2 of its layers:
    sequences with overflow events (1), repeated triggers at periods 12 and 2 (20, 47), a long
    context at budget 8192 (9) and a short one below its budget (4)."""
    from paper_2604_10044_amd.synth import ragged
    trig, ors, _ = _compare_traj(ragged(steps=256, n_layers=2), [1, 20, 47, 9, 4], check_every=16)
    assert trig >= 10
    assert [s for s, d in enumerate(ors[1].history) if d["new_len"] >= 0] == [127, 255]
