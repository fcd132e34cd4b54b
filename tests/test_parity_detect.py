"""GPU parity of lg_detect_loop against the oracle's monitor (Sec. 5.2, Eq. (8)/(9), App. B.2).

Every decision field (votes, gates, distinct count, LZ cost, novelty, P*, span, trigger, level,
interventions) and the carried state must be bit-identical, step after step, on token streams
that plant loops of many periods (short, mid, long, nested, interrupted), random text over large
and tiny alphabets, with a circular token ring smaller than the stream, several t0 and parameter
sets. Confidence values are inputs here (including the exact float threshold).
"""
import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu


def _streams(n_total, rng):
    out = []
    fresh = iter(range(100000, 10 ** 7))

    def loop(P, length):
        u = [next(fresh) for _ in range(P)]
        return [u[i % P] for i in range(length)]

    out.append(list(rng.integers(0, 32000, n_total)))                    # i.i.d. text
    out.append(list(rng.integers(0, 3, n_total)))                        # tiny alphabet
    out.append(list(rng.integers(0, 2, n_total)))
    for P in [1, 2, 4, 12, 28, 29, 40, 51, 52, 100, 200, 256, 300]:
        s0 = int(rng.integers(20, 400))
        out.append(list(rng.integers(0, 32000, s0)) + loop(P, n_total - s0))
    motif = [next(fresh) for _ in range(16)]
    unit = motif * 12 + [next(fresh) for _ in range(8)]
    out.append(list(rng.integers(0, 32000, 300)) + [unit[i % 200] for i in range(n_total - 300)])
    # a loop that breaks for a while and resumes
    a = loop(7, 500)
    s = list(rng.integers(0, 32000, 100)) + a + list(rng.integers(0, 32000, 150))
    out.append(s + loop(7, n_total - len(s)))
    # repeated fragment with a one-token mutation every 50 tokens
    base = loop(9, n_total)
    for i in range(0, n_total, 50):
        base[i] = next(fresh)
    out.append(base)
    assert all(len(s) >= n_total for s in out)
    return [np.asarray(s[:n_total], np.int32) for s in out]


def _run(params, n_total=2600, ring=2048, phases=((1, 220), (1900, 2060)), t0s=None, seed=0,
         conf_mode="mixed"):
    from paper_2604_10044_amd import lg
    rng = np.random.default_rng(seed)
    ys = _streams(n_total, rng)
    B = len(ys)
    t0 = np.zeros(B, np.int32) if t0s is None else np.asarray(t0s(B), np.int32)
    dev = torch.device("cuda")
    gp = lg.params_from_dict(params)
    state = torch.zeros(B, lg.STATE_INTS, dtype=torch.int32, device=dev)
    dec = torch.zeros(B, lg.DECISION_INTS, dtype=torch.int32, device=dev)
    conf_d = torch.zeros(B, dtype=torch.float32, device=dev)
    t0_d = torch.from_numpy(t0).to(dev)
    dets = [oracle.Detector(params) for _ in range(B)]
    steps_checked = 0
    n_trig = 0
    for lo, hi in phases:
        for k in range(lo, hi):
            n = t0 + k                                   # per-sequence stream length
            if conf_mode == "mixed":
                conf = np.where(rng.random(B) < 0.7, rng.uniform(0.91, 1.0, B), rng.uniform(0, 0.95, B))
                conf[rng.random(B) < 0.05] = np.float32(0.9)
            else:
                conf = np.zeros(B)
            conf = conf.astype(np.float32)
            ring_h = np.zeros((B, ring), np.int32)
            for b in range(B):
                idx = np.arange(max(0, n[b] - ring), n[b])
                ring_h[b, idx % ring] = ys[b][idx]
            conf_d.copy_(torch.from_numpy(conf))
            lg.lg_detect_loop(gp, torch.from_numpy(ring_h).to(dev), ring,
                              torch.from_numpy((n - 1).astype(np.int32)).to(dev), t0_d, conf_d,
                              state, dec)
            d_h = dec.cpu().numpy()
            s_h = state.cpu().numpy()
            assert np.all(conf_d.cpu().numpy() == 0)     # consumed
            for b in range(B):
                ref = dets[b].step(ys[b], int(t0[b]), int(n[b]), float(conf[b]))
                got = {f: int(d_h[b, i]) for i, f in enumerate(lg.DECISION_FIELDS)}
                assert got == ref, (b, int(n[b]), {f: (got[f], ref[f]) for f in ref if got[f] != ref[f]})
                st = dets[b].state_dict()
                gst = {f: int(s_h[b, i]) for i, f in enumerate(lg.STATE_FIELDS)}
                assert gst == st, (b, int(n[b]))
                n_trig += ref["trigger"]
                steps_checked += 1
    return steps_checked, n_trig


def test_detect_parity_paper_params():
    steps, trig = _run(oracle.paper_params())
    assert trig > 0


def test_detect_parity_small_window_and_t0():
    p = oracle.paper_params(W=64, cooldown=16, t_min=32)
    _run(p, t0s=lambda B: np.arange(B) * 7 % 50, phases=((1, 150), (1500, 1600)), seed=1)


def test_detect_parity_max_window_horizon():
    p = oracle.paper_params(W=512, rep_horizon=2048, rep_pmax=512, nov_span=200, nov_ngram=3)
    _run(p, n_total=3000, ring=2600, phases=((1, 60), (2500, 2600)), seed=2)


@pytest.mark.parametrize("over", [dict(cr_interval=5), dict(mode=1), dict(mode=2), dict(K=1),
                                  dict(K=3), dict(rep_min_copies=2, rep_min_len=8, rep_debounce=1)])
def test_detect_parity_variants(over):
    _run(oracle.paper_params(**over), phases=((1, 120), (2000, 2050)), seed=3)


def test_detect_parity_minimum_ring():
    """The token ring at its minimum length max(W, rep_horizon): every token the monitor reads is
    still in the ring (the oracle reads the whole stream, so a read past the documented span would
    see an overwritten token and disagree)."""
    _run(oracle.paper_params(), ring=1024, phases=((1, 80), (1900, 2000)), seed=4)
    _run(oracle.paper_params(W=512, rep_horizon=256, rep_pmax=200), ring=512,
         phases=((1, 60), (2000, 2060)), seed=5)


@pytest.mark.parametrize("i", range(8))
def test_detect_parity_random_params(i):
    """Seeded random parameter sets over the whole valid range (window 8-512, horizon up to 2048,
    periods up to 512, n-gram order up to 16, thresholds, debounces, level cap, modes), the ring
    a little above its minimum."""
    rng = np.random.default_rng(5000 + i)
    ri = lambda lo, hi: int(rng.integers(lo, hi + 1))
    W, H = ri(8, 512), ri(1, 2048)
    p = oracle.paper_params(
        W=W, rep_horizon=H, rep_pmax=ri(1, 512), nov_ngram=ri(1, 16), nov_span=ri(1, 300),
        t_min=ri(0, 100), cooldown=ri(0, 64), streak_min=ri(0, 10), stall_min=ri(0, 8),
        cr_interval=ri(1, 8), rep_min_copies=ri(1, 5), rep_min_len=ri(0, 64), rep_debounce=ri(0, 6),
        level_max=ri(0, 5), retrigger_window=ri(0, 128), K=ri(0, 3), ttr_num=ri(0, 3), ttr_den=ri(1, 10),
        cr_num=ri(0, 5), cr_den=ri(1, 30), nov_num=ri(0, 3), nov_den=ri(1, 60), mode=ri(0, 2))
    _run(p, ring=max(W, H) + ri(0, 64), phases=((1, 90), (2000, 2050)), seed=10 + i,
         t0s=lambda B: rng.integers(0, 40, B))


def _forced_state(rng, p, n):
    """Detector counters written directly, biased to the boundaries of the rule: cooldown and
    re-trigger window distances, the level cap, the streak / stall / debounce thresholds, a held
    compression value."""
    pick = lambda opts: int(opts[int(rng.integers(0, len(opts)))])
    d = pick([1, p["cooldown"] - 1, p["cooldown"], p["cooldown"] + 1, p["retrigger_window"],
              p["retrigger_window"] + 1, int(rng.integers(1, 400))])
    st = dict(streak=pick([0, p["streak_min"] - 1, p["streak_min"], int(rng.integers(0, 50))]),
              stall=pick([0, p["stall_min"] - 1, p["stall_min"], int(rng.integers(0, 50))]),
              rep=pick([0, p["rep_debounce"] - 1, p["rep_debounce"], int(rng.integers(0, 50))]),
              n_int=pick([0, 1, int(rng.integers(2, 9))]),
              n_last=max(0, n - d),
              level=pick([0, p["level_max"] - 1, p["level_max"]]),
              cr_valid=pick([0, 1]), cr_cost=int(rng.integers(1, 300)), cr_m=int(rng.integers(1, 300)))
    if st["n_int"] == 0:
        st["n_last"], st["level"] = 0, 0
    return st


@pytest.mark.parametrize("cr_interval", [1, 4])
def test_detect_forced_states(cr_interval):
    """One step from counters written directly into the state (the tail-run cache left empty, so
    the kernel recomputes it): decisions and the updated counters equal the oracle's for 40 rounds
    of random stream lengths and boundary-biased states (level at its cap, cooldown and re-trigger
    distances at their edges, held compression values)."""
    from paper_2604_10044_amd import lg
    rng = np.random.default_rng(90 + cr_interval)
    p = oracle.paper_params(cr_interval=cr_interval)
    ys = _streams(2600, rng)
    B = len(ys)
    ring = 2048
    dev = torch.device("cuda")
    gp = lg.params_from_dict(p)
    dec = torch.zeros(B, lg.DECISION_INTS, dtype=torch.int32, device=dev)
    t0_d = torch.zeros(B, dtype=torch.int32, device=dev)
    n_trig = 0
    for _ in range(40):
        n = rng.integers(2, 2600, B).astype(np.int64)
        conf = np.where(rng.random(B) < 0.5, np.float32(0.9), rng.uniform(0.5, 1.0, B)).astype(np.float32)
        state_h = np.zeros((B, lg.STATE_INTS), np.int32)
        ring_h = np.zeros((B, ring), np.int32)
        refs, dets = [], []
        for b in range(B):
            st = _forced_state(rng, p, int(n[b]))
            for i, f in enumerate(lg.STATE_FIELDS):
                state_h[b, i] = st[f]
            det = oracle.Detector(p)
            for f in oracle.STATE_FIELDS:
                setattr(det.state, f, st[f])
            refs.append(det.step(ys[b], 0, int(n[b]), float(conf[b])))
            dets.append(det)
            idx = np.arange(max(0, n[b] - ring), n[b])
            ring_h[b, idx % ring] = ys[b][idx]
        state = torch.from_numpy(state_h).to(dev)
        conf_d = torch.from_numpy(conf).to(dev)
        lg.lg_detect_loop(gp, torch.from_numpy(ring_h).to(dev), ring,
                          torch.from_numpy((n - 1).astype(np.int32)).to(dev), t0_d, conf_d, state, dec)
        d_h, s_h = dec.cpu().numpy(), state.cpu().numpy()
        for b in range(B):
            got = {f: int(d_h[b, i]) for i, f in enumerate(lg.DECISION_FIELDS)}
            assert got == refs[b], (b, int(n[b]), {f: (got[f], refs[b][f]) for f in refs[b] if got[f] != refs[b][f]})
            gst = {f: int(s_h[b, i]) for i, f in enumerate(lg.STATE_FIELDS)}
            assert gst == dets[b].state_dict(), (b, int(n[b]))
            n_trig += refs[b]["trigger"]
    assert n_trig > 0
