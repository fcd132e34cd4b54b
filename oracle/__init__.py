"""CPU oracle of the LoopGuard guarded-decode step (arXiv 2604.10044).

TEST INFRASTRUCTURE ONLY: only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package. It shares no code with the GPU path (``paper_2604_10044_amd``)
and never imports it; the two meet only in the seeded input generator.

The arithmetic lives in ``lg_oracle.c`` (plain C, double precision); this module is a thin ctypes
wrapper plus the paper's hyperparameters. ``trajectory.py`` strings the pieces together in the
order of one guarded decode step.

Parity notes: the compression-ratio and novelty readings are pinned only by their closed forms and
invariants; their calibration against the paper's unnamed compressor and undefined novelty score
is parity unpinned (the paper prints no worked example).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Dict, Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "lg_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")


def build(force: bool = False) -> str:
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-ffp-contract=off", "-shared", "-fPIC", "-o", tmp,
                               _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


PARAM_FIELDS = ["W", "K", "n_anchor", "t_min", "cooldown", "streak_min", "stall_min",
                "cr_interval", "nov_ngram", "nov_span", "rep_pmax", "rep_horizon",
                "rep_min_copies", "rep_min_len", "rep_debounce", "level_max", "retrigger_window",
                "recent_div", "sparse_div", "ttr_num", "ttr_den", "cr_num", "cr_den", "nov_num",
                "nov_den"]
STATE_FIELDS = ["streak", "stall", "rep", "n_int", "n_last", "level", "cr_valid", "cr_cost", "cr_m"]
DECISION_FIELDS = ["trigger", "warn", "votes", "stall_gate", "tailrep_gate", "n", "distinct",
                   "lz_cost", "novel", "nov_r", "period", "span_lo", "level", "n_int"]


POLICY_LOOPGUARD, POLICY_H2O, POLICY_STREAMING = 0, 1, 2


class Params(ctypes.Structure):
    _fields_ = [(f, ctypes.c_int32) for f in PARAM_FIELDS] + [
        ("conf_threshold", ctypes.c_float), ("mode", ctypes.c_int32), ("policy", ctypes.c_int32)]


class State(ctypes.Structure):
    _fields_ = [(f, ctypes.c_int32) for f in STATE_FIELDS]


class Decision(ctypes.Structure):
    _fields_ = [(f, ctypes.c_int32) for f in DECISION_FIELDS]


def paper_params(**over) -> Dict[str, float]:
    """The paper's constants (Sec. 6.1: W=256, K=2, 32 anchors; App. B.2: theta_ttr=0.2,
    theta_cr=0.12, theta_conf=0.9, theta_streak=6, theta_nov=0.02, theta_stall=4, t_min=64,
    cooldown 32) and the readings for what it leaves open."""
    p = dict(W=256, K=2, n_anchor=32, t_min=64, cooldown=32, streak_min=6, stall_min=4,
             cr_interval=1, nov_ngram=4, nov_span=64, rep_pmax=256, rep_horizon=1024,
             rep_min_copies=3, rep_min_len=32, rep_debounce=4, level_max=3, retrigger_window=64,
             recent_div=4, sparse_div=2, ttr_num=1, ttr_den=5, cr_num=3, cr_den=25, nov_num=1,
             nov_den=50, conf_threshold=0.9, mode=0, policy=POLICY_LOOPGUARD)
    p.update(over)
    return p


def make_params(d: Dict[str, float]) -> Params:
    return Params(*[int(d[f]) for f in PARAM_FIELDS], float(d["conf_threshold"]), int(d["mode"]),
                  int(d.get("policy", POLICY_LOOPGUARD)))


_lib_handle = None


def lib():
    global _lib_handle
    if _lib_handle is None:
        if not os.path.exists(_LIB):
            build()
        L = ctypes.CDLL(_LIB)
        vp, i32 = ctypes.c_void_p, ctypes.c_int32
        L.or_attend_group.restype = None
        L.or_attend_group.argtypes = [i32, i32, i32, vp, vp, vp, vp, i32, i32, vp, vp, vp, vp]
        L.or_distinct.restype = i32
        L.or_distinct.argtypes = [vp, i32, i32]
        L.or_lz_cost.restype = i32
        L.or_lz_cost.argtypes = [vp, i32, i32, i32]
        L.or_novelty.restype = i32
        L.or_novelty.argtypes = [vp, i32, i32, i32, i32, ctypes.POINTER(i32)]
        L.or_tail_align.restype = None
        L.or_tail_align.argtypes = [vp, i32, i32, i32, i32, vp]
        L.or_tail_best.restype = i32
        L.or_tail_best.argtypes = [vp, i32, i32, i32, i32, i32, i32, ctypes.POINTER(i32)]
        L.or_detect_step.restype = None
        L.or_detect_step.argtypes = [ctypes.POINTER(Params), vp, i32, i32, ctypes.c_double,
                                     ctypes.POINTER(State), ctypes.POINTER(Decision)]
        L.or_keep_set.restype = i32
        L.or_keep_set.argtypes = [ctypes.POINTER(Params), vp, i32, i32, i32, i32, vp]
        L.or_h2o_score.restype = None
        L.or_h2o_score.argtypes = [i32, i32, i32, i32, vp, vp]
        L.or_keep_set_baseline.restype = i32
        L.or_keep_set_baseline.argtypes = [ctypes.POINTER(Params), vp, i32, i32, vp, vp]
        _lib_handle = L
    return _lib_handle


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _f32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.float32))


# ---------------------------------------------------------------------------------------------
def attend_group(q, K, V, pos, t: int, w_s: int):
    """Eq. (1) for the G query heads of one KV head. q [G][d], K/V [n][d], pos [n].
    Returns (o [G][d], lse [G], sigma [G], alpha_sum [n]) in float64."""
    q, K, V, pos = _f32(q), _f32(K), _f32(V), _i32(pos)
    G, d = q.shape
    n = K.shape[0]
    o = np.zeros((G, d)); lse = np.zeros(G); sg = np.zeros(G); asum = np.zeros(max(n, 1))
    lib().or_attend_group(n, G, d, q.ctypes.data, K.ctypes.data, V.ctypes.data, pos.ctypes.data,
                          int(t), int(w_s), o.ctypes.data, lse.ctypes.data, sg.ctypes.data,
                          asum.ctypes.data)
    return o, lse, sg, asum[:n]


def distinct(y, lo: int, hi: int) -> int:
    y = _i32(y)
    return int(lib().or_distinct(y.ctypes.data, lo, hi))


def lz_cost(y, lo: int, hi: int, min_match: int = 3) -> int:
    y = _i32(y)
    return int(lib().or_lz_cost(y.ctypes.data, lo, hi, min_match))


def novelty(y, w0: int, n: int, g: int = 4, span: int = 64):
    y = _i32(y)
    r = ctypes.c_int32(0)
    nov = lib().or_novelty(y.ctypes.data, w0, n, g, span, ctypes.byref(r))
    return int(nov), int(r.value)


def tail_align(y, t0: int, n: int, pmax: int = 256, H: int = 1024) -> np.ndarray:
    y = _i32(y)
    L = np.zeros(pmax + 1, np.int32)
    lib().or_tail_align(y.ctypes.data, t0, n, pmax, H, L.ctypes.data)
    return L


def tail_best(y, t0: int, n: int, pmax: int = 256, H: int = 1024, copies: int = 3,
              min_len: int = 32):
    y = _i32(y)
    T = ctypes.c_int32(0)
    P = lib().or_tail_best(y.ctypes.data, t0, n, pmax, H, copies, min_len, ctypes.byref(T))
    return int(P), int(T.value)


class Detector:
    """The monitor of one sequence (Sec. 5.2), stepping over a token stream."""

    def __init__(self, params: Dict[str, float]):
        self.params = dict(params)
        self._p = make_params(self.params)
        self.state = State()

    def step(self, y, t0: int, n: int, conf: float) -> Dict[str, int]:
        y = _i32(y)
        assert len(y) >= n
        dec = Decision()
        lib().or_detect_step(ctypes.byref(self._p), y.ctypes.data, int(t0), int(n), float(conf),
                             ctypes.byref(self.state), ctypes.byref(dec))
        return {f: int(getattr(dec, f)) for f in DECISION_FIELDS}

    def state_dict(self) -> Dict[str, int]:
        return {f: int(getattr(self.state, f)) for f in STATE_FIELDS}


def keep_set(params: Dict[str, float], pos, budget: int, span_lo: int = -1,
             level: int = 0) -> np.ndarray:
    """Eq. (10)/(11): kept slot indices (ascending) of one sequence."""
    pos = _i32(pos)
    keep = np.zeros(max(1, len(pos)), np.int32)
    p = make_params(params)
    n = lib().or_keep_set(ctypes.byref(p), pos.ctypes.data, len(pos), int(budget), int(span_lo),
                          int(level), keep.ctypes.data)
    return keep[:n].copy()


def h2o_score(acc) -> np.ndarray:
    """H2O importance of each slot of one sequence: acc [L][H][n] summed over layers and KV heads in
    float32, in ascending layer then head order (the heavy-hitter score of Sec. 6.1's H2O)."""
    acc = _f32(acc)
    L, H, n = acc.shape
    score = np.zeros(max(n, 1), np.float32)
    lib().or_h2o_score(L, H, n, n, acc.ctypes.data, score.ctypes.data)
    return score[:n].copy()


def keep_set_baseline(params: Dict[str, float], pos, budget: int, score=None) -> np.ndarray:
    """Kept slot indices (ascending) of a sequence at its budget under the H2O or StreamingLLM
    policy (params["policy"]); score [n] float32 is the H2O importance (ignored by StreamingLLM,
    zeros when None)."""
    pos = _i32(pos)
    n = len(pos)
    sc = _f32(np.zeros(max(n, 1)) if score is None else score)
    assert len(sc) >= n
    keep = np.zeros(max(1, n), np.int32)
    p = make_params(params)
    m = lib().or_keep_set_baseline(ctypes.byref(p), pos.ctypes.data, n, int(budget),
                                   sc.ctypes.data, keep.ctypes.data)
    return keep[:m].copy()
