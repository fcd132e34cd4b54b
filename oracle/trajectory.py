"""The oracle's guarded decode of one sequence, in the order of one LoopGuard step.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

One step at newest position t (Sec. 3.1, Sec. 5.1-5.3):
  1. append the step's key/value row at position t to every layer's cache (the query attends to
     its own key, standard decoding);
  2. attend, every layer and head (Eq. (1)); accumulate the H2O importance; conf = the largest
     suffix attention mass over layers and heads (stand-in for p_max);
  3. the stream now holds n = t + 1 tokens; run the monitor (Eq. (8), Eq. (9));
  4. on a trigger build I_keep with I_bad and level l (Eq. (10), Eq. (11)); otherwise, when the
     cache has reached its budget, build I_keep with I_bad empty and l = 0; gather every layer's
     rows with I_keep (index selection across layers, Sec. 5.3). Under a baseline policy (H2O,
     StreamingLLM; Sec. 6.1) only the budget prunes, with that policy's keep set; the H2O score
     is the float32 sum over layers and KV heads of the accumulated importance.
Prefill: a context of ctx >= budget tokens is reduced once by the same keep rule at t = ctx - 1
(I_bad empty, l = 0); only the kept rows exist afterwards and their importance starts at 0.

Inputs come from the seeded generator module; nothing here reads the GPU path.
"""
from __future__ import annotations

from concurrent.futures import ThreadPoolExecutor
from typing import Dict, List, Optional

import numpy as np

from . import (POLICY_H2O, POLICY_LOOPGUARD, Detector, attend_group, h2o_score, keep_set,
               keep_set_baseline, paper_params)

_POOL: Optional[ThreadPoolExecutor] = None


def _pool(threads: int) -> ThreadPoolExecutor:
    global _POOL
    if _POOL is None or _POOL._max_workers != threads:
        _POOL = ThreadPoolExecutor(max_workers=threads)
    return _POOL


def prefill_positions(params: Dict[str, float], ctx: int, budget: int) -> np.ndarray:
    """Positions left by reducing a context of ctx tokens to the budget (no attention history: the
    H2O scores are all zero)."""
    pos = np.arange(ctx, dtype=np.int32)
    if ctx >= budget:
        if int(params.get("policy", POLICY_LOOPGUARD)) == POLICY_LOOPGUARD:
            pos = pos[keep_set(params, pos, budget, -1, 0)]
        else:
            pos = pos[keep_set_baseline(params, pos, budget)]
    return pos


def h2o_margin(params: Dict[str, float], score: np.ndarray, L: int, budget: int) -> float:
    """Relative gap between the last kept and the first evicted H2O score (inf when the policy
    keeps every older slot or the two are tied exactly); decisions closer than the arithmetic's
    rounding are not unique."""
    rd, sd = int(params["recent_div"]), int(params["sparse_div"])
    R = min(budget // rd, L)
    older = L - R
    heavy = budget // sd + budget // rd - R
    if older <= heavy:
        return float("inf")
    s = np.sort(score[:older].astype(np.float64))[::-1]
    a, b = s[heavy - 1], s[heavy]
    if a == b:
        return float("inf")
    return float((a - b) / max(abs(a), 1e-30))


class SequenceOracle:
    """Guarded decode of sequence ``b`` of a workload (see the module docstring)."""

    def __init__(self, wl, b: int, params: Optional[Dict[str, float]] = None,
                 threads: int = 1, keep_outputs: bool = False):
        from paper_2604_10044_amd.synth import KIND_K, KIND_V, to_f32  # seeded inputs only
        self._KK, self._KV, self._f32 = KIND_K, KIND_V, to_f32
        self.wl, self.b = wl, b
        self.params = paper_params() if params is None else dict(params)
        self.threads = threads
        self.keep_outputs = keep_outputs
        self.ctx = int(wl.ctx[b])
        self.budget = int(wl.budget[b])
        self.R = self.budget // int(self.params["recent_div"])
        self.y = wl.tokens(b)
        self.pos = prefill_positions(self.params, self.ctx, self.budget)
        n = len(self.pos)
        L, H, d = wl.n_layers, wl.n_kv_heads, wl.head_dim
        cap = self.budget
        self.K = np.zeros((L, H, cap, d), np.float32)
        self.V = np.zeros((L, H, cap, d), np.float32)
        self.acc = np.zeros((L, H, cap), np.float64)
        if n:
            self.K[:, :, :n] = to_f32(wl.rows(KIND_K, 0, L, [b], self.pos[None, :]))[:, 0]
            self.V[:, :, :n] = to_f32(wl.rows(KIND_V, 0, L, [b], self.pos[None, :]))[:, 0]
        self.len = n
        self.det = Detector(self.params)
        self.history: List[Dict] = []
        self.outputs: List[Dict] = []

    # -------------------------------------------------------------------------------------
    def step(self, s: int, q_rows=None, k_rows=None, v_rows=None) -> Dict:
        from paper_2604_10044_amd.synth import KIND_Q
        wl, b = self.wl, self.b
        t = self.ctx + s
        L, H, G, d = wl.n_layers, wl.n_kv_heads, wl.group, wl.head_dim
        tp = np.array([[t]], np.int32)
        if q_rows is None:
            q_rows = self._f32(wl.rows(KIND_Q, 0, L, [b], tp))[:, 0, :, 0]   # [L][Hq][d]
            k_rows = self._f32(wl.rows(self._KK, 0, L, [b], tp))[:, 0, :, 0]  # [L][Hkv][d]
            v_rows = self._f32(wl.rows(self._KV, 0, L, [b], tp))[:, 0, :, 0]
        # 1. append
        j = self.len
        assert j < self.K.shape[2], "cache full before append"
        self.K[:, :, j] = k_rows
        self.V[:, :, j] = v_rows
        self.acc[:, :, j] = 0.0
        pos = np.append(self.pos, np.int32(t)).astype(np.int32)
        n_slots = j + 1

        # 2. attention and statistics
        def one(args):
            l, h = args
            return attend_group(q_rows[l, h * G:(h + 1) * G], self.K[l, h, :n_slots],
                                self.V[l, h, :n_slots], pos, t, self.R)

        jobs = [(l, h) for l in range(L) for h in range(H)]
        if self.threads > 1:
            res = list(_pool(self.threads).map(one, jobs))
        else:
            res = [one(a) for a in jobs]
        conf = 0.0
        outs = {}
        for (l, h), (o, lse, sg, asum) in zip(jobs, res):
            self.acc[l, h, :n_slots] += asum
            conf = max(conf, float(sg.max()))
            if self.keep_outputs:
                outs[(l, h)] = (o, lse, sg)
        self.pos = pos
        self.len = n_slots

        # 3. monitor
        n = t + 1
        dec = self.det.step(self.y, 0, n, conf)
        dec["conf"] = conf

        # 4. prune
        keep = None
        policy = int(self.params.get("policy", POLICY_LOOPGUARD))
        if policy == POLICY_LOOPGUARD:
            if dec["trigger"]:
                keep = keep_set(self.params, self.pos, self.budget, dec["span_lo"], dec["level"])
            elif self.len >= self.budget:
                keep = keep_set(self.params, self.pos, self.budget, -1, 0)
        elif self.len >= self.budget:
            score = None
            if policy == POLICY_H2O:
                score = h2o_score(self.acc[:, :, :self.len].astype(np.float32))
                dec["h2o_margin"] = h2o_margin(self.params, score, self.len, self.budget)
            keep = keep_set_baseline(self.params, self.pos, self.budget, score)
        dec["new_len"] = -1
        if keep is not None:
            m = len(keep)
            self.K[:, :, :m] = self.K[:, :, keep]
            self.V[:, :, :m] = self.V[:, :, keep]
            self.acc[:, :, :m] = self.acc[:, :, keep]
            self.pos = self.pos[keep]
            self.len = m
            dec["new_len"] = m
            dec["keep"] = keep
        self.history.append(dec)
        if self.keep_outputs:
            self.outputs.append(outs)
        return dec
