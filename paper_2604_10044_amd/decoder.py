"""GuardedDecoder: device buffers for a batch of sequences and the per-step call sequence.

One guarded decode step (Sec. 5.1-5.3 of the paper) is
    for every layer: lg_decode_attend  (append + attention + suffix mass + H2O + conf)
    lg_detect_and_prune                (onset rule on the token tail and conf; commit the append;
                                        keep set + compaction if flagged)
all enqueued on one stream with no host synchronisation (the separate lg_detect_loop and
lg_prune_compact calls give the same results). PyTorch only allocates device memory
and provides the stream; every step of the path runs in liblg's kernels.

Inputs (the context cache, per-step q/k/v rows and tokens) come from the seeded workload
generator; they are produced on the host before timing and uploaded once.
"""
from __future__ import annotations

from typing import Dict, List, Optional

import numpy as np
import torch

from . import lg
from .synth import KIND_K, KIND_Q, KIND_V, Workload


def _to_torch(a: np.ndarray, bf16: bool, device) -> torch.Tensor:
    if bf16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


class GuardedDecoder:
    def __init__(self, wl: Workload, params: Optional[Dict] = None, device="cuda",
                 form: int = 0, max_split: int = 0, attend_flags: int = 0,
                 keep_layer_outputs: bool = False):
        """form / max_split / attend_flags: the attention kernel form, split length and flags of
        the test hook (lg_testing.h); 0 / 0 / 0 is what lg_decode_attend runs."""
        self.wl = wl
        self.device = torch.device(device)
        self.form = form
        self.max_split = max_split
        self.attend_flags = attend_flags
        self.params = lg.lg_guard_params_default()
        for k, v in (params or {}).items():
            setattr(self.params, k, v)
        B, L, Hq, Hkv, D = wl.batch, wl.n_layers, wl.n_q_heads, wl.n_kv_heads, wl.head_dim
        self.B, self.L, self.Hq, self.Hkv, self.D = B, L, Hq, Hkv, D
        self.cap = wl.cap
        self.bf16 = wl.dtype == "bf16"
        self.dt = torch.bfloat16 if self.bf16 else torch.float32
        dev = self.device
        self.K = [torch.zeros(B, Hkv, self.cap, D, dtype=self.dt, device=dev) for _ in range(L)]
        self.V = [torch.zeros(B, Hkv, self.cap, D, dtype=self.dt, device=dev) for _ in range(L)]
        self.acc = [torch.zeros(B, Hkv, self.cap, dtype=torch.float32, device=dev) for _ in range(L)]
        self.layers = [lg.layer_cache(self.K[l], self.V[l], self.acc[l], Hq) for l in range(L)]
        self.pos = torch.zeros(B, self.cap, dtype=torch.int32, device=dev)
        self.len = torch.zeros(B, dtype=torch.int32, device=dev)
        self.budget = torch.as_tensor(np.asarray(wl.budget, np.int32), device=dev)
        self.suffix_w = torch.div(self.budget, int(self.params.recent_div), rounding_mode="floor").to(torch.int32)
        self.t0 = torch.zeros(B, dtype=torch.int32, device=dev)
        self.state = torch.zeros(B, lg.STATE_INTS, dtype=torch.int32, device=dev)
        self.decision = torch.zeros(B, lg.DECISION_INTS, dtype=torch.int32, device=dev)
        self.conf = torch.zeros(B, dtype=torch.float32, device=dev)
        self.keep_idx = torch.zeros(B, self.cap, dtype=torch.int32, device=dev)
        self.new_len = torch.zeros(B, dtype=torch.int32, device=dev)
        ws = lg.lg_test_attend_workspace(self.layers[0], form, max_split)
        self.workspace = torch.empty(ws, dtype=torch.uint8, device=dev)
        self.init_workspace()
        nout = L if keep_layer_outputs else 1
        self.out = torch.zeros(nout, B, Hq, D, dtype=self.dt, device=dev)
        self.lse = torch.zeros(nout, B, Hq, dtype=torch.float32, device=dev)
        self.smass = torch.zeros(nout, B, Hq, dtype=torch.float32, device=dev)
        self.keep_layer_outputs = keep_layer_outputs
        ctx = np.asarray(wl.ctx, np.int64)
        self.ctx = ctx
        self.ring = int(max(ctx.max() + wl.steps, max(self.params.W, self.params.rep_horizon)))
        toks = np.zeros((B, self.ring), np.int32)
        for b in range(B):
            y = wl.tokens(b)
            toks[b, :len(y)] = y
        self.tokens = torch.from_numpy(toks).to(dev)
        self.t_steps = torch.as_tensor((ctx[None, :] + np.arange(wl.steps)[:, None]).astype(np.int32),
                                       device=dev)
        self.step_inputs = None
        self.prefill_positions: List[np.ndarray] = []

    # ------------------------------------------------------------------------------------------
    def prefill(self):
        """Reduce each context to the budget with the keep rule (on the GPU), then fill the cache
        with the generator's rows for the kept positions."""
        B, dev = self.B, self.device
        cmax = int(self.ctx.max())
        pos_full = torch.arange(cmax, dtype=torch.int32, device=dev).repeat(B, 1).contiguous()
        len_full = torch.as_tensor(self.ctx.astype(np.int32), device=dev)
        kidx = torch.zeros(B, cmax, dtype=torch.int32, device=dev)
        nlen = torch.zeros(B, dtype=torch.int32, device=dev)
        lg.lg_prune_compact(self.params, B, cmax, [], pos_full, len_full, self.budget, None, None,
                            kidx, nlen)
        torch.cuda.synchronize()
        lens = len_full.cpu().numpy()
        P = pos_full.cpu().numpy()
        self.prefill_positions = [P[b, :lens[b]].copy() for b in range(B)]
        pos_h = np.zeros((B, self.cap), np.int32)
        for b in range(B):
            pos_h[b, :lens[b]] = P[b, :lens[b]]
        self.pos.copy_(torch.from_numpy(pos_h))
        self.len.copy_(torch.from_numpy(lens.astype(np.int32)))
        cnt = lens.astype(np.int32)
        chunk = max(1, 4 if self.L > 4 else self.L)
        for l0 in range(0, self.L, chunk):
            l1 = min(self.L, l0 + chunk)
            kr = self.wl.rows(KIND_K, l0, l1, range(B), pos_h, cnt)
            vr = self.wl.rows(KIND_V, l0, l1, range(B), pos_h, cnt)
            for l in range(l0, l1):
                self.K[l].copy_(_to_torch(kr[l - l0], self.bf16, dev))
                self.V[l].copy_(_to_torch(vr[l - l0], self.bf16, dev))
        for a in self.acc:
            a.zero_()
        torch.cuda.synchronize()

    def load_steps(self, steps: Optional[int] = None):
        """Generate and upload q, k_new, v_new for decode steps [0, steps)."""
        S = self.wl.steps if steps is None else steps
        B = self.B
        pos = (self.ctx[:, None] + np.arange(S)[None, :]).astype(np.int32)   # [B][S]
        q = self.wl.rows(KIND_Q, 0, self.L, range(B), pos)        # [L][B][Hq][S][D]
        k = self.wl.rows(KIND_K, 0, self.L, range(B), pos)
        v = self.wl.rows(KIND_V, 0, self.L, range(B), pos)
        tr = lambda a: np.ascontiguousarray(a.transpose(3, 0, 1, 2, 4))   # [S][L][B][H][D]
        self.step_inputs = (_to_torch(tr(q), self.bf16, self.device),
                            _to_torch(tr(k), self.bf16, self.device),
                            _to_torch(tr(v), self.bf16, self.device))
        torch.cuda.synchronize()

    # ------------------------------------------------------------------------------------------
    def init_workspace(self, stream=None):
        """(Re)initialise the attention workspace shared by every layer."""
        if self.form == 0 and self.max_split == 0:
            lg.lg_decode_attend_workspace_init(self.layers[0], self.workspace, stream)
        else:
            lg.lg_test_attend_workspace_init(self.layers[0], self.form, self.max_split,
                                             self.workspace, stream)

    def attend_layer(self, s: int, l: int, stream=None, flags: Optional[int] = None):
        q, kn, vn = self.step_inputs
        o = l if self.keep_layer_outputs else 0
        args = (self.layers[l], q[s, l], kn[s, l], vn[s, l], self.out[o], self.pos, self.len,
                self.t_steps[s], self.suffix_w, self.lse[o], self.smass[o], self.conf,
                self.workspace)
        flags = self.attend_flags if flags is None else flags
        if self.form == 0 and self.max_split == 0 and flags == 0:
            lg.lg_decode_attend(*args, stream=stream)
        else:
            lg.lg_test_decode_attend(*args, form=self.form, max_split=self.max_split, flags=flags,
                                     stream=stream)

    def detect(self, s: int, stream=None):
        lg.lg_detect_loop(self.params, self.tokens, self.ring, self.t_steps[s], self.t0, self.conf,
                          self.state, self.decision, stream)

    def prune(self, s: int, stream=None):
        lg.lg_prune_compact(self.params, self.B, self.cap, self.layers, self.pos, self.len,
                            self.budget, self.t_steps[s], self.decision, self.keep_idx,
                            self.new_len, stream)

    def detect_prune(self, s: int, stream=None):
        """detect + prune in one call (the detector and the keep set share a launch)."""
        lg.lg_detect_and_prune(self.params, self.tokens, self.ring, self.t_steps[s], self.t0,
                               self.conf, self.state, self.decision, self.cap, self.layers,
                               self.pos, self.len, self.budget, self.t_steps[s], self.keep_idx,
                               self.new_len, stream)

    def step(self, s: int, stream=None, fused: bool = True):
        for l in range(self.L):
            self.attend_layer(s, l, stream)
        if fused:
            self.detect_prune(s, stream)
        else:
            self.detect(s, stream)
            self.prune(s, stream)

    def snapshot(self):
        """Device copy of every array a step modifies (cache, scores, positions, detector)."""
        return {"K": [k.clone() for k in self.K], "V": [v.clone() for v in self.V],
                "acc": [a.clone() for a in self.acc], "pos": self.pos.clone(),
                "len": self.len.clone(), "state": self.state.clone(),
                "decision": self.decision.clone(), "conf": self.conf.clone()}

    def restore(self, snap):
        for dst, src in zip(self.K + self.V + self.acc, snap["K"] + snap["V"] + snap["acc"]):
            dst.copy_(src)
        for name in ("pos", "len", "state", "decision", "conf"):
            getattr(self, name).copy_(snap[name])

    # ------------------------------------------------------------------------------------------
    def decisions(self) -> List[Dict[str, int]]:
        d = self.decision.cpu().numpy()
        return [{f: int(d[b, i]) for i, f in enumerate(lg.DECISION_FIELDS)} for b in range(self.B)]
