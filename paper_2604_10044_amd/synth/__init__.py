"""Seeded synthetic workloads for the guarded-decode path.

This module produces inputs only: token streams and query/key/value rows, as pure functions of a
seed (see ``lg_synth.c`` for the generator). It contains none of the method's arithmetic, so both
the GPU path's harness and the CPU oracle's harness can draw identical inputs from it.

The five workloads imitate the paper's loop-inducing regime (Sec. 3.3, Sec. 4.1) at the shapes of
the benchmarked models; the paper's datasets and checkpoints are not used (synthetic stand-ins).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "lg_synth.c")
_LIB = os.path.join(_HERE, "libsynth.so")

KIND_K, KIND_V, KIND_Q = 0, 1, 2


def build(force: bool = False) -> str:
    """Compile the generator (gcc, OpenMP, no FP contraction)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-shared", "-fPIC",
                               "-o", tmp, _SRC])
        os.replace(tmp, _LIB)
    return _LIB


class _Cfg(ctypes.Structure):
    _fields_ = [("seed", ctypes.c_uint64), ("n_layers", ctypes.c_int32),
                ("n_q_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("vocab", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("lock_gain", ctypes.c_float),
                ("lock_noise", ctypes.c_float), ("lock_every", ctypes.c_int32),
                ("lock_layer_min", ctypes.c_int32), ("dup_rate", ctypes.c_float),
                ("reserved", ctypes.c_int32)]


class _Seg(ctypes.Structure):
    _fields_ = [("start", ctypes.c_int32), ("end", ctypes.c_int32), ("unit_len", ctypes.c_int32),
                ("unit_off", ctypes.c_int32), ("noise0", ctypes.c_float),
                ("noise1", ctypes.c_float), ("ramp_lo", ctypes.c_int32),
                ("ramp_hi", ctypes.c_int32)]


class _Seq(ctypes.Structure):
    _fields_ = [("n_seg", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("seg", ctypes.POINTER(_Seg)), ("unit_tokens", ctypes.POINTER(ctypes.c_int32))]


_lib_handle = None


def _lib():
    global _lib_handle
    if _lib_handle is None:
        if not os.path.exists(_LIB):
            build()
        L = ctypes.CDLL(_LIB)
        P = ctypes.POINTER
        L.synth_token.restype = ctypes.c_int32
        L.synth_token.argtypes = [P(_Cfg), P(_Seq), ctypes.c_int32, ctypes.c_int32]
        L.synth_tokens.restype = None
        L.synth_tokens.argtypes = [P(_Cfg), P(_Seq), ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p]
        L.synth_unit_tokens.restype = None
        L.synth_unit_tokens.argtypes = [P(_Cfg), ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                        ctypes.c_int32, ctypes.c_void_p]
        L.synth_fill.restype = None
        L.synth_fill.argtypes = [P(_Cfg), P(_Seq), ctypes.c_void_p, ctypes.c_int32, ctypes.c_int,
                                 ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                 ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
        L.synth_bf16_to_f32.restype = None
        L.synth_bf16_to_f32.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64]
        _lib_handle = L
    return _lib_handle


@dataclass
class Segment:
    """Positions [start, end) repeat a unit of ``len(unit)`` tokens (the first copy)."""
    start: int
    end: int
    unit: np.ndarray
    noise0: float = 0.05
    noise1: float = 0.05
    ramp_lo: int = 0
    ramp_hi: int = 0


@dataclass
class Workload:
    name: str
    seed: int
    batch: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    dtype: str            # "f32" or "bf16"
    n_layers: int
    ctx: np.ndarray       # [B] context length (positions 0..ctx-1 precede decoding)
    budget: np.ndarray    # [B] KV budget
    steps: int
    vocab: int
    segments: List[List[Segment]] = field(default_factory=list)
    lock_gain: float = 1.0
    lock_noise: float = 0.25
    lock_every: int = 4
    lock_layer_min: int = 0
    dup_rate: float = 0.0

    # ----------------------------------------------------------------------------------------
    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def cap(self) -> int:
        return int(self.budget.max())

    @property
    def elem_bytes(self) -> int:
        return 2 if self.dtype == "bf16" else 4

    def _cfg(self) -> _Cfg:
        return _Cfg(self.seed, self.n_layers, self.n_q_heads, self.n_kv_heads, self.head_dim,
                    self.vocab, 1 if self.dtype == "bf16" else 0, self.lock_gain, self.lock_noise,
                    self.lock_every, self.lock_layer_min, self.dup_rate, 0)

    def _seq(self, b: int):
        segs = self.segments[b] if b < len(self.segments) else []
        arr = (_Seg * max(1, len(segs)))()
        units = [np.asarray(s.unit, dtype=np.int32) for s in segs]
        flat = np.concatenate(units).astype(np.int32) if units else np.zeros(1, np.int32)
        off = 0
        for i, s in enumerate(segs):
            arr[i] = _Seg(s.start, s.end, len(s.unit), off, s.noise0, s.noise1, s.ramp_lo,
                          s.ramp_hi)
            off += len(s.unit)
        keep = (arr, flat)
        seq = _Seq(len(segs), 0, ctypes.cast(arr, ctypes.POINTER(_Seg)),
                   flat.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)))
        return seq, keep

    # ----------------------------------------------------------------------------------------
    def tokens(self, b: int, n: Optional[int] = None) -> np.ndarray:
        """Token stream y[0..n) of sequence b (default: context plus every decode step)."""
        n = int(self.ctx[b]) + self.steps if n is None else int(n)
        out = np.zeros(n, np.int32)
        cfg = self._cfg()
        seq, keep = self._seq(b)
        _lib().synth_tokens(ctypes.byref(cfg), ctypes.byref(seq), b, n, out.ctypes.data)
        return out

    def rows(self, kind: int, layer_lo: int, layer_hi: int, b_list: Sequence[int],
             pos: np.ndarray, cnt: Optional[np.ndarray] = None) -> np.ndarray:
        """Rows for sequences ``b_list`` at positions pos[i, :cnt[i]].

        Returns [layer_hi-layer_lo][len(b_list)][heads][P][head_dim] as uint16 (bf16 bits) or
        float32; heads is n_q_heads for queries, n_kv_heads otherwise.
        """
        b_list = np.ascontiguousarray(np.asarray(b_list, dtype=np.int32))
        pos = np.ascontiguousarray(np.asarray(pos, dtype=np.int32))
        nb = len(b_list)
        if pos.ndim == 1:
            pos = pos.reshape(nb, -1)
        P = pos.shape[1]
        cnt = np.full(nb, P, np.int32) if cnt is None else np.ascontiguousarray(cnt, np.int32)
        heads = self.n_q_heads if kind == KIND_Q else self.n_kv_heads
        dt = np.uint16 if self.dtype == "bf16" else np.float32
        out = np.empty((layer_hi - layer_lo, nb, heads, P, self.head_dim), dt)
        cfg = self._cfg()
        seqs = (_Seq * nb)()
        keep = []
        for i, b in enumerate(b_list):
            s, k = self._seq(int(b))
            seqs[i] = s
            keep.append(k)
        _lib().synth_fill(ctypes.byref(cfg), seqs, b_list.ctypes.data, nb, kind, layer_lo,
                          layer_hi, heads, P, pos.ctypes.data, cnt.ctypes.data, out.ctypes.data)
        return out


def to_f32(a: np.ndarray) -> np.ndarray:
    """Exact float32 view of generator rows (bf16 bits are widened, float32 is returned as is)."""
    if a.dtype == np.float32:
        return a
    a = np.ascontiguousarray(a)
    out = np.empty(a.shape, np.float32)
    _lib().synth_bf16_to_f32(a.ctypes.data, out.ctypes.data, a.size)
    return out


def unit_tokens(wl_seed: int, vocab: int, b: int, idx: int, length: int, avoid: int = -1):
    cfg = _Cfg(wl_seed, 1, 1, 1, 64, vocab, 0, 0.0, 0.0, 0, 0, 0.0, 0)
    out = np.zeros(length, np.int32)
    _lib().synth_unit_tokens(ctypes.byref(cfg), b, idx, length, avoid, out.ctypes.data)
    return out


def _base_token(seed: int, vocab: int, b: int, p: int) -> int:
    cfg = _Cfg(seed, 1, 1, 1, 64, vocab, 0, 0.0, 0.0, 0, 0, 0.0, 0)
    seq = _Seq(0, 0, None, None)
    return int(_lib().synth_token(ctypes.byref(cfg), ctypes.byref(seq), b, p))


def loop_segment(seed: int, vocab: int, b: int, idx: int, start: int, period: int, end: int,
                 noise: float = 0.05, **kw) -> Segment:
    """A primitive period-`period` loop: distinct unit tokens, none equal to y[start-1]."""
    avoid = _base_token(seed, vocab, b, start - 1) if start > 0 else -1
    return Segment(start, end, unit_tokens(seed, vocab, b, idx, period, avoid), noise, noise, **kw)


# ------------------------------------------------------------------------------------------------
# The five workloads (shapes of the benchmarked configurations).
# ------------------------------------------------------------------------------------------------
def tiny(steps: int = 16, seed: int = 1, period: int = 12) -> Workload:
    """Single layer, batch 1, 4/4 heads, head_dim 64, float32, cache 256 = budget 256; the last 96
    context positions repeat a 12-token period that continues through decoding."""
    ctx, st = 256, steps
    seg = loop_segment(seed, 1000, 0, 0, 160, period, ctx + st)
    return Workload("tiny-1layer-fp32", seed, 1, 4, 4, 64, "f32", 1, np.array([ctx]),
                    np.array([256]), st, 1000, [[seg]], lock_every=2, lock_layer_min=0)


def qwen15b(steps: int = 256, seed: int = 2, n_layers: int = 28) -> Workload:
    """1.5B-shaped: batch 1, 12/2 heads, head_dim 128, bf16, 28 layers, context 4096, budget 1024;
    one loop (period U{8..64}) starting in the last 30% of the context."""
    rng = np.random.default_rng(seed)
    ctx = 4096
    P = int(rng.integers(8, 65))
    s0 = int(rng.integers(2868, 4096))
    seg = loop_segment(seed, 32000, 0, 0, s0, P, ctx + steps)
    return Workload("1.5B-shaped-b1", seed, 1, 12, 2, 128, "bf16", n_layers, np.array([ctx]),
                    np.array([1024]), steps, 32000, [[seg]], lock_layer_min=n_layers // 2)


def llama7b(steps: int = 128, seed: int = 9003, batch: int = 32, n_layers: int = 28) -> Workload:
    """7B-shaped: batch 32, 28/4 heads, head_dim 128, bf16, 28 layers, context 8192, budget 2048;
    even sequences carry a loop (period U{4..128}, key noise 0.05) starting in the last 30% of the
    context, odd sequences are i.i.d. Seed 9003: seeds 3 to 8003 (in steps of 1000) each put
    some oracle confidence of the 128 steps within 0.018 of the 0.9 threshold, the band that
    tests/golden/conf_margins.py rejects (3 and 1003 even within 2e-3: sequence 20 at 3.5e-4,
    sequence 10 at 3.9e-5)."""
    rng = np.random.default_rng(seed)
    ctx = 8192
    segs = []
    for b in range(batch):
        if b % 2 == 0:
            P = int(rng.integers(4, 129))
            s0 = int(rng.integers(5734, 8192))
            segs.append([loop_segment(seed, 32000, b, 0, s0, P, ctx + steps)])
        else:
            segs.append([])
    return Workload("7B-shaped-b32", seed, batch, 28, 4, 128, "bf16", n_layers,
                    np.full(batch, ctx), np.full(batch, 2048), steps, 32000, segs,
                    lock_layer_min=n_layers // 2)


def llama8b_long(steps: int = 512, seed: int = 4, batch: int = 8, n_layers: int = 32) -> Workload:
    """8B-shaped long context: batch 8, 32/8 heads, head_dim 128, bf16, 32 layers, context 32768,
    budget 4096. From the first decode step the stream repeats a 200-token unit made of a
    16-token motif repeated 12 times plus 8 fresh tokens (a period-16 loop nested in a period-200
    loop); repeated-key noise ramps from 0.2 down to 0.02 over the 512 decode steps."""
    ctx = 32768
    segs = []
    for b in range(batch):
        motif = unit_tokens(seed, 32000, b, 0, 16, _base_token(seed, 32000, b, ctx - 1))
        fresh = unit_tokens(seed, 32000, b, 1, 24, -1)
        fresh = np.array([x for x in fresh if x not in set(motif.tolist())][:8], np.int32)
        unit = np.concatenate([np.tile(motif, 12), fresh]).astype(np.int32)
        segs.append([Segment(ctx, ctx + steps, unit, 0.2, 0.02, ctx, ctx + 512)])
    return Workload("8B-shaped-long-b8", seed, batch, 32, 8, 128, "bf16", n_layers,
                    np.full(batch, ctx), np.full(batch, 4096), steps, 32000, segs,
                    lock_layer_min=n_layers // 2)


def ragged(steps: int = 256, seed: int = 5, batch: int = 64, n_layers: int = 32) -> Workload:
    """Ragged stress: batch 64, context lengths log-uniform in [512, 65536], budgets in
    {512, 2048, 8192}, 32/8 heads, head_dim 128, bf16; 0-3 loops per sequence (period U{2..256})
    on disjoint spans, the last one running through the decode steps; 1% of key rows are exact
    duplicates of an earlier row."""
    rng = np.random.default_rng(seed)
    ctx = np.floor(np.exp(rng.uniform(np.log(512), np.log(65536), batch))).astype(np.int64)
    budget = rng.choice(np.array([512, 2048, 8192]), batch)
    segs = []
    for b in range(batch):
        nl = int(rng.integers(0, 4))
        lst = []
        end = int(ctx[b]) + steps
        hi = int(ctx[b])
        for k in range(nl):
            P = int(rng.integers(2, 257))
            if k == 0:
                length = int(rng.integers(3 * P + 32, 3 * P + 800))
                s0 = max(1, hi - length)
                lst.append(loop_segment(seed, 32000, b, k, s0, P, end))
            else:
                length = int(rng.integers(3 * P, 3 * P + 400))
                e = hi - int(rng.integers(8, 200))
                s0 = e - length
                if s0 < 64:
                    break
                lst.append(loop_segment(seed, 32000, b, k, s0, P, e))
            hi = s0 - 1
            end = s0
        segs.append(sorted(lst, key=lambda s: s.start))
    return Workload("ragged-b64", seed, batch, 32, 8, 128, "bf16", n_layers, ctx, budget, steps,
                    32000, segs, lock_layer_min=n_layers // 2, dup_rate=0.01)


CONFIGS = {0: tiny, 1: qwen15b, 2: llama7b, 3: llama8b_long, 4: ragged}


def config(i: int, **kw) -> Workload:
    return CONFIGS[i](**kw)
