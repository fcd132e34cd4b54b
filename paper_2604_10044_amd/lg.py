"""Python binding of liblg (the C ABI in include/lg.h): argument marshalling only.

Every function here has the name of the C entry point it calls and takes torch tensors (device
memory) in place of raw pointers. Importing this module loads liblg.so and raises if it is
missing: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "liblg.so")

if not os.path.exists(LIB_PATH):
    raise ImportError("liblg.so is not built (run __graft_entry__.build() or "
                      "python -m paper_2604_10044_amd.build)")
_lib = ctypes.CDLL(LIB_PATH)

LG_F32, LG_BF16 = 0, 1
LG_ATTEND_STATUS_WAIT, LG_ATTEND_STATUS_WORKSPACE = 1, 2
# test hooks (include/lg_testing.h)
FORM_AUTO, FORM_PORTABLE, FORM_MERGE, FORM_ONE_LAUNCH = 0, 1, 2, 3
TEST_FORCE_HANDOVER, TEST_NO_WAIT, TEST_WHOLE_DIMS = 1, 2, 4
LG_MODE_FULL, LG_MODE_ALWAYS_ON, LG_MODE_P1_ONLY = 0, 1, 2
LG_POLICY_LOOPGUARD, LG_POLICY_H2O, LG_POLICY_STREAMING = 0, 1, 2
STATUS = {0: "LG_OK", 1: "LG_ERR_NULL", 2: "LG_ERR_SHAPE", 3: "LG_ERR_UNSUPPORTED",
          4: "LG_ERR_PARAM", 5: "LG_ERR_WORKSPACE", 6: "LG_ERR_HIP", 7: "LG_ERR_ALIGN",
          8: "LG_ERR_TOO_LARGE"}
NOALLOC_SCRATCH_BYTES = 64 << 20   # LG_NOALLOC_SCRATCH_BYTES

PARAM_FIELDS = ["W", "K", "n_anchor", "t_min", "cooldown", "streak_min", "stall_min",
                "cr_interval", "nov_ngram", "nov_span", "rep_pmax", "rep_horizon",
                "rep_min_copies", "rep_min_len", "rep_debounce", "level_max", "retrigger_window",
                "recent_div", "sparse_div", "ttr_num", "ttr_den", "cr_num", "cr_den", "nov_num",
                "nov_den"]
STATE_FIELDS = ["streak", "stall", "rep", "n_int", "n_last", "level", "cr_valid", "cr_cost",
                "cr_m"]
DECISION_FIELDS = ["trigger", "warn", "votes", "stall_gate", "tailrep_gate", "n", "distinct",
                   "lz_cost", "novel", "nov_r", "period", "span_lo", "level", "n_int"]
ATTEND_ERROR_COL = 14  # lg_decision.attend_error (not a decision of the paper's rule)
HEADER_FIELDS = ["magic", "version", "batch", "n_q_heads", "n_kv_heads", "head_dim", "cap",
                 "dtype", "form", "split", "status"]
STATE_INTS = 528     # lg_guard_state is 528 int32 (16 fields + 512 tail runs)
DECISION_INTS = 16   # lg_decision is 16 int32


class LayerCache(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("cap", ctypes.c_int32), ("dtype", ctypes.c_int), ("k", ctypes.c_void_p),
                ("v", ctypes.c_void_p), ("acc", ctypes.c_void_p)]


class GuardParams(ctypes.Structure):
    _fields_ = [(f, ctypes.c_int32) for f in PARAM_FIELDS] + [
        ("conf_threshold", ctypes.c_float), ("mode", ctypes.c_int32), ("policy", ctypes.c_int32)]

    def as_dict(self):
        d = {f: int(getattr(self, f)) for f in PARAM_FIELDS}
        d["conf_threshold"] = float(self.conf_threshold)
        d["mode"] = int(self.mode)
        d["policy"] = int(self.policy)
        return d


_vp, _i32, _sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
_lib.lg_guard_params_default.restype = GuardParams
_lib.lg_guard_params_default.argtypes = []
_lib.lg_status_string.restype = ctypes.c_char_p
_lib.lg_status_string.argtypes = [ctypes.c_int]
_lib.lg_state_bytes.restype = _sz
_lib.lg_decision_bytes.restype = _sz
_LP = ctypes.POINTER(LayerCache)
_lib.lg_decode_attend_workspace.restype = _sz
_lib.lg_decode_attend_workspace.argtypes = [_LP]
_lib.lg_decode_attend_workspace_init.restype = ctypes.c_int
_lib.lg_decode_attend_workspace_init.argtypes = [_LP, _vp, _sz, _vp]
_ATT = [_LP, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _sz]
_lib.lg_decode_attend.restype = ctypes.c_int
_lib.lg_decode_attend.argtypes = _ATT + [_vp]
_lib.lg_decode_attend_noalloc.restype = ctypes.c_int
_lib.lg_decode_attend_noalloc.argtypes = _ATT[:-2] + [_i32, _vp]
_lib.lg_test_attend_workspace.restype = _sz
_lib.lg_test_attend_workspace.argtypes = [_LP, _i32, _i32]
_lib.lg_test_attend_workspace_init.restype = ctypes.c_int
_lib.lg_test_attend_workspace_init.argtypes = [_LP, _i32, _i32, _vp, _sz, _vp]
_lib.lg_test_decode_attend.restype = ctypes.c_int
_lib.lg_test_decode_attend.argtypes = _ATT + [_i32, _i32, _i32, _vp]
_lib.lg_detect_loop.restype = ctypes.c_int
_lib.lg_detect_loop.argtypes = [ctypes.POINTER(GuardParams), _i32, _vp, _i32, _vp, _vp, _vp, _vp,
                                _vp, _vp]
_lib.lg_prune_compact.restype = ctypes.c_int
_lib.lg_prune_compact.argtypes = [ctypes.POINTER(GuardParams), _i32, _i32, _i32,
                                  ctypes.POINTER(LayerCache), _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                  _vp]
_lib.lg_detect_and_prune.restype = ctypes.c_int
_lib.lg_detect_and_prune.argtypes = [ctypes.POINTER(GuardParams), _i32, _vp, _i32, _vp, _vp, _vp,
                                     _vp, _vp, _i32, _i32, ctypes.POINTER(LayerCache), _vp, _vp,
                                     _vp, _vp, _vp, _vp, _vp]
_lib.lg_copy_bandwidth.restype = ctypes.c_int
_lib.lg_copy_bandwidth.argtypes = [_vp, _vp, _sz, _vp]


class LGError(RuntimeError):
    pass


def _check(status: int, what: str):
    if status != 0:
        raise LGError("%s: %s (%s)" % (what, STATUS.get(status, status),
                                       _lib.lg_status_string(status).decode()))


def _ptr(x) -> Optional[int]:
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return stream if isinstance(stream, int) else stream.cuda_stream


def lg_guard_params_default() -> GuardParams:
    return _lib.lg_guard_params_default()


def lg_status_string(status: int) -> str:
    return _lib.lg_status_string(status).decode()


def lg_state_bytes() -> int:
    return int(_lib.lg_state_bytes())


def lg_decision_bytes() -> int:
    return int(_lib.lg_decision_bytes())


def lg_decode_attend_workspace(layer: "LayerCache") -> int:
    return int(_lib.lg_decode_attend_workspace(ctypes.byref(layer)))


def lg_decode_attend_workspace_init(layer: "LayerCache", workspace, stream=None):
    ws = workspace.numel() * workspace.element_size()
    _check(_lib.lg_decode_attend_workspace_init(ctypes.byref(layer), _ptr(workspace), ws,
                                                _stream(stream)), "lg_decode_attend_workspace_init")


def lg_test_attend_workspace(layer: "LayerCache", form: int, max_split: int = 0) -> int:
    return int(_lib.lg_test_attend_workspace(ctypes.byref(layer), form, max_split))


def lg_test_attend_workspace_init(layer: "LayerCache", form: int, max_split: int, workspace,
                                  stream=None):
    ws = workspace.numel() * workspace.element_size()
    _check(_lib.lg_test_attend_workspace_init(ctypes.byref(layer), form, max_split,
                                              _ptr(workspace), ws, _stream(stream)),
           "lg_test_attend_workspace_init")


def workspace_header(workspace) -> dict:
    """The lg_attend_workspace_header at the start of a workspace, read back to the host."""
    h = workspace[:64].cpu().numpy().view("<i4")
    return {f: int(h[i]) & 0xffffffff if f in ("magic", "version", "status") else int(h[i])
            for i, f in enumerate(HEADER_FIELDS)}


def layer_cache(k: torch.Tensor, v: torch.Tensor, acc: torch.Tensor, n_q_heads: int) -> LayerCache:
    """View of one layer's cache: k, v [B][Hkv][cap][D] (float32 or bfloat16), acc [B][Hkv][cap]."""
    B, Hkv, cap, D = k.shape
    dt = LG_BF16 if k.dtype == torch.bfloat16 else LG_F32
    return LayerCache(B, n_q_heads, Hkv, D, cap, dt, k.data_ptr(), v.data_ptr(), acc.data_ptr())


def lg_decode_attend(layer: LayerCache, q, k_new, v_new, out, pos, len_, t, suffix_w, lse,
                     suffix_mass, conf, workspace, stream=None):
    ws = workspace.numel() * workspace.element_size()
    _check(_lib.lg_decode_attend(ctypes.byref(layer), _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(out),
                                 _ptr(pos), _ptr(len_), _ptr(t), _ptr(suffix_w), _ptr(lse),
                                 _ptr(suffix_mass), _ptr(conf), _ptr(workspace), ws,
                                 _stream(stream)), "lg_decode_attend")


def lg_decode_attend_noalloc(layer: LayerCache, q, k_new, v_new, out, pos, len_, t, suffix_w, lse,
                             suffix_mass, conf, reinit: int = 0, stream=None):
    _check(_lib.lg_decode_attend_noalloc(ctypes.byref(layer), _ptr(q), _ptr(k_new), _ptr(v_new),
                                         _ptr(out), _ptr(pos), _ptr(len_), _ptr(t),
                                         _ptr(suffix_w), _ptr(lse), _ptr(suffix_mass), _ptr(conf),
                                         int(reinit), _stream(stream)),
           "lg_decode_attend_noalloc")


def lg_test_decode_attend(layer: LayerCache, q, k_new, v_new, out, pos, len_, t, suffix_w, lse,
                          suffix_mass, conf, workspace, form: int, max_split: int = 0,
                          flags: int = 0, stream=None):
    ws = workspace.numel() * workspace.element_size()
    _check(_lib.lg_test_decode_attend(ctypes.byref(layer), _ptr(q), _ptr(k_new), _ptr(v_new),
                                      _ptr(out), _ptr(pos), _ptr(len_), _ptr(t), _ptr(suffix_w),
                                      _ptr(lse), _ptr(suffix_mass), _ptr(conf), _ptr(workspace),
                                      ws, form, max_split, flags, _stream(stream)),
           "lg_test_decode_attend")


def lg_detect_loop(params: GuardParams, tokens, ring: int, t, t0, conf, state, decision,
                   stream=None):
    batch = t.shape[0]
    _check(_lib.lg_detect_loop(ctypes.byref(params), batch, _ptr(tokens), ring, _ptr(t), _ptr(t0),
                               _ptr(conf), _ptr(state), _ptr(decision), _stream(stream)),
           "lg_detect_loop")


def lg_prune_compact(params: GuardParams, batch: int, cap: int, layers: Sequence[LayerCache],
                     pos, len_, budget, t_append, decision, keep_idx, new_len, stream=None):
    n = len(layers)
    arr = (LayerCache * max(1, n))(*layers) if n else None
    _check(_lib.lg_prune_compact(ctypes.byref(params), batch, cap, n, arr, _ptr(pos), _ptr(len_),
                                 _ptr(budget), _ptr(t_append), _ptr(decision), _ptr(keep_idx),
                                 _ptr(new_len), _stream(stream)), "lg_prune_compact")


def lg_detect_and_prune(params: GuardParams, tokens, ring: int, t, t0, conf, state, decision,
                        cap: int, layers: Sequence[LayerCache], pos, len_, budget, t_append,
                        keep_idx, new_len, stream=None):
    batch = t.shape[0]
    n = len(layers)
    arr = (LayerCache * max(1, n))(*layers) if n else None
    _check(_lib.lg_detect_and_prune(ctypes.byref(params), batch, _ptr(tokens), ring, _ptr(t),
                                    _ptr(t0), _ptr(conf), _ptr(state), _ptr(decision), cap, n,
                                    arr, _ptr(pos), _ptr(len_), _ptr(budget), _ptr(t_append),
                                    _ptr(keep_idx), _ptr(new_len), _stream(stream)),
           "lg_detect_and_prune")


def lg_copy_bandwidth(src, dst, nbytes: int, stream=None):
    _check(_lib.lg_copy_bandwidth(_ptr(src), _ptr(dst), nbytes, _stream(stream)),
           "lg_copy_bandwidth")


def params_from_dict(d) -> GuardParams:
    p = lg_guard_params_default()
    for k, v in d.items():
        setattr(p, k, v)
    return p
