"""The C ABI library: it loads, exports every entry point include/lg.h declares, and rejects bad
arguments on the host (nothing is enqueued, so these run without a GPU)."""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = [os.path.join(ROOT, "include", h) for h in ("lg.h", "lg_testing.h")]


def _declared():
    names = set()
    for h in HEADERS:
        src = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names |= set(re.findall(r"\b(lg_[a-z_0-9]+)\s*\(", src))
    return sorted(names)


def test_exports_every_declared_symbol():
    from paper_2604_10044_amd import lg
    names = _declared()
    assert len(names) >= 10
    out = subprocess.run(["nm", "-D", "--defined-only", lg.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\s[TW]\s+(lg_\w+)", out))
    missing = [n for n in names if n not in exported]
    assert not missing, missing
    for n in names:
        assert hasattr(lg._lib, n)


def test_defaults_and_sizes():
    from paper_2604_10044_amd import lg
    import oracle
    p = lg.lg_guard_params_default().as_dict()
    ref = oracle.paper_params()
    for k, v in ref.items():
        if k == "conf_threshold":
            assert abs(p[k] - v) < 1e-7
        else:
            assert p[k] == v, k
    assert lg.lg_state_bytes() == 4 * lg.STATE_INTS
    assert lg.lg_decision_bytes() == 4 * lg.DECISION_INTS
    big = _layer(lg, batch=32, n_q_heads=28, n_kv_heads=4, cap=2048)
    assert lg.lg_decode_attend_workspace(big) > 0
    # the automatic form of a bf16 layer is the one-launch form
    assert lg.lg_decode_attend_workspace(big) == lg.lg_test_attend_workspace(big, lg.FORM_ONE_LAUNCH, 0)
    assert lg.lg_decode_attend_workspace(_layer(lg, n_q_heads=3)) == 0   # 3 % 2 != 0
    assert lg.lg_test_attend_workspace(big, lg.FORM_MERGE, 100) == 0       # not a multiple of 32
    assert lg.lg_test_attend_workspace(_layer(lg, dtype=lg.LG_F32), lg.FORM_ONE_LAUNCH, 0) == 0
    # shorter splits need more exchange words
    assert lg.lg_test_attend_workspace(big, lg.FORM_ONE_LAUNCH, 128) > lg.lg_decode_attend_workspace(big)
    for s in range(9):
        assert lg.lg_status_string(s) and lg.lg_status_string(s) != "unknown status"


def _layer(lg, **kw):
    d = dict(batch=2, n_q_heads=8, n_kv_heads=2, head_dim=128, cap=64, dtype=lg.LG_BF16,
             k=0x1000, v=0x2000, acc=0x3000)
    d.update(kw)
    return lg.LayerCache(**d)


def _attend(lg, layer, ws_bytes=1 << 30, form=0, max_split=0, flags=0, **kw):
    args = dict(q=0x10, k_new=0x20, v_new=0x30, out=0x40, pos=0x50, len=0x60, t=0x70,
                suffix_w=0x80, lse=0x90, sm=0xa0, conf=0xb0, ws=0xc0)
    args.update(kw)
    a = (ctypes.byref(layer), args["q"], args["k_new"], args["v_new"], args["out"], args["pos"],
         args["len"], args["t"], args["suffix_w"], args["lse"], args["sm"], args["conf"],
         args["ws"], ws_bytes)
    if form == 0 and max_split == 0 and flags == 0:
        return lg._lib.lg_decode_attend(*a, None)
    return lg._lib.lg_test_decode_attend(*a, form, max_split, flags, None)


def test_attend_rejects_bad_arguments():
    from paper_2604_10044_amd import lg
    assert _attend(lg, _layer(lg), q=None) == 1
    assert _attend(lg, _layer(lg), k_new=None) == 1          # k_new without v_new
    assert _attend(lg, _layer(lg, k=None)) == 1
    assert _attend(lg, _layer(lg, n_q_heads=7)) == 2          # 7 % 2 != 0
    assert _attend(lg, _layer(lg, batch=0)) == 2
    assert _attend(lg, _layer(lg, head_dim=96)) == 3
    assert _attend(lg, _layer(lg, n_q_heads=34)) == 3         # group of 17 > 16
    assert _attend(lg, _layer(lg, dtype=7)) == 3
    assert _attend(lg, _layer(lg, dtype=lg.LG_F32), form=lg.FORM_ONE_LAUNCH) == 3   # MFMA: bf16 only
    assert _attend(lg, _layer(lg, dtype=lg.LG_F32), form=lg.FORM_MERGE) == 3
    assert _attend(lg, _layer(lg), form=4) == 3
    assert _attend(lg, _layer(lg, cap=48), form=lg.FORM_MERGE) == 3      # MFMA blocks: cap % 32 == 0
    assert _attend(lg, _layer(lg, cap=32800), form=lg.FORM_ONE_LAUNCH) == 3
    for bad in (96, 100, 2080, 4096):
        assert _attend(lg, _layer(lg), form=lg.FORM_ONE_LAUNCH, max_split=bad) == 4, bad
    # beyond 1024 slots only a one-launch split that covers the cap (groups of <= 8 heads)
    assert _attend(lg, _layer(lg, cap=2048), form=lg.FORM_ONE_LAUNCH, max_split=1056) == 4
    assert _attend(lg, _layer(lg, cap=2048, n_q_heads=32), form=lg.FORM_ONE_LAUNCH,
                   max_split=2048) == 4
    assert _attend(lg, _layer(lg, cap=1024), form=lg.FORM_MERGE, max_split=2048) == 4
    assert _attend(lg, _layer(lg), form=lg.FORM_PORTABLE, max_split=256) == 4
    assert _attend(lg, _layer(lg, dtype=lg.LG_F32), max_split=256) == 4  # auto = portable for f32
    assert _attend(lg, _layer(lg), form=lg.FORM_ONE_LAUNCH, flags=8) == 4
    assert _attend(lg, _layer(lg), form=lg.FORM_ONE_LAUNCH, flags=-1) == 4
    assert _attend(lg, _layer(lg, acc=0x3004)) == 7          # 16-byte alignment
    assert _attend(lg, _layer(lg), q=0x18) == 7
    assert _attend(lg, _layer(lg), ws=0xc8) == 7
    assert _attend(lg, _layer(lg), ws_bytes=16) == 5
    assert _attend(lg, _layer(lg), ws=None) == 5


def _noalloc(lg, layer, reinit=0, **kw):
    args = dict(q=0x10, k_new=0x20, v_new=0x30, out=0x40, pos=0x50, len=0x60, t=0x70,
                suffix_w=0x80, lse=0x90, sm=0xa0, conf=0xb0)
    args.update(kw)
    return lg._lib.lg_decode_attend_noalloc(
        ctypes.byref(layer), args["q"], args["k_new"], args["v_new"], args["out"], args["pos"],
        args["len"], args["t"], args["suffix_w"], args["lse"], args["sm"], args["conf"], reinit,
        None)


def test_noalloc_rejects_bad_arguments():
    """The allocation-free attention entry point checks its arguments like lg_decode_attend, and
    refuses a layer whose workspace does not fit its static scratch (all before any HIP call)."""
    from paper_2604_10044_amd import lg
    assert _noalloc(lg, _layer(lg), q=None) == 1
    assert _noalloc(lg, _layer(lg), v_new=None) == 1
    assert _noalloc(lg, _layer(lg, n_q_heads=7)) == 2
    assert _noalloc(lg, _layer(lg, head_dim=96)) == 3
    assert _noalloc(lg, _layer(lg), out=0x48) == 7
    fits = _layer(lg, batch=32, n_q_heads=28, n_kv_heads=4, cap=2048)
    assert lg.lg_decode_attend_workspace(fits) <= lg.NOALLOC_SCRATCH_BYTES
    for big in (_layer(lg, batch=128, n_q_heads=32, n_kv_heads=8, cap=4096),
                _layer(lg, batch=256, n_q_heads=28, n_kv_heads=4, cap=32768),
                _layer(lg, batch=4096, n_q_heads=8, n_kv_heads=8, cap=2048, dtype=lg.LG_F32)):
        assert lg.lg_decode_attend_workspace(big) > lg.NOALLOC_SCRATCH_BYTES
        assert _noalloc(lg, big) == 8
        assert _noalloc(lg, big, reinit=1) == 8


def test_workspace_init_rejects_bad_arguments():
    from paper_2604_10044_amd import lg
    layer = _layer(lg)
    n = lg.lg_decode_attend_workspace(layer)
    f = lg._lib.lg_decode_attend_workspace_init
    assert f(ctypes.byref(layer), 0x1000, n - 16, None) == 5
    assert f(ctypes.byref(layer), None, n, None) == 1
    assert f(ctypes.byref(layer), 0x1008, n, None) == 7
    assert f(ctypes.byref(_layer(lg, head_dim=96)), 0x1000, n, None) == 3
    g = lg._lib.lg_test_attend_workspace_init
    assert g(ctypes.byref(layer), lg.FORM_ONE_LAUNCH, 100, 0x1000, 1 << 30, None) == 4
    assert g(ctypes.byref(layer), 9, 0, 0x1000, 1 << 30, None) == 3


def _detect(lg, p, ring=2048, **kw):
    args = dict(tokens=0x10, t=0x20, t0=0x30, conf=0x40, state=0x50, dec=0x60, batch=4)
    args.update(kw)
    return lg._lib.lg_detect_loop(ctypes.byref(p), args["batch"], args["tokens"], ring, args["t"],
                                  args["t0"], args["conf"], args["state"], args["dec"], None)


def test_detect_rejects_bad_arguments():
    from paper_2604_10044_amd import lg
    p = lg.lg_guard_params_default()
    assert _detect(lg, p, tokens=None) == 1
    assert _detect(lg, p, state=None) == 1
    assert _detect(lg, p, batch=0) == 2
    assert _detect(lg, p, ring=1000) == 2                     # ring < rep_horizon
    for field, bad in [("W", 0), ("W", 513), ("K", 4), ("rep_horizon", 4096), ("rep_pmax", 0),
                       ("nov_ngram", 0), ("ttr_den", 0), ("cr_interval", 0), ("mode", 3), ("policy", 3), ("policy", -1),
                       ("level_max", 31), ("recent_div", 0)]:
        q = lg.lg_guard_params_default()
        setattr(q, field, bad)
        assert _detect(lg, q) == 4, field
    assert lg._lib.lg_detect_loop(None, 4, 0x10, 2048, 0x20, 0x30, 0x40, 0x50, 0x60, None) == 1


def test_prune_rejects_bad_arguments():
    from paper_2604_10044_amd import lg
    p = lg.lg_guard_params_default()
    f = lg._lib.lg_prune_compact
    L = (lg.LayerCache * 2)(_layer(lg), _layer(lg))
    ok = dict(pos=0x10, len=0x20, budget=0x30, keep=0x40, nl=0x50)

    def call(batch=2, cap=64, n=2, layers=L, **kw):
        a = dict(ok)
        a.update(kw)
        return f(ctypes.byref(p), batch, cap, n, layers, a["pos"], a["len"], a["budget"], None,
                 None, a["keep"], a["nl"], None)

    assert call(pos=None) == 1
    assert call(keep=None) == 1
    assert call(layers=None) == 1
    assert call(batch=0) == 2
    assert call(cap=32) == 2                                   # layer cap differs
    L2 = (lg.LayerCache * 2)(_layer(lg), _layer(lg, head_dim=64))
    assert call(layers=L2) == 2
    q = lg.lg_guard_params_default()
    q.recent_div = 0
    assert f(ctypes.byref(q), 2, 64, 0, None, 0x10, 0x20, 0x30, None, None, 0x40, 0x50, None) == 4
    assert lg._lib.lg_copy_bandwidth(0x10, 0x20, 17, None) == 2
    assert lg._lib.lg_copy_bandwidth(None, 0x20, 16, None) == 1


def test_prune_rejects_unknown_policy():
    from paper_2604_10044_amd import lg
    f = lg._lib.lg_prune_compact
    for bad in (-1, 3):
        q = lg.lg_guard_params_default()
        q.policy = bad
        assert f(ctypes.byref(q), 2, 64, 0, None, 0x10, 0x20, 0x30, None, None, 0x40, 0x50, None) == 4
    assert lg.lg_guard_params_default().policy == lg.LG_POLICY_LOOPGUARD
