"""Device-side values the host cannot check (lengths, positions, widths, budgets, t0): the kernels
clamp them as include/lg.h states, so out-of-range values give defined results and no access
outside the caller's buffers. Rows with valid values in the same launch are unaffected and equal
the oracle; rows with out-of-range values are checked against the oracle under the documented
clamping where it defines the result."""
import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu
I32_MIN, I32_MAX = -2 ** 31, 2 ** 31 - 1


def _bf16(x):
    return torch.from_numpy(x).to(torch.bfloat16).float().numpy()


def test_attend_clamps_lengths_and_saturates_the_suffix_threshold():
    from paper_2604_10044_amd import lg
    rng = np.random.default_rng(3)
    B, Hq, Hkv, D, cap = 4, 8, 2, 128, 256
    G = Hq // Hkv
    dev = torch.device("cuda")
    K = _bf16(rng.standard_normal((B, Hkv, cap, D)).astype(np.float32))
    V = _bf16(rng.standard_normal((B, Hkv, cap, D)).astype(np.float32))
    q = _bf16(rng.standard_normal((B, Hq, D)).astype(np.float32))
    kn = _bf16(rng.standard_normal((B, Hkv, D)).astype(np.float32))
    vn = _bf16(rng.standard_normal((B, Hkv, D)).astype(np.float32))
    pos = np.tile(np.arange(cap, dtype=np.int32) * 3, (B, 1))
    lens = np.array([100, -7, cap + 50, I32_MAX], np.int32)
    t = np.array([3 * 99 + 3, 5, 3 * cap, I32_MIN], np.int32)
    sw = np.array([64, 2, 100, I32_MAX], np.int32)
    acc0 = rng.uniform(0, 5, (B, Hkv, cap)).astype(np.float32)
    accd = torch.from_numpy(acc0).to(dev)
    Kd = torch.from_numpy(K).to(dev).to(torch.bfloat16)
    Vd = torch.from_numpy(V).to(dev).to(torch.bfloat16)
    out = torch.zeros(B, Hq, D, dtype=torch.bfloat16, device=dev)
    lse = torch.zeros(B, Hq, device=dev)
    sm = torch.zeros(B, Hq, device=dev)
    conf = torch.zeros(B, device=dev)
    to = lambda a, dt=torch.bfloat16: torch.from_numpy(a).to(dev).to(dt)
    for form in (0, 1, 2):   # the automatic (one-launch) form, the portable and the merge form
        accd.copy_(torch.from_numpy(acc0))
        Kd.copy_(torch.from_numpy(K).to(torch.bfloat16))
        Vd.copy_(torch.from_numpy(V).to(torch.bfloat16))
        layer = lg.layer_cache(Kd, Vd, accd, Hq)
        ws = torch.empty(lg.lg_test_attend_workspace(layer, form, 0), dtype=torch.uint8, device=dev)
        lg.lg_test_attend_workspace_init(layer, form, 0, ws)
        lg.lg_test_decode_attend(layer, to(q), to(kn), to(vn), out, to(pos, torch.int32),
                                 to(lens, torch.int32), to(t, torch.int32), to(sw, torch.int32),
                                 lse, sm, conf, ws, form=form)
        torch.cuda.synchronize()
        o_h, l_h, s_h, a_h = out.float().cpu().numpy(), lse.cpu().numpy(), sm.cpu().numpy(), accd.cpu().numpy()
        # the documented clamp: L = min(max(len, 0), cap); the row is appended only if L < cap
        for b in range(B):
            L = min(max(int(lens[b]), 0), cap)
            app = L < cap
            for h in range(Hkv):
                Ke, Ve, pe = K[b, h, :L], V[b, h, :L], pos[b, :L]
                if app:
                    Ke = np.concatenate([Ke, kn[b, h][None]])
                    Ve = np.concatenate([Ve, vn[b, h][None]])
                    pe = np.append(pe, t[b])
                o, ls, sg, asum = oracle.attend_group(q[b, h * G:(h + 1) * G], Ke, Ve, pe, int(t[b]), int(sw[b]))
                go = o_h[b, h * G:(h + 1) * G]
                rowmax = np.abs(o).max(axis=1, keepdims=True)
                assert np.all(np.abs(go - o) <= 2e-2 * np.abs(o) + 1e-3 * rowmax), (form, b, h)
                assert np.all(np.abs(l_h[b, h * G:(h + 1) * G] - ls) <= 2e-4 * np.maximum(1, np.abs(ls)))
                assert np.all(np.abs(s_h[b, h * G:(h + 1) * G] - sg) <= 2e-4), (form, b, h)
                n = L + (1 if app else 0)
                ref = acc0[b, h, :n].astype(np.float64)
                if app:
                    ref[L] = 0.0
                ref += asum
                assert np.all(np.abs(a_h[b, h, :n] - ref) <= 1e-4 * np.maximum(1, np.abs(ref))), (form, b, h)
        # threshold saturated at the int32 minimum: every slot counts (S * (1/Z) with S = Z)
        np.testing.assert_allclose(s_h[3], 1.0, rtol=0, atol=1e-6)


def test_detect_clamps_positions():
    from paper_2604_10044_amd import lg
    rng = np.random.default_rng(4)
    p = oracle.paper_params()
    B, ring, N = 8, 1100, 1500      # a ring length that is not a power of two (>= max(W, H))
    ys = [rng.integers(0, 50, N).astype(np.int32) for _ in range(B)]
    n_valid = np.array([1200, 700, 1500, 900, 1, 1, 1, 1], np.int64)
    t = (n_valid - 1).astype(np.int32)
    t0 = np.zeros(B, np.int32)
    # out-of-range rows: the smallest and largest positions, a t0 far past the stream, a negative t0
    t[4], t[5] = I32_MIN, I32_MAX
    t0[6], t0[7] = I32_MAX, -9
    t[6], t[7] = 500, 400
    dev = torch.device("cuda")
    ring_h = np.zeros((B, ring), np.int32)
    for b in range(4):
        idx = np.arange(max(0, n_valid[b] - ring), n_valid[b])
        ring_h[b, idx % ring] = ys[b][idx]
    ring_h[4:] = rng.integers(0, 50, (4, ring))
    state = torch.zeros(B, lg.STATE_INTS, dtype=torch.int32, device=dev)
    dec = torch.zeros(B, lg.DECISION_INTS, dtype=torch.int32, device=dev)
    conf = torch.full((B,), 0.95, dtype=torch.float32, device=dev)
    lg.lg_detect_loop(lg.params_from_dict(p), torch.from_numpy(ring_h).to(dev), ring,
                      torch.from_numpy(t).to(dev), torch.from_numpy(t0).to(dev), conf, state, dec)
    torch.cuda.synchronize()
    d_h = dec.cpu().numpy()
    F = lg.DECISION_FIELDS
    for b in range(4):
        ref = oracle.Detector(p).step(ys[b], 0, int(n_valid[b]), 0.95)
        got = {f: int(d_h[b, i]) for i, f in enumerate(F)}
        assert got == ref, (b, {f: (got[f], ref[f]) for f in F if got[f] != ref[f]})
    n_col = F.index("n")
    assert d_h[4, n_col] == 0 and d_h[5, n_col] == 2 ** 30      # t clamped to [-1, 2^30 - 1]
    assert d_h[6, n_col] == 501
    for b in (4, 6):                                             # empty monitored stream
        assert d_h[b, F.index("trigger")] == 0 and d_h[b, F.index("distinct")] == 0
    # t0 = -9 clamps to 0: the stream is the first 401 ring entries
    ref7 = oracle.Detector(p).step(ring_h[7][:401], 0, 401, 0.95)
    got7 = {f: int(d_h[7, i]) for i, f in enumerate(F)}
    assert got7 == ref7, {f: (got7[f], ref7[f]) for f in F if got7[f] != ref7[f]}


def test_prune_clamps_lengths_and_budgets():
    from paper_2604_10044_amd import lg
    rng = np.random.default_rng(5)
    p = oracle.paper_params()
    B, cap, D = 6, 512, 128
    dev = torch.device("cuda")
    lens = np.array([511, 300, -4, I32_MAX, 200, 512], np.int32)
    budget = np.array([512, 256, 256, 512, I32_MIN, I32_MAX], np.int32)
    pos = np.tile(np.arange(cap, dtype=np.int32) * 2, (B, 1))
    tapp = np.array([2 * 511 + 1, 2 * 300 + 1, 1, I32_MAX, 2 * 200 + 1, 5000], np.int32)
    K = torch.randn(B, 2, cap, D, device=dev).to(torch.bfloat16)
    V = torch.randn(B, 2, cap, D, device=dev).to(torch.bfloat16)
    A = torch.rand(B, 2, cap, device=dev)
    K0, V0 = K.clone(), V.clone()
    pos_d, len_d = torch.from_numpy(pos).to(dev), torch.from_numpy(lens).to(dev)
    kidx = torch.full((B, cap), -7, dtype=torch.int32, device=dev)
    nlen = torch.zeros(B, dtype=torch.int32, device=dev)
    lg.lg_prune_compact(lg.params_from_dict(p), B, cap, [lg.layer_cache(K, V, A, 4)], pos_d, len_d,
                        torch.from_numpy(budget).to(dev), torch.from_numpy(tapp).to(dev), None,
                        kidx, nlen)
    torch.cuda.synchronize()
    len_h, nlen_h, pos_h = len_d.cpu().numpy(), nlen.cpu().numpy(), pos_d.cpu().numpy()
    # valid rows: row 0 overflows its 512 budget after the append and is reduced by the keep rule
    for b in (0, 1):
        L = int(lens[b]) + 1
        p_ref = np.append(pos[b, :L - 1], tapp[b]).astype(np.int32)
        if L >= budget[b]:
            keep = oracle.keep_set(p, p_ref, int(budget[b]), -1, 0)
            assert nlen_h[b] == len(keep) and len_h[b] == len(keep)
            np.testing.assert_array_equal(pos_h[b, :len(keep)], p_ref[keep])
            kt = torch.from_numpy(keep.astype(np.int64)).to(dev)
            assert torch.equal(K[b, :, :len(keep)], K0[b].index_select(1, kt))
        else:
            assert nlen_h[b] == -1 and len_h[b] == L
    # out-of-range rows: every length stays inside [0, cap]
    assert np.all((len_h >= 0) & (len_h <= cap))
    assert len_h[2] == 1                    # len -4 clamps to 0, then the append
