"""GPU parity of lg_decode_attend against the oracle (Eq. (1) and the fused statistics).

Tolerances (bf16/fp32 inputs, fp32 accumulation in the kernels, fp64 in the oracle):
  out          |gpu - ref| <= 2e-2 |ref| + 1e-3 max|ref row|   (2e-2 relative; bf16 output rounding
               is 2^-9 relative)
  lse          |gpu - ref| <= 2e-4 max(1, |ref|)
  suffix mass  |gpu - ref| <= 2e-4 (a sum of probabilities, each within ~1e-6 relative)
  acc          |gpu - ref| <= 1e-4 max(1, |ref|)
  conf         equals the largest GPU suffix mass bit for bit; within 2e-4 of the oracle's
"""
import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu


def _round_bf16(x: np.ndarray) -> np.ndarray:
    return torch.from_numpy(x).to(torch.bfloat16).float().numpy()


def attend_form(ws, B, Hq, Hkv, D, cap):
    """Which MFMA attention form a launch used, read from its zero-filled workspace (the layout of
    lg_decode_attend_workspace): the split form with its merging launch writes the logit stash, the
    one-launch form leaves it untouched and writes its tagged partials instead."""
    G, bh, al = Hq // Hkv, B * Hkv, (lambda x: (x + 255) // 256 * 256)
    ns_max, cap_s, nsq = (cap + 63) // 64, al(cap), min(32, (cap + 127) // 128)
    o_stash = al(al(al(bh * ns_max * G * 8) + bh * ns_max * G * 4) + bh * ns_max * G * D * 4)
    o_tag = al(o_stash + bh * G * cap_s * 4)
    stash_used = bool(ws[o_stash:o_tag].any())
    tags_used = bool(ws[o_tag:o_tag + bh * nsq * G * (D + 3) * 8].any())
    return {(True, False): "merge-launch", (False, True): "one-launch"}.get((stash_used, tags_used),
                                                                           "unknown")


def run_case(B, Hq, Hkv, D, cap, lens, dtype, variant, append=True, seed=0, t_gap=3,
             suffix_w=None, q_scale=None):
    from paper_2604_10044_amd import lg
    rng = np.random.default_rng(seed)
    G = Hq // Hkv
    dev = torch.device("cuda")
    K = rng.standard_normal((B, Hkv, cap, D)).astype(np.float32)
    V = rng.standard_normal((B, Hkv, cap, D)).astype(np.float32)
    q = (rng.standard_normal((B, Hq, D)) * (rng.uniform(0.5, 3.0) if q_scale is None else q_scale)).astype(np.float32)
    kn = rng.standard_normal((B, Hkv, D)).astype(np.float32)
    vn = rng.standard_normal((B, Hkv, D)).astype(np.float32)
    if dtype == "bf16":
        K, V, q, kn, vn = (_round_bf16(x) for x in (K, V, q, kn, vn))
    # slots past the live ones (and past the append) hold NaN: no kernel may let them leak
    for b in range(B):
        K[b, :, lens[b] + 1:] = np.nan
        V[b, :, lens[b] + 1:] = np.nan
    pos = np.zeros((B, cap), np.int32)
    t = np.zeros(B, np.int32)
    for b in range(B):
        L = lens[b]
        p = np.sort(rng.choice(4 * cap + 10, L, replace=False)).astype(np.int32) if L else np.zeros(0, np.int32)
        pos[b, :L] = p
        t[b] = (p[-1] if L else 0) + t_gap
    suffix_w = (rng.integers(0, cap, B) if suffix_w is None else np.full(B, suffix_w)).astype(np.int32)
    acc0 = rng.uniform(0, 50, (B, Hkv, cap)).astype(np.float32)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    to = lambda a: torch.from_numpy(a).to(dev).to(tdt)
    Kd, Vd, qd, knd, vnd = to(K), to(V), to(q), to(kn), to(vn)
    accd = torch.from_numpy(acc0).to(dev)
    layer = lg.layer_cache(Kd, Vd, accd, Hq)
    out = torch.zeros(B, Hq, D, dtype=tdt, device=dev)
    lse = torch.zeros(B, Hq, device=dev)
    sm = torch.zeros(B, Hq, device=dev)
    conf = torch.zeros(B, device=dev)
    ws = torch.zeros(lg.lg_decode_attend_workspace(B, Hq, Hkv, D, cap), dtype=torch.uint8, device=dev)
    lg.lg_decode_attend(layer, qd, knd if append else None, vnd if append else None, out,
                        torch.from_numpy(pos).to(dev), torch.tensor(lens, dtype=torch.int32, device=dev),
                        torch.from_numpy(t).to(dev), torch.from_numpy(suffix_w).to(dev), lse, sm, conf,
                        ws, variant=variant)
    torch.cuda.synchronize()
    out_h, lse_h, sm_h = out.float().cpu().numpy(), lse.cpu().numpy(), sm.cpu().numpy()
    conf_h, acc_h = conf.cpu().numpy(), accd.cpu().numpy()
    K_h, V_h = Kd.float().cpu().numpy(), Vd.float().cpu().numpy()
    for b in range(B):
        L = lens[b]
        n = L + (1 if append else 0)
        for h in range(Hkv):
            Ke, Ve, pe = K[b, h, :L], V[b, h, :L], pos[b, :L]
            if append:
                Ke = np.concatenate([Ke, kn[b, h][None]])
                Ve = np.concatenate([Ve, vn[b, h][None]])
                pe = np.append(pe, t[b])
                # the appended row lands in slot L of the cache
                np.testing.assert_array_equal(K_h[b, h, L], kn[b, h])
                np.testing.assert_array_equal(V_h[b, h, L], vn[b, h])
            o, ls, sg, asum = oracle.attend_group(q[b, h * G:(h + 1) * G], Ke, Ve, pe, int(t[b]),
                                                  int(suffix_w[b]))
            go = out_h[b, h * G:(h + 1) * G]
            if n == 0:
                assert np.all(go == 0) and np.all(np.isneginf(lse_h[b, h * G:(h + 1) * G]))
                assert np.all(sm_h[b, h * G:(h + 1) * G] == 0)
                continue
            rowmax = np.abs(o).max(axis=1, keepdims=True)
            err = np.abs(go - o)
            assert np.all(err <= 2e-2 * np.abs(o) + 1e-3 * rowmax), (b, h, err.max())
            assert np.all(np.abs(lse_h[b, h * G:(h + 1) * G] - ls) <= 2e-4 * np.maximum(1, np.abs(ls)))
            assert np.all(np.abs(sm_h[b, h * G:(h + 1) * G] - sg) <= 2e-4), (b, h)
            ref_acc = acc0[b, h, :n].astype(np.float64)
            if append:
                ref_acc[L] = 0.0
            ref_acc += asum
            assert np.all(np.abs(acc_h[b, h, :n] - ref_acc) <= 1e-4 * np.maximum(1, np.abs(ref_acc))), (b, h)
            # slots beyond the live ones are untouched
            np.testing.assert_array_equal(acc_h[b, h, n:], acc0[b, h, n:])
            assert np.all(np.isnan(K_h[b, h, L + 1:])) and np.all(np.isnan(V_h[b, h, L + 1:]))
        if n:
            assert conf_h[b] == sm_h[b].max()
    return out_h, lse_h, sm_h, acc_h


SHAPES = [
    # B, Hq, Hkv, D, cap, lens
    (3, 4, 4, 64, 256, [0, 191, 255]),
    (2, 12, 2, 128, 1024, [767, 1023]),
    (4, 28, 4, 128, 600, [1, 31, 257, 599]),
    (2, 16, 1, 128, 300, [64, 299]),
    (3, 8, 8, 64, 130, [32, 33, 129]),
    (2, 7, 7, 128, 97, [96, 5]),
]


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("dtype,variant", [("f32", 1), ("bf16", 1), ("bf16", 2), ("bf16", 4),
                                           ("bf16", 9), ("bf16", 14), ("bf16", 15), ("bf16", 16)])
def test_attend_parity(shape, dtype, variant):
    B, Hq, Hkv, D, cap, lens = shape
    if variant >= 2:
        cap = (cap + 31) // 32 * 32   # the MFMA kernels take whole 32-slot blocks
    run_case(B, Hq, Hkv, D, cap, lens, dtype, variant, append=True, seed=sum(lens) + Hq)


@pytest.mark.parametrize("variant", list(range(2, 18)))
def test_attend_every_mfma_variant(variant):
    """Every MFMA configuration the library exposes (lg_decode_attend_variant 2..17: split forms with
    other split lengths, pipelining, occupancy targets, dynamic block assignment, load kinds, the
    fused form and the one-launch split form) on one ragged 7B-like launch, including an empty and a
    full row."""
    run_case(4, 28, 4, 128, 1024, [0, 31, 700, 1023], "bf16", variant, seed=77)


@pytest.mark.parametrize("Hq,Hkv,D", [(16, 1, 128), (8, 1, 64), (4, 1, 128)])
def test_attend_long_splits(Hq, Hkv, D):
    """64 rows over a 2048-slot cache: the automatic choice cuts each row into 512-slot splits,
    long enough that the split form stages its logits in LDS (group bounds 16, 8 and 4); ragged
    lengths include a single live slot, a full cache and a split boundary."""
    rng = np.random.default_rng(Hq + D)
    lens = rng.integers(600, 2047, 64).tolist()
    lens[0], lens[1], lens[2], lens[3] = 0, 2047, 511, 1024
    run_case(64, Hq, Hkv, D, 2048, lens, "bf16", 0, append=True, seed=Hq * 7 + D)


def _random_shape(i):
    rng = np.random.default_rng(1000 + i)
    G = int(rng.choice([1, 2, 4, 7, 8, 16]))
    Hkv = int(rng.integers(1, 5))
    B = int(rng.integers(1, 9))
    D = int(rng.choice([64, 128]))
    cap = 32 * int(rng.integers(1, 129))
    lens = [int(rng.integers(0, cap)) for _ in range(B)]
    if B > 1:
        lens[int(rng.integers(0, B))] = cap - 1     # a row that fills the cache with the append
    if B > 2:
        lens[int(rng.integers(0, B))] = 0           # a row whose only live slot is the append
    return B, G * Hkv, Hkv, D, cap, lens, int(rng.integers(0, cap + 1))


@pytest.mark.parametrize("variant", [0, 1, 15])
@pytest.mark.parametrize("i", range(24))
def test_attend_random_shapes(i, variant):
    """Seeded random launches (group sizes 1-16, 1-4 KV heads, head_dim 64/128, caches of 32-4096
    slots, ragged lengths with a full row and a row holding only the appended slot, random suffix
    widths) under the automatic choice, the portable kernel and the fused form."""
    B, Hq, Hkv, D, cap, lens, sw = _random_shape(i)
    run_case(B, Hq, Hkv, D, cap, lens, "bf16", variant, seed=i, suffix_w=sw)


@pytest.mark.parametrize("variant", [0, 1, 15])
def test_attend_max_cache(variant):
    """The longest cache the MFMA kernels take (cap 32768): the split form at its limit of 32
    splits of 1024 slots (logits staged in LDS), the fused form sweeping 1024 blocks in one
    workgroup, and the portable kernel; one row fills the cache with the appended slot."""
    run_case(2, 8, 2, 128, 32768, [32767, 1000], "bf16", variant, seed=11)


@pytest.mark.parametrize("variant", [1, 2, 15])
@pytest.mark.parametrize("q_scale", [40.0, 1e-3])
def test_attend_extreme_logits(variant, q_scale):
    """Logits spanning hundreds (softmax rows nearly one-hot, every exponent far below the running
    max) and logits near zero (nearly uniform rows)."""
    run_case(3, 8, 2, 128, 512, [511, 300, 37], "bf16", variant, seed=11, q_scale=q_scale)


@pytest.mark.parametrize("variant", [1, 2, 15])
def test_attend_without_append_and_empty(variant):
    run_case(3, 8, 2, 128, 512, [0, 1, 300], "bf16", variant, append=False, seed=5)


@pytest.mark.parametrize("variant", [1, 2, 15])
def test_attend_suffix_extremes(variant):
    # a suffix wider than every position: mass 1; width 0: mass 0
    _, _, sm, _ = run_case(2, 4, 1, 128, 128, [100, 126], "bf16", variant, seed=9, suffix_w=10 ** 6)
    np.testing.assert_allclose(sm, 1.0, atol=2e-6)
    _, _, sm, _ = run_case(2, 4, 1, 128, 128, [100, 126], "bf16", variant, seed=9, suffix_w=0)
    assert np.all(sm == 0)


@pytest.mark.parametrize("variant", [1, 2, 15])
def test_attend_without_conf(variant):
    """conf may be NULL: every other output is unchanged."""
    from paper_2604_10044_amd import lg
    dev = torch.device("cuda")
    B, Hq, Hkv, D, cap = 2, 8, 2, 128, 256
    g = torch.Generator(device="cpu").manual_seed(3)
    K = torch.randn(B, Hkv, cap, D, generator=g).to(dev).to(torch.bfloat16)
    V = torch.randn(B, Hkv, cap, D, generator=g).to(dev).to(torch.bfloat16)
    q = torch.randn(B, Hq, D, generator=g).to(dev).to(torch.bfloat16)
    pos = torch.arange(cap, dtype=torch.int32).repeat(B, 1).contiguous().to(dev)
    lens = torch.tensor([100, 255], dtype=torch.int32, device=dev)
    t = lens + 1
    sw = torch.full((B,), 64, dtype=torch.int32, device=dev)
    ws = torch.zeros(lg.lg_decode_attend_workspace(B, Hq, Hkv, D, cap), dtype=torch.uint8, device=dev)
    res = []
    for with_conf in (True, False):
        acc = torch.zeros(B, Hkv, cap, device=dev)
        out = torch.zeros(B, Hq, D, dtype=torch.bfloat16, device=dev)
        lse = torch.zeros(B, Hq, device=dev)
        sm = torch.zeros(B, Hq, device=dev)
        conf = torch.zeros(B, device=dev) if with_conf else None
        lg.lg_decode_attend(lg.layer_cache(K, V, acc, Hq), q, None, None, out, pos, lens, t, sw,
                            lse, sm, conf, ws, variant=variant)
        torch.cuda.synchronize()
        res.append((out.float().cpu(), lse.cpu(), sm.cpu(), acc.cpu()))
    for a, b in zip(res[0], res[1]):
        assert torch.equal(a, b)


def test_variants_agree():
    a = run_case(2, 28, 4, 128, 704, [500, 699], "bf16", 1, seed=21)
    b = run_case(2, 28, 4, 128, 704, [500, 699], "bf16", 2, seed=21)
    np.testing.assert_allclose(a[2], b[2], atol=2e-5)
    np.testing.assert_allclose(a[1], b[1], atol=1e-4)


def test_bench_shape_sampled_against_oracle():
    """The 7B-shaped layer at full size (batch 32, 28/4 heads, head_dim 128, budget 2048, the
    prefill length of 1536 slots) in the launch configuration the benchmark uses, with the
    generator's rows (locked heads included); every (sequence, kv head) is compared."""
    from paper_2604_10044_amd import lg
    from paper_2604_10044_amd.synth import KIND_K, KIND_Q, KIND_V, llama7b
    from oracle.trajectory import prefill_positions
    wl = llama7b(steps=1)
    B, Hq, Hkv, D, cap = 32, 28, 4, 128, 2048
    G = Hq // Hkv
    layer_id = 20
    p = oracle.paper_params()
    pos0 = prefill_positions(p, 8192, 2048)
    n0 = len(pos0)
    pos = np.zeros((B, cap), np.int32)
    pos[:, :n0] = pos0
    K = wl.rows(KIND_K, layer_id, layer_id + 1, range(B), pos, np.full(B, n0, np.int32))[0]
    V = wl.rows(KIND_V, layer_id, layer_id + 1, range(B), pos, np.full(B, n0, np.int32))[0]
    tp = np.full((B, 1), 8192, np.int32)
    q = wl.rows(KIND_Q, layer_id, layer_id + 1, range(B), tp)[0][:, :, 0]
    kn = wl.rows(KIND_K, layer_id, layer_id + 1, range(B), tp)[0][:, :, 0]
    vn = wl.rows(KIND_V, layer_id, layer_id + 1, range(B), tp)[0][:, :, 0]
    dev = torch.device("cuda")
    tb = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(torch.bfloat16)
    f32 = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).float().numpy()
    Kd, Vd = tb(K), tb(V)
    accd = torch.zeros(B, Hkv, cap, device=dev)
    layer = lg.layer_cache(Kd, Vd, accd, Hq)
    out = torch.zeros(B, Hq, D, dtype=torch.bfloat16, device=dev)
    lse = torch.zeros(B, Hq, device=dev)
    sm = torch.zeros(B, Hq, device=dev)
    conf = torch.zeros(B, device=dev)
    ws = torch.zeros(lg.lg_decode_attend_workspace(B, Hq, Hkv, D, cap), dtype=torch.uint8, device=dev)
    lens = torch.full((B,), n0, dtype=torch.int32, device=dev)
    t = torch.full((B,), 8192, dtype=torch.int32, device=dev)
    sw = torch.full((B,), 512, dtype=torch.int32, device=dev)
    lg.lg_decode_attend(layer, tb(q), tb(kn), tb(vn), out, torch.from_numpy(pos).to(dev), lens, t,
                        sw, lse, sm, conf, ws)
    torch.cuda.synchronize()
    out_h, sm_h, acc_h = out.float().cpu().numpy(), sm.cpu().numpy(), accd.cpu().numpy()
    Kf, Vf, qf, knf, vnf = f32(K), f32(V), f32(q), f32(kn), f32(vn)
    pe = np.append(pos0, 8192).astype(np.int32)
    worst = 0.0
    for b in range(B):
        for h in range(Hkv):
            Ke = np.concatenate([Kf[b, h, :n0], knf[b, h][None]])
            Ve = np.concatenate([Vf[b, h, :n0], vnf[b, h][None]])
            o, ls, sg, asum = oracle.attend_group(qf[b, h * G:(h + 1) * G], Ke, Ve, pe, 8192, 512)
            go = out_h[b, h * G:(h + 1) * G]
            rowmax = np.abs(o).max(axis=1, keepdims=True)
            assert np.all(np.abs(go - o) <= 2e-2 * np.abs(o) + 1e-3 * rowmax)
            assert np.all(np.abs(sm_h[b, h * G:(h + 1) * G] - sg) <= 2e-4)
            assert np.all(np.abs(acc_h[b, h, :n0 + 1] - asum) <= 1e-4 * np.maximum(1, asum))
            worst = max(worst, float(np.abs(sm_h[b, h * G:(h + 1) * G] - sg).max()))
    print("worst suffix-mass error", worst)


def _full_size_layer_case(wl, layer_id, pairs, variant=0):
    """One layer of a workload at full size in its first decode step: every sequence holds its own
    prefill-reduced context (ragged lengths and budgets), the step's row is appended, and the
    (sequence, kv head) pairs listed are compared with the oracle."""
    from paper_2604_10044_amd import lg
    from paper_2604_10044_amd.synth import KIND_K, KIND_Q, KIND_V
    from oracle.trajectory import prefill_positions
    B, Hq, Hkv, D, cap = wl.batch, wl.n_q_heads, wl.n_kv_heads, wl.head_dim, wl.cap
    G = Hq // Hkv
    p = oracle.paper_params()
    ctx = np.asarray(wl.ctx, np.int64)
    budget = np.asarray(wl.budget, np.int32)
    pos = np.zeros((B, cap), np.int32)
    lens = np.zeros(B, np.int32)
    for b in range(B):
        pb = prefill_positions(p, int(ctx[b]), int(budget[b]))
        pos[b, :len(pb)] = pb
        lens[b] = len(pb)
    K = wl.rows(KIND_K, layer_id, layer_id + 1, range(B), pos, lens)[0]
    V = wl.rows(KIND_V, layer_id, layer_id + 1, range(B), pos, lens)[0]
    tp = ctx.astype(np.int32)[:, None]
    q = wl.rows(KIND_Q, layer_id, layer_id + 1, range(B), tp)[0][:, :, 0]
    kn = wl.rows(KIND_K, layer_id, layer_id + 1, range(B), tp)[0][:, :, 0]
    vn = wl.rows(KIND_V, layer_id, layer_id + 1, range(B), tp)[0][:, :, 0]
    dev = torch.device("cuda")
    tb = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(torch.bfloat16)
    f32 = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).float().numpy()
    Kd, Vd = tb(K), tb(V)
    acc0 = np.random.default_rng(layer_id).uniform(0, 4, (B, Hkv, cap)).astype(np.float32)
    accd = torch.from_numpy(acc0).to(dev)
    layer = lg.layer_cache(Kd, Vd, accd, Hq)
    out = torch.zeros(B, Hq, D, dtype=torch.bfloat16, device=dev)
    lse = torch.zeros(B, Hq, device=dev)
    sm = torch.zeros(B, Hq, device=dev)
    conf = torch.zeros(B, device=dev)
    ws = torch.zeros(lg.lg_decode_attend_workspace(B, Hq, Hkv, D, cap), dtype=torch.uint8, device=dev)
    sw = (budget // int(p["recent_div"])).astype(np.int32)
    lg.lg_decode_attend(layer, tb(q), tb(kn), tb(vn), out, torch.from_numpy(pos).to(dev),
                        torch.from_numpy(lens).to(dev), torch.from_numpy(tp[:, 0].copy()).to(dev),
                        torch.from_numpy(sw).to(dev), lse, sm, conf, ws, variant=variant)
    torch.cuda.synchronize()
    out_h, sm_h, lse_h = out.float().cpu().numpy(), sm.cpu().numpy(), lse.cpu().numpy()
    conf_h = conf.cpu().numpy()
    qf, knf, vnf = f32(q), f32(kn), f32(vn)
    for b, h in pairs:
        n0 = int(lens[b])
        Ke = np.concatenate([f32(K[b, h, :n0]), knf[b, h][None]])
        Ve = np.concatenate([f32(V[b, h, :n0]), vnf[b, h][None]])
        # the appended row lands in slot n0 of the cache
        np.testing.assert_array_equal(Kd[b, h, n0].float().cpu().numpy(), knf[b, h])
        np.testing.assert_array_equal(Vd[b, h, n0].float().cpu().numpy(), vnf[b, h])
        pe = np.append(pos[b, :n0], tp[b, 0]).astype(np.int32)
        o, ls, sg, asum = oracle.attend_group(qf[b, h * G:(h + 1) * G], Ke, Ve, pe, int(tp[b, 0]),
                                              int(sw[b]))
        go = out_h[b, h * G:(h + 1) * G]
        rowmax = np.abs(o).max(axis=1, keepdims=True)
        assert np.all(np.abs(go - o) <= 2e-2 * np.abs(o) + 1e-3 * rowmax), (b, h)
        assert np.all(np.abs(lse_h[b, h * G:(h + 1) * G] - ls) <= 2e-4 * np.maximum(1, np.abs(ls)))
        assert np.all(np.abs(sm_h[b, h * G:(h + 1) * G] - sg) <= 2e-4), (b, h)
        ref_acc = acc0[b, h, :n0 + 1].astype(np.float64)
        ref_acc[n0] = 0.0
        ref_acc += asum
        got_acc = accd[b, h, :n0 + 1].cpu().numpy()
        assert np.all(np.abs(got_acc - ref_acc) <= 1e-4 * np.maximum(1, np.abs(ref_acc))), (b, h)
        np.testing.assert_array_equal(accd[b, h, n0 + 1:].cpu().numpy(), acc0[b, h, n0 + 1:])
    # conf = max suffix mass over all heads of the sequence (every head, not only the sampled ones)
    np.testing.assert_array_equal(conf_h, sm_h.max(axis=1))
    if variant == 0:
        # the automatic choice: the one-launch form when the grid has at most one workgroup per CU
        # (the library's split choice: ~256 workgroups, 128..1024 slots, at most 32 splits per row)
        rows = B * Hkv
        want = max(128, ((cap * rows + 255) // 256 + 31) // 32 * 32)
        min_split = ((cap + 31) // 32 + 31) // 32 * 32
        split = max(min(1024, want), min_split)
        grid = rows * -(-cap // split)
        want = "one-launch" if grid <= torch.cuda.get_device_properties(0).multi_processor_count \
            else "merge-launch"
        assert attend_form(ws, B, Hq, Hkv, D, cap) == want, (grid, want)
    return lens


@pytest.mark.parametrize("variant", [0, 15])
def test_7b_layer_full_size(variant):
    """7B-shaped batch 32 (28/4 heads, budget 2048, context 8192): layer 3, every (sequence, kv
    head), with the default kernel choice and with the fused one-workgroup-per-row sweep."""
    from paper_2604_10044_amd.synth import llama7b
    wl = llama7b(steps=1)
    pairs = [(b, h) for b in range(wl.batch) for h in range(wl.n_kv_heads)]
    lens = _full_size_layer_case(wl, 3, pairs, variant)
    assert np.all(lens == 1536)


@pytest.mark.parametrize("variant", [0, 15])
def test_8b_long_context_layer_full_size(variant):
    """8B-shaped long context (batch 8, 32/8 heads, budget 4096, context 32768): layer 20 (a locked
    layer), every (sequence, kv head)."""
    from paper_2604_10044_amd.synth import llama8b_long
    wl = llama8b_long(steps=1)
    pairs = [(b, h) for b in range(wl.batch) for h in range(wl.n_kv_heads)]
    lens = _full_size_layer_case(wl, 20, pairs, variant)
    assert np.all(lens == 3072)


@pytest.mark.parametrize("variant", [0, 15])
def test_ragged_layer_full_size(variant):
    """Ragged stress (batch 64, contexts 512..65536, budgets 512/2048/8192 in one cap-8192 launch,
    duplicate key rows): layer 17, kv heads 0 and 7 of every sequence."""
    from paper_2604_10044_amd.synth import ragged
    wl = ragged(steps=1, n_layers=32)
    pairs = [(b, h) for b in range(wl.batch) for h in (0, 7)]
    lens = _full_size_layer_case(wl, 17, pairs, variant)
    assert len(set(lens.tolist())) > 3 and lens.max() > 4096 and lens.min() < 512


def test_one_launch_form_matches_merge_launch():
    """The one-launch split form (variant 17: the splits of a row exchange tagged partials through
    memory) and the split form with its merging launch (variant 9) run the same sweep and merge the
    same partials in the same order, so over consecutive launches on one workspace their outputs,
    lse, suffix mass and conf are identical bit for bit; acc differs only by the rounding of the
    factored probability (exp2(s - m_split) * exp2(m_split - M) / Z). The row lengths change from
    launch to launch (rows of 1 to 16 splits of 128 slots, a row that drops to one split and grows
    back, an empty row), so stale partials of an earlier launch must never be taken for current
    ones. The grid (4 KV heads x 4 sequences x 16 splits) is one workgroup per CU, so variant 17
    runs the one-launch form: its logit stash stays untouched and its tagged partials are written."""
    from paper_2604_10044_amd import lg
    dev = torch.device("cuda")
    B, Hq, Hkv, D, cap = 4, 28, 4, 128, 2048
    g = torch.Generator(device="cpu").manual_seed(12)
    K = torch.randn(B, Hkv, cap, D, generator=g).to(torch.bfloat16).to(dev)
    V = torch.randn(B, Hkv, cap, D, generator=g).to(torch.bfloat16).to(dev)
    steps = [[1500, 2040, 64, 0], [1501, 2041, 65, 0], [300, 100, 66, 0], [301, 2042, 67, 0],
             [1502, 2043, 68, 0]]
    pos = torch.arange(cap, dtype=torch.int32).repeat(B, 1).contiguous().to(dev)
    sw = torch.full((B,), 300, dtype=torch.int32, device=dev)
    acc0 = torch.rand(B, Hkv, cap, generator=g).to(dev)
    wsn = lg.lg_decode_attend_workspace(B, Hq, Hkv, D, cap)
    res = {}
    for variant in (9, 17):
        Kc, Vc, acc = K.clone(), V.clone(), acc0.clone()
        ws = torch.zeros(wsn, dtype=torch.uint8, device=dev)
        outs = []
        for step, lens_l in enumerate(steps):
            gs = torch.Generator(device="cpu").manual_seed(100 + step)
            q = (2 * torch.randn(B, Hq, D, generator=gs)).to(torch.bfloat16).to(dev)
            kn = torch.randn(B, Hkv, D, generator=gs).to(torch.bfloat16).to(dev)
            vn = torch.randn(B, Hkv, D, generator=gs).to(torch.bfloat16).to(dev)
            lens = torch.tensor(lens_l, dtype=torch.int32, device=dev)
            t = lens.clone()
            out = torch.zeros(B, Hq, D, dtype=torch.bfloat16, device=dev)
            lse = torch.zeros(B, Hq, device=dev)
            sm = torch.zeros(B, Hq, device=dev)
            conf = torch.zeros(B, device=dev)
            lg.lg_decode_attend(lg.layer_cache(Kc, Vc, acc, Hq), q, kn, vn, out, pos, lens, t, sw,
                                lse, sm, conf, ws, variant=variant)
            torch.cuda.synchronize()
            outs.append((out.cpu(), lse.cpu(), sm.cpu(), conf.cpu(), acc.cpu()))
        assert all(torch.isfinite(o[4]).all() and torch.isfinite(o[0].float()).all() for o in outs)
        assert attend_form(ws, B, Hq, Hkv, D, cap) == ("merge-launch" if variant == 9 else "one-launch")
        res[variant] = outs
    for a, b in zip(res[9], res[17]):
        for x, y in zip(a[:4], b[:4]):
            assert torch.equal(x, y)
        torch.testing.assert_close(a[4], b[4], rtol=1e-6, atol=1e-6)


def test_one_launch_form_many_launches():
    """120 consecutive launches of the one-launch form on one workspace, each with freshly drawn row
    lengths (1 to 16 splits per row, rows that grow, shrink and empty), compared after every launch
    with the split form and its merging launch on the same inputs: outputs, lse and suffix mass bit
    for bit, acc within 1e-6. Exercises the generation word and the tags over many launches."""
    from paper_2604_10044_amd import lg
    dev = torch.device("cuda")
    B, Hq, Hkv, D, cap = 4, 28, 4, 128, 2048
    g = torch.Generator(device="cpu").manual_seed(31)
    K = torch.randn(B, Hkv, cap, D, generator=g).to(torch.bfloat16).to(dev)
    V = torch.randn(B, Hkv, cap, D, generator=g).to(torch.bfloat16).to(dev)
    pos = torch.arange(cap, dtype=torch.int32).repeat(B, 1).contiguous().to(dev)
    sw = torch.full((B,), 200, dtype=torch.int32, device=dev)
    wsn = lg.lg_decode_attend_workspace(B, Hq, Hkv, D, cap)
    ws = {v: torch.zeros(wsn, dtype=torch.uint8, device=dev) for v in (9, 17)}
    acc = {v: torch.zeros(B, Hkv, cap, device=dev) for v in (9, 17)}
    rng = np.random.default_rng(5)
    for step in range(120):
        lens = torch.tensor(rng.integers(0, cap - 1, B), dtype=torch.int32, device=dev)
        q = (2 * torch.randn(B, Hq, D, generator=g)).to(torch.bfloat16).to(dev)
        res = {}
        for v in (9, 17):
            out = torch.zeros(B, Hq, D, dtype=torch.bfloat16, device=dev)
            lse = torch.zeros(B, Hq, device=dev)
            sm = torch.zeros(B, Hq, device=dev)
            lg.lg_decode_attend(lg.layer_cache(K, V, acc[v], Hq), q, None, None, out, pos, lens, lens,
                                sw, lse, sm, None, ws[v], variant=v)
            res[v] = (out, lse, sm)
        torch.cuda.synchronize()
        for x, y in zip(res[9], res[17]):
            assert torch.equal(x, y), step
        torch.testing.assert_close(acc[9], acc[17], rtol=1e-6, atol=1e-6)
    assert attend_form(ws[17], B, Hq, Hkv, D, cap) == "one-launch"
