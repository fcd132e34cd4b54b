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


FORMS = {"auto": 0, "portable": 1, "merge": 2, "one": 3}


def auto_is_single_split(cap, rows, G):
    """The automatic choice runs the one-launch form (one split per row, no exchange) for launches
    of >= 128 rows whose cap fits one split, the merge form otherwise."""
    return rows >= 128 and cap <= (2048 if G <= 8 else 1024)


def split_plan(cap, rows, max_split, n_eff, G=7, one_launch=True):
    """Splits of a row of n_eff live slots in an MFMA launch (the library's plan: the given split
    length; by default, in the one-launch form, one split per row for launches of >= 128 rows
    whose cap fits one (2048 slots for groups of <= 8 heads, else 1024), otherwise ~256
    workgroups with splits of 128..1024 slots; at most 32 per row, balanced and 32-aligned,
    except 128-slot splits, which are fixed)."""
    if max_split:
        split = max_split
    elif one_launch and rows >= 128 and cap <= (2048 if G <= 8 else 1024):
        split = max(cap, 128)
    else:
        split = min(1024, max(128, ((cap * rows + 255) // 256 + 31) // 32 * 32))
    split = max(split, ((cap + 31) // 32 + 31) // 32 * 32)
    if n_eff == 0:
        return split, 0
    if split == 128:  # one block per wave: fixed 128-slot chunks
        return split, -(-n_eff // split)
    ns0 = -(-n_eff // split)
    chunk = (-(-n_eff // ns0) + 31) // 32 * 32
    return split, -(-n_eff // chunk)


def make_ws(lg, layer, form=0, max_split=0):
    ws = torch.empty(lg.lg_test_attend_workspace(layer, form, max_split), dtype=torch.uint8,
                     device="cuda")
    lg.lg_test_attend_workspace_init(layer, form, max_split, ws)
    return ws


def attend(lg, layer, q, kn, vn, out, pos, lens, t, sw, lse, sm, conf, ws, form=0, max_split=0,
           flags=0):
    if form == 0 and max_split == 0 and flags == 0:
        lg.lg_decode_attend(layer, q, kn, vn, out, pos, lens, t, sw, lse, sm, conf, ws)
    else:
        lg.lg_test_decode_attend(layer, q, kn, vn, out, pos, lens, t, sw, lse, sm, conf, ws,
                                 form=form, max_split=max_split, flags=flags)


def run_case(B, Hq, Hkv, D, cap, lens, dtype, form=0, append=True, seed=0, t_gap=3,
             suffix_w=None, q_scale=None, max_split=0, flags=0):
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
    ws = make_ws(lg, layer, form, max_split)
    attend(lg, layer, qd, knd if append else None, vnd if append else None, out,
           torch.from_numpy(pos).to(dev), torch.tensor(lens, dtype=torch.int32, device=dev),
           torch.from_numpy(t).to(dev), torch.from_numpy(suffix_w).to(dev), lse, sm, conf, ws,
           form, max_split, flags)
    torch.cuda.synchronize()
    assert lg.workspace_header(ws)["status"] == 0
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
@pytest.mark.parametrize("dtype,form,max_split", [("f32", "portable", 0), ("bf16", "portable", 0),
                                                  ("bf16", "auto", 0), ("bf16", "one", 0),
                                                  ("bf16", "one", 128), ("bf16", "merge", 0),
                                                  ("bf16", "merge", 256)])
def test_attend_parity(shape, dtype, form, max_split):
    B, Hq, Hkv, D, cap, lens = shape
    if form in ("one", "merge") or (form == "auto" and dtype == "bf16"):
        cap = (cap + 31) // 32 * 32   # the MFMA kernels take whole 32-slot blocks
    run_case(B, Hq, Hkv, D, cap, lens, dtype, FORMS[form], append=True, seed=sum(lens) + Hq,
             max_split=max_split)


@pytest.mark.parametrize("form", ["one", "merge"])
@pytest.mark.parametrize("max_split", [0, 128, 256, 512, 1024])
def test_attend_every_form_and_split(form, max_split):
    """Both MFMA forms at every split bound on one ragged 7B-like launch, including an empty and a
    full row: 1 to 8 splits per row, one-split rows (merged without an exchange) and multi-split
    rows side by side."""
    run_case(4, 28, 4, 128, 1024, [0, 31, 700, 1023], "bf16", FORMS[form], seed=77,
             max_split=max_split)


@pytest.mark.parametrize("Hq,Hkv,D,cap,lens", [
    (12, 2, 128, 1024, [0, 1]), (12, 2, 128, 1024, [31, 100]), (12, 2, 128, 1024, [288, 289]),
    (12, 2, 128, 1024, [300, 769]), (12, 2, 128, 1024, [1000, 1023]),
    (16, 1, 64, 512, [130, 511]), (32, 2, 128, 1024, [97, 700]), (4, 4, 128, 256, [255, 129])])
def test_fixed_chunk_rows(Hq, Hkv, D, cap, lens):
    """Launches of a few rows (batch 2 or less): the automatic choice cuts rows into 128-slot
    splits, which start at fixed slots, and the merging launch's grid has more workgroups than
    most rows have splits; those past a row's last split still merge their slice of the output.
    Lengths around the 288-slot point below which a balanced plan would have used shorter
    splits; group sizes 6, 16 (head_dim 64 and 128) and 1 cover the three compiled group
    bounds of the merging kernel."""
    from paper_2604_10044_amd import lg
    kv = torch.zeros(1, Hkv, cap, D, dtype=torch.bfloat16, device="cuda")
    hdr = lg.workspace_header(make_ws(lg, lg.layer_cache(kv, kv, torch.zeros(1, Hkv, cap,
                                                                              device="cuda"), Hq)))
    assert (hdr["form"], hdr["split"]) == (FORMS["merge"], 128)
    run_case(len(lens), Hq, Hkv, D, cap, lens, "bf16", 0, append=True, seed=sum(lens) + Hq)


@pytest.mark.parametrize("Hq,Hkv,D", [(16, 1, 128), (8, 1, 64), (4, 1, 128)])
def test_attend_long_splits(Hq, Hkv, D):
    """64 rows over a 2048-slot cache: the automatic choice cuts each row into 512-slot splits,
    long enough that the split form stages its logits in LDS (group bounds 16, 8 and 4); ragged
    lengths include a single live slot, a full cache and a split boundary."""
    rng = np.random.default_rng(Hq + D)
    lens = rng.integers(600, 2047, 64).tolist()
    lens[0], lens[1], lens[2], lens[3] = 0, 2047, 511, 1024
    run_case(64, Hq, Hkv, D, 2048, lens, "bf16", 0, append=True, seed=Hq * 7 + D)


@pytest.mark.parametrize("B,Hq,Hkv,D,cap", [(32, 28, 4, 128, 2048), (32, 32, 4, 64, 2048),
                                             (32, 64, 4, 128, 1024), (16, 8, 8, 128, 1056),
                                             (40, 28, 4, 128, 1536)])
@pytest.mark.parametrize("whole_dims", [False, True])
def test_single_split_rows(B, Hq, Hkv, D, cap, whole_dims):
    """Launches of >= 128 rows whose cap fits one split (up to 2048 slots for groups of <= 8 heads,
    1024 for 16): each row is finished without an exchange, by one workgroup or, for at most 128
    rows of head_dim 128 and splits over 1024 slots, by two that each form half of the output dims
    (whole_dims forces one). Ragged lengths with an empty row, a single slot, a full cache, and
    lengths around 1024."""
    from paper_2604_10044_amd import lg
    rng = np.random.default_rng(B * Hq + cap)
    lens = rng.integers(0, cap, B).tolist()
    lens[0], lens[1], lens[2], lens[3] = 0, 1, cap - 1, min(cap - 1, 1024)
    assert split_plan(cap, B * Hkv, 0, 1, Hq // Hkv)[0] == cap
    run_case(B, Hq, Hkv, D, cap, lens, "bf16", 0, seed=cap + Hq,
             flags=lg.TEST_WHOLE_DIMS if whole_dims else 0)


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


@pytest.mark.parametrize("form,max_split", [("auto", 0), ("portable", 0), ("one", 128),
                                            ("merge", 0)])
@pytest.mark.parametrize("i", range(24))
def test_attend_random_shapes(i, form, max_split):
    """Seeded random launches (group sizes 1-16, 1-4 KV heads, head_dim 64/128, caches of 32-4096
    slots, ragged lengths with a full row and a row holding only the appended slot, random suffix
    widths) under the automatic choice, the portable kernels, the one-launch form with the shortest
    splits (the most splits per row) and the merge form."""
    B, Hq, Hkv, D, cap, lens, sw = _random_shape(i)
    run_case(B, Hq, Hkv, D, cap, lens, "bf16", FORMS[form], seed=i, suffix_w=sw,
             max_split=max_split)


@pytest.mark.parametrize("form", ["auto", "portable", "merge"])
def test_attend_max_cache(form):
    """The longest cache the MFMA kernels take (cap 32768): 32 splits of 1024 slots (logits staged
    in LDS) in the one-launch and the merge form, and the portable kernels; one row fills the cache
    with the appended slot."""
    run_case(2, 8, 2, 128, 32768, [32767, 1000], "bf16", FORMS[form], seed=11)


@pytest.mark.parametrize("form", ["portable", "merge", "one"])
@pytest.mark.parametrize("q_scale", [40.0, 1e-3])
def test_attend_extreme_logits(form, q_scale):
    """Logits spanning hundreds (softmax rows nearly one-hot, every exponent far below the running
    max) and logits near zero (nearly uniform rows)."""
    run_case(3, 8, 2, 128, 512, [511, 300, 37], "bf16", FORMS[form], seed=11, q_scale=q_scale,
             max_split=128 if form == "one" else 0)


@pytest.mark.parametrize("form", ["portable", "merge", "one"])
def test_attend_without_append_and_empty(form):
    run_case(3, 8, 2, 128, 512, [0, 1, 300], "bf16", FORMS[form], append=False, seed=5)


@pytest.mark.parametrize("form", ["portable", "merge", "one"])
def test_attend_suffix_extremes(form):
    # a suffix wider than every position: mass 1; width 0: mass 0
    _, _, sm, _ = run_case(2, 4, 1, 128, 128, [100, 126], "bf16", FORMS[form], seed=9,
                           suffix_w=10 ** 6)
    np.testing.assert_allclose(sm, 1.0, atol=2e-6)
    _, _, sm, _ = run_case(2, 4, 1, 128, 128, [100, 126], "bf16", FORMS[form], seed=9, suffix_w=0)
    assert np.all(sm == 0)


def _rand_layer(B, Hq, Hkv, D, cap, seed):
    g = torch.Generator(device="cpu").manual_seed(seed)
    dev = torch.device("cuda")
    K = torch.randn(B, Hkv, cap, D, generator=g).to(torch.bfloat16).to(dev)
    V = torch.randn(B, Hkv, cap, D, generator=g).to(torch.bfloat16).to(dev)
    return g, K, V


@pytest.mark.parametrize("form", ["portable", "merge", "one"])
def test_attend_without_conf(form):
    """conf may be NULL: every other output is unchanged."""
    from paper_2604_10044_amd import lg
    dev = torch.device("cuda")
    B, Hq, Hkv, D, cap = 2, 8, 2, 128, 256
    g, K, V = _rand_layer(B, Hq, Hkv, D, cap, 3)
    q = torch.randn(B, Hq, D, generator=g).to(dev).to(torch.bfloat16)
    pos = torch.arange(cap, dtype=torch.int32).repeat(B, 1).contiguous().to(dev)
    lens = torch.tensor([100, 255], dtype=torch.int32, device=dev)
    t = lens + 1
    sw = torch.full((B,), 64, dtype=torch.int32, device=dev)
    res = []
    for with_conf in (True, False):
        acc = torch.zeros(B, Hkv, cap, device=dev)
        layer = lg.layer_cache(K, V, acc, Hq)
        ws = make_ws(lg, layer, FORMS[form], 128 if form == "one" else 0)
        out = torch.zeros(B, Hq, D, dtype=torch.bfloat16, device=dev)
        lse = torch.zeros(B, Hq, device=dev)
        sm = torch.zeros(B, Hq, device=dev)
        conf = torch.zeros(B, device=dev) if with_conf else None
        attend(lg, layer, q, None, None, out, pos, lens, t, sw, lse, sm, conf, ws, FORMS[form],
               128 if form == "one" else 0)
        torch.cuda.synchronize()
        res.append((out.float().cpu(), lse.cpu(), sm.cpu(), acc.cpu()))
    for a, b in zip(res[0], res[1]):
        assert torch.equal(a, b)


def test_forms_agree():
    a = run_case(2, 28, 4, 128, 704, [500, 699], "bf16", FORMS["portable"], seed=21)
    b = run_case(2, 28, 4, 128, 704, [500, 699], "bf16", FORMS["one"], seed=21, max_split=128)
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
    ws = make_ws(lg, layer)
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


def _full_size_layer_case(wl, layer_id, pairs, form=0, max_split=0, flags=0):
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
    ws = make_ws(lg, layer, form, max_split)
    sw = (budget // int(p["recent_div"])).astype(np.int32)
    attend(lg, layer, tb(q), tb(kn), tb(vn), out, torch.from_numpy(pos).to(dev),
           torch.from_numpy(lens).to(dev), torch.from_numpy(tp[:, 0].copy()).to(dev),
           torch.from_numpy(sw).to(dev), lse, sm, conf, ws, form, max_split, flags)
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
    hd = lg.workspace_header(ws)
    assert hd["status"] == 0
    if form == 0:
        # bfloat16 layers run the one-launch form when every row is one split, else the merge
        # form, with the library's split plan
        G = wl.n_q_heads // wl.n_kv_heads
        rows = wl.batch * wl.n_kv_heads
        one = auto_is_single_split(wl.cap, rows, G)
        assert hd["form"] == FORMS["one" if one else "merge"], hd
        want = split_plan(wl.cap, rows, 0, 1, G, one_launch=one)[0]
        assert hd["split"] == want, (hd, want)
    return lens


@pytest.mark.parametrize("whole_dims", [False, True])
def test_7b_layer_full_size(whole_dims):
    """7B-shaped batch 32 (28/4 heads, budget 2048, context 8192): layer 3, every (sequence, kv
    head), in the launch configuration of the benchmark (the one-launch form, one 2048-slot split
    per row, two workgroups per row each forming half of the output dims: 256 workgroups, no
    exchange), and with one workgroup per row (whole_dims)."""
    from paper_2604_10044_amd import lg
    from paper_2604_10044_amd.synth import llama7b
    wl = llama7b(steps=1)
    pairs = [(b, h) for b in range(wl.batch) for h in range(wl.n_kv_heads)]
    lens = _full_size_layer_case(wl, 3, pairs, flags=lg.TEST_WHOLE_DIMS if whole_dims else 0)
    assert np.all(lens == 1536)


@pytest.mark.parametrize("max_split", [512, 1024])
def test_7b_layer_full_size_exchange(max_split):
    """The same layer with the exchange: 1024-slot splits (2 per row, 256 workgroups) and 512-slot
    splits (3 per row, 384 workgroups: more than one per CU, so the grid is ordered row-major);
    every (sequence, kv head) compared."""
    from paper_2604_10044_amd.synth import llama7b
    wl = llama7b(steps=1)
    pairs = [(b, h) for b in range(wl.batch) for h in range(wl.n_kv_heads)]
    _full_size_layer_case(wl, 3, pairs, FORMS["one"], max_split)


@pytest.mark.parametrize("form", ["auto", "merge"])
def test_8b_long_context_layer_full_size(form):
    """8B-shaped long context (batch 8, 32/8 heads, budget 4096, context 32768): layer 20 (a locked
    layer), every (sequence, kv head)."""
    from paper_2604_10044_amd.synth import llama8b_long
    wl = llama8b_long(steps=1)
    pairs = [(b, h) for b in range(wl.batch) for h in range(wl.n_kv_heads)]
    lens = _full_size_layer_case(wl, 20, pairs, FORMS[form])
    assert np.all(lens == 3072)


def test_ragged_layer_full_size():
    """Ragged stress (batch 64, contexts 512..65536, budgets 512/2048/8192 in one cap-8192 launch,
    duplicate key rows): layer 17, every (sequence, kv head). 4096 workgroups, many more than the
    device holds at once."""
    from paper_2604_10044_amd.synth import ragged
    wl = ragged(steps=1, n_layers=32)
    pairs = [(b, h) for b in range(wl.batch) for h in range(wl.n_kv_heads)]
    lens = _full_size_layer_case(wl, 17, pairs)
    assert len(set(lens.tolist())) > 3 and lens.max() > 4096 and lens.min() < 512


# ------------------------------------------------------------------------------------------------
# The one-launch form's exchange over many launches, its rare paths and its error paths.
# ------------------------------------------------------------------------------------------------

def _launch_seq(lg, K, V, acc, ws, steps, Hq, form, max_split, flags=0, seed=100, sw_w=300,
                append=True):
    """Consecutive launches on one workspace (row lengths per launch from `steps`); returns the
    outputs of every launch."""
    dev = torch.device("cuda")
    B, Hkv, cap, D = K.shape
    pos = torch.arange(cap, dtype=torch.int32).repeat(B, 1).contiguous().to(dev)
    sw = torch.full((B,), sw_w, dtype=torch.int32, device=dev)
    outs = []
    for step, lens_l in enumerate(steps):
        gs = torch.Generator(device="cpu").manual_seed(seed + step)
        q = (2 * torch.randn(B, Hq, D, generator=gs)).to(torch.bfloat16).to(dev)
        kn = torch.randn(B, Hkv, D, generator=gs).to(torch.bfloat16).to(dev)
        vn = torch.randn(B, Hkv, D, generator=gs).to(torch.bfloat16).to(dev)
        lens = torch.tensor(lens_l, dtype=torch.int32, device=dev)
        out = torch.zeros(B, Hq, D, dtype=torch.bfloat16, device=dev)
        lse = torch.zeros(B, Hq, device=dev)
        sm = torch.zeros(B, Hq, device=dev)
        conf = torch.zeros(B, device=dev)
        attend(lg, lg.layer_cache(K, V, acc, Hq), q, kn if append else None,
               vn if append else None, out, pos, lens, lens, sw, lse, sm, conf, ws, form,
               max_split, flags)
        torch.cuda.synchronize()
        outs.append((out.cpu(), lse.cpu(), sm.cpu(), conf.cpu(), acc.cpu()))
    return outs


# Row lengths that move between 1 and 16 splits of 128 slots, a row that drops to one split and
# grows back, and an empty row.
STEPS16 = [[1500, 2040, 64, 0], [1501, 2041, 65, 0], [300, 100, 66, 0], [301, 2042, 67, 0],
           [1502, 2043, 68, 0], [2045, 90, 1200, 5]]


def test_one_launch_matches_merge_launch():
    """Over consecutive launches on one workspace the one-launch form (the splits of a row exchange
    their partials through memory) agrees with the merge form (the same sweep, partials merged by a
    second launch): the two merge the partials in different orders (per wave here, per split
    there), so out may differ by one bf16 ulp and lse, suffix mass and acc by rounding. A stale
    partial of an earlier launch taken for a current one would break this by far."""
    from paper_2604_10044_amd import lg
    B, Hq, Hkv, D, cap = 4, 28, 4, 128, 2048
    _, K, V = _rand_layer(B, Hq, Hkv, D, cap, 12)
    acc0 = torch.rand(B, Hkv, cap, device="cuda")
    res = {}
    for form in ("merge", "one"):
        Kc, Vc, acc = K.clone(), V.clone(), acc0.clone()
        ws = make_ws(lg, lg.layer_cache(Kc, Vc, acc, Hq), FORMS[form], 128)
        res[form] = _launch_seq(lg, Kc, Vc, acc, ws, STEPS16, Hq, FORMS[form], 128)
        assert lg.workspace_header(ws)["status"] == 0
    for a, b in zip(res["merge"], res["one"]):
        torch.testing.assert_close(a[0].float(), b[0].float(), rtol=8e-3, atol=1e-3)
        torch.testing.assert_close(a[1], b[1], rtol=2e-6, atol=2e-6)
        torch.testing.assert_close(a[2], b[2], rtol=2e-6, atol=2e-6)
        torch.testing.assert_close(a[3], b[3], rtol=2e-6, atol=2e-6)
        torch.testing.assert_close(a[4], b[4], rtol=2e-6, atol=2e-6)


def test_forced_handover_is_bit_identical():
    """Every split that is not its row's closer hands its share over (the path a split takes when
    some split of its row has not started): the closer then finishes those shares from the same
    words in the same order, so every output is identical bit for bit to the default exchange, over
    consecutive launches with changing split counts."""
    from paper_2604_10044_amd import lg
    B, Hq, Hkv, D, cap = 4, 28, 4, 128, 2048
    _, K, V = _rand_layer(B, Hq, Hkv, D, cap, 14)
    acc0 = torch.rand(B, Hkv, cap, device="cuda")
    res = {}
    for flags in (0, lg.TEST_FORCE_HANDOVER):
        Kc, Vc, acc = K.clone(), V.clone(), acc0.clone()
        ws = make_ws(lg, lg.layer_cache(Kc, Vc, acc, Hq), FORMS["one"], 128)
        res[flags] = _launch_seq(lg, Kc, Vc, acc, ws, STEPS16, Hq, FORMS["one"], 128, flags)
        assert lg.workspace_header(ws)["status"] == 0
    for a, b in zip(res[0], res[lg.TEST_FORCE_HANDOVER]):
        for x, y in zip(a, b):
            assert torch.equal(x, y)


def test_one_launch_many_launches():
    """120 consecutive launches of the one-launch form on one workspace, each with freshly drawn row
    lengths (1 to 16 splits per row; rows that grow, shrink and empty), every third one with forced
    handovers, compared after every launch with the merge form on the same inputs."""
    from paper_2604_10044_amd import lg
    dev = torch.device("cuda")
    B, Hq, Hkv, D, cap = 4, 28, 4, 128, 2048
    g, K, V = _rand_layer(B, Hq, Hkv, D, cap, 31)
    pos = torch.arange(cap, dtype=torch.int32).repeat(B, 1).contiguous().to(dev)
    sw = torch.full((B,), 200, dtype=torch.int32, device=dev)
    acc = {f: torch.zeros(B, Hkv, cap, device=dev) for f in ("merge", "one")}
    ws = {f: make_ws(lg, lg.layer_cache(K, V, acc[f], Hq), FORMS[f], 128) for f in ("merge", "one")}
    rng = np.random.default_rng(5)
    for step in range(120):
        lens = torch.tensor(rng.integers(0, cap - 1, B), dtype=torch.int32, device=dev)
        q = (2 * torch.randn(B, Hq, D, generator=g)).to(torch.bfloat16).to(dev)
        res = {}
        for f in ("merge", "one"):
            out = torch.zeros(B, Hq, D, dtype=torch.bfloat16, device=dev)
            lse = torch.zeros(B, Hq, device=dev)
            sm = torch.zeros(B, Hq, device=dev)
            flags = lg.TEST_FORCE_HANDOVER if (f == "one" and step % 3 == 2) else 0
            attend(lg, lg.layer_cache(K, V, acc[f], Hq), q, None, None, out, pos, lens, lens, sw,
                   lse, sm, None, ws[f], FORMS[f], 128, flags)
            res[f] = (out, lse, sm)
        torch.cuda.synchronize()
        torch.testing.assert_close(res["merge"][0].float(), res["one"][0].float(), rtol=8e-3,
                                   atol=1e-3, msg=str(step))
        for x, y in zip(res["merge"][1:], res["one"][1:]):
            torch.testing.assert_close(x, y, rtol=2e-6, atol=2e-6, msg=str(step))
        torch.testing.assert_close(acc["merge"], acc["one"], rtol=2e-6, atol=2e-6)
    assert lg.workspace_header(ws["one"])["status"] == 0


@pytest.mark.parametrize("max_split", [128, 1024])
def test_generation_wrap(max_split):
    """The arrival words start at the last generation before the wrap (2^32 - 2): the tags of the
    next launches are 2^32 - 1, then 1, 2, ... (never 0, the tag of a zero-filled word). Launches
    with growing split counts (so every statistics word of the later splits is still zero-tagged)
    and forced handovers agree with a workspace whose generations start at 0, bit for bit; with
    1024-slot splits the rows move between one and two splits as they grow."""
    from paper_2604_10044_amd import lg
    B, Hq, Hkv, D, cap = 4, 28, 4, 128, 2048
    _, K, V = _rand_layer(B, Hq, Hkv, D, cap, 41)
    acc0 = torch.rand(B, Hkv, cap, device="cuda")
    steps = [[130, 129, 0, 5], [400, 600, 130, 300], [900, 1300, 700, 800], [1500, 2000, 1600, 2040],
             [2040, 2041, 2042, 2043], [100, 2044, 3, 1000]]
    res = {}
    for preset in (False, True):
        Kc, Vc, acc = K.clone(), V.clone(), acc0.clone()
        ws = make_ws(lg, lg.layer_cache(Kc, Vc, acc, Hq), FORMS["one"], max_split)
        if preset:
            # arrival words: u64 per row right after the 256-byte header ([63:32] generation)
            rows = ws[256:256 + 8 * B * Hkv].view(torch.int64)
            rows.fill_((0xfffffffe << 32) - (1 << 64))
            torch.cuda.synchronize()
        outs = []
        for i in range(len(steps)):
            flags = lg.TEST_FORCE_HANDOVER if i % 2 else 0
            outs += _launch_seq(lg, Kc, Vc, acc, ws, steps[i:i + 1], Hq, FORMS["one"], max_split,
                                flags, seed=200 + i)
        assert lg.workspace_header(ws)["status"] == 0
        gen = (ws[256:256 + 8 * B * Hkv].view(torch.int64).cpu().numpy() >> 32) & 0xffffffff
        res[preset] = (outs, gen)
    # a row's generation advances at every launch in which it has more than one split: from 0 to
    # k, or from 2^32 - 2 through the wrap to k - 1
    k = np.array([sum(split_plan(cap, B * Hkv, max_split, st[b] + 1)[1] > 1 for st in steps)
                  for b in range(B)])
    assert np.all(k >= (4 if max_split == 128 else 1))
    np.testing.assert_array_equal(res[False][1].reshape(B, Hkv), np.repeat(k[:, None], Hkv, 1))
    np.testing.assert_array_equal(res[True][1].reshape(B, Hkv), np.repeat(k[:, None] - 1, Hkv, 1))
    for a, b in zip(res[False][0], res[True][0]):
        for x, y in zip(a, b):
            assert torch.equal(x, y)


def test_no_wait_error_path():
    """Every wait of the exchange gives up at once (test flag): each row with more than one split
    writes nothing (out, lse, suffix mass and acc untouched), its sequence's conf is NaN and the
    header status carries LG_ATTEND_STATUS_WAIT; rows with one split are finished normally; every
    kernel exits. The next call on the workspace refuses (sticky status); after the workspace is
    initialised again the same launch is correct."""
    from paper_2604_10044_amd import lg
    dev = torch.device("cuda")
    B, Hq, Hkv, D, cap = 4, 28, 4, 128, 2048
    g, K, V = _rand_layer(B, Hq, Hkv, D, cap, 51)
    lens_l = [100, 1500, 60, 2000]   # 512-slot splits: 1 / 3 / 1 / 4 per row
    pos = torch.arange(cap, dtype=torch.int32).repeat(B, 1).contiguous().to(dev)
    lens = torch.tensor(lens_l, dtype=torch.int32, device=dev)
    sw = torch.full((B,), 64, dtype=torch.int32, device=dev)
    q = torch.randn(B, Hq, D, generator=g).to(torch.bfloat16).to(dev)
    acc0 = torch.rand(B, Hkv, cap, device=dev)

    def launch(ws, acc, flags):
        out = torch.full((B, Hq, D), 7.0, dtype=torch.bfloat16, device=dev)
        lse = torch.full((B, Hq), 7.0, device=dev)
        sm = torch.full((B, Hq), 7.0, device=dev)
        conf = torch.zeros(B, device=dev)
        attend(lg, lg.layer_cache(K, V, acc, Hq), q, None, None, out, pos, lens, lens, sw, lse, sm,
               conf, ws, FORMS["one"], 512, flags)
        torch.cuda.synchronize()
        return out.float().cpu(), lse.cpu(), sm.cpu(), conf.cpu()

    acc_ref = acc0.clone()
    ws_ref = make_ws(lg, lg.layer_cache(K, V, acc_ref, Hq), FORMS["one"], 512)
    ref = launch(ws_ref, acc_ref, 0)
    acc = acc0.clone()
    ws = make_ws(lg, lg.layer_cache(K, V, acc, Hq), FORMS["one"], 512)
    got = launch(ws, acc, lg.TEST_NO_WAIT)
    assert lg.workspace_header(ws)["status"] == lg.LG_ATTEND_STATUS_WAIT
    for b in range(B):
        ns = split_plan(cap, B * Hkv, 512, lens_l[b])[1]
        if ns > 1:
            assert torch.isnan(got[3][b]), b
            assert torch.all(got[0][b] == 7.0) and torch.all(got[1][b] == 7.0) and torch.all(got[2][b] == 7.0)
            assert torch.equal(acc[b].cpu(), acc0[b].cpu()), b
        else:
            for x, y in zip(got[:3], ref[:3]):
                assert torch.equal(x[b], y[b]), b
            assert got[3][b] == ref[3][b]
            assert torch.equal(acc[b].cpu(), acc_ref[b].cpu()), b
    assert [split_plan(cap, B * Hkv, 512, n)[1] for n in lens_l] == [1, 3, 1, 4]
    # sticky: the next call refuses every sequence
    acc1 = acc.clone()
    got = launch(ws, acc, 0)
    assert torch.all(torch.isnan(got[3])) and torch.equal(acc.cpu(), acc1.cpu())
    assert torch.all(got[0] == 7.0)
    # initialised again: correct
    lg.lg_test_attend_workspace_init(lg.layer_cache(K, V, acc, Hq), FORMS["one"], 512, ws)
    acc.copy_(acc0)
    got = launch(ws, acc, 0)
    for x, y in zip(got, ref):
        assert torch.equal(x, y)
    assert torch.equal(acc.cpu(), acc_ref.cpu())
    assert lg.workspace_header(ws)["status"] == 0


@pytest.mark.parametrize("form", ["auto", "portable", "merge"])
def test_workspace_refused(form):
    """A workspace that was never initialised, or was initialised for another shape or form, is
    refused: conf NaN for every sequence, status LG_ATTEND_STATUS_WORKSPACE, out / lse / suffix
    mass / acc untouched."""
    from paper_2604_10044_amd import lg
    dev = torch.device("cuda")
    B, Hq, Hkv, D, cap = 3, 8, 2, 128, 512
    g, K, V = _rand_layer(B, Hq, Hkv, D, cap, 61)
    acc = torch.rand(B, Hkv, cap, device=dev)
    acc0 = acc.clone()
    layer = lg.layer_cache(K, V, acc, Hq)
    q = torch.randn(B, Hq, D, generator=g).to(torch.bfloat16).to(dev)
    pos = torch.arange(cap, dtype=torch.int32).repeat(B, 1).contiguous().to(dev)
    lens = torch.tensor([0, 300, 511], dtype=torch.int32, device=dev)
    sw = torch.full((B,), 64, dtype=torch.int32, device=dev)
    nbytes = lg.lg_test_attend_workspace(layer, FORMS[form], 0)
    other = lg.layer_cache(K[:2].contiguous(), V[:2].contiguous(), acc[:2].contiguous(), Hq)
    other_form = FORMS["portable"] if form != "portable" else FORMS["merge"]
    cases = {"zeros": None, "other shape": (other, FORMS[form]), "other form": (layer, other_form)}
    for name, init in cases.items():
        size = nbytes if init is None else max(nbytes, lg.lg_test_attend_workspace(init[0], init[1], 0))
        ws = torch.zeros(size, dtype=torch.uint8, device=dev)
        if init is not None:
            lg.lg_test_attend_workspace_init(init[0], init[1], 0, ws)
        out = torch.full((B, Hq, D), 7.0, dtype=torch.bfloat16, device=dev)
        lse = torch.full((B, Hq), 7.0, device=dev)
        sm = torch.full((B, Hq), 7.0, device=dev)
        conf = torch.zeros(B, device=dev)
        attend(lg, layer, q, None, None, out, pos, lens, lens, sw, lse, sm, conf, ws, FORMS[form],
               0, 0 if form == "auto" else 0)
        torch.cuda.synchronize()
        assert torch.all(torch.isnan(conf)), name
        assert lg.workspace_header(ws)["status"] & lg.LG_ATTEND_STATUS_WORKSPACE, name
        assert torch.all(out.float() == 7.0) and torch.all(lse == 7.0) and torch.all(sm == 7.0), name
        assert torch.equal(acc, acc0), name


# Rows of 1540 and 1600 live slots (two 1024-slot splits of 24 + 25 and 24 + 26 blocks, uneven over
# the waves), 1536 and 2040 (24 + 24 and 32 + 32 blocks); one slot of each is the appended row.
UNEVEN_LENS = [1539, 1599, 1535, 2039]


def test_uneven_two_split_rows_oracle():
    """Two-split rows whose blocks divide unevenly over the splits' waves, beside even ones, every
    (sequence, kv head) against the oracle."""
    run_case(4, 28, 4, 128, 2048, UNEVEN_LENS, "bf16", FORMS["one"], seed=81, max_split=1024)
