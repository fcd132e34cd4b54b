"""GPU parity of lg_prune_compact against the oracle's keep set (Eq. (10), Eq. (11), Sec. 5.3;
the H2O and StreamingLLM baselines of Sec. 6.1) and index-select compaction: keep lists, lengths,
positions and the compacted K/V/acc rows must be bit-identical."""
import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu


def _decisions(B, trig, span, level):
    from paper_2604_10044_amd import lg
    d = np.zeros((B, lg.DECISION_INTS), np.int32)
    F = lg.DECISION_FIELDS
    d[:, F.index("trigger")] = trig
    d[:, F.index("span_lo")] = span
    d[:, F.index("level")] = level
    return d


def _case(B, cap, D, dtype, n_layers, seed, with_decision=True, append=True, params=None,
          tied_acc=False, budgets=None):
    from paper_2604_10044_amd import lg
    rng = np.random.default_rng(seed)
    params = params or oracle.paper_params()
    dev = torch.device("cuda")
    budget = rng.choice([128, 256, 512, cap], B).astype(np.int32)
    if budgets is not None:
        budget = np.asarray(budgets, np.int32)
    budget = np.minimum(budget, cap)
    lens = np.array([int(rng.integers(0, bb)) if rng.random() < 0.5 else int(bb) - (1 if append else 0)
                     for bb in budget], np.int32)
    lens[0] = budget[0] - 1 if append else budget[0]       # overflow after the commit
    pos = np.zeros((B, cap), np.int32)
    tapp = np.zeros(B, np.int32)
    for b in range(B):
        L = lens[b]
        if L:
            gap = int(rng.integers(1, 6))
            pos[b, :L] = np.sort(rng.choice(gap * (L + 40), L, replace=False))
        tapp[b] = (pos[b, L - 1] if L else 0) + int(rng.integers(1, 4))
    trig = (rng.random(B) < 0.5).astype(np.int32) if with_decision else np.zeros(B, np.int32)
    span = np.zeros(B, np.int32)
    level = rng.integers(0, 4, B).astype(np.int32)
    for b in range(B):
        newest = tapp[b] if append else (pos[b, lens[b] - 1] if lens[b] else 0)
        R = budget[b] // 4
        span[b] = -1 if rng.random() < 0.25 else int(rng.integers(max(0, newest - 2 * R), newest + 1))
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    K = [torch.randn(B, 2, cap, D, device=dev).to(tdt) for _ in range(n_layers)]
    V = [torch.randn(B, 2, cap, D, device=dev).to(tdt) for _ in range(n_layers)]
    if tied_acc:   # few distinct values: H2O ties across the selection threshold
        A = [torch.randint(0, 3, (B, 2, cap), device=dev).float() * 0.5 for _ in range(n_layers)]
    else:
        A = [torch.rand(B, 2, cap, device=dev) * 10 for _ in range(n_layers)]
    K0 = [k.clone() for k in K]
    V0 = [v.clone() for v in V]
    A0 = [a.clone() for a in A]
    layers = [lg.layer_cache(K[l], V[l], A[l], 4) for l in range(n_layers)]
    pos_d = torch.from_numpy(pos).to(dev)
    len_d = torch.from_numpy(lens).to(dev)
    kidx = torch.full((B, cap), -7, dtype=torch.int32, device=dev)
    nlen = torch.zeros(B, dtype=torch.int32, device=dev)
    dec = torch.from_numpy(_decisions(B, trig, span, level)).to(dev) if with_decision else None
    gp = lg.params_from_dict(params)
    lg.lg_prune_compact(gp, B, cap, layers, pos_d, len_d, torch.from_numpy(budget).to(dev),
                        torch.from_numpy(tapp).to(dev) if append else None, dec, kidx, nlen)
    torch.cuda.synchronize()
    kidx_h, nlen_h = kidx.cpu().numpy(), nlen.cpu().numpy()
    pos_h, len_h = pos_d.cpu().numpy(), len_d.cpu().numpy()
    n_flag = 0
    policy = int(params.get("policy", 0))
    A0h = [a.cpu().numpy() for a in A0]
    for b in range(B):
        L = int(lens[b])
        p_ref = pos[b, :L].copy()
        if append and L < cap:
            p_ref = np.append(p_ref, tapp[b]).astype(np.int32)
            L += 1
        if policy != 0:
            keep = None
            if L >= budget[b]:
                score = None
                if policy == oracle.POLICY_H2O and n_layers:
                    score = oracle.h2o_score(np.stack([a[b, :, :L] for a in A0h]))
                keep = oracle.keep_set_baseline(params, p_ref, int(budget[b]), score)
        elif trig[b]:
            keep = oracle.keep_set(params, p_ref, int(budget[b]), int(span[b]), int(level[b]))
        elif L >= budget[b]:
            keep = oracle.keep_set(params, p_ref, int(budget[b]), -1, 0)
        else:
            keep = None
        if keep is None:
            assert nlen_h[b] == -1
            assert len_h[b] == L
            np.testing.assert_array_equal(pos_h[b, :L], p_ref)
            for l in range(n_layers):
                assert torch.equal(K[l][b], K0[l][b]) and torch.equal(A[l][b], A0[l][b])
            continue
        n_flag += 1
        m = len(keep)
        assert m <= max(0, int(budget[b]) - 1)                 # room for the next append
        assert nlen_h[b] == m and len_h[b] == m
        np.testing.assert_array_equal(kidx_h[b, :m], keep)
        np.testing.assert_array_equal(pos_h[b, :m], p_ref[keep])
        kt = torch.from_numpy(keep.astype(np.int64)).to(dev)
        for l in range(n_layers):
            assert torch.equal(K[l][b, :, :m], K0[l][b].index_select(1, kt))
            assert torch.equal(V[l][b, :, :m], V0[l][b].index_select(1, kt))
            assert torch.equal(A[l][b, :, :m], A0[l][b].index_select(1, kt))
    return n_flag


@pytest.mark.parametrize("D,dtype", [(128, "bf16"), (64, "bf16"), (128, "f32"), (64, "f32")])
def test_prune_parity(D, dtype):
    assert _case(24, 1024, D, dtype, 3, seed=D) > 0


def test_prune_parity_many_layers_and_no_append():
    assert _case(8, 2048, 128, "bf16", 70, seed=7, append=False) > 0   # > 64 layers: two launches


@pytest.mark.parametrize("policy", [1, 2])
@pytest.mark.parametrize("tied", [False, True])
def test_baseline_policy_parity(policy, tied):
    # decisions with triggers are passed and must be ignored by the baseline policies
    p = oracle.paper_params(policy=policy)
    assert _case(24, 1024, 128, "bf16", 3, seed=31 + policy, params=p, tied_acc=tied) > 0


def test_h2o_parity_many_layers():
    # > 64 layers: the score is accumulated over two launches in layer order
    p = oracle.paper_params(policy=1)
    assert _case(6, 512, 64, "f32", 70, seed=5, params=p, tied_acc=True) > 0


@pytest.mark.parametrize("policy", [0, 1, 2])
def test_prune_parity_max_cache(policy):
    """Rows at the 32768-slot maximum cache (budgets up to the cap): keep sets, the H2O radix
    select over tied scores and the compaction of full rows."""
    p = oracle.paper_params(policy=policy)
    assert _case(4, 32768, 128, "bf16", 2, seed=41 + policy, params=p, tied_acc=policy == 1,
                 budgets=[32768, 32768, 8192, 512]) > 0


@pytest.mark.parametrize("i", range(12))
def test_prune_parity_random_shapes(i):
    """Seeded random prune calls: batch 1-12, caches of 128-4096 slots (any size, not only multiples
    of 32), head_dim 64/128, bf16 or f32, 1-5 layers, each keep policy, with and without the append."""
    rng = np.random.default_rng(2000 + i)
    B = int(rng.integers(1, 13))
    cap = int(rng.integers(128, 4097))
    D = int(rng.choice([64, 128]))
    dtype = str(rng.choice(["bf16", "f32"]))
    n_layers = int(rng.integers(1, 6))
    policy = i % 3
    append = bool(rng.integers(0, 2))
    p = oracle.paper_params(policy=policy)
    _case(B, cap, D, dtype, n_layers, seed=3000 + i, append=append, params=p,
          tied_acc=policy == 1 and i % 2 == 0)


def test_budget_upkeep_without_decisions():
    assert _case(16, 512, 128, "bf16", 2, seed=11, with_decision=False) > 0


@pytest.mark.parametrize("policy", [0, 1, 2])
def test_prefill_reduction_matches_oracle(policy):
    """A context longer than the budget is reduced by the keep rule (no decision, no append; no
    layers, so the H2O scores are all zero)."""
    from paper_2604_10044_amd import lg
    dev = torch.device("cuda")
    ctx = np.array([100, 256, 4096, 8192, 70000, 9000], np.int32)
    budget = np.array([256, 256, 1024, 2048, 8192, 512], np.int32)
    B, cap = len(ctx), int(ctx.max())
    pos = torch.arange(cap, dtype=torch.int32, device=dev).repeat(B, 1).contiguous()
    lens = torch.from_numpy(ctx).to(dev)
    kidx = torch.zeros(B, cap, dtype=torch.int32, device=dev)
    nlen = torch.zeros(B, dtype=torch.int32, device=dev)
    params = oracle.paper_params(policy=policy)
    gp = lg.params_from_dict(params)
    lg.lg_prune_compact(gp, B, cap, [], pos, lens, torch.from_numpy(budget).to(dev), None, None,
                        kidx, nlen)
    torch.cuda.synchronize()
    from oracle.trajectory import prefill_positions
    P, Lh = pos.cpu().numpy(), lens.cpu().numpy()
    for b in range(B):
        ref = prefill_positions(params, int(ctx[b]), int(budget[b]))
        assert Lh[b] == len(ref)
        np.testing.assert_array_equal(P[b, :Lh[b]], ref)


@pytest.mark.parametrize("policy", [0, 1, 2])
@pytest.mark.parametrize("divs", [(1, 1), (1, 2), (2, 1), (4, 2)])
def test_prune_parity_keep_cap(policy, divs):
    """Budgets too small for the anchors and divisors whose keep sizes exceed the budget: every
    keep set is capped at budget - 1 slots (LoopGuard: anchors, then the recent window, then the
    sparse history; the baselines: their keep size), as in the oracle."""
    rd, sd = divs
    p = oracle.paper_params(policy=policy, recent_div=rd, sparse_div=sd)
    _case(8, 128, 64, "bf16", 2, seed=70 + 7 * policy + 3 * rd + sd, params=p,
          budgets=[2, 3, 17, 33, 40, 64, 100, 128])


def test_budget_above_cap_acts_as_cap():
    """A budget larger than the cache: a full cache is pruned as if the budget were the cap (so
    the next append fits), and a cache below the cap is left alone."""
    from paper_2604_10044_amd import lg
    dev = torch.device("cuda")
    B, cap = 4, 128
    p = oracle.paper_params()
    budget = np.array([4096, 129, 200, 4096], np.int32)
    lens = np.array([cap - 1, cap - 1, cap - 1, 60], np.int32)   # the append fills rows 0-2
    pos = np.zeros((B, cap), np.int32)
    for b in range(B):
        pos[b, :lens[b]] = 3 * np.arange(lens[b])
    tapp = (3 * lens + 1).astype(np.int32)
    K = [torch.randn(B, 2, cap, 64, device=dev).to(torch.bfloat16)]
    V = [torch.randn(B, 2, cap, 64, device=dev).to(torch.bfloat16)]
    A = [torch.rand(B, 2, cap, device=dev)]
    layers = [lg.layer_cache(K[0], V[0], A[0], 4)]
    pos_d, len_d = torch.from_numpy(pos).to(dev), torch.from_numpy(lens).to(dev)
    kidx = torch.zeros(B, cap, dtype=torch.int32, device=dev)
    nlen = torch.zeros(B, dtype=torch.int32, device=dev)
    lg.lg_prune_compact(lg.params_from_dict(p), B, cap, layers, pos_d, len_d,
                        torch.from_numpy(budget).to(dev), torch.from_numpy(tapp).to(dev), None,
                        kidx, nlen)
    torch.cuda.synchronize()
    for b in range(B):
        L = int(lens[b]) + 1
        p_ref = np.append(pos[b, :lens[b]], tapp[b]).astype(np.int32)
        if L >= min(int(budget[b]), cap):
            keep = oracle.keep_set(p, p_ref, cap, -1, 0)
            assert int(nlen[b]) == len(keep) <= cap - 1
            np.testing.assert_array_equal(pos_d[b, :len(keep)].cpu().numpy(), p_ref[keep])
        else:
            assert int(nlen[b]) == -1 and int(len_d[b]) == L
