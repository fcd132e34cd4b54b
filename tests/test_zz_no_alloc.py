"""lg_decode_attend_noalloc (the attention entry point that allocates nothing; its workspace is a
static device array of the library) against lg_decode_attend on a workspace of the caller: the
same launches on the same inputs give the same bits in every output (out, lse, suffix mass, conf,
acc and the appended cache rows). Consecutive calls change the layer shape (the scratch is
initialised again), keep it (the scratch carries its exchange words over), and force a reinit."""
import pytest
import torch

pytestmark = pytest.mark.gpu


def _layer_inputs(B, Hq, Hkv, D, cap, seed):
    g = torch.Generator(device="cpu").manual_seed(seed)
    dev = torch.device("cuda")
    K = torch.randn(B, Hkv, cap, D, generator=g).to(torch.bfloat16).to(dev)
    V = torch.randn(B, Hkv, cap, D, generator=g).to(torch.bfloat16).to(dev)
    acc = torch.rand(B, Hkv, cap, generator=g).to(dev)
    return g, K, V, acc


def _call_pair(lg, state, lens, seed, append=True, reinit=0):
    """One launch through each entry point on its own copy of the layer; returns both results."""
    K, V, acc, ws, Hq = state["K"], state["V"], state["acc"], state["ws"], state["Hq"]
    B, Hkv, cap, D = K.shape
    dev = K.device
    g = torch.Generator(device="cpu").manual_seed(seed)
    q = torch.randn(B, Hq, D, generator=g).to(torch.bfloat16).to(dev)
    kn = torch.randn(B, Hkv, D, generator=g).to(torch.bfloat16).to(dev) if append else None
    vn = torch.randn(B, Hkv, D, generator=g).to(torch.bfloat16).to(dev) if append else None
    lens_t = torch.tensor(lens, dtype=torch.int32, device=dev)
    # positions with gaps (a pruned cache), strictly increasing; t beyond the last live one
    pos = (torch.arange(cap, dtype=torch.int32) * 3).repeat(B, 1).contiguous().to(dev)
    t = (3 * lens_t + 5).to(torch.int32)
    sw = torch.full((B,), cap // 4, dtype=torch.int32, device=dev)
    res = []
    for which in ("workspace", "noalloc"):
        if which == "workspace":
            Kc, Vc, ac = K, V, acc
        else:
            Kc, Vc, ac = state["K2"], state["V2"], state["acc2"]
        layer = lg.layer_cache(Kc, Vc, ac, Hq)
        out = torch.full((B, Hq, D), 7.0, dtype=torch.bfloat16, device=dev)
        lse = torch.full((B, Hq), 7.0, device=dev)
        sm = torch.full((B, Hq), 7.0, device=dev)
        conf = torch.full((B,), 0.25, device=dev)
        if which == "workspace":
            lg.lg_decode_attend(layer, q, kn, vn, out, pos, lens_t, t, sw, lse, sm, conf, ws)
        else:
            lg.lg_decode_attend_noalloc(layer, q, kn, vn, out, pos, lens_t, t, sw, lse, sm, conf,
                                        reinit=reinit)
        torch.cuda.synchronize()
        res.append((out, lse, sm, conf, ac.clone(), Kc.clone(), Vc.clone()))
    assert lg.workspace_header(ws)["status"] == 0
    return res


def _new_state(lg, B, Hq, Hkv, D, cap, seed):
    _, K, V, acc = _layer_inputs(B, Hq, Hkv, D, cap, seed)
    layer = lg.layer_cache(K, V, acc, Hq)
    ws = torch.empty(lg.lg_decode_attend_workspace(layer), dtype=torch.uint8, device="cuda")
    lg.lg_decode_attend_workspace_init(layer, ws)
    return {"K": K, "V": V, "acc": acc, "K2": K.clone(), "V2": V.clone(), "acc2": acc.clone(),
            "ws": ws, "Hq": Hq}


def _assert_same(res, what):
    a, b = res
    names = ("out", "lse", "suffix_mass", "conf", "acc", "K", "V")
    for n, x, y in zip(names, a, b):
        assert torch.equal(x.view(torch.uint8) if x.dtype == torch.bfloat16 else x,
                           y.view(torch.uint8) if y.dtype == torch.bfloat16 else y), (what, n)
    assert not torch.isnan(b[3]).any(), what


def test_noalloc_matches_workspace_entry_point():
    from paper_2604_10044_amd import lg
    print("noalloc: 7B-shaped layer, batch 32, cap 2048", flush=True)
    big = _new_state(lg, 32, 28, 4, 128, 2048, seed=11)
    lens = [2047 - (37 * b) % 520 for b in range(32)]
    lens[3], lens[9] = 0, 1
    _assert_same(_call_pair(lg, big, lens, seed=1), "first call, batch 32")
    print("noalloc: smaller layer, batch 3, 8 / 2 heads, cap 512", flush=True)
    small = _new_state(lg, 3, 8, 2, 128, 512, seed=12)
    _assert_same(_call_pair(lg, small, [300, 511, 17], seed=2), "second call, smaller layer")
    _assert_same(_call_pair(lg, small, [301, 100, 0], seed=3, append=False),
                 "third call, same shape (scratch carried over)")
    _assert_same(_call_pair(lg, small, [450, 200, 60], seed=4, reinit=1), "fourth call, reinit")
    print("noalloc: back to the batch-32 layer", flush=True)
    lens = [min(2047, n + 1) for n in lens]
    _assert_same(_call_pair(lg, big, lens, seed=5), "fifth call, the first shape again")
    _assert_same(_call_pair(lg, big, [n // 2 for n in lens], seed=6), "sixth call, same shape")


def test_noalloc_rejects_oversize_layer():
    """A layer whose workspace exceeds the scratch is refused before anything is enqueued, and the
    next call of a fitting shape still matches the workspace entry point."""
    from paper_2604_10044_amd import lg
    dev = torch.device("cuda")
    K = torch.zeros(1, 1, 32, 128, dtype=torch.bfloat16, device=dev)
    acc = torch.zeros(1, 1, 32, device=dev)
    big = lg.LayerCache(batch=256, n_q_heads=28, n_kv_heads=4, head_dim=128, cap=32768,
                        dtype=lg.LG_BF16, k=K.data_ptr(), v=K.data_ptr(), acc=acc.data_ptr())
    assert lg.lg_decode_attend_workspace(big) > lg.NOALLOC_SCRATCH_BYTES
    x = torch.zeros(256 * 28 * 128, dtype=torch.bfloat16, device=dev)
    i = torch.zeros(256 * 32768, dtype=torch.int32, device=dev)
    f = torch.zeros(256 * 28, device=dev)
    with pytest.raises(lg.LGError, match="LG_ERR_TOO_LARGE"):
        lg.lg_decode_attend_noalloc(big, x, None, None, x, i, i, i, i, f, f, f)
    small = _new_state(lg, 2, 8, 2, 128, 256, seed=13)
    _assert_same(_call_pair(lg, small, [255, 40], seed=7), "after a refused call")
