"""The guarded step captured as a HIP graph (the way bench.py times it) gives the same results as the
same steps launched eagerly: decisions, lengths, positions, caches, scores and layer outputs bit for
bit. Each graph is replayed several times from a restored snapshot, with eager work between the
replays, and every replay is checked."""
import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu


def _state(dec):
    return {"decision": dec.decision.cpu().numpy().copy(), "len": dec.len.cpu().numpy().copy(),
            "pos": dec.pos.cpu().numpy().copy(), "state": dec.state.cpu().numpy().copy(),
            "K": [k.float().cpu().numpy() for k in dec.K], "V": [v.float().cpu().numpy() for v in dec.V],
            "acc": [a.cpu().numpy() for a in dec.acc], "out": dec.out.float().cpu().numpy(),
            "lse": dec.lse.cpu().numpy()}


def _assert_same(a, b, what):
    for k in a:
        if isinstance(a[k], list):
            for i, (x, y) in enumerate(zip(a[k], b[k])):
                np.testing.assert_array_equal(x, y, err_msg="%s %s[%d]" % (what, k, i))
        else:
            np.testing.assert_array_equal(a[k], b[k], err_msg="%s %s" % (what, k))


# portable kernels (automatic for float32), the one-launch form (automatic for bf16), the merge form
@pytest.mark.parametrize("dtype,form", [("f32", 0), ("bf16", 0), ("bf16", 2)])
@pytest.mark.parametrize("policy", [oracle.POLICY_LOOPGUARD, oracle.POLICY_H2O])
def test_step_graph_replay_matches_eager(policy, dtype, form):
    import dataclasses
    from paper_2604_10044_amd.decoder import GuardedDecoder
    from paper_2604_10044_amd.synth import tiny
    # W = 64 makes the tiny workload trigger within the captured steps (pruning inside the graph)
    wl = dataclasses.replace(tiny(steps=80, period=4), dtype=dtype)
    p = oracle.paper_params(W=64, policy=policy)
    dec = GuardedDecoder(wl, params=p, form=form, keep_layer_outputs=True)
    dec.prefill()
    dec.load_steps(80)
    for s in range(60):
        dec.step(s)
    torch.cuda.synchronize()
    snap = dec.snapshot()
    steps = range(60, 80)
    # eager reference
    ref = []
    for s in steps:
        dec.step(s)
        torch.cuda.synchronize()
        ref.append(_state(dec))
    assert any(d[0][0] for d in [r["decision"] for r in ref]), "no trigger inside the captured steps"
    # one graph per step, captured from the snapshot state
    dec.restore(snap)
    torch.cuda.synchronize()
    graphs = []
    cap = torch.cuda.Stream()
    for s in steps:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=cap):
            dec.step(s)
        graphs.append(g)
    torch.cuda.synchronize()
    for rep in range(3):
        dec.restore(snap)
        scratch = torch.randn(1 << 20, device="cuda").sum()   # eager work between replays
        torch.cuda.synchronize()
        for i, g in enumerate(graphs):
            g.replay()
            torch.cuda.synchronize()
            _assert_same(ref[i], _state(dec), "replay %d step %d" % (rep, steps[i]))
        del scratch
