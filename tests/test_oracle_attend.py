"""Pins of the oracle's attention (Eq. (1), Sec. 3.1) and its fused statistics.

Checked against an independent library routine (torch.softmax / logsumexp in float64), closed
forms and invariants that a dropped term, a wrong index or a transposed operand would break.
"""
import numpy as np
import pytest
import torch

import oracle


def _rand(rng, *shape):
    return rng.standard_normal(shape).astype(np.float32)


@pytest.mark.parametrize("G,d,n", [(1, 64, 1), (4, 64, 37), (7, 128, 129), (6, 128, 300)])
def test_against_torch_softmax(G, d, n):
    rng = np.random.default_rng(G * 1000 + n)
    q, K, V = _rand(rng, G, d), _rand(rng, n, d), _rand(rng, n, d)
    pos = np.sort(rng.choice(5 * n, n, replace=False)).astype(np.int32)
    t = int(pos[-1]) + 3
    w = max(1, (t - int(pos[0])) // 3)
    o, lse, sg, asum = oracle.attend_group(q, K, V, pos, t, w)
    qt, Kt, Vt = (torch.from_numpy(x).double() for x in (q, K, V))
    s = (qt @ Kt.T) / np.sqrt(d)
    a = torch.softmax(s, dim=1)
    np.testing.assert_allclose(o, (a @ Vt).numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(lse, torch.logsumexp(s, dim=1).numpy(), rtol=1e-12)
    mask = torch.from_numpy(pos > t - w)
    np.testing.assert_allclose(sg, a[:, mask].sum(1).numpy(), rtol=1e-10, atol=1e-14)
    np.testing.assert_allclose(asum, a.sum(0).numpy(), rtol=1e-10, atol=1e-14)


def test_invariants_sum_and_bounds():
    rng = np.random.default_rng(7)
    G, d, n = 5, 64, 90
    q, K, V = _rand(rng, G, d) * 3, _rand(rng, n, d), _rand(rng, n, d)
    pos = np.arange(n, dtype=np.int32) * 2
    o, lse, sg, asum = oracle.attend_group(q, K, V, pos, 2 * n, 40)
    assert abs(asum.sum() - G) < 1e-12          # every head's weights sum to one
    assert np.all((sg >= 0) & (sg <= 1))
    _, _, s_all, _ = oracle.attend_group(q, K, V, pos, 2 * n, 10 ** 6)
    _, _, s_none, _ = oracle.attend_group(q, K, V, pos, 2 * n, 0)
    np.testing.assert_allclose(s_all, 1.0, atol=1e-14)
    np.testing.assert_allclose(s_none, 0.0, atol=0)


def test_single_slot_and_equal_keys():
    rng = np.random.default_rng(3)
    G, d = 3, 64
    q, V1 = _rand(rng, G, d), _rand(rng, 1, d)
    K1 = _rand(rng, 1, d)
    o, lse, _, asum = oracle.attend_group(q, K1, V1, np.array([5]), 5, 1)
    np.testing.assert_allclose(o, np.repeat(V1.astype(np.float64), G, 0), rtol=0, atol=1e-15)
    np.testing.assert_allclose(lse, (q.astype(np.float64) @ K1[0].astype(np.float64)) / 8.0,
                               rtol=1e-12)
    n = 17
    K = np.repeat(_rand(rng, 1, d), n, 0)
    V = _rand(rng, n, d)
    o, lse, _, asum = oracle.attend_group(q, K, V, np.arange(n), n, 4)
    np.testing.assert_allclose(o, np.repeat(V.astype(np.float64).mean(0, keepdims=True), G, 0),
                               rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(asum, np.full(n, G / n), rtol=1e-12)


def test_permutation_invariance_and_dominant_logit():
    rng = np.random.default_rng(11)
    G, d, n = 2, 128, 50
    q, K, V = _rand(rng, G, d), _rand(rng, n, d), _rand(rng, n, d)
    pos = np.arange(n, dtype=np.int32)
    o, lse, _, asum = oracle.attend_group(q, K, V, pos, n - 1, 10)
    perm = rng.permutation(n)
    o2, lse2, _, asum2 = oracle.attend_group(q, K[perm], V[perm], pos[perm], n - 1, 10)
    np.testing.assert_allclose(o2, o, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(asum2, asum[perm], rtol=1e-12, atol=1e-15)
    # One key aligned with the query so its logit leads the rest by > 40: output = its value row.
    K2 = K.copy()
    K2[17] = q[0] * 8.0
    o3, _, s3, _ = oracle.attend_group(q[:1], K2, V, pos, n - 1, n - 17)
    np.testing.assert_allclose(o3[0], V[17].astype(np.float64), rtol=0, atol=1e-12)
    np.testing.assert_allclose(s3, 1.0, atol=1e-12)
    o4, _, s4, _ = oracle.attend_group(q[:1], K2, V, pos, n - 1, n - 1 - 17)
    np.testing.assert_allclose(s4, 0.0, atol=1e-12)   # slot 17 sits just outside the suffix


def test_suffix_threshold_is_integer_exact():
    """The suffix set {j : pos_j > t - w_s} is taken over the integers: t - w_s below every
    int32 position gives sigma = 1, above every position sigma = 0, even at the ends of the int32
    range where a 32-bit difference would wrap."""
    rng = np.random.default_rng(8)
    q, K, V = (rng.standard_normal(s).astype(np.float32) for s in ((2, 16), (9, 16), (9, 16)))
    pos = np.arange(9, dtype=np.int32) * 5
    _, _, s_all, _ = oracle.attend_group(q, K, V, pos, -2 ** 31, 2 ** 31 - 1)
    np.testing.assert_allclose(s_all, 1.0, atol=1e-12)
    _, _, s_none, _ = oracle.attend_group(q, K, V, pos, 2 ** 31 - 1, -2 ** 31)
    np.testing.assert_allclose(s_none, 0.0, atol=1e-12)
