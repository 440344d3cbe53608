"""Pins of the oracle's primitive operations against facts other than the oracle itself:
closed forms, invariants, special cases, brute force on tiny inputs and finite differences."""
import math

import numpy as np
import pytest

from oracle import ops

R = np.random.default_rng(1234)


def _fd_check(f, x, dx_analytic, n_coords=20, h=1e-6, rtol=1e-6):
    """Central differences of the scalar f at random coordinates of x vs the analytic gradient."""
    flat = x.reshape(-1)
    idx = R.choice(flat.size, size=min(n_coords, flat.size), replace=False)
    for i in idx:
        old = flat[i]
        flat[i] = old + h
        fp = f()
        flat[i] = old - h
        fm = f()
        flat[i] = old
        num = (fp - fm) / (2 * h)
        ana = dx_analytic.reshape(-1)[i]
        assert abs(num - ana) <= rtol * max(1.0, abs(num)) + 1e-9, (i, num, ana)


# ------------------------------------------------------------------ RMSNorm
def test_rmsnorm_unit_gain_mean_square_closed_form():
    x = R.standard_normal((7, 13))
    eps = 1e-5
    y, r = ops.rmsnorm_fwd(x, np.ones(13), eps)
    ms = np.mean(x * x, axis=1)
    np.testing.assert_allclose(np.mean(y * y, axis=1), ms / (ms + eps), rtol=1e-12)
    np.testing.assert_allclose(r, 1 / np.sqrt(ms + eps), rtol=1e-14)


def test_rmsnorm_scale_invariance_and_gain_per_feature():
    x = R.standard_normal((5, 9))
    g = R.standard_normal(9)
    y1, _ = ops.rmsnorm_fwd(x, g, 0.0)
    y2, _ = ops.rmsnorm_fwd(3.7 * x, g, 0.0)
    np.testing.assert_allclose(y1, y2, rtol=1e-12)
    # gain acts per feature: doubling gain of feature 4 doubles column 4 only
    g2 = g.copy()
    g2[4] *= 2
    y3, _ = ops.rmsnorm_fwd(x, g2, 0.0)
    np.testing.assert_allclose(y3[:, 4], 2 * y1[:, 4], rtol=1e-12)
    np.testing.assert_allclose(np.delete(y3, 4, 1), np.delete(y1, 4, 1), rtol=1e-12)


def test_rmsnorm_bwd_finite_differences():
    x = R.standard_normal((4, 6))
    g = R.standard_normal(6)
    dy = R.standard_normal((4, 6))
    f = lambda: float(np.sum(ops.rmsnorm_fwd(x, g, 1e-5)[0] * dy))
    y, r = ops.rmsnorm_fwd(x, g, 1e-5)
    dx, dg = ops.rmsnorm_bwd(dy, x, r, g)
    _fd_check(f, x, dx)
    _fd_check(f, g, dg)


# ------------------------------------------------------------------ linear
def test_linear_one_hot_input_selects_weight_column():
    W = R.standard_normal((5, 3))  # N=5 outputs, K=3 inputs: a transposed operand cannot fit
    for j in range(3):
        e = np.zeros((1, 3))
        e[0, j] = 1.0
        np.testing.assert_array_equal(ops.linear_fwd(e, W)[0], W[:, j])


def test_linear_bwd_finite_differences():
    x = R.standard_normal((4, 3))
    W = R.standard_normal((5, 3))
    dy = R.standard_normal((4, 5))
    f = lambda: float(np.sum(ops.linear_fwd(x, W) * dy))
    dx, dW = ops.linear_bwd(dy, x, W)
    _fd_check(f, x, dx)
    _fd_check(f, W, dW)


# ------------------------------------------------------------------ RoPE
def test_rope_closed_form_two_pairs():
    # hd = 4: pair (0, 2) turns by p * 1, pair (1, 3) by p * theta^(-1/2)
    theta = 10000.0
    s = 6
    x = np.zeros((1, s, 1, 4))
    x[..., 0] = 1.0   # unit vector on the first element of pair (0, 2)
    x[..., 3] = 1.0   # unit vector on the second element of pair (1, 3)
    y = ops.rope_apply(x, theta)
    p = np.arange(s)
    w1 = p * theta ** (-0.5)
    np.testing.assert_allclose(y[0, :, 0, 0], np.cos(p), atol=1e-15)
    np.testing.assert_allclose(y[0, :, 0, 2], np.sin(p), atol=1e-15)
    np.testing.assert_allclose(y[0, :, 0, 1], -np.sin(w1), atol=1e-15)
    np.testing.assert_allclose(y[0, :, 0, 3], np.cos(w1), atol=1e-15)


def test_rope_position_zero_identity_norm_and_relative_position():
    x = R.standard_normal((2, 9, 3, 8))
    y = ops.rope_apply(x, 10000.0)
    np.testing.assert_allclose(y[:, 0], x[:, 0], rtol=0, atol=0)
    np.testing.assert_allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-13)
    # <R_m q, R_n k> depends on m - n only
    q = R.standard_normal(8)
    k = R.standard_normal(8)
    seq = np.zeros((1, 9, 2, 8))
    seq[0, :, 0, :] = q
    seq[0, :, 1, :] = k
    rot = ops.rope_apply(seq, 10000.0)[0]
    d1 = rot[5, 0] @ rot[2, 1]
    d2 = rot[7, 0] @ rot[4, 1]
    d3 = rot[3, 0] @ rot[0, 1]
    np.testing.assert_allclose([d2, d3], [d1, d1], rtol=1e-12)
    np.testing.assert_allclose(ops.rope_apply(y, 10000.0, inverse=True), x, atol=1e-14)


# ------------------------------------------------------------------ attention
def test_attention_zero_queries_give_causal_running_mean():
    B, s, H, hd = 2, 7, 3, 4
    q = np.zeros((B, s, H, hd))
    k = R.standard_normal((B, s, H, hd))
    v = R.standard_normal((B, s, H, hd))
    o, lse = ops.attention_fwd(q, k, v)
    mean = np.cumsum(v, axis=1) / np.arange(1, s + 1)[None, :, None, None]
    np.testing.assert_allclose(o, mean, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(lse, np.broadcast_to(np.log(np.arange(1, s + 1)), (B, H, s)), rtol=1e-13)


def test_attention_single_position_returns_value_and_causality():
    q = R.standard_normal((1, 1, 2, 4))
    k = R.standard_normal((1, 1, 2, 4))
    v = R.standard_normal((1, 1, 2, 4))
    o, _ = ops.attention_fwd(q, k, v)
    np.testing.assert_allclose(o, v, rtol=1e-14)
    q = R.standard_normal((1, 8, 2, 4))
    k = R.standard_normal((1, 8, 2, 4))
    v = R.standard_normal((1, 8, 2, 4))
    o1, _ = ops.attention_fwd(q, k, v)
    k2, v2 = k.copy(), v.copy()
    k2[:, 5:] += 3.0
    v2[:, 5:] -= 2.0
    o2, _ = ops.attention_fwd(q, k2, v2)
    np.testing.assert_array_equal(o1[:, :5], o2[:, :5])
    assert np.abs(o1[:, 5:] - o2[:, 5:]).max() > 1e-3


def test_attention_brute_force_scalar_loops():
    B, s, Hq, Hkv, hd = 1, 5, 4, 2, 3
    q = R.standard_normal((B, s, Hq, hd))
    k = R.standard_normal((B, s, Hkv, hd))
    v = R.standard_normal((B, s, Hkv, hd))
    o, _ = ops.attention_fwd(q, k, v)
    for h in range(Hq):
        g = h // (Hq // Hkv)
        for i in range(s):
            w = [math.exp(sum(q[0, i, h, c] * k[0, j, g, c] for c in range(hd)) / math.sqrt(hd))
                 for j in range(i + 1)]
            for c in range(hd):
                ref = sum(w[j] * v[0, j, g, c] for j in range(i + 1)) / sum(w)
                assert abs(o[0, i, h, c] - ref) < 1e-12


def test_attention_gqa_equals_mha_with_repeated_kv_heads():
    B, s, Hq, Hkv, hd = 2, 6, 6, 2, 4
    q = R.standard_normal((B, s, Hq, hd))
    k = R.standard_normal((B, s, Hkv, hd))
    v = R.standard_normal((B, s, Hkv, hd))
    o, lse = ops.attention_fwd(q, k, v)
    krep = np.repeat(k, Hq // Hkv, axis=2)  # consecutive query heads share a kv head
    vrep = np.repeat(v, Hq // Hkv, axis=2)
    o2, lse2 = ops.attention_fwd(q, krep, vrep)
    np.testing.assert_allclose(o, o2, rtol=1e-13)
    np.testing.assert_allclose(lse, lse2, rtol=1e-13)


def test_attention_bwd_finite_differences_gqa():
    B, s, Hq, Hkv, hd = 2, 5, 4, 2, 4
    q = R.standard_normal((B, s, Hq, hd))
    k = R.standard_normal((B, s, Hkv, hd))
    v = R.standard_normal((B, s, Hkv, hd))
    do = R.standard_normal((B, s, Hq, hd))
    f = lambda: float(np.sum(ops.attention_fwd(q, k, v)[0] * do))
    dq, dk, dv = ops.attention_bwd(do, q, k, v)
    _fd_check(f, q, dq, n_coords=30)
    _fd_check(f, k, dk, n_coords=30)
    _fd_check(f, v, dv, n_coords=30)


# ------------------------------------------------------------------ SwiGLU
def test_swiglu_known_values_and_fd():
    a = np.array([0.0, 1.0, -1.0, 20.0])
    b = np.array([3.0, 1.0, 1.0, 2.0])
    z = ops.swiglu_fwd(a, b)
    s1 = 1 / (1 + math.exp(-1))
    np.testing.assert_allclose(z, [0.0, s1, -(1 - s1), 2 * 20 / (1 + math.exp(-20))], rtol=1e-14)
    da, db = ops.swiglu_bwd(np.ones(4), np.zeros(4), np.ones(4))
    np.testing.assert_allclose(da, 0.5)  # d silu / da at 0 is 1/2
    np.testing.assert_allclose(db, 0.0)
    a = R.standard_normal((3, 5))
    b = R.standard_normal((3, 5))
    dz = R.standard_normal((3, 5))
    f = lambda: float(np.sum(ops.swiglu_fwd(a, b) * dz))
    da, db = ops.swiglu_bwd(dz, a, b)
    _fd_check(f, a, da)
    _fd_check(f, b, db)


# ------------------------------------------------------------------ embedding
def test_embedding_gather_and_brute_force_scatter():
    V, d = 11, 3
    E = R.standard_normal((V, d))
    tok = np.array([[3, 7, 3, 0], [10, 3, 7, 7]], dtype=np.int32)
    x0 = ops.embed_fwd(E, tok)
    for b in range(2):
        for i in range(4):
            np.testing.assert_array_equal(x0[b, i], E[tok[b, i]])
    dx0 = R.standard_normal((2, 4, d))
    de, ids, counts = ops.embed_bwd(dx0, tok, V)
    ref = np.zeros((V, d))
    for b in range(2):
        for i in range(4):
            ref[tok[b, i]] += dx0[b, i]
    np.testing.assert_allclose(de, ref, rtol=1e-15)
    assert list(ids) == [0, 3, 7, 10]
    assert list(counts) == [1, 3, 3, 1]
    untouched = [v for v in range(V) if v not in ids]
    assert np.all(de[untouched] == 0.0)


# ------------------------------------------------------------------ cross-entropy
def test_ce_zero_logits_closed_form():
    N, V = 6, 512
    tg = R.integers(0, V, N)
    loss, lse = ops.ce_fwd(np.zeros((N, V)), tg)
    assert abs(loss - math.log(V)) < 1e-14
    dl = ops.ce_bwd(np.zeros((N, V)), tg, lse, 1.0 / N)
    ref = np.full((N, V), 1.0 / V / N)
    ref[np.arange(N), tg] -= 1.0 / N
    np.testing.assert_allclose(dl, ref, rtol=1e-13)


def test_ce_fd():
    N, V = 4, 7
    z = R.standard_normal((N, V))
    tg = R.integers(0, V, N)
    f = lambda: float(ops.ce_fwd(z, tg)[0])
    _, lse = ops.ce_fwd(z, tg)
    _fd_check(f, z, ops.ce_bwd(z, tg, lse, 1.0 / N))
