"""Pins of the oracle's delayed Muon (Alg. 2 of §4) and its Newton-Schulz step, against routes
that share nothing with the oracle's matrix iteration: the SVD of M with the Newton-Schulz
polynomial applied to each singular value, closed forms, invariances, and the delay / Error-
Feedback identities of Alg. 1 and §3.2."""
import math

import numpy as np
import pytest

from oracle.update import (NS_COEFFS, NS_EPS, HParams, OptState, is_muon_matrix, iteration_update,
                           muon_scale, newton_schulz)


def svd_route(M, steps=5):
    """U q(S / (||M||_F + eps)) V^T with q the scalar quintic iterated `steps` times: the same map
    as Newton-Schulz, computed on the singular values instead of with matrix products."""
    a, b, c = NS_COEFFS
    U, S, Vt = np.linalg.svd(M, full_matrices=False)
    s = S / (np.linalg.norm(M) + NS_EPS)
    for _ in range(steps):
        s = a * s + b * s ** 3 + c * s ** 5
    return (U * s) @ Vt


def rel(a, b):
    return float(np.linalg.norm(a - b) / np.linalg.norm(b))


@pytest.mark.parametrize("shape", [(48, 48), (32, 96), (96, 32), (7, 5)])
def test_newton_schulz_equals_singular_value_route(shape):
    M = np.random.default_rng(1).standard_normal(shape)
    assert rel(newton_schulz(M), svd_route(M)) < 1e-12


@pytest.mark.parametrize("steps", [1, 2, 5])
def test_newton_schulz_step_count(steps):
    M = np.random.default_rng(2).standard_normal((24, 40))
    assert rel(newton_schulz(M, steps), svd_route(M, steps)) < 1e-12


def test_newton_schulz_output_is_nearly_orthogonal():
    # the published property of these coefficients: after 5 steps every singular value of a
    # well-conditioned input lands in about (0.68, 1.13), not at exactly 1
    rng = np.random.default_rng(3)
    Q1, _ = np.linalg.qr(rng.standard_normal((96, 96)))
    Q2, _ = np.linalg.qr(rng.standard_normal((96, 96)))
    square = (Q1 * rng.uniform(1.0, 10.0, 96)) @ Q2   # condition number <= 10
    for M in [rng.standard_normal((64, 128)), rng.standard_normal((128, 64)), square]:
        s = np.linalg.svd(newton_schulz(M), compute_uv=False)
        assert s.min() > 0.6 and s.max() < 1.2, (M.shape, s.min(), s.max())


def test_newton_schulz_invariances():
    rng = np.random.default_rng(4)
    M = rng.standard_normal((20, 36))
    O = newton_schulz(M)
    # scale (up to the normalisation epsilon) and sign
    assert rel(newton_schulz(7.3 * M), O) < 1e-6
    assert np.array_equal(newton_schulz(-M), -O)
    # transposition
    assert rel(newton_schulz(M.T), O.T) < 1e-12
    # orthogonal equivariance: NS(Q1 M Q2) = Q1 NS(M) Q2
    Q1, _ = np.linalg.qr(rng.standard_normal((20, 20)))
    Q2, _ = np.linalg.qr(rng.standard_normal((36, 36)))
    assert rel(newton_schulz(Q1 @ M @ Q2), Q1 @ O @ Q2) < 1e-10


def test_muon_matrix_selection():
    assert all(is_muon_matrix(f"blk3.{n}") for n in ("wq", "wk", "wv", "wo", "wgate", "wup", "wdown"))
    assert not any(is_muon_matrix(n) for n in ("embed", "final_norm", "blk0.attn_norm", "blk1.ffn_norm"))


def toy_params(rng):
    return {"embed": rng.standard_normal((6, 8)) * 0.02, "blk0.attn_norm": np.ones(8),
            "blk0.wq": rng.standard_normal((8, 8)) * 0.02, "blk0.wgate": rng.standard_normal((12, 8)) * 0.02,
            "blk0.wdown": rng.standard_normal((8, 12)) * 0.02}


def run(hp, x0, grads):
    st = OptState.create(x0)
    xs = [{k: v.copy() for k, v in st.x.items()}]
    for g in grads:
        iteration_update(st, g, hp)
        xs.append({k: v.copy() for k, v in st.x.items()})
    return st, xs


@pytest.mark.parametrize("lam", [0.0, 1.0])
def test_muon_constant_gradient_closed_form(lam):
    # constant gradient, no decay, no clipping: M_k = (1 - mu^k) G, Newton-Schulz ignores the scale,
    # so every update is lr s NS(G) and the delay-1 run moves by (T - 1) of them (t = 0 is a no-op;
    # with a constant update the EF form x - 2u + u_prev reduces to x - u)
    rng = np.random.default_rng(5)
    x0 = toy_params(rng)
    G = {k: rng.standard_normal(v.shape) for k, v in x0.items()}
    hp = HParams(lr=1e-2, weight_decay=0.0, clip_norm=0.0, ef_lambda=lam, optimizer="muon")
    T = 6
    st, _ = run(hp, x0, [G] * T)
    for k in ("blk0.wq", "blk0.wgate", "blk0.wdown"):
        expect = x0[k] - (T - 1) * hp.lr * muon_scale(x0[k].shape, hp.update_rms) * svd_route(G[k])
        assert rel(st.x[k], expect) < 1e-6, k


def test_muon_delay_is_the_synchronous_run_one_step_late():
    rng = np.random.default_rng(6)
    x0 = toy_params(rng)
    grads = [{k: rng.standard_normal(v.shape) for k, v in x0.items()} for _ in range(5)]
    _, x1 = run(HParams(lr=1e-2, optimizer="muon", delay=1), x0, grads)
    _, x0s = run(HParams(lr=1e-2, optimizer="muon", delay=0), x0, grads)
    for t in range(1, len(grads)):
        for k in x0:
            assert rel(x1[t + 1][k], x0s[t][k]) < 1e-12, (t, k)


def test_non_muon_parameters_follow_adamw():
    rng = np.random.default_rng(7)
    x0 = toy_params(rng)
    grads = [{k: rng.standard_normal(v.shape) for k, v in x0.items()} for _ in range(4)]
    # no clipping: the clip coefficient is the only coupling between parameters
    sm, _ = run(HParams(lr=1e-2, clip_norm=0.0, optimizer="muon", ef_lambda=1.0), x0, grads)
    sa, _ = run(HParams(lr=1e-2, clip_norm=0.0, optimizer="adamw", ef_lambda=1.0), x0, grads)
    for k in ("embed", "blk0.attn_norm"):
        assert np.array_equal(sm.x[k], sa.x[k])
    assert not np.allclose(sm.x["blk0.wq"], sa.x["blk0.wq"])


@pytest.mark.parametrize("lam", [0.0, 0.5, 1.0])
def test_muon_replay(lam):
    # every x_{t+1} of a delay-1 Muon run equals x_t - u_{t-1} - lam (u_{t-1} - u_{t-2}) (the first
    # applied update standard), with u rebuilt from scratch: the momentum as an explicit weighted
    # sum of the clipped gradient history, O by the singular-value route, decay on x_t
    rng = np.random.default_rng(8)
    x0 = toy_params(rng)
    grads = [{k: rng.standard_normal(v.shape) * 3 for k, v in x0.items()} for _ in range(6)]
    hp = HParams(lr=2e-2, weight_decay=0.1, clip_norm=1.0, ef_lambda=lam, optimizer="muon", momentum=0.9)
    _, xs = run(hp, x0, grads)
    clips = []
    for g in grads:
        nrm = math.sqrt(sum(float(np.sum(v * v)) for v in g.values()))
        clips.append(min(1.0, hp.clip_norm / (nrm + 1e-6)))
    for k in ("blk0.wq", "blk0.wgate", "blk0.wdown"):
        us = []
        for t in range(1, len(grads)):
            # iteration t consumes g_{t-1}; the momentum has seen g_0 .. g_{t-1}
            M = sum((1 - hp.momentum) * hp.momentum ** (t - 1 - j) * clips[j] * grads[j][k] for j in range(t))
            u = hp.lr * (muon_scale(x0[k].shape, hp.update_rms) * svd_route(M) + hp.weight_decay * xs[t][k])
            expect = xs[t][k] - u - (lam * (u - us[-1]) if us and lam else 0.0)
            assert rel(xs[t + 1][k], expect) < 1e-9, (t, k)
            us.append(u)


def _semi_orthogonal(shape, seed):
    """An exactly semi-orthogonal matrix (orthonormal rows or columns) from a QR factorisation."""
    m, n = shape
    Q, _ = np.linalg.qr(np.random.default_rng(seed).standard_normal((max(m, n), min(m, n))))
    return Q if m >= n else Q.T


@pytest.mark.parametrize("shape", [(96, 32), (32, 96), (48, 48), (768, 3072)])
def test_muon_scale_gives_update_rms(shape):
    """The update RMS of §3 (0.2): s O has RMS 0.2 for an exactly semi-orthogonal O of any shape,
    measured directly, not through the formula muon_scale implements."""
    O = _semi_orthogonal(shape, 3)
    np.testing.assert_allclose(O @ O.T if shape[0] <= shape[1] else O.T @ O, np.eye(min(shape)), atol=1e-12)
    s = muon_scale(shape, 0.2)
    assert abs(math.sqrt(np.mean((s * O) ** 2)) - 0.2) < 1e-12
    s3 = muon_scale(shape, 0.35)
    assert abs(math.sqrt(np.mean((s3 * O) ** 2)) - 0.35) < 1e-12


@pytest.mark.parametrize("shape", [(96, 32), (32, 96), (40, 40)])
def test_muon_update_rms_on_semi_orthogonal_momentum(shape):
    """A first Muon update (wd 0, no clip) whose momentum is semi-orthogonal: Newton-Schulz maps
    every singular value 1 / sqrt(min(m, n)) of the normalised momentum through the scalar quintic
    to the same value q, so RMS(u) = lr 0.2 q exactly (the scalar recurrence computed here)."""
    G = _semi_orthogonal(shape, 4)
    hp = HParams(lr=3e-3, weight_decay=0.0, clip_norm=0.0, optimizer="muon", momentum=0.95, delay=0)
    name = "blk0.wq"
    st = OptState.create({name: np.zeros(shape)})
    iteration_update(st, {name: G}, hp)
    u = -st.x[name]
    a, b, c = NS_COEFFS
    M_fro = (1 - hp.momentum) * math.sqrt(min(shape))     # ||(1 - mu) G||_F
    q = (1 - hp.momentum) / (M_fro + NS_EPS)
    for _ in range(hp.ns_steps):
        q = a * q + b * q ** 3 + c * q ** 5
    rms = math.sqrt(np.mean(u ** 2))
    assert abs(rms - hp.lr * 0.2 * q) < 1e-12 * hp.lr
    # and u is parallel to G: every element scaled by the same factor
    np.testing.assert_allclose(u, hp.lr * 0.2 * math.sqrt(max(shape)) * q * G, rtol=1e-10, atol=1e-16)
