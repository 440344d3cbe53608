"""Pins of the oracle's fixed delay tau >= 2 (the delayed-gradient method of App. C with
prev(k) = k - tau, and its tau-step Error Feedback x_{k+1} = x_k - (tau + 1) u_k + tau u_{k-tau}).

Independent facts used: torch's own AdamW and global-norm clipping (a tau-delayed run under an
x-independent gradient sequence is the synchronous run tau iterations late), the closed forms of
Adam and of Newton-Schulz under a constant gradient, and a replay in which every update is rebuilt
from scratch (Adam's moments as explicit weighted sums of the clipped gradient history) and the
EF term takes the update formed tau iterations earlier."""
import math

import numpy as np
import pytest
import torch

from oracle.update import HParams, OptState, flat_update, iteration_update, muon_scale
from test_oracle_muon import svd_route

R = np.random.default_rng(11)


def _run(hp, x0, grads):
    st = OptState.create(x0)
    xs = [{k: v.copy() for k, v in st.x.items()}]
    for g in grads:
        iteration_update(st, g, hp)
        xs.append({k: v.copy() for k, v in st.x.items()})
    return st, xs


@pytest.mark.parametrize("tau", [2, 3])
def test_first_tau_iterations_change_nothing(tau):
    x0 = {"w": R.standard_normal(12)}
    grads = [{"w": R.standard_normal(12)} for _ in range(tau + 2)]
    st, xs = _run(HParams(lr=1e-2, delay=tau, ef_lambda=1.0), x0, grads)
    for t in range(tau + 1):
        assert np.array_equal(xs[t]["w"], x0["w"])
    assert not np.array_equal(xs[tau + 1]["w"], x0["w"])
    assert st.n_updates == 2


@pytest.mark.parametrize("tau", [2, 3, 5])
def test_delay_tau_lags_torch_synchronous_adamw_by_tau_steps(tau):
    # no weight decay: u depends on the gradient history only, so with gradients that do not depend
    # on x the delayed run replays the synchronous one tau iterations late
    hp = HParams(lr=1e-2, weight_decay=0.0, clip_norm=1.0, ef_lambda=0.0, delay=tau)
    x0 = R.standard_normal(30)
    G = [R.standard_normal(30) * (0.05 if t % 3 else 2.0) for t in range(12)]
    _, xs = _run(hp, {"w": x0}, [{"w": g} for g in G])
    p = torch.nn.Parameter(torch.tensor(x0, dtype=torch.float64))
    opt = torch.optim.AdamW([p], lr=hp.lr, betas=(hp.beta1, hp.beta2), eps=hp.eps, weight_decay=0.0,
                            foreach=False)
    sync = [x0.copy()]
    for g in G:
        p.grad = torch.tensor(g.copy())
        torch.nn.utils.clip_grad_norm_([p], hp.clip_norm)
        opt.step()
        sync.append(p.detach().numpy().copy())
    for t in range(len(G) + 1 - tau):
        np.testing.assert_allclose(xs[t + tau]["w"], sync[t], rtol=1e-12, atol=1e-15)


@pytest.mark.parametrize("tau", [2, 3])
@pytest.mark.parametrize("lam_of_tau", [0.0, 1.0, "tau"])
def test_constant_gradient_closed_form(tau, lam_of_tau):
    # constant g, no decay, no clipping: every update is lr g / (|g| + eps) (bias-corrected moments
    # equal g and g^2 exactly), the EF term lam (u - u_{t-tau}) vanishes, and the run moves by
    # (T - tau) updates
    lam = float(tau) if lam_of_tau == "tau" else lam_of_tau
    hp = HParams(lr=3e-3, weight_decay=0.0, clip_norm=0.0, ef_lambda=lam, delay=tau)
    x0 = R.standard_normal(16)
    g = R.standard_normal(16)
    T = 9
    st, _ = _run(hp, {"w": x0}, [{"w": g}] * T)
    u = hp.lr * g / (np.abs(g) + hp.eps)
    np.testing.assert_allclose(st.x["w"], x0 - (T - tau) * u, rtol=1e-10, atol=1e-14)


@pytest.mark.parametrize("tau", [2, 3])
def test_muon_constant_gradient_closed_form(tau):
    rng = np.random.default_rng(12)
    x0 = {"blk0.wq": rng.standard_normal((8, 8)) * 0.02, "blk0.wdown": rng.standard_normal((8, 12)) * 0.02}
    G = {k: rng.standard_normal(v.shape) for k, v in x0.items()}
    hp = HParams(lr=1e-2, weight_decay=0.0, clip_norm=0.0, ef_lambda=float(tau), optimizer="muon", delay=tau)
    T = 8
    st, _ = _run(hp, x0, [G] * T)
    for k in x0:
        expect = x0[k] - (T - tau) * hp.lr * muon_scale(x0[k].shape, hp.update_rms) * svd_route(G[k])
        assert np.linalg.norm(st.x[k] - expect) / np.linalg.norm(expect) < 1e-6, k


def _replay_u(hp, grads, clips, k, x_now):
    """The k-th AdamW update (k >= 1) from scratch: moments as explicit weighted sums of the clipped
    gradients g_0 .. g_{k-1}, bias-corrected, decay on the current weights."""
    b1, b2 = hp.beta1, hp.beta2
    m = sum((1 - b1) * b1 ** (k - 1 - j) * clips[j] * grads[j] for j in range(k))
    v = sum((1 - b2) * b2 ** (k - 1 - j) * (clips[j] * grads[j]) ** 2 for j in range(k))
    mhat, vhat = m / (1 - b1 ** k), v / (1 - b2 ** k)
    return hp.lr * (mhat / (np.sqrt(vhat) + hp.eps) + hp.weight_decay * x_now)


@pytest.mark.parametrize("tau", [2, 3])
@pytest.mark.parametrize("lam", [0.0, 0.5, "tau"])
def test_replay_from_scratch(tau, lam):
    lam = float(tau) if lam == "tau" else lam
    hp = HParams(lr=2e-2, weight_decay=0.1, clip_norm=1.0, ef_lambda=lam, delay=tau)
    x0 = R.standard_normal(20)
    G = [R.standard_normal(20) * (3.0 if t % 2 else 0.02) for t in range(11)]
    _, xs = _run(hp, {"w": x0}, [{"w": g} for g in G])
    clips = [min(1.0, hp.clip_norm / (math.sqrt(float(np.sum(g * g))) + 1e-6)) for g in G]
    us = {}
    for t in range(len(G)):
        if t < tau:
            np.testing.assert_array_equal(xs[t + 1]["w"], xs[t]["w"])
            continue
        k = t - tau + 1                       # iteration t applies the k-th update, from g_{t-tau}
        u = _replay_u(hp, G, clips, k, xs[t]["w"])
        expect = xs[t]["w"] - u
        if lam and k > tau:                   # the update formed tau iterations earlier
            expect = expect - lam * (u - us[k - tau])
        us[k] = u
        np.testing.assert_allclose(xs[t + 1]["w"], expect, rtol=1e-11, atol=1e-15)


@pytest.mark.parametrize("tau", [1, 2, 3])
def test_flat_update_replays_from_scratch(tau):
    # the elementwise form the flat update kernel follows: iteration t gets g_{t-tau} and the EF
    # buffer of the update formed tau iterations earlier (a ring of tau buffers, slot t mod tau)
    hp = HParams(lr=1e-2, weight_decay=0.1, clip_norm=0.0, ef_lambda=1.0, delay=tau)
    x = R.standard_normal(24)
    G = [R.standard_normal(24) for _ in range(10)]
    m = np.zeros(24); v = np.zeros(24)
    ring = [np.zeros(24) for _ in range(tau)]
    xs = [x.copy()]
    for t in range(len(G)):
        g = G[t - tau] if t >= tau else np.zeros(24)
        x, m, v, ring[t % tau] = flat_update(x, g, m, v, ring[t % tau], t, hp)
        xs.append(x.copy())
    us = {}
    for t in range(tau, len(G)):
        k = t - tau + 1
        u = _replay_u(hp, G, [1.0] * len(G), k, xs[t])
        expect = xs[t] - u - ((u - us[k - tau]) if k > tau else 0.0)
        us[k] = u
        np.testing.assert_allclose(xs[t + 1], expect, rtol=1e-11, atol=1e-15)
