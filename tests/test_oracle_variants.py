"""Pins of the oracle's elementwise update variants: NAdam and Lion as u, and SAPipe weight
prediction with the updated optimizer state (App. B.1).

Independent facts used: torch's own NAdam (decoupled weight decay, its momentum-decay schedule) and
AdamW stepped a second time from a copy of its state, global-norm clipping, a delayed run being the
synchronous one a step late under an x-independent gradient sequence, the closed form of Lion under
a constant gradient, Lion's invariance to a positive gradient scale, and a Lion replay with the
momentum rebuilt as an explicit weighted sum of the gradient history."""
import copy

import numpy as np
import pytest
import torch

from oracle.update import HParams, OptState, iteration_update

R = np.random.default_rng(23)


@pytest.fixture(autouse=True)
def _torch_float64_scalars():
    # torch keeps NAdam's running momentum product in the default dtype: float64 for the pins
    old = torch.get_default_dtype()
    torch.set_default_dtype(torch.float64)
    yield
    torch.set_default_dtype(old)


def _run(hp, x0, grads):
    st = OptState.create({"w": x0})
    xs, xc = [x0.copy()], [None]
    for g in grads:
        iteration_update(st, {"w": g}, hp)
        xs.append(st.x["w"].copy())
        xc.append(None if st.x_compute is None else st.x_compute["w"].copy())
    return st, xs, xc


def _torch_nadam(x0, hp):
    p = torch.nn.Parameter(torch.tensor(x0, dtype=torch.float64))
    opt = torch.optim.NAdam([p], lr=hp.lr, betas=(hp.beta1, hp.beta2), eps=hp.eps,
                            weight_decay=hp.weight_decay, momentum_decay=hp.nadam_psi,
                            decoupled_weight_decay=True, foreach=False)
    return p, opt


def test_nadam_delay0_equals_torch_with_clipping():
    hp = HParams(lr=1e-2, beta2=0.999, weight_decay=0.1, clip_norm=1.0, delay=0, optimizer="nadam")
    x0 = R.standard_normal(40)
    G = [R.standard_normal(40) * (0.05 if t % 2 else 3.0) for t in range(14)]
    _, xs, _ = _run(hp, x0, G)
    p, opt = _torch_nadam(x0, hp)
    for t, g in enumerate(G):
        p.grad = torch.tensor(g.copy())
        torch.nn.utils.clip_grad_norm_([p], hp.clip_norm)
        opt.step()
        np.testing.assert_allclose(xs[t + 1], p.detach().numpy(), rtol=1e-12, atol=1e-15)


def test_nadam_delay1_lags_torch_by_one_step():
    hp = HParams(lr=1e-2, beta2=0.999, weight_decay=0.0, clip_norm=0.0, delay=1, optimizer="nadam")
    x0 = R.standard_normal(30)
    G = [R.standard_normal(30) for _ in range(10)]
    _, xs, _ = _run(hp, x0, G)
    p, opt = _torch_nadam(x0, hp)
    sync = [x0.copy()]
    for g in G:
        p.grad = torch.tensor(g.copy())
        opt.step()
        sync.append(p.detach().numpy().copy())
    for t in range(len(G)):
        np.testing.assert_allclose(xs[t + 1], sync[t], rtol=1e-12, atol=1e-15)


@pytest.mark.parametrize("lam", [0.0, 1.0])
def test_lion_constant_gradient_closed_form(lam):
    hp = HParams(lr=5e-4, beta1=0.9, beta2=0.99, weight_decay=0.0, clip_norm=0.0, ef_lambda=lam,
                 optimizer="lion")
    x0 = R.standard_normal(16)
    g = R.standard_normal(16)
    T = 7
    st, _, _ = _run(hp, x0, [g] * T)
    np.testing.assert_allclose(st.x["w"], x0 - (T - 1) * hp.lr * np.sign(g), rtol=1e-13, atol=1e-15)


def test_lion_is_invariant_to_a_positive_gradient_scale():
    hp = HParams(lr=5e-4, beta1=0.9, beta2=0.99, weight_decay=0.5, clip_norm=0.0, ef_lambda=1.0,
                 optimizer="lion")
    x0 = R.standard_normal(25)
    G = [R.standard_normal(25) for _ in range(9)]
    _, a, _ = _run(hp, x0, G)
    _, b, _ = _run(hp, x0, [7.5 * g for g in G])
    for xa, xb in zip(a, b):
        np.testing.assert_allclose(xa, xb, rtol=1e-12, atol=1e-15)


@pytest.mark.parametrize("lam", [0.0, 1.0])
def test_lion_replay_from_scratch(lam):
    hp = HParams(lr=5e-4, beta1=0.9, beta2=0.99, weight_decay=0.5, clip_norm=1.0, ef_lambda=lam,
                 optimizer="lion")
    x0 = R.standard_normal(20)
    G = [R.standard_normal(20) * (3.0 if t % 2 else 0.02) for t in range(9)]
    G[3][5] = 0.0                                    # sign(0) = 0 in the first update that sees it
    _, xs, _ = _run(hp, x0, G)
    clips = [min(1.0, hp.clip_norm / (float(np.linalg.norm(g)) + 1e-6)) for g in G]
    u_prev = None
    for t in range(1, len(G)):
        k = t                                        # iteration t applies the k-th update, from g_{t-1}
        m_before = sum((1 - hp.beta2) * hp.beta2 ** (k - 2 - j) * clips[j] * G[j] for j in range(k - 1)) \
            if k > 1 else np.zeros(20)
        c = hp.beta1 * m_before + (1 - hp.beta1) * clips[k - 1] * G[k - 1]
        u = hp.lr * (np.sign(c) + hp.weight_decay * xs[t])
        expect = xs[t] - u - (lam * (u - u_prev) if (lam and u_prev is not None) else 0.0)
        np.testing.assert_allclose(xs[t + 1], expect, rtol=1e-12, atol=1e-15)
        u_prev = u


def test_sapipe_updated_state_prediction_matches_torch_second_step():
    # master: torch AdamW one step late; prediction: the same torch optimizer stepped once more with
    # the same (clipped) gradient from a copy of its updated state
    hp = HParams(lr=1e-2, weight_decay=0.1, clip_norm=1.0, ef_lambda=0.0, delay=1, predict="updated")
    x0 = R.standard_normal(30)
    G = [R.standard_normal(30) * (0.05 if t % 2 else 3.0) for t in range(10)]
    _, xs, xc = _run(hp, x0, G)
    p = torch.nn.Parameter(torch.tensor(x0, dtype=torch.float64))
    opt = torch.optim.AdamW([p], lr=hp.lr, betas=(hp.beta1, hp.beta2), eps=hp.eps,
                            weight_decay=hp.weight_decay, foreach=False)
    assert xc[1] is None   # t = 0 applies nothing and predicts nothing
    for t in range(1, len(G)):
        with torch.no_grad():
            p.copy_(torch.tensor(xs[t]))
        p.grad = torch.tensor(G[t - 1].copy())
        torch.nn.utils.clip_grad_norm_([p], hp.clip_norm)
        opt.step()
        np.testing.assert_allclose(xs[t + 1], p.detach().numpy(), rtol=1e-12, atol=1e-15)
        q = torch.nn.Parameter(p.detach().clone())
        o2 = torch.optim.AdamW([q], lr=hp.lr, betas=(hp.beta1, hp.beta2), eps=hp.eps,
                               weight_decay=hp.weight_decay, foreach=False)
        o2.load_state_dict(copy.deepcopy(opt.state_dict()))
        q.grad = p.grad.clone()
        o2.step()
        np.testing.assert_allclose(xc[t + 1], q.detach().numpy(), rtol=1e-12, atol=1e-15)


def test_sapipe_master_is_the_standard_delayed_run():
    x0 = R.standard_normal(12)
    G = [R.standard_normal(12) for _ in range(8)]
    _, a, _ = _run(HParams(lr=1e-2, ef_lambda=0.0, predict="updated"), x0, G)
    _, b, _ = _run(HParams(lr=1e-2, ef_lambda=0.0), x0, G)
    for xa, xb in zip(a, b):
        np.testing.assert_array_equal(xa, xb)


# ---------------------------------------------------------------------------------------- Adan
ADAN = dict(optimizer="adan", beta1=0.98, beta2=0.92, beta3=0.99)


def test_adan_with_beta2_zero_is_adamw():
    """beta2 = 0 takes the difference terms out: d is fed back with weight 0 and n averages g^2,
    so Adan(beta1, 0, beta3) is AdamW(beta1, beta3) -- torch's AdamW with clipping, synchronous."""
    hp = HParams(lr=1e-2, weight_decay=0.1, clip_norm=1.0, delay=0, **dict(ADAN, beta2=0.0))
    x0 = R.standard_normal(30)
    G = [R.standard_normal(30) * (0.05 if t % 2 else 3.0) for t in range(12)]
    _, xs, _ = _run(hp, x0, G)
    p = torch.nn.Parameter(torch.tensor(x0))
    opt = torch.optim.AdamW([p], lr=hp.lr, betas=(hp.beta1, hp.beta3), eps=hp.eps,
                            weight_decay=hp.weight_decay, foreach=False)
    for t, g in enumerate(G):
        p.grad = torch.tensor(g.copy())
        torch.nn.utils.clip_grad_norm_([p], hp.clip_norm)
        opt.step()
        np.testing.assert_allclose(xs[t + 1], p.detach().numpy(), rtol=1e-12, atol=1e-15)


@pytest.mark.parametrize("lam", [0.0, 1.0])
def test_adan_constant_gradient_closed_form(lam):
    """A constant gradient has zero differences: d = 0, n / (1 - b3^k) = g^2, m / (1 - b1^k) = g,
    so every update is lr (g / (|g| + eps) + wd x_t); delay 1: x_{t+1} = x_t - u (EF: - lam (u -
    u_prev)), with x_1 = x_0."""
    hp = HParams(lr=5e-3, weight_decay=0.0, clip_norm=0.0, ef_lambda=lam, delay=1, **ADAN)
    g = R.standard_normal(16)
    x0 = R.standard_normal(16)
    _, xs, _ = _run(hp, x0, [g] * 8)
    u = hp.lr * g / (np.abs(g) + hp.eps)
    expect = [x0, x0]
    for t in range(1, 8):
        step = u if t == 1 or lam == 0 else u + lam * (u - u)
        expect.append(expect[-1] - step)
    for a, b in zip(xs, expect):
        np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("lam", [0.0, 1.0])
def test_adan_replay_with_explicit_sums(lam):
    """Delay-1 Adan with clipping and decay, against a from-scratch rebuild of every update: the
    three averages as explicit weighted sums over the clipped history of consumed gradients
    (differences from the second consumed gradient on), with the bias corrections of the count."""
    hp = HParams(lr=2e-3, weight_decay=0.1, clip_norm=0.5, ef_lambda=lam, delay=1, **ADAN)
    T = 9
    G = [R.standard_normal(12) * (0.1 if t % 3 else 2.0) for t in range(T)]
    x0 = R.standard_normal(12)
    _, xs, _ = _run(hp, x0, G)
    clipped = []
    x = x0.copy()
    u_prev = None
    assert np.array_equal(xs[1], x0)
    for t in range(1, T):
        g = G[t - 1]
        clipped.append(g * min(1.0, hp.clip_norm / (np.linalg.norm(g) + 1e-6)))
        k = len(clipped)
        diffs = [np.zeros(12)] + [clipped[j] - clipped[j - 1] for j in range(1, k)]
        m = sum((1 - hp.beta1) * hp.beta1 ** (k - 1 - j) * clipped[j] for j in range(k))
        d = sum((1 - hp.beta2) * hp.beta2 ** (k - 1 - j) * diffs[j] for j in range(k))
        n = sum((1 - hp.beta3) * hp.beta3 ** (k - 1 - j) * (clipped[j] + hp.beta2 * diffs[j]) ** 2
                for j in range(k))
        u = hp.lr * ((m / (1 - hp.beta1 ** k) + hp.beta2 * d / (1 - hp.beta2 ** k)) /
                     (np.sqrt(n / (1 - hp.beta3 ** k)) + hp.eps) + hp.weight_decay * x)
        x = x - u if (u_prev is None or lam == 0) else x - u - lam * (u - u_prev)
        u_prev = u
        np.testing.assert_allclose(xs[t + 1], x, rtol=1e-11, atol=1e-14)


def test_adan_delay1_lags_synchronous_by_one_step():
    hp0 = HParams(lr=1e-2, clip_norm=1.0, delay=0, **ADAN)
    hp1 = HParams(lr=1e-2, clip_norm=1.0, delay=1, **ADAN)
    x0 = R.standard_normal(20)
    G = [R.standard_normal(20) for _ in range(10)]
    _, xs0, _ = _run(hp0, x0, G)
    _, xs1, _ = _run(hp1, x0, G)
    for t in range(1, 10):
        np.testing.assert_allclose(xs1[t + 1], xs0[t], rtol=1e-13, atol=1e-15)
