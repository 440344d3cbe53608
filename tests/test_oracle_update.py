"""Pins of the oracle's delayed update (Alg. 1, Error Feedback of §3.2 and App. A.4).

Independent facts used: torch's own AdamW and global-norm clipping (library routines, float64 CPU),
the one-step lag of a delayed run under an x-independent gradient sequence, the closed form of Adam
under a constant gradient, the telescoping sum of the lambda-EF recurrence, and a brute-force
replay of the delayed rule on the tiny stage with gradients recomputed from scratch."""
import math

import numpy as np
import pytest
import torch

from datagen import Workload, init_params, step_inputs
from oracle import model, run
from oracle.update import HParams, OptState, flat_update, global_norm, iteration_update

R = np.random.default_rng(7)


def _torch_adamw(x0, hp):
    p = torch.nn.Parameter(torch.tensor(x0, dtype=torch.float64))
    opt = torch.optim.AdamW([p], lr=hp.lr, betas=(hp.beta1, hp.beta2), eps=hp.eps,
                            weight_decay=hp.weight_decay, foreach=False)
    return p, opt


def _torch_u(p, opt, x_now, g, clip):
    """One torch AdamW step taken at x_now with gradient g (torch's own clipping applied);
    returns u = x_now - x_after."""
    with torch.no_grad():
        p.copy_(torch.tensor(x_now))
    p.grad = torch.tensor(g.copy())
    if clip > 0:
        torch.nn.utils.clip_grad_norm_([p], clip)
    opt.step()
    return x_now - p.detach().numpy().copy()


def test_delay0_equals_torch_adamw_with_clipping():
    hp = HParams(lr=1e-2, weight_decay=0.1, clip_norm=1.0, ef_lambda=0.0, delay=0)
    x0 = R.standard_normal(40)
    st = OptState.create({"w": x0})
    p, opt = _torch_adamw(x0, hp)
    for t in range(12):
        g = R.standard_normal(40) * (0.05 if t % 2 else 3.0)  # alternate clipped / unclipped
        iteration_update(st, {"w": g}, hp)
        p.grad = torch.tensor(g.copy())
        torch.nn.utils.clip_grad_norm_([p], hp.clip_norm)
        opt.step()
        np.testing.assert_allclose(st.x["w"], p.detach().numpy(), rtol=1e-12, atol=1e-15)


def test_delay1_lags_synchronous_by_one_step_for_fixed_gradient_sequence():
    hp1 = HParams(lr=1e-2, weight_decay=0.1, clip_norm=0.0, ef_lambda=0.0, delay=1)
    x0 = R.standard_normal(30)
    G = [R.standard_normal(30) for _ in range(10)]
    st = OptState.create({"w": x0})
    p, opt = _torch_adamw(x0, hp1)
    sync = [x0.copy()]
    for g in G:
        p.grad = torch.tensor(g.copy())
        opt.step()
        sync.append(p.detach().numpy().copy())
    for t, g in enumerate(G):
        iteration_update(st, {"w": g}, hp1)          # x_{t+1}
        np.testing.assert_allclose(st.x["w"], sync[t], rtol=1e-12)   # x^delayed_{t+1} = x^sync_t


def test_constant_gradient_closed_form_with_and_without_ef():
    # constant g, no weight decay: m_hat = g, v_hat = g^2, u = lr g / (|g| + eps) every update;
    # delayed: x_T = x_0 - (T-1) u; lambda-EF adds -lam (u - u) = 0.
    g = R.standard_normal(25)
    x0 = R.standard_normal(25)
    for lam in (0.0, 1.0, 2.5):
        hp = HParams(lr=3e-3, weight_decay=0.0, clip_norm=0.0, ef_lambda=lam, delay=1)
        st = OptState.create({"w": x0})
        u = hp.lr * g / (np.abs(g) + hp.eps)
        for t in range(8):
            iteration_update(st, {"w": g}, hp)
            np.testing.assert_allclose(st.x["w"], x0 - max(t, 0) * u, rtol=1e-10, atol=1e-14)


def test_ef_telescoping_against_torch_updates():
    # With weight decay 0 the update sequence u_j does not depend on x, and the lambda-EF
    # recurrence sums to x_T = x_0 - sum_{j<=T-2} u_j - lam (u_{T-2} - u_0).
    T = 9
    G = [R.standard_normal(20) for _ in range(T)]
    x0 = R.standard_normal(20)
    for lam in (0.0, 1.0, 1.7):
        hp = HParams(lr=1e-2, weight_decay=0.0, clip_norm=0.0, ef_lambda=lam, delay=1)
        p, opt = _torch_adamw(np.zeros(20), hp)
        us = [_torch_u(p, opt, np.zeros(20), G[j], 0.0) for j in range(T - 1)]
        st = OptState.create({"w": x0})
        for t in range(T):
            iteration_update(st, {"w": G[t]}, hp)
        Tn = T  # state now holds x_T
        ref = x0 - sum(us[: Tn - 1]) - lam * (us[Tn - 2] - us[0])
        np.testing.assert_allclose(st.x["w"], ref, rtol=1e-11, atol=1e-14)


def test_sapipe_same_state_prediction_displacement_equals_ef():
    # App. B.1: predicted points x~_{t+1} = x_{t+1} - u(g_{t-1}) of the standard delayed run move
    # by -2u(g_{t-1}) + u(g_{t-2}), the EF displacement, when the updates are fixed in advance.
    T = 7
    G = [R.standard_normal(10) for _ in range(T)]
    hp0 = HParams(lr=1e-2, weight_decay=0.0, clip_norm=0.0, ef_lambda=0.0, delay=1)
    hp1 = HParams(lr=1e-2, weight_decay=0.0, clip_norm=0.0, ef_lambda=1.0, delay=1)
    x0 = R.standard_normal(10)
    a, b = OptState.create({"w": x0}), OptState.create({"w": x0})
    xs_std, us, xs_ef = [x0], [], [x0]
    for t in range(T):
        iteration_update(a, {"w": G[t]}, hp0)
        iteration_update(b, {"w": G[t]}, hp1)
        xs_std.append(a.x["w"].copy())
        us.append(a.u_prev["w"].copy() if a.n_updates else np.zeros(10))
        xs_ef.append(b.x["w"].copy())
    for t in range(3, T):
        pred_next = xs_std[t + 1] - us[t]
        pred_now = xs_std[t] - us[t - 1]
        np.testing.assert_allclose(pred_next - pred_now, xs_ef[t + 1] - xs_ef[t], rtol=1e-10, atol=1e-15)


def test_lambda_zero_is_standard_and_clipping_bound():
    hp0 = HParams(ef_lambda=0.0)
    st = OptState.create({"w": np.ones(5)})
    st2 = OptState.create({"w": np.ones(5)})
    for t in range(5):
        g = {"w": R.standard_normal(5) * 10}
        iteration_update(st, g, hp0)
        iteration_update(st2, {"w": g["w"].copy()}, HParams(ef_lambda=0.0))
    np.testing.assert_array_equal(st.x["w"], st2.x["w"])
    from oracle.update import clip_coefficient
    g = R.standard_normal(100) * 5
    n = float(np.linalg.norm(g))
    c = clip_coefficient(n, 1.0)
    assert np.linalg.norm(c * g) <= 1.0 * (1 + 1e-6)
    assert clip_coefficient(0.5, 1.0) == 1.0


def _grad_seq(n, T, bad):
    """x-independent gradient sequence; g_bad holds an infinity in one element."""
    gs = [R.standard_normal(n) for _ in range(T)]
    gs[bad] = gs[bad].copy()
    gs[bad][3] = np.inf
    return gs


def test_nonfinite_gradient_is_skipped_with_k_advanced():
    """A non-finite g_{t-1} leaves x, m, v and u_prev as they are, and the next update takes the
    bias correction of the following index: torch AdamW (its own step counter advanced by hand,
    no step taken for the bad gradient) on the same delayed sequence, lambda = 0."""
    n, T, bad = 12, 8, 3
    hp = HParams(lr=1e-2, clip_norm=0.0, ef_lambda=0.0, delay=1)
    gs = _grad_seq(n, T, bad)
    x0 = R.standard_normal(n)
    st = OptState.create({"w": x0})
    p, opt = _torch_adamw(x0, hp)
    for t in range(T):
        before = st.copy()
        info = iteration_update(st, {"w": gs[t]}, hp)
        if t == 0:
            continue
        if t - 1 == bad:   # consumes the bad gradient
            assert info["skipped"] and not info["applied"] and st.n_skipped == 1
            for f in ("x", "m", "v", "u_prev"):
                np.testing.assert_array_equal(getattr(st, f)["w"], getattr(before, f)["w"])
            opt.state[p]["step"] += 1      # torch: the iteration is counted, no step is taken
            continue
        p.grad = torch.tensor(gs[t - 1])
        opt.step()
        np.testing.assert_allclose(st.x["w"], p.detach().numpy(), rtol=1e-12, atol=1e-15)
    assert st.n_updates == T - 1


def test_nonfinite_gradient_ef_reads_last_applied_update():
    """With Error Feedback after a skip, the EF term takes the update of the last applied
    iteration (the EF buffer kept its contents): x_{t+1} = x_t - u - lambda (u - u_last)."""
    n, T, bad, lam = 10, 7, 2, 1.0
    hp = HParams(lr=1e-2, clip_norm=0.0, ef_lambda=lam, delay=1)
    gs = _grad_seq(n, T, bad)
    x0 = R.standard_normal(n)
    st = OptState.create({"w": x0})
    p, opt = _torch_adamw(np.zeros(n), hp)
    u_last = None
    for t in range(T):
        x_t = st.x["w"].copy()
        iteration_update(st, {"w": gs[t]}, hp)
        if t == 0:
            continue
        if t - 1 == bad:
            opt.state[p]["step"] += 1
            np.testing.assert_array_equal(st.x["w"], x_t)
            continue
        u = _torch_u(p, opt, x_t, gs[t - 1], 0.0)
        ref = x_t - u if u_last is None else x_t - u - lam * (u - u_last)
        np.testing.assert_allclose(st.x["w"], ref, rtol=1e-12, atol=1e-15)
        u_last = u


@pytest.mark.parametrize("tau", [2, 3])
def test_nonfinite_gradient_tau_keeps_ef_slot(tau):
    """Delay tau: the skipped iteration's EF slot keeps its contents, so the iteration tau later
    reads the update formed 2 tau iterations before it (zero before the ring's first write)."""
    n, T = 9, 4 * tau + 3
    hp = HParams(lr=1e-2, clip_norm=0.0, ef_lambda=float(tau), delay=tau)
    for bad in (1, tau + 1):      # consumed at iteration bad + tau (ring still filling, ring full)
        gs = _grad_seq(n, T, bad)
        st = OptState.create({"w": R.standard_normal(n)})
        slots = [np.zeros(n) for _ in range(tau)]     # the device ring: iteration t uses t mod tau
        p, opt = _torch_adamw(np.zeros(n), hp)
        for t in range(T):
            x_t = st.x["w"].copy()
            iteration_update(st, {"w": gs[t]}, hp)
            if t < tau:
                np.testing.assert_array_equal(st.x["w"], x_t)
                continue
            j = t - tau                 # the gradient consumed
            if j == bad:
                opt.state[p]["step"] += 1
                np.testing.assert_array_equal(st.x["w"], x_t)
                continue
            u = _torch_u(p, opt, x_t, gs[j], 0.0)
            ef = j >= tau              # tau gradients consumed before this one
            ref = x_t - u - tau * (u - slots[t % tau]) if ef else x_t - u
            np.testing.assert_allclose(st.x["w"], ref, rtol=1e-12, atol=1e-15)
            slots[t % tau] = u


@pytest.mark.parametrize("kind", ["tau2-ef", "predict", "delay1-ef"])
def test_optstate_copy_round_trip(kind):
    """copy() reproduces every field, shares no array with the original, and a run continued from
    the copy equals the run continued from the original."""
    hp = {"tau2-ef": HParams(lr=1e-2, ef_lambda=2.0, delay=2),
          "predict": HParams(lr=1e-2, predict="updated"),
          "delay1-ef": HParams(lr=1e-2, ef_lambda=1.0)}[kind]
    gs = [{"w": R.standard_normal(6), "b": R.standard_normal(3)} for _ in range(9)]
    st = OptState.create({"w": R.standard_normal(6), "b": R.standard_normal(3)})
    for t in range(5):
        iteration_update(st, gs[t], hp)
    cp = st.copy()

    def same(a, b):
        if isinstance(a, dict):
            assert a.keys() == b.keys()
            for k in a:
                np.testing.assert_array_equal(a[k], b[k])
                assert a[k] is not b[k]
        elif isinstance(a, list):
            assert len(a) == len(b)
            for u, v in zip(a, b):
                same(u, v)
        else:
            assert a == b

    import dataclasses
    for f in dataclasses.fields(OptState):
        a, b = getattr(st, f.name), getattr(cp, f.name)
        assert (a is None) == (b is None), f.name
        if a is not None:
            same(a, b)
    if kind == "tau2-ef":
        assert len(cp.u_ring) == 2 and len(cp.queue) == 2 and cp.x_compute is None
    if kind == "predict":
        assert isinstance(cp.x_compute, dict) and cp.u_ring == []
    for t in range(5, 9):
        iteration_update(st, gs[t], hp)
        iteration_update(cp, gs[t], hp)
    same(st.x, cp.x)
    same(st.m, cp.m)


def test_flat_update_matches_iteration_update():
    hp = HParams(lr=1e-3, ef_lambda=1.0, clip_norm=0.0)
    x0 = R.standard_normal(50)
    g = R.standard_normal(50)
    st = OptState.create({"w": x0})
    x, m, v, up = x0.copy(), np.zeros(50), np.zeros(50), np.zeros(50)
    for t in range(6):
        iteration_update(st, {"w": g}, hp)
        x, m, v, up = flat_update(x, g, m, v, up, t, hp)
        np.testing.assert_allclose(x, st.x["w"], rtol=1e-15)


TINYT = Workload("replay", 2, 8, 4, 2, 4, 12, 11, True, True, True, 6, 2, 1, "f32", 6, 21)


@pytest.mark.parametrize("lam", [0.0, 1.0])
def test_brute_force_replay_delay1_uses_gradient_at_previous_weights(lam):
    """Run the delayed oracle, store every x_t; then recompute g_{t-1} from scratch at x_{t-1}
    and check x_{t+1} = x_t - u_{t-1}(g_{t-1}) (- lam (u_{t-1} - u_{t-2})) with u from torch."""
    w = TINYT
    hp = HParams(lr=5e-3, weight_decay=0.1, clip_norm=0.05, ef_lambda=lam, delay=1)
    p0 = {k: v.astype(np.float64) for k, v in init_params(w).items()}
    xs = [dict(p0)]
    recs = []

    def rec(t, info):
        recs.append(info)

    inputs = lambda t, i: step_inputs(w, t, i)
    st = OptState.create(p0)
    for t in range(w.steps):
        grads, _ = model.stage_step_grads(st.x, [inputs(t, 0)], w)
        iteration_update(st, grads, hp)
        xs.append({k: v.copy() for k, v in st.x.items()})
    names = sorted(p0)
    flat = lambda d: np.concatenate([d[k].reshape(-1) for k in names])
    p, opt = _torch_adamw(np.zeros(sum(p0[k].size for k in names)), hp)
    u_prev = None
    assert np.array_equal(flat(xs[1]), flat(xs[0]))          # t = 0 changes nothing
    for t in range(1, w.steps):
        g_prev, _ = model.stage_step_grads(xs[t - 1], [inputs(t - 1, 0)], w)   # fresh, at x_{t-1}
        u = _torch_u(p, opt, flat(xs[t]), flat(g_prev), hp.clip_norm)
        ref = flat(xs[t]) - u
        if u_prev is not None:
            ref = ref - lam * (u - u_prev)
        np.testing.assert_allclose(flat(xs[t + 1]), ref, rtol=1e-10, atol=1e-13)
        u_prev = u


def test_run_checkpoint_resume_bit_identical():
    w = TINYT
    hp = HParams(lr=5e-3, ef_lambda=1.0)
    p0 = init_params(w)
    inputs = lambda t, i: step_inputs(w, t, i)
    full = run(w, 6, hp, p0, inputs)
    st = OptState.create(p0)
    for t in range(3):
        g, _ = model.stage_step_grads(st.x, [inputs(t, 0)], w)
        iteration_update(st, g, hp)
    saved = st.copy()
    for t in range(3, 6):
        g, _ = model.stage_step_grads(saved.x, [inputs(t, 0)], w)
        iteration_update(saved, g, hp)
    for k in p0:
        np.testing.assert_array_equal(saved.x[k], full.x[k])
        np.testing.assert_array_equal(saved.u_prev[k], full.u_prev[k])
