"""Pins of the oracle's stage forward/backward: finite differences through the whole stage (float64),
closed forms and invariants that a dropped term, a wrong sign or a swapped operand would break."""
import math

import numpy as np
import pytest

from datagen import Workload, init_params, param_specs, step_inputs
from oracle import model

R = np.random.default_rng(99)

HEAD = Workload("test-head", 2, 8, 4, 2, 4, 12, 11, True, True, True, 5, 2, 1, "f32", 3, 7)
MIDDLE = Workload("test-mid", 2, 8, 4, 2, 4, 12, 0, False, False, False, 5, 2, 1, "f32", 3, 8)
FIRST = Workload("test-first", 1, 8, 2, 2, 4, 12, 11, True, False, False, 5, 2, 1, "f32", 3, 9)
LAST = Workload("test-last", 2, 8, 4, 2, 4, 12, 11, False, True, False, 5, 2, 1, "f32", 3, 10)


def _params(w, scale=0.5):
    p = {}
    for name, shape, init in param_specs(w):
        base = 1.0 if init == "ones" else 0.0
        p[name] = base + scale * R.standard_normal(shape)
    return p


def _loss(w, p, inp):
    out, _ = model.stage_forward(p, inp, w)
    return float(out["loss"])


@pytest.mark.parametrize("w", [HEAD, MIDDLE, FIRST, LAST], ids=["head", "middle", "first", "last-untied"])
def test_stage_gradients_finite_differences(w):
    p = _params(w)
    inp = {k: (v.astype(np.float64) if v.dtype != np.int32 else v) for k, v in step_inputs(w, 0).items()}
    if "dy" in inp:
        inp["dy"] = R.standard_normal(inp["dy"].shape)
    out, sv = model.stage_forward(p, inp, w)
    grads, dx_in = model.stage_backward(p, inp, sv, w)
    assert set(grads) == set(p)
    h = 1e-6
    for name, arr in p.items():
        flat = arr.reshape(-1)
        for i in R.choice(flat.size, size=min(6, flat.size), replace=False):
            old = flat[i]
            flat[i] = old + h
            fp = _loss(w, p, inp)
            flat[i] = old - h
            fm = _loss(w, p, inp)
            flat[i] = old
            num = (fp - fm) / (2 * h)
            ana = grads[name].reshape(-1)[i]
            assert abs(num - ana) <= 1e-6 * max(1.0, abs(num)), (name, i, num, ana)
    # a random direction through all parameters at once
    dirs = {k: R.standard_normal(v.shape) for k, v in p.items()}
    eps = 1e-6
    pp = {k: p[k] + eps * dirs[k] for k in p}
    pm = {k: p[k] - eps * dirs[k] for k in p}
    num = (_loss(w, pp, inp) - _loss(w, pm, inp)) / (2 * eps)
    ana = sum(float(np.sum(grads[k] * dirs[k])) for k in p)
    assert abs(num - ana) <= 1e-6 * max(1.0, abs(num))
    if not w.first_stage:
        x = inp["x_in"]
        flat = x.reshape(-1)
        for i in R.choice(flat.size, size=6, replace=False):
            old = flat[i]
            flat[i] = old + h
            fp = _loss(w, p, inp)
            flat[i] = old - h
            fm = _loss(w, p, inp)
            flat[i] = old
            assert abs((fp - fm) / (2 * h) - dx_in.reshape(-1)[i]) <= 1e-6 * max(1.0, abs(fp))


def test_block_is_identity_when_output_projections_are_zero():
    w = MIDDLE
    p = _params(w)
    for i in range(w.n_blocks):
        p[f"blk{i}.wo"][:] = 0.0
        p[f"blk{i}.wdown"][:] = 0.0
    x = R.standard_normal((2, 5, 8))
    out, _ = model.stage_forward(p, {"x_in": x}, w)
    np.testing.assert_array_equal(out["y"], x)


def test_attention_only_block_adds_mean_of_values_when_queries_vanish():
    # wq = 0 makes every causal attention row uniform; with wdown = 0 the block output is
    # x + mean_{j<=i}(v_j) Wo^T, v = RMSNorm(x) Wv^T: a closed form through norm, projections,
    # causal mean and residual.
    w = MIDDLE.with_(n_blocks=1, n_heads=2, n_kv_heads=2)
    p = _params(w)
    p["blk0.wq"][:] = 0.0
    p["blk0.wdown"][:] = 0.0
    x = R.standard_normal((1, 5, 8))
    out, _ = model.stage_forward(p, {"x_in": x}, w)
    xf = x[0]
    n1 = xf / np.sqrt(np.mean(xf * xf, axis=1, keepdims=True) + w.rms_eps) * p["blk0.attn_norm"]
    vv = n1 @ p["blk0.wv"].T
    cm = np.cumsum(vv, axis=0) / np.arange(1, 6)[:, None]
    ref = xf + cm @ p["blk0.wo"].T
    np.testing.assert_allclose(out["y"][0], ref, rtol=1e-12, atol=1e-12)


def test_stage_causality_over_tokens():
    w = HEAD
    p = _params(w)
    inp = step_inputs(w, 0)
    out1, _ = model.stage_forward(p, inp, w)
    inp2 = {k: v.copy() for k, v in inp.items()}
    inp2["tokens"][:, 3:] = (inp2["tokens"][:, 3:] + 1) % w.vocab
    out2, _ = model.stage_forward(p, inp2, w)
    l1 = out1["logits"].reshape(2, 5, -1)
    l2 = out2["logits"].reshape(2, 5, -1)
    np.testing.assert_array_equal(l1[:, :3], l2[:, :3])
    assert np.abs(l1[:, 3:] - l2[:, 3:]).max() > 1e-6


def test_zero_embedding_gives_uniform_loss_log_vocab():
    w = HEAD
    p = _params(w)
    p["embed"][:] = 0.0
    out, _ = model.stage_forward(p, step_inputs(w, 0), w)
    assert abs(float(out["loss"]) - math.log(w.vocab)) < 1e-14


def test_zero_untied_head_gives_uniform_loss_log_vocab():
    w = LAST
    p = _params(w)
    p["head"][:] = 0.0
    out, _ = model.stage_forward(p, step_inputs(w, 0), w)
    assert abs(float(out["loss"]) - math.log(w.vocab)) < 1e-14


def test_untied_head_equal_to_embedding_matches_tied():
    # a stage holding both ends with a separate head matrix equal to the embedding computes the
    # tied stage's logits, and its two matrix gradients sum to the tied embedding gradient
    wt = HEAD
    wu = HEAD.with_(tie_embedding=False)
    p = _params(wt)
    pu = dict(p, head=p["embed"].copy())
    inp = step_inputs(wt, 0)
    ot, st = model.stage_forward(p, inp, wt)
    ou, su = model.stage_forward(pu, inp, wu)
    np.testing.assert_array_equal(ot["logits"], ou["logits"])
    gt, _ = model.stage_backward(p, inp, st, wt)
    gu, _ = model.stage_backward(pu, inp, su, wu)
    np.testing.assert_allclose(gu["embed"] + gu["head"], gt["embed"], rtol=1e-12, atol=1e-15)
    assert np.abs(gu["head"]).max() > 0 and np.abs(gu["embed"]).max() > 0


def test_tiny_workload_initial_loss_near_log_vocab():
    from datagen import TINY
    p = init_params(TINY)
    out, _ = model.stage_forward(p, step_inputs(TINY, 0), TINY)
    assert abs(float(out["loss"]) - math.log(512)) < 0.1


def test_microbatch_gradients_sum():
    w = MIDDLE
    p = _params(w)
    i0 = {"x_in": R.standard_normal((2, 5, 8)), "dy": R.standard_normal((2, 5, 8))}
    i1 = {"x_in": R.standard_normal((2, 5, 8)), "dy": R.standard_normal((2, 5, 8))}
    g, _ = model.stage_step_grads(p, [i0, i1], w)
    o0, s0 = model.stage_forward(p, i0, w)
    g0, _ = model.stage_backward(p, i0, s0, w)
    o1, s1 = model.stage_forward(p, i1, w)
    g1, _ = model.stage_backward(p, i1, s1, w)
    for k in g:
        np.testing.assert_allclose(g[k], g0[k] + g1[k], rtol=1e-13)
