"""GPU checks of the stage's run state, through the C ABI:

* a non-finite gradient (an infinity written into one element of a gradient buffer before the
  update that consumes it) is skipped on the device exactly as the oracle reads it: x, m, v and the
  EF buffers untouched, the compute copy written from x_t, the skip counted (stage_poll_nonfinite),
  the bias-correction index still advancing; the whole trajectory against the oracle run with the
  same gradient, with clipping on and off, AdamW and Muon, delay 1 and 2, fp32 and bf16;
* resume: a run of 10 iterations against 5 + a copy of the state into a fresh stage
  (stage_resume) + 5, bit for bit;
* determinism: the same steps run twice on two stages give bit-identical outputs, gradients and
  weights (no float atomics anywhere on the path);
* dx_out, the gradient a non-first stage hands upstream, against the oracle's gradient of the
  stage input at the same weights (every microbatch of a 1F1B step).
Tolerances: fp32 workload 1e-4, bf16 workloads 2e-2 (norm-wise relative)."""
import numpy as np
import pytest

import datagen
import oracle
from gpu_common import hp_of, log, rel, run_gpu, schedule_1f1b, shape_of, to_device
from oracle import model
from oracle.update import OptState, iteration_update
from test_gpu_stage import LARGE_R, MID_R, SMALL_R, TINY_LAST

pytestmark = pytest.mark.gpu

BAD_ELEM = ("blk0.wq", 7)


def _oracle_with_bad(w, steps, hpo, p0, bad_step):
    """The oracle's run with g_bad_step's element BAD_ELEM set to +inf."""
    st = OptState.create(p0, np.float64)
    losses, loss_abs, skipped = [], [], 0
    for t in range(steps):
        inps = [datagen.step_inputs(w, t, i) for i in range(w.microbatches_per_step)]
        g, outs = model.stage_step_grads(st.x, inps, w, np.float64)
        if t == bad_step:
            g[BAD_ELEM[0]].reshape(-1)[BAD_ELEM[1]] = np.inf
        info = iteration_update(st, g, hpo)
        skipped += int(info["skipped"])
        losses.append([o["loss"] for o in outs])
        loss_abs.append([o.get("loss_abs") for o in outs])
    return st, losses, loss_abs, skipped


NONFINITE = {
    "tiny-adamw-ef": (datagen.TINY, dict(ef_lambda=1.0), 1e-4),
    "tiny-adamw-noclip": (datagen.TINY, dict(ef_lambda=1.0, clip_norm=0.0), 1e-4),
    "tiny-muon-ef": (datagen.TINY, dict(ef_lambda=1.0, optimizer="muon", momentum=0.95, update_rms=0.2,
                                        ns_steps=5), 1e-4),
    "tiny-delay2": (datagen.TINY, dict(ef_lambda=2.0, delay=2), 1e-4),
    "small-reduced-bf16": (SMALL_R, dict(ef_lambda=1.0), 2e-2),
}


@pytest.mark.parametrize("case", sorted(NONFINITE))
def test_nonfinite_gradient_skipped(case):
    import torch
    w, kw, tol = NONFINITE[case]
    steps, bad = 8, 2
    tau = kw.get("delay", 1)
    p0 = datagen.init_params(w)
    hp = hp_of(w, **kw)
    hpo = oracle.hparams_of(w, **kw)
    muon = kw.get("optimizer") == "muon"
    consume = bad + tau
    copy_ok = []

    def inject(t, st):
        torch.cuda.synchronize()
        if t == bad:   # the gradient of step `bad`, before the update that consumes it
            st.view(f"grad{bad % (tau + 1)}.{BAD_ELEM[0]}")[BAD_ELEM[1]] = float("inf")
            torch.cuda.synchronize()
        if t == consume + 1:   # step consume + 1 ran at the compute copy the skipped update wrote
            v = (consume + 1) % 2
            copy_ok.append(torch.equal(st.view(f"flat.w{v}"), st.view("flat.master").to(st.view(f"flat.w{v}").dtype)))

    log(f"non-finite {case}: {steps} steps, inf in g_{bad} (consumed at iteration {consume})")
    g = run_gpu(w, steps, hp, p0, upd_steps=(consume,), muon=muon, after_backward=inject)
    assert g["skipped"] == 1, g["skipped"]
    assert copy_ok == [True], "compute copy after the skipped update is not x_t"
    pre, post = g["upd"][consume]
    for key in ("", "m.", "v.", "u_prev.", "u_slot"):
        for n in pre.get(key, {}):
            assert np.array_equal(pre[key][n], post[key][n]), f"{key}{n} changed by the skipped update"
    st_o, losses_o, loss_abs_o, skipped_o = _oracle_with_bad(w, steps, hpo, p0, bad)
    assert skipped_o == 1
    errs = {}
    for t in range(steps):
        for i, (a, b) in enumerate(zip(g["losses"][t], losses_o[t])):
            scale = abs(b) if w.last_stage else loss_abs_o[t][i]
            errs[f"loss[{t}][{i}]"] = abs(a - b) / max(scale, 1e-30)
    for pre_k, ref in (("", st_o.x), ("m.", st_o.m), ("v.", st_o.v)):
        for n in ref:
            errs[f"final.{pre_k}{n}"] = rel(g["final"][pre_k][n], ref[n])
    state_tol = tol if w.dtype == "f32" else 5e-2   # free-running bf16 m, v (as the reduced stages)
    over = {k: e for k, e in errs.items()
            if not e <= (state_tol if k.startswith(("final.m.", "final.v.")) else tol)}
    worst = sorted(errs, key=errs.get, reverse=True)[:5]
    log(f"non-finite {case}: worst " + ", ".join(f"{k}={errs[k]:.2e}" for k in worst))
    assert not over, over


def _flat_state(st, delay):
    import torch
    torch.cuda.synchronize()
    keys = ["flat.master", "flat.m", "flat.v", "flat.u_prev"] + [f"flat.u_prev{j}" for j in range(1, delay)]
    keys += [f"flat.grad{j}" for j in range(delay + 1)]
    return {k: st.view(k).clone() for k in keys}


def _iterate(st, w, t0, t1, hp, dev):
    M = w.microbatches_per_step
    for t in range(t0, t1):
        inps = [to_device(datagen.step_inputs(w, t, i), w, dev) for i in range(M)]
        order = schedule_1f1b(M, w.max_inflight - 1) if M > 1 else [("F", 0), ("B", 0)]
        loss = __import__("torch").zeros(1, device=dev)
        for kind, i in order:
            if kind == "F":
                st.forward(i % w.max_inflight, t, tokens=inps[i].get("tokens"), x_in=inps[i].get("x_in"),
                           targets=inps[i].get("targets"), loss=loss if w.last_stage else None)
            else:
                st.backward(i % w.max_inflight, dy=inps[i].get("dy"), microbatches_per_step=M)
        st.update(t, hp)


RESUME = {"tiny-ef": (datagen.TINY, dict(ef_lambda=1.0)),
          "tiny-delay2": (datagen.TINY, dict(ef_lambda=2.0, delay=2)),
          "small-reduced-bf16": (SMALL_R, dict(ef_lambda=1.0)),
          "large-reduced-1f1b": (LARGE_R, dict(ef_lambda=1.0))}


@pytest.mark.parametrize("case", sorted(RESUME))
def test_resume_bit_identical(case):
    import torch
    from paper_2606_30634_amd.stage import Stage
    w, kw = RESUME[case]
    tau = kw.get("delay", 1)
    dev = torch.device("cuda:0")
    hp = hp_of(w, **kw)
    p0 = datagen.init_params(w)
    log(f"resume {case}: 10 iterations straight")
    a = Stage(shape_of(w, max_delay=tau), "cuda:0")
    a.load_master(p0)
    _iterate(a, w, 0, 10, hp, dev)
    full = _flat_state(a, tau)
    a.close()
    log(f"resume {case}: 5 iterations, state copied into a fresh stage, 5 more")
    b = Stage(shape_of(w, max_delay=tau), "cuda:0")
    b.load_master(p0)
    _iterate(b, w, 0, 5, hp, dev)
    saved = _flat_state(b, tau)
    b.close()
    c = Stage(shape_of(w, max_delay=tau), "cuda:0")
    for k, v in saved.items():
        c.view(k).copy_(v)
    c.resume(5, tau)
    _iterate(c, w, 5, 10, hp, dev)
    res = _flat_state(c, tau)
    c.close()
    for k in ("flat.master", "flat.m", "flat.v", "flat.u_prev"):
        assert torch.equal(res[k], full[k]), f"{k} differs after resume"
    # the pending gradient of step 9 too (it lives in buffer 9 mod (tau + 1))
    j = 9 % (tau + 1)
    assert torch.equal(res[f"flat.grad{j}"], full[f"flat.grad{j}"])


@pytest.mark.parametrize("wname", ["small", "large-reduced"])
def test_run_twice_bit_identical(wname):
    """The full small workload's step (and a GQA 1F1B stage): two stages, same inputs, bit-identical
    outputs, gradients and updated weights."""
    import torch
    from paper_2606_30634_amd.stage import Stage
    w = datagen.SMALL if wname == "small" else LARGE_R
    dev = torch.device("cuda:0")
    hp = hp_of(w)
    p0 = datagen.init_params(w)
    runs = []
    for r in range(2):
        log(f"determinism {wname}: run {r}")
        st = Stage(shape_of(w), "cuda:0")
        st.load_master(p0)
        M = w.microbatches_per_step
        ys = []
        for t in range(3):
            inps = [to_device(datagen.step_inputs(w, t, i), w, dev) for i in range(M)]
            order = schedule_1f1b(M, w.max_inflight - 1) if M > 1 else [("F", 0), ("B", 0)]
            for kind, i in order:
                if kind == "F":
                    y = torch.empty_like(inps[i]["dy"])
                    st.forward(i % w.max_inflight, t, tokens=inps[i].get("tokens"), x_in=inps[i].get("x_in"), y_out=y)
                    ys.append(y)
                else:
                    st.backward(i % w.max_inflight, dy=inps[i]["dy"], microbatches_per_step=M)
            st.update(t, hp)
        st_ = _flat_state(st, 1)
        runs.append((ys, st_))
        st.close()
    (ya, sa), (yb, sb) = runs
    assert all(torch.equal(a, b) for a, b in zip(ya, yb)), "outputs differ between runs"
    for k in sa:
        assert torch.equal(sa[k], sb[k]), f"{k} differs between runs"


@pytest.mark.parametrize("w", [MID_R, LARGE_R, TINY_LAST], ids=lambda w: w.name)
def test_dx_out_against_oracle(w):
    """dx_out of every microbatch of one step (a 1F1B step on the GQA stage) against the oracle's
    gradient of the stage input at the same weights x_0 (a last stage: of its mean cross-entropy
    divided by the microbatches per step)."""
    import torch
    from paper_2606_30634_amd.stage import Stage
    dev = torch.device("cuda:0")
    p0 = datagen.init_params(w)
    st = Stage(shape_of(w), "cuda:0")
    st.load_master(p0)
    M = w.microbatches_per_step
    inps_h = [datagen.step_inputs(w, 0, i) for i in range(M)]
    inps = [to_device(x, w, dev) for x in inps_h]
    order = schedule_1f1b(M, w.max_inflight - 1) if M > 1 else [("F", 0), ("B", 0)]
    dxs = [torch.empty_like(inps[i]["x_in"]) for i in range(M)]
    loss = torch.zeros(1, device=dev)
    for kind, i in order:
        if kind == "F":
            st.forward(i % w.max_inflight, 0, x_in=inps[i]["x_in"], targets=inps[i].get("targets"),
                       loss=loss if w.last_stage else None)
        else:
            st.backward(i % w.max_inflight, dy=inps[i].get("dy"), dx_out=dxs[i], microbatches_per_step=M)
    torch.cuda.synchronize()
    tol = 1e-4 if w.dtype == "f32" else 2e-2
    errs = {}
    for i in range(M):
        _, sv = model.stage_forward(p0, inps_h[i], w, np.float64)
        _, dx_ref = model.stage_backward(p0, inps_h[i], sv, w, np.float64, loss_scale=1.0 / M)
        errs[f"dx[{i}]"] = rel(dxs[i].float().cpu().numpy().reshape(dx_ref.shape), dx_ref)
    st.close()
    log(f"dx_out {w.name}: " + ", ".join(f"{k}={v:.2e}" for k, v in errs.items()))
    assert max(errs.values()) <= tol, errs
