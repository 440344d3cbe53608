"""GPU parity at the workloads' full sizes against stored float64 oracle values (tests/golden/,
written by the scripts beside them, which call only the oracle and the seeded input generators).

* one-block stages at the full width of the mid workload (d_model 2048, heads of 128, SwiGLU 8192,
  seq 2048 x 4) and of the large one (d_model 4096, 32 query / 8 key-value heads, SwiGLU 14336,
  seq 4096 x 2, eight microbatches per step in a 1F1B order with 4 activation slots): step 0's
  output rows, the gradient handed upstream (dx_out) of every microbatch, the step's parameter
  gradient (seeded slices and whole-tensor norms), then the delayed updates of iterations 1 and 2
  (Error Feedback active at 2) in place on slices of the flat vector;
* the small workload (3 blocks, d_model 768, seq 1024 x 8, vocab-32000 embedding) free-running for
  100 iterations of Alg. 1 with Error Feedback against the stored float64 trajectory (every step's
  surrogate loss; outputs and gradients at x_0; weights and state norms through step 10; moments
  through step 3); at every later point (and for the EF buffer from step 2), the median error of
  each quantity within 1.5 times that of the same oracle run whose gradients carry noise of bf16
  size; then iteration 100 teacher-forced: the oracle's gradient at the GPU's weights and its
  update from the GPU's state;
* the mid workload (a middle stage of 4 blocks, d_model 2048) free-running for 10 iterations, with
  the same bars.
Tolerance: 2e-2 norm-wise relative (the bf16 bar), except where a comparison says otherwise."""
import json
import os

import numpy as np
import pytest

import datagen
from gpu_common import hp_of, log, rel, schedule_1f1b, shape_of, to_device
from test_gpu_fullsize import _update_in_place

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
TOL = 2e-2


def _load(name):
    path = os.path.join(GOLDEN, name)
    if not os.path.exists(path):
        pytest.skip(f"{name} not generated (tests/golden/make_*.py)")
    return np.load(path)


def _report(label, errs, tols):
    over = {k: e for k, e in errs.items() if not e <= tols.get(k, TOL)}
    worst = sorted(errs, key=lambda k: errs[k] / tols.get(k, TOL), reverse=True)[:8]
    log(f"{label}: {len(errs)} comparisons; worst " + ", ".join(f"{k}={errs[k]:.2e}" for k in worst))
    assert not over, f"{label}: {len(over)} over tolerance: " + ", ".join(
        f"{k}={e:.2e}" for k, e in sorted(over.items(), key=lambda kv: -kv[1])[:12])


@pytest.mark.parametrize("wname", ["mid", "large"])
def test_one_block_full_width_step(wname):
    import torch
    from paper_2606_30634_amd.stage import Stage
    z = _load(f"{wname}_1block_step0.npz")
    w = datagen.WORKLOADS[wname].with_(n_blocks=1)
    dev = torch.device("cuda:0")
    M = w.microbatches_per_step
    log(f"golden {wname}: one block at full width, {M} microbatch(es), slots {w.max_inflight}")
    st = Stage(shape_of(w), "cuda:0")
    p0 = datagen.init_params(w)
    st.load_master(p0)
    inps = [to_device(datagen.step_inputs(w, 0, i), w, dev) for i in range(M)]
    ys = [torch.empty_like(inps[i]["dy"]) for i in range(M)]
    dxs = [torch.empty_like(inps[i]["x_in"]) for i in range(M)]
    order = schedule_1f1b(M, w.max_inflight - 1) if M > 1 else [("F", 0), ("B", 0)]
    for kind, i in order:
        if kind == "F":
            st.forward(i % w.max_inflight, 0, x_in=inps[i]["x_in"], y_out=ys[i])
        else:
            st.backward(i % w.max_inflight, dy=inps[i]["dy"], dx_out=dxs[i], microbatches_per_step=M)
    torch.cuda.synchronize()
    T = w.micro_batch * w.seq_len
    errs = {}
    for i in range(M):
        rows = [r for r in (0, 1, 2047, 2048, 4095, 4096, 8191) if r < T]
        y = ys[i].float().reshape(T, w.d_model)
        dx = dxs[i].float().reshape(T, w.d_model)
        errs[f"y[{i}].rows"] = rel(y[rows].cpu().numpy(), z[f"y/{i}"])
        errs[f"y[{i}].norm"] = abs(float(y.double().norm()) - float(z[f"ynorm/{i}"])) / float(z[f"ynorm/{i}"])
        errs[f"dx[{i}].rows"] = rel(dx[rows].cpu().numpy(), z[f"dx/{i}"])
        errs[f"dx[{i}].norm"] = abs(float(dx.double().norm()) - float(z[f"dxnorm/{i}"])) / float(z[f"dxnorm/{i}"])
    for n in p0:
        g = st.view(f"grad0.{n}").double()
        offs = z[f"offsets/{n}"]
        sl = np.stack([g[int(o):int(o) + z[f"g/{n}"].shape[1]].cpu().numpy() for o in offs])
        errs[f"g.{n}.slices"] = rel(sl, z[f"g/{n}"])
        errs[f"g.{n}.norm"] = abs(float(g.norm()) - float(z[f"gnorm/{n}"])) / float(z[f"gnorm/{n}"])
    _report(f"golden {wname} step 0", errs, {})
    # iterations 1 (the first update, consuming g_0) and 2 (Error Feedback) in place on 16 slices
    st.update(0, hp_of(w))
    n = st.tensors["flat.master"][1]
    rng = np.random.default_rng(5)
    sample = [(int(a) // 64 * 64, 65536) for a in rng.integers(0, n - 65536, size=16)]
    for t in (1, 2):
        inps = [to_device(datagen.step_inputs(w, t, i), w, dev) for i in range(M)]
        for kind, i in order:
            if kind == "F":
                st.forward(i % w.max_inflight, t, x_in=inps[i]["x_in"], y_out=ys[i])
            else:
                st.backward(i % w.max_inflight, dy=inps[i]["dy"], microbatches_per_step=M)
        e = _update_in_place(st, w, hp_of(w), t, sample)
        log(f"golden {wname}: update {t} in place on 16 slices, worst rel {e:.3e}")
        assert e < 1e-5
    st.close()


def _slice(st, key, n, off, cnt):
    return st.view(key + n)[off:off + cnt].double().cpu().numpy()


# Free-running comparison points of the small workload.  Steps 0 and 1 both run at x_0 (the first
# update, at t = 1, consumes g_0), so their outputs and gradients differ from the oracle's by the
# bf16 arithmetic alone.  From t = 1 on, each Adam update turns the gradient's bf16 error into sign
# flips of m/sqrt(v) in its smallest elements (about 1.2 % norm-wise gradient error moves ~10 % of the
# first update's norm), and the trajectories separate at a rate the method itself sets, about doubling
# every 8 steps.  So the free-running 2e-2 bar applies where it is well-posed: the loss of every
# step, the weights and the whole-tensor norms of the state through step 10, the moments through
# step 3.  Later iterations are compared teacher-forced, one oracle iteration from the GPU's own
# state: the gradient at step 50 to 2e-2; at step 100 this run's gradient has grown about 30-fold
# and a few positions carry most of it, so that rounding the weights alone to bf16 moves the exact
# gradient by more than 2e-2 there, and the bar is 2e-2 plus twice that measured move (the GPU
# computes with bf16 weight copies by design); the update of step 100 from the GPU's state to 1e-5.
FREE_STATE_AT = (2, 3, 10)
FREE_MOMENT_AT = (2, 3)
FREE_GRAD_AT = (0, 1)
# v is quadratic in the gradient: a gradient within 2e-2 gives v within about 4e-2
V_TOL = 2 * TOL
# Beyond the window, the free-running values are held against the method's own sensitivity: the
# float64 oracle run of the same iterations with every gradient element perturbed by 1.2 % of its
# tensor's rms (make_trajectory.py --grad-noise 0.012 --noise-kind additive, an error of the size
# and kind of bf16 accumulation: the smallest elements change sign) separates from the clean run by
# the medians in <workload>_<steps>_noise_profile.json; the GPU's median error at each point may not
# exceed that by more than this factor.
NOISE_ENVELOPE = 1.5


def _trajectory(w, z, label, at_step=None):
    """Runs the stage free for len(z["loss"]) iterations on the workload's inputs, comparing with the
    stored trajectory z: returns the stage (after its last update), the comparisons held to the bar
    (errs, with their tolerances in tols) and those beyond the 2e-2 window (diag), which the caller
    holds against the noise-perturbed oracle run.  at_step(t, st, y, inp_h)
    runs after step t's backward, before its update."""
    import torch
    from paper_2606_30634_amd.stage import Stage
    dev = torch.device("cuda:0")
    p0 = datagen.init_params(w)
    names = list(p0)
    offs = {n: int(z[f"offsets/{n}"]) for n in names}
    cnt = 512
    steps = len(z["loss"])
    state_pts = sorted(int(k.split("@")[1].split("/")[0]) for k in z.files
                       if k.startswith("norm.dx@") and k.split("/", 1)[1] == names[0])
    grad_pts = sorted(int(k.split("@")[1]) for k in z.files if k.startswith("y@"))
    x0 = {n: torch.from_numpy(p0[n].reshape(-1)).double() for n in names}
    st = Stage(shape_of(w), "cuda:0")
    st.load_master(p0)
    hp = hp_of(w)
    errs, diag = {}, {}
    y = torch.empty(w.micro_batch, w.seq_len, w.d_model, dtype=torch.bfloat16, device=dev)
    rows = [0, 1, 1023, 1024, 4095, 8191]
    log(f"golden {label}: {steps} free-running iterations")

    def state_at(k):
        # held to the bar: weights and whole-tensor norms through step 10, m and v slices through
        # step 3; the rest is reported
        torch.cuda.synchronize()
        free = k in FREE_STATE_AT
        for n in names:
            x = st.view(n).double()
            (errs if free else diag)[f"x@{k}.{n}"] = rel(x[offs[n]:offs[n] + cnt].cpu().numpy(), z[f"x@{k}/{n}"])
            ref = float(z[f"norm.dx@{k}/{n}"])
            if ref > 0:
                (errs if free else diag)[f"|dx|@{k}.{n}"] = abs(float((x.cpu() - x0[n]).norm()) - ref) / ref
            for pre in ("m", "v", "u_prev"):
                full = st.view(f"{pre}.{n}").double()
                ref_n = float(z[f"norm.{pre}@{k}/{n}"])
                if ref_n == 0:
                    continue
                (errs if free else diag)[f"|{pre}|@{k}.{n}"] = abs(float(full.norm()) - ref_n) / ref_n
                e = rel(full[offs[n]:offs[n] + cnt].cpu().numpy(), z[f"{pre}@{k}/{n}"])
                (errs if pre != "u_prev" and k in FREE_MOMENT_AT else diag)[f"{pre}@{k}.{n}"] = e

    for t in range(steps):
        if t in state_pts:
            state_at(t)
        inp_h = datagen.step_inputs(w, t, 0)
        inp = to_device(inp_h, w, dev)
        if w.first_stage:
            st.forward(0, t, tokens=inp["tokens"], y_out=y)
        else:
            st.forward(0, t, x_in=inp["x_in"], y_out=y)
        st.backward(0, dy=inp["dy"])
        if at_step is not None:
            at_step(t, st, y, inp_h)
        if t in grad_pts:
            torch.cuda.synchronize()
            out = errs if t in FREE_GRAD_AT else diag
            for n in names:
                g = st.view(f"grad{t % 2}.{n}").double()[offs[n]:offs[n] + cnt].cpu().numpy()
                if np.linalg.norm(z[f"g@{t}/{n}"]) > 0:
                    out[f"g@{t}.{n}"] = rel(g, z[f"g@{t}/{n}"])
            yr = y.float().reshape(-1, w.d_model)[rows].cpu().numpy()
            out[f"y@{t}"] = rel(yr, z[f"y@{t}"])
        loss = float((y.double() * inp["dy"].double()).sum())
        errs[f"loss@{t}"] = abs(loss - float(z["loss"][t])) / float(z["loss_abs"][t])
        st.update(t, hp)
    if steps in state_pts:
        state_at(steps)
    tols = {key: V_TOL for key in errs if key.startswith(("v@", "|v|@"))}
    for k in sorted({int(key.split("@")[1].split(".")[0]) for key in diag}):
        ks = {key: e for key, e in diag.items() if int(key.split("@")[1].split(".")[0]) == k}
        log(f"  free-running step {k} (beyond the 2e-2 window): {len(ks)} values, median "
            f"{float(np.median(list(ks.values()))):.2e}, max {max(ks.values()):.2e}")
    return st, y, errs, tols, diag


def _noise_envelope(diag, errs, profile, label):
    """The median over the parameters of each free-running point's errors (diag: keys
    "<quantity>@<step>.<parameter>") against NOISE_ENVELOPE times the median of the noise-perturbed
    oracle run at the same point.  The perturbed run's outputs carry no rounding of their own (its
    gradients carry the injected noise, its forward is exact), so an output's error is first reduced
    by the GPU's output error where both run at x_0 (errs "y@0", "y@1": the forward's bf16
    arithmetic alone)."""
    with open(os.path.join(GOLDEN, profile)) as f:
        ref = json.load(f)["additive"]
    y_floor = max(errs.get("y@0", 0.0), errs.get("y@1", 0.0))
    groups = {}
    for key, e in diag.items():
        groups.setdefault(key.split(".", 1)[0], []).append(e)
    ratios = {}
    for point, es in sorted(groups.items()):
        if point not in ref or ref[point]["median"] <= 0:
            continue
        own = y_floor if point.startswith("y@") else 0.0
        ratios[point] = (float(np.median(es)) - own) / ref[point]["median"]
    assert ratios, "no free-running point to compare"
    log(f"{label}, free-running median error / noise-perturbed oracle's (outputs less their step-0 "
        f"error {y_floor:.2e}): " + ", ".join(f"{p}={r:.2f}" for p, r in ratios.items()))
    over = {p: r for p, r in ratios.items() if not r <= NOISE_ENVELOPE}
    assert not over, f"free-running error above {NOISE_ENVELOPE}x the noise-perturbed oracle's: {over}"


@pytest.mark.timeout(900)
def test_small_workload_100_steps():
    import torch
    from oracle import model
    z = _load("small_100_steps.npz")
    w = datagen.SMALL
    dev = torch.device("cuda:0")
    p0 = datagen.init_params(w)
    names = list(p0)
    steps = len(z["loss"])
    tf_errs = {}

    def teacher_forced(st, y, t, inp_h, sensitivity):
        # the oracle's gradient at the GPU's own weights x_t (float64, from the fp32 master); with
        # `sensitivity`, also at the weights rounded to bf16, whose distance from the first is the
        # bf16 move the bar allows for
        torch.cuda.synchronize()
        xt = {n: st.view(n).double().cpu().numpy().reshape(p0[n].shape) for n in names}
        log(f"golden small: oracle gradient at the GPU's weights of step {t} (float64)")
        ref, outs = model.stage_step_grads(xt, [inp_h], w, np.float64)
        e = {f"y@{t}": rel(y.float().cpu().numpy(), outs[0]["y"])}
        bars = {}
        if sensitivity:
            xb = {n: datagen.bf16_values(a.astype(np.float32)).astype(np.float64) for n, a in xt.items()}
            refb, _ = model.stage_step_grads(xb, [inp_h], w, np.float64)
        for n in names:
            g = st.view(f"grad{t % 2}.{n}").double().cpu().numpy().reshape(p0[n].shape)
            e[f"g@{t}.{n}"] = rel(g, ref[n])
            if sensitivity:
                move = rel(refb[n], ref[n])
                bars[f"g@{t}.{n}"] = TOL + 2 * move
                log(f"  {n}: GPU {e[f'g@{t}.{n}']:.2e}, bf16-weight move of the exact gradient {move:.2e}")
        return e, bars

    def at_step(t, st, y, inp_h):
        if t == 50:
            e, _ = teacher_forced(st, y, t, inp_h, False)
            tf_errs.update({f"teacher-forced {k}": v for k, v in e.items()})

    st, y, errs, tols, diag = _trajectory(w, z, "small", at_step)
    errs.update(tf_errs)
    _report(f"golden small {steps} free-running steps", errs, tols)
    _noise_envelope(diag, errs, "small_100_noise_profile.json", "golden small")

    # iteration `steps` teacher-forced: the gradient against the bar above, then the update
    t = steps
    inp_h = datagen.step_inputs(w, t, 0)
    inp = to_device(inp_h, w, dev)
    st.forward(0, t, tokens=inp["tokens"], y_out=y)
    st.backward(0, dy=inp["dy"])
    tf, bars = teacher_forced(st, y, t, inp_h, True)
    _report(f"golden small teacher-forced gradient {t}", tf, bars)
    rng = np.random.default_rng(11)
    nflat = st.tensors["flat.master"][1]
    sample = [(int(a) // 64 * 64, 65536) for a in rng.integers(0, nflat - 65536, size=16)]
    e = _update_in_place(st, w, hp_of(w), t, sample)
    log(f"golden small: teacher-forced update {t} on 16 slices, worst rel {e:.3e}")
    assert e < 1e-5
    st.close()


@pytest.mark.timeout(600)
def test_mid_workload_10_steps():
    # the mid workload at full size (a middle stage: d_model 2048, heads of 128, SwiGLU 8192, seq
    # 2048 x 4) free-running over 10 iterations, within the window where the bf16 bar is well-posed
    z = _load("mid_10_steps.npz")
    st, _, errs, tols, diag = _trajectory(datagen.MID, z, "mid")
    st.close()
    _report(f"golden mid {len(z['loss'])} free-running steps", errs, tols)
    _noise_envelope(diag, errs, "mid_10_noise_profile.json", "golden mid")
