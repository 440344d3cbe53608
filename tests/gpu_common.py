"""Helpers of the GPU parity tests: drive the HIP stage through the C ABI for T iterations of
Alg. 1 and record what the oracle records (losses, outputs, gradients, final state)."""
from __future__ import annotations

import sys
from typing import Dict, Iterable, List, Optional

import numpy as np

import datagen
import oracle


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def rel(a, b) -> float:
    """Norm-wise relative error ||a - b|| / max(||b||, 1e-30), in float64."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.linalg.norm((a - b).ravel()) / max(np.linalg.norm(b.ravel()), 1e-30))


def shape_of(w, muon=False, max_delay=1, adan=False):
    from paper_2606_30634_amd.stage import make_shape
    return make_shape(w.n_blocks, w.d_model, w.n_heads, w.n_kv_heads, w.head_dim, w.d_ffn, w.vocab,
                      w.first_stage, w.last_stage, w.tie_embedding, w.seq_len, w.micro_batch,
                      w.max_inflight, bf16=(w.dtype == "bf16"), rms_eps=w.rms_eps,
                      rope_theta=w.rope_theta, muon=muon, max_delay=max_delay, adan=adan)


def hp_of(w, **kw):
    from paper_2606_30634_amd.stage import hparams
    base = dict(lr=w.lr, beta1=w.beta1, beta2=w.beta2, eps=w.eps, weight_decay=w.weight_decay,
                clip_norm=w.clip_norm, ef_lambda=w.ef_lambda, delay=1)
    base.update(kw)
    return hparams(**base)


def to_device(inp: Dict[str, np.ndarray], w, dev):
    import torch
    out = {}
    for k, v in inp.items():
        if v.dtype == np.int32:
            out[k] = torch.from_numpy(v).to(dev)
        else:
            t = torch.from_numpy(np.ascontiguousarray(v, dtype=np.float32))
            out[k] = t.to(dev).to(torch.bfloat16 if w.dtype == "bf16" else torch.float32)
    return out


def schedule_1f1b(M: int, warm: int):
    """Order of (kind, microbatch) on one stage for one step of a 1F1B schedule with `warm` forwards
    ahead of the first backward (no cross-step overlap)."""
    order = []
    f = b = 0
    for _ in range(min(warm, M)):
        order.append(("F", f)); f += 1
    while b < M:
        if f < M:
            order.append(("F", f)); f += 1
        order.append(("B", b)); b += 1
    return order


def run_gpu(w, steps: int, hp, params0, grad_steps: Iterable[int] = (), y_steps: Iterable[int] = (),
            device: str = "cuda:0", upd_steps: Iterable[int] = (), muon: bool = False,
            early_update: bool = False, after_backward=None, overlap_mode: int = 1):
    """T iterations of Alg. 1 on the GPU stage.  Returns losses (per step, per microbatch), outputs
    at y_steps, and at grad_steps the gradient g_t together with the master weights x_t it was taken
    at, at upd_steps the whole optimizer state before and after delayed_update(t) with the gradient
    it consumed (and, under "u_slot", the EF buffer iteration t uses), plus the final master / m / v /
    u_prev and every EF buffer ("u_ring", buffer j = iterations j mod tau).

    early_update: the stage in overlap mode (overlap_mode 1, or 2 with the update's elementwise pass
    deferred beside the attention backwards), and delayed_update(t) issued before step t's forwards
    and backwards (it consumes g_{t-1}), so that it runs beside them.
    after_backward(t, stage): called after step t's backwards, before delayed_update(t)."""
    import torch
    from paper_2606_30634_amd.stage import Stage
    dev = torch.device(device)
    tau = max(hp.delay, 1)
    ng = tau + 1
    st = Stage(shape_of(w, muon=muon or hp.optimizer == 1, max_delay=tau, adan=hp.optimizer == 4), device)
    st.load_master(params0)
    if early_update:
        st.set_update_overlap(overlap_mode)
    names = list(params0)
    grad_steps, y_steps = set(grad_steps), set(y_steps)
    M = w.microbatches_per_step
    upd_steps = set(upd_steps)
    res = dict(losses=[], ys={}, grads={}, x_at={}, upd={})

    def ef_name(j):
        return "u_prev." if j == 0 else f"u_prev{j}."

    def grab(pre):
        return {n: st.view(pre + n).float().cpu().numpy().reshape(params0[n].shape).copy() for n in names}

    def state(g_idx=None, u_slot=None):
        if early_update and overlap_mode == 2:
            st.join_update()          # launches the deferred chunks
        torch.cuda.synchronize(dev)   # the update stream too (overlap mode)
        d = {pre: grab(pre) for pre in ("", "m.", "v.", "u_prev.")}
        if g_idx is not None:
            d["g"] = grab(f"grad{g_idx}.")
        if u_slot is not None:
            d["u_slot"] = grab(ef_name(u_slot))
        return d

    def update(t):
        if t in upd_steps:
            pre = state((t - hp.delay) % ng, t % tau)
        st.update(t, hp)
        if t in upd_steps:
            res["upd"][t] = (pre, state(None, t % tau))

    for t in range(steps):
        if t in grad_steps:   # x_t, before an early update(t) starts writing x_{t+1}
            if early_update and overlap_mode == 2:
                st.join_update()
            torch.cuda.synchronize(dev)
            res["x_at"][t] = {n: st.view(n).float().cpu().numpy().reshape(params0[n].shape).copy() for n in names}
        if early_update:
            update(t)
        inps = [to_device(datagen.step_inputs(w, t, i), w, dev) for i in range(M)]
        losses = [None] * M
        ys = [None] * M
        loss_t = [torch.zeros(1, device=dev) for _ in range(M)]
        y_t = [None] * M
        order = schedule_1f1b(M, w.max_inflight - 1) if M > 1 else [("F", 0), ("B", 0)]
        for kind, i in order:
            slot = i % w.max_inflight
            inp = inps[i]
            if kind == "F":
                if not w.last_stage:
                    y_t[i] = torch.empty_like(inp["dy"])
                st.forward(slot, t, tokens=inp.get("tokens"), x_in=inp.get("x_in"),
                           targets=inp.get("targets"), y_out=y_t[i],
                           loss=loss_t[i] if w.last_stage else None)
            else:
                st.backward(slot, dy=inp.get("dy"), microbatches_per_step=M)
        if after_backward is not None:
            after_backward(t, st)
        if t in grad_steps:
            res["grads"][t] = grab(f"grad{t % ng}.")
        for i in range(M):
            if w.last_stage:
                losses[i] = float(loss_t[i].item())
            else:
                yv = y_t[i].float().cpu().numpy().astype(np.float64)
                losses[i] = float(np.sum(yv * inps[i]["dy"].float().cpu().numpy().astype(np.float64)))
                if t in y_steps:
                    ys[i] = yv
        if t in y_steps:
            res["ys"][t] = ys
        res["losses"].append(losses)
        if not early_update:
            update(t)
    if early_update and overlap_mode == 2:
        st.join_update()
    torch.cuda.synchronize(dev)
    final = {}
    for pre in ("", "m.", "v.", "u_prev."):
        final[pre] = {n: st.view(pre + n).float().cpu().numpy().reshape(params0[n].shape) for n in names}
    final["u_ring"] = [grab(ef_name(j)) for j in range(tau)]
    res["final"] = final
    rc, skipped = __import__("paper_2606_30634_amd.binding", fromlist=["x"]).stage_poll_nonfinite(st.handle)
    res["skipped"] = skipped
    st.close()
    return res


def run_oracle_noisy(w, steps: int, hp_oracle, params0, eps=0.012, seed=7, dt=np.float64):
    """The oracle's iterations with every gradient perturbed before its update by additive noise of
    eps times its tensor's rms (xi standard normal from a generator seeded with (seed, t)): an error
    of the size and kind of bf16 accumulation, which changes the signs of a tensor's smallest
    elements.  How far this run ends from the clean one is how far the method itself carries such
    an error.  Returns the final x, m, v and EF buffer."""
    from oracle import model
    from oracle.update import OptState, iteration_update
    st = OptState.create(params0, dt)
    for t in range(steps):
        x_t = st.x if st.x_compute is None else st.x_compute
        inps = [datagen.step_inputs(w, t, i) for i in range(w.microbatches_per_step)]
        grads, _ = model.stage_step_grads(x_t, inps, w, dt)
        rng = np.random.default_rng([seed, t])
        grads = {n: a + eps * np.sqrt(np.mean(a * a)) * rng.standard_normal(a.shape) for n, a in grads.items()}
        iteration_update(st, grads, hp_oracle)
    return {"": st.x, "m.": st.m, "v.": st.v, "u_prev.": st.u_prev}


def oracle_grads_at(w, t, x_t, dt=np.float64):
    """The oracle's gradient g_t of step t's microbatches, taken at the given weights (teacher forcing)."""
    from oracle import model
    g, _ = model.stage_step_grads(x_t, [datagen.step_inputs(w, t, i) for i in range(w.microbatches_per_step)], w, dt)
    return g


def run_oracle(w, steps: int, hp_oracle, params0, grad_steps=(), y_steps=(), dt=np.float64):
    grad_steps, y_steps = set(grad_steps), set(y_steps)
    res = dict(losses=[], ys={}, grads={})

    def rec(t, info):
        res["losses"].append([float(l) for l in info["losses"]])
        res.setdefault("loss_abs", []).append([o.get("loss_abs") for o in info["outs"]])
        if t in grad_steps:
            res["grads"][t] = info["grads"]
        if t in y_steps:
            res["ys"][t] = [o.get("y") for o in info["outs"]]

    st = oracle.run(w, steps, hp_oracle, params0, lambda t, i: datagen.step_inputs(w, t, i), dt, rec)
    res["final"] = {"": st.x, "m.": st.m, "v.": st.v, "u_prev.": st.u_prev, "u_ring": st.u_ring}
    return res
