"""Writes the float64 oracle's trajectory of a bf16 workload at full size under Alg. 1 (§2) with the
Error-Feedback step of §3.2 (AdamW, delay 1, lambda 1, clip 1.0, lr 1e-3): tests/golden/small_100_steps.npz,
the small workload (3 decoder blocks, d_model 768, 12 heads, SwiGLU 3072, seq 1024 x 8, vocab-32000
embedding on a first stage) over 100 iterations, and tests/golden/mid_10_steps.npz, the mid workload
(a middle stage of 4 blocks, d_model 2048, 16 heads of 128, SwiGLU 8192, seq 2048 x 4, fed N(0, 1)
activations) over 10 iterations.

Only the oracle and the seeded input generators are used; nothing comes from the HIP path.

Stored (every array float64 unless noted):
  loss[t], loss_abs[t]        surrogate loss sum(Y dY) of step t and sum |Y dY| (its condition)
  offsets[name]               int64: start of the stored slice of each parameter (seeded)
  {x,m,v,u_prev}@k/<name>     the slice of the master weights and optimizer state x_k, m_k, v_k,
                              u_prev_k before iteration k's forward, k in STATE_AT
  g@t/<name>                  the slice of the oracle's own gradient g_t (at its own x_t), t in GRAD_AT
  norm.{dx,m,v,u_prev}@k/<name>  whole-tensor norms ||x_k - x_0||, ||m_k||, ||v_k||, ||u_prev_k||
  y@t                         rows Y_ROWS of the stage output of step t (flattened tokens), t in Y_AT

  python tests/golden/make_trajectory.py [--workload small|mid] [--checkpoint DIR]
      small: state before iterations 2, 3, 10, 50, 100; gradients and output rows of steps 0, 1,
      10, 50, 99.  mid: state before iterations 2, 3, 10; gradients and output rows of steps 0, 1, 9.

With --grad-noise EPS every gradient element g is perturbed before the update, by xi standard
normal from a generator seeded with (--noise-seed, t) at step t: multiplied by (1 + EPS xi)
(--noise-kind relative, which keeps every element's sign), or added EPS rms xi with rms the tensor's
root mean square (--noise-kind additive: the shape of an accumulated rounding error, which can flip
the sign of the tensor's smallest elements).  It is the same method with a perturbation of the size
of bf16 arithmetic, whose trajectory shows how far such perturbations alone carry two runs apart
(--out names its file).
"""
from __future__ import annotations

import argparse
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import datagen  # noqa: E402
import oracle  # noqa: E402
from oracle import model  # noqa: E402
from oracle.update import OptState, iteration_update  # noqa: E402

SLICE = 512
SLICE_SEED = 20250611
Y_ROWS = (0, 1, 1023, 1024, 4095, 8191)
HERE = os.path.dirname(os.path.abspath(__file__))
# per workload: iterations, state / gradient / output points, output file
PLANS = {
    "small": dict(steps=100, state_at=(2, 3, 10, 50, 100), grad_at=(0, 1, 10, 50, 99), y_at=(0, 1, 10, 50, 99),
                  out=os.path.join(HERE, "small_100_steps.npz")),
    "mid": dict(steps=10, state_at=(2, 3, 10), grad_at=(0, 1, 9), y_at=(0, 1, 9),
                out=os.path.join(HERE, "mid_10_steps.npz")),
}


def slice_offsets(params):
    rng = np.random.default_rng(SLICE_SEED)
    return {n: int(rng.integers(0, v.size - SLICE + 1)) for n, v in params.items()}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="small", choices=sorted(PLANS))
    ap.add_argument("--steps", type=int, default=0)
    ap.add_argument("--checkpoint", default="")
    ap.add_argument("--out", default="")
    ap.add_argument("--grad-noise", type=float, default=0.0)
    ap.add_argument("--noise-seed", type=int, default=0)
    ap.add_argument("--noise-kind", default="relative", choices=("relative", "additive"))
    args = ap.parse_args()
    plan = PLANS[args.workload]
    args.steps = args.steps or plan["steps"]
    args.out = args.out or plan["out"]
    STATE_AT, GRAD_AT, Y_AT = plan["state_at"], plan["grad_at"], plan["y_at"]
    w = datagen.WORKLOADS[args.workload]
    p0 = datagen.init_params(w)
    offs = slice_offsets(p0)
    hp = oracle.hparams_of(w)
    st = OptState.create(p0, np.float64)
    rec = {"loss": np.zeros(args.steps), "loss_abs": np.zeros(args.steps)}
    for n, o in offs.items():
        rec[f"offsets/{n}"] = np.array(o, dtype=np.int64)
    x0 = {n: v.astype(np.float64) for n, v in p0.items()}
    t0 = 0
    ck = os.path.join(args.checkpoint, f"{args.workload}_ckpt.npz") if args.checkpoint else ""
    if ck and os.path.exists(ck):
        z = np.load(ck)
        t0 = int(z["t"])
        for pre, d in (("x", st.x), ("m", st.m), ("v", st.v), ("u_prev", st.u_prev)):
            for n in d:
                d[n] = z[f"{pre}/{n}"].copy()
        st.pending = {n: z[f"pending/{n}"].copy() for n in st.x}
        st.n_updates, st.t = int(z["n_updates"]), t0
        for k in z.files:
            if k.startswith("rec/"):
                rec[k[4:]] = z[k].copy()
        print(f"resumed at t = {t0}", flush=True)

    def save_state(k):
        for pre, d in (("x", st.x), ("m", st.m), ("v", st.v), ("u_prev", st.u_prev)):
            for n, a in d.items():
                rec[f"{pre}@{k}/{n}"] = a.ravel()[offs[n]:offs[n] + SLICE].copy()
        for n in st.x:
            rec[f"norm.dx@{k}/{n}"] = np.array(np.linalg.norm((st.x[n] - x0[n]).ravel()))
            rec[f"norm.m@{k}/{n}"] = np.array(np.linalg.norm(st.m[n].ravel()))
            rec[f"norm.v@{k}/{n}"] = np.array(np.linalg.norm(st.v[n].ravel()))
            rec[f"norm.u_prev@{k}/{n}"] = np.array(np.linalg.norm(st.u_prev[n].ravel()))

    for t in range(t0, args.steps):
        tic = time.time()
        if t in STATE_AT:
            save_state(t)
        inp = datagen.step_inputs(w, t, 0)
        grads, outs = model.stage_step_grads(st.x, [inp], w, np.float64)
        if args.grad_noise > 0:
            noise = np.random.default_rng([args.noise_seed, t])
            if args.noise_kind == "relative":
                grads = {n: a * (1.0 + args.grad_noise * noise.standard_normal(a.shape)) for n, a in grads.items()}
            else:
                grads = {n: a + args.grad_noise * np.sqrt(np.mean(a * a)) * noise.standard_normal(a.shape)
                         for n, a in grads.items()}
        rec["loss"][t] = outs[0]["loss"]
        rec["loss_abs"][t] = outs[0]["loss_abs"]
        if t in GRAD_AT:
            for n, a in grads.items():
                rec[f"g@{t}/{n}"] = a.ravel()[offs[n]:offs[n] + SLICE].copy()
        if t in Y_AT:
            rec[f"y@{t}"] = outs[0]["y"].reshape(-1, w.d_model)[list(Y_ROWS)].copy()
        iteration_update(st, grads, hp)
        print(f"t = {t}: loss {rec['loss'][t]:.6e}, {time.time() - tic:.1f} s", flush=True)
        if ck and (t + 1) % 5 == 0:
            tmp = {f"{pre}/{n}": a for pre, d in (("x", st.x), ("m", st.m), ("v", st.v),
                                                    ("u_prev", st.u_prev), ("pending", st.pending))
                   for n, a in d.items()}
            tmp.update({f"rec/{k}": v for k, v in rec.items()})
            np.savez(ck + ".tmp.npz", t=t + 1, n_updates=st.n_updates, **tmp)
            os.replace(ck + ".tmp.npz", ck)
    if args.steps in STATE_AT:
        save_state(args.steps)
    store = {k: (v.astype(np.float32) if v.ndim and k.split("@")[0] in ("x", "m", "v", "u_prev", "g", "y")
                 else v) for k, v in rec.items()}
    np.savez_compressed(args.out, **store)
    print(f"wrote {args.out}: {len(store)} arrays", flush=True)


if __name__ == "__main__":
    main()
