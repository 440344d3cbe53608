"""GPU parity of delayed Muon with Error Feedback (Alg. 2 of §4) against the oracle, through the C
ABI: the update in place (the oracle's rule on the GPU's own state and gradient before
delayed_update(t), against the GPU's state after it) and free-running trajectories.  Muon runs on
the blocks' weight matrices, AdamW on the embedding and the gains.  Tolerances: fp32 workload 1e-4;
bf16 workloads 2e-2 on the Muon update and on losses (Newton-Schulz keeps its iterate in fp32, or
as a hi + lo pair of bf16 matrices on shapes of whole tiles, and takes bf16 Gram products: a bf16
emulation of either scheme on these workloads' momenta stays under 1e-2 of float64 Newton-Schulz,
where rounding the iterate itself to bf16 gives up to 8e-2); 1e-5 on the momentum and on the AdamW
parameters (fp32 arithmetic against float64).  The reduced workloads have whole-tile matrix shapes
(the carried pair); the mixed one adds an FFN width of 320, whose [256, 320] matrices take the fp32
iterate; the small workload's update is also checked in place at full size."""
import numpy as np
import pytest

import datagen
import oracle
from gpu_common import hp_of, log, rel, run_gpu, run_oracle
from oracle.update import OptState, is_muon_matrix, iteration_update
from test_gpu_stage import MID_R, LARGE_R, SMALL_R, TILED_R

pytestmark = pytest.mark.gpu

# one group of whole-tile shapes ([256, 256]) and one of the others ([256, 320])
MIXED_R = SMALL_R.with_(name="small-mixed-muon", d_ffn=320)

MUON = dict(optimizer="muon", momentum=0.95, update_rms=0.2, ns_steps=5)


def _update_in_place(w, g, lam, tol):
    errs, tols = {}, {}
    for t, (pre, post) in g["upd"].items():
        ost = OptState({n: v.astype(np.float64) for n, v in pre[""].items()},
                       {n: v.astype(np.float64) for n, v in pre["m."].items()},
                       {n: v.astype(np.float64) for n, v in pre["v."].items()},
                       {n: v.astype(np.float64) for n, v in pre["u_prev."].items()},
                       pending={n: v.astype(np.float64) for n, v in pre["g"].items()},
                       n_updates=max(t - 1, 0), t=t)
        iteration_update(ost, {n: np.zeros_like(v) for n, v in ost.x.items()},
                         oracle.hparams_of(w, ef_lambda=lam, **MUON))
        for n in ost.x:
            muon = is_muon_matrix(n)
            if muon:  # the step taken, x_{t+1} - x_t, against the oracle's
                errs[f"step[{t}].{n}"] = rel(post[""][n] - pre[""][n], ost.x[n] - pre[""][n])
                tols[f"step[{t}].{n}"] = tol
            else:     # AdamW: x itself (a gain near 1 holds its small step only to fp32 resolution)
                errs[f"x[{t}].{n}"] = rel(post[""][n], ost.x[n])
                tols[f"x[{t}].{n}"] = 1e-5
            errs[f"m[{t}].{n}"] = rel(post["m."][n], ost.m[n])
            tols[f"m[{t}].{n}"] = 1e-5
            if lam:
                errs[f"u_prev[{t}].{n}"] = rel(post["u_prev."][n], ost.u_prev[n])
                tols[f"u_prev[{t}].{n}"] = tol if muon else 1e-5
            if not muon:
                errs[f"v[{t}].{n}"] = rel(post["v."][n], ost.v[n])
                tols[f"v[{t}].{n}"] = 1e-5
    return errs, tols


def _report(label, errs, tols):
    bad = {k: v for k, v in errs.items() if not v <= tols[k]}
    worst = sorted(errs, key=lambda k: errs[k] / tols[k], reverse=True)[:6]
    log(f"{label}: {len(errs)} comparisons; worst " + ", ".join(f"{k}={errs[k]:.2e}" for k in worst))
    assert not bad, f"{label}: {len(bad)} over tolerance: " + ", ".join(
        f"{k}={v:.2e}" for k, v in sorted(bad.items(), key=lambda kv: -kv[1])[:12])


@pytest.mark.parametrize("lam", [0.0, 1.0])
def test_muon_tiny_fp32(lam):
    w = datagen.TINY
    p0 = datagen.init_params(w)
    steps = 10
    log(f"muon tiny fp32 {steps} steps lambda={lam}")
    g = run_gpu(w, steps, hp_of(w, ef_lambda=lam, **MUON), p0, upd_steps=(1, 2, steps - 1))
    o = run_oracle(w, steps, oracle.hparams_of(w, ef_lambda=lam, **MUON), p0)
    errs, tols = _update_in_place(w, g, lam, 1e-4)
    for t, (lg, lo) in enumerate(zip(g["losses"], o["losses"])):
        errs[f"loss[{t}]"] = abs(lg[0] - lo[0]) / abs(lo[0])
        tols[f"loss[{t}]"] = 1e-4
    for n, ref in o["final"][""].items():
        errs[f"final.{n}"] = rel(g["final"][""][n], ref)
        tols[f"final.{n}"] = 1e-4
    _report(f"muon tiny lambda={lam}", errs, tols)


@pytest.mark.parametrize("w", [SMALL_R, MID_R, LARGE_R, TILED_R, MIXED_R], ids=lambda w: w.name)
def test_muon_reduced_bf16(w):
    steps = 6
    p0 = datagen.init_params(w)
    log(f"muon {w.name}: {steps} steps")
    g = run_gpu(w, steps, hp_of(w, **MUON), p0, upd_steps=(1, 2, steps - 1))
    o = run_oracle(w, steps, oracle.hparams_of(w, **MUON), p0)
    errs, tols = _update_in_place(w, g, w.ef_lambda, 2e-2)
    for t, (lg, lo) in enumerate(zip(g["losses"], o["losses"])):
        for i, (a, b) in enumerate(zip(lg, lo)):
            scale = abs(b) if w.last_stage else o["loss_abs"][t][i]
            errs[f"loss[{t}][{i}]"] = abs(a - b) / max(scale, 1e-30)
            tols[f"loss[{t}][{i}]"] = 2e-2
    for n, ref in o["final"][""].items():
        errs[f"final.{n}"] = rel(g["final"][""][n], ref)
        tols[f"final.{n}"] = 2e-2
    _report(f"muon {w.name}", errs, tols)


def test_muon_update_small_full_size():
    """The small workload at its full size: one step, then delayed_update(1), which consumes g_0, in
    place on the GPU's own state.  Its two Newton-Schulz groups (twelve 768 x 768 matrices, nine
    768 x 3072 ones) have whole tiles: the carried hi/lo pair, and symmetric Gram products that
    compute 21 of their 36 tiles and mirror 15."""
    w = datagen.SMALL
    p0 = datagen.init_params(w)
    log(f"muon {w.name}: 2 steps at full size")
    g = run_gpu(w, 2, hp_of(w, **MUON), p0, upd_steps=(1,))
    errs, tols = _update_in_place(w, g, w.ef_lambda, 2e-2)
    _report("muon small full size", errs, tols)
