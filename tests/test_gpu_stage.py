"""GPU parity of the whole stage step (forward, backward, delayed update) against the oracle, through
the C ABI.  Tolerances: fp32 workload 1e-4, bf16 workloads 2e-2, relative, norm-wise per tensor
(losses: scalar relative)."""
import numpy as np
import pytest

import datagen
import oracle
from gpu_common import hp_of, log, rel, run_gpu, run_oracle

pytestmark = pytest.mark.gpu


def _compare(w, g, o, tol, grad_steps, label, lam=1.0):
    """Losses per step (a head's mean CE: scalar relative; a middle stage's surrogate sum(Y dY):
    error relative to sum |Y dY|, the sum's condition), outputs Y, gradients at grad_steps and the
    final master / m / v / u_prev, all norm-wise relative.  Every failure is reported."""
    errs, bad = {}, []
    for t, (lg, lo) in enumerate(zip(g["losses"], o["losses"])):
        for i, (a, b) in enumerate(zip(lg, lo)):
            scale = abs(b) if w.last_stage else o["loss_abs"][t][i]
            errs[f"loss[{t}][{i}]"] = abs(a - b) / max(scale, 1e-30)
    for t in o["ys"]:
        for i, y in enumerate(o["ys"][t]):
            errs[f"y[{t}][{i}]"] = rel(g["ys"][t][i], y)
    for t in grad_steps:
        for n in o["grads"][t]:
            errs[f"grad[{t}].{n}"] = rel(g["grads"][t][n], o["grads"][t][n])
    for pre in ("", "m.", "v.", "u_prev."):
        if pre == "u_prev." and not lam:
            continue  # standard async keeps no EF buffer
        for n, ref in o["final"][pre].items():
            errs[f"final.{pre}{n}"] = rel(g["final"][pre][n], ref)
    bad = {k: v for k, v in errs.items() if not v <= tol}
    worst = max(errs, key=errs.get)
    log(f"{label}: {len(errs)} comparisons, worst {worst} = {errs[worst]:.3e} (tol {tol})")
    assert not bad, f"{label}: {len(bad)} over tolerance: " + ", ".join(f"{k}={v:.2e}" for k, v in sorted(bad.items(), key=lambda kv: -kv[1])[:12])


@pytest.mark.parametrize("lam", [0.0, 1.0])
def test_tiny_fp32_20_steps(lam):
    w = datagen.TINY
    p0 = datagen.init_params(w)
    log(f"tiny fp32 20 steps lambda={lam}")
    g = run_gpu(w, 20, hp_of(w, ef_lambda=lam), p0, grad_steps=(0, 1, 19))
    o = run_oracle(w, 20, oracle.hparams_of(w, ef_lambda=lam), p0, grad_steps=(0, 1, 19))
    _compare(w, g, o, 1e-4, (0, 1, 19), f"tiny lambda={lam}", lam)


# Reduced bf16 stages: the shapes of the bf16 workloads at sizes the oracle finishes in seconds,
# with ragged sequence lengths (not multiples of 64) and GQA.
SMALL_R = datagen.SMALL.with_(name="small-reduced", n_blocks=2, d_model=256, n_heads=4, n_kv_heads=4,
                              head_dim=64, d_ffn=512, vocab=1000, seq_len=96, micro_batch=2)
MID_R = datagen.MID.with_(name="mid-reduced", n_blocks=2, d_model=256, n_heads=2, n_kv_heads=2,
                          head_dim=128, d_ffn=640, seq_len=80, micro_batch=2)
LARGE_R = datagen.LARGE.with_(name="large-reduced", n_blocks=2, d_model=256, n_heads=4, n_kv_heads=2,
                              head_dim=64, d_ffn=384, seq_len=72, micro_batch=2,
                              microbatches_per_step=4, max_inflight=3)


@pytest.mark.parametrize("w", [SMALL_R, MID_R, LARGE_R], ids=lambda w: w.name)
def test_reduced_bf16_stages(w):
    steps = 12
    p0 = datagen.init_params(w)
    log(f"{w.name}: {steps} steps")
    ys = (0, steps - 1) if not w.last_stage else ()
    g = run_gpu(w, steps, hp_of(w), p0, grad_steps=(0, 1, steps - 1), y_steps=ys)
    o = run_oracle(w, steps, oracle.hparams_of(w), p0, grad_steps=(0, 1, steps - 1), y_steps=ys)
    _compare(w, g, o, 2e-2, (0, 1, steps - 1), w.name)
