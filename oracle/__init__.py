"""CPU oracle of one pipeline stage's training step under a one-step gradient delay.

TEST INFRASTRUCTURE.  This package is the plain, slow, obviously correct reference that the HIP
path is checked against.  Only the tests, the smoke check and the bench's CPU-baseline leg may
import it; the product path never does.  It shares no code with the HIP path: it imports only
numpy and the seeded input generators in `datagen`.

Precision: every routine works in the dtype it is handed (float64 for the pins and the parity
checks, float32 for the timed CPU baseline).

Contents
  ops     primitive operations of a decoder block (App. E.2) and the tied head
  model   stage forward / backward (stack of blocks, embedding, head)
  update  Alg. 1 of §2 with AdamW and the Error-Feedback correction of §3.2 / App. A.4
  run()   the training loop: fwd/bwd at x_t, then the delayed update, for T iterations
"""
from __future__ import annotations

from typing import Callable, Dict, List, Optional

import numpy as np

from . import model, ops, update  # noqa: F401
from .update import HParams, OptState, iteration_update


def hparams_of(w, **kw) -> HParams:
    base = dict(lr=w.lr, beta1=w.beta1, beta2=w.beta2, eps=w.eps, weight_decay=w.weight_decay,
                clip_norm=w.clip_norm, ef_lambda=w.ef_lambda, delay=1)
    base.update(kw)
    return HParams(**base)


def run(w, steps: int, hp: HParams, params0: Dict[str, np.ndarray],
        inputs: Callable[[int, int], Dict[str, np.ndarray]], dt=np.float64,
        record: Optional[Callable[[int, dict], None]] = None) -> OptState:
    """Alg. 1 for `steps` iterations from params0.

    inputs(t, i) returns microbatch i of iteration t.  record(t, info) is called after each
    iteration with the losses, the gradient g_t (float arrays, summed over microbatches) and the
    update diagnostics."""
    st = OptState.create(params0, dt)
    M = w.microbatches_per_step
    for t in range(steps):
        x_t = st.x if st.x_compute is None else st.x_compute   # the compute weights of step t
        grads, outs = model.stage_step_grads(x_t, [inputs(t, i) for i in range(M)], w, dt)
        info = iteration_update(st, grads, hp)
        if record is not None:
            record(t, dict(losses=[o.get("loss") for o in outs], outs=outs, grads=grads, **info))
    return st
