"""Writes tests/golden/{mid,large}_1block_step0.npz: the float64 oracle's step 0 of a one-block
stage at the full width of the mid workload (d_model 2048, 16 heads of 128, SwiGLU 8192, seq 2048
x 4, one microbatch) or of the large one (d_model 4096, 32 query / 8 key-value heads of 128,
SwiGLU 14336, seq 4096 x 2, eight microbatches per optimizer step: a 1F1B step of the stage), at
the initial weights, with the seeded input activations and upstream gradients of step 0.  One
block keeps every kernel shape of the workload while the stage input stays the seeded x_in, so
the oracle needs nothing from the GPU (App. E.2 block; §2 Alg. 1 gradient of step 0).

Only the oracle and the seeded input generators are used.

Stored (float64 unless noted; slices float32):
  offsets/<name>             int64 [NS]: starts of the stored slices of each parameter (seeded)
  g/<name>                   float32 [NS, SLICE]: those slices of g_0 (summed over microbatches)
  gnorm/<name>               ||g_0|| of each parameter
  dx/<i>                     float32 rows DX_ROWS of the gradient of microbatch i's stage input
  dxnorm/<i>                 its whole norm
  y/<i>                      float32 rows DX_ROWS of microbatch i's stage output
  ynorm/<i>                  its whole norm

  python tests/golden/make_wide_step.py --workload mid|large
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
from oracle import model  # noqa: E402

SLICE = 512
NS = 4
SLICE_SEED = 20250612
DX_ROWS = (0, 1, 2047, 2048, 4095, 4096, 8191)
HERE = os.path.dirname(os.path.abspath(__file__))


def workload(name):
    return datagen.WORKLOADS[name].with_(n_blocks=1)


def slice_offsets(params):
    rng = np.random.default_rng(SLICE_SEED)
    return {n: np.sort(rng.integers(0, v.size - SLICE + 1, size=NS)).astype(np.int64) for n, v in params.items()}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", choices=("mid", "large"), required=True)
    args = ap.parse_args()
    w = workload(args.workload)
    p0 = datagen.init_params(w)
    offs = slice_offsets(p0)
    P = {k: v.astype(np.float64) for k, v in p0.items()}
    M = w.microbatches_per_step
    rec = {}
    total = None
    for i in range(M):
        tic = time.time()
        inp = datagen.step_inputs(w, 0, i)
        out, sv = model.stage_forward(P, inp, w, np.float64)
        g, dx = model.stage_backward(P, inp, sv, w, np.float64)
        T = w.micro_batch * w.seq_len
        rows = [r for r in DX_ROWS if r < T]
        rec[f"dx/{i}"] = dx.reshape(T, w.d_model)[rows].astype(np.float32)
        rec[f"dxnorm/{i}"] = np.array(np.linalg.norm(dx.ravel()))
        rec[f"y/{i}"] = out["y"].reshape(T, w.d_model)[rows].astype(np.float32)
        rec[f"ynorm/{i}"] = np.array(np.linalg.norm(out["y"].ravel()))
        if total is None:
            total = g
        else:
            for k in total:
                total[k] = total[k] + g[k]
        del out, sv, g, dx
        print(f"{args.workload}: microbatch {i}: {time.time() - tic:.1f} s", flush=True)
    for n, a in total.items():
        flat = a.ravel()
        rec[f"offsets/{n}"] = offs[n]
        rec[f"g/{n}"] = np.stack([flat[o:o + SLICE] for o in offs[n]]).astype(np.float32)
        rec[f"gnorm/{n}"] = np.array(np.linalg.norm(flat))
    out_path = os.path.join(HERE, f"{args.workload}_1block_step0.npz")
    np.savez_compressed(out_path, **rec)
    print(f"wrote {out_path}: {len(rec)} arrays", flush=True)


if __name__ == "__main__":
    main()
