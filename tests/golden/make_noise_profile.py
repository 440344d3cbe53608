"""Writes tests/golden/<workload>_<steps>_noise_profile.json: how far a workload's float64 oracle
trajectory (small: 100 iterations of Alg. 1 with Error Feedback, mid: 10) moves when every
gradient is perturbed by an error of the size of bf16 arithmetic, measured with the comparisons the
GPU test makes against the clean trajectory (norm-wise relative errors of the stored slices,
relative errors of the whole-tensor norms), as the median and the maximum over the parameters at
every stored point.  Perturbations (make_trajectory.py --grad-noise 0.012 --noise-seed 7): additive
(0.012 times the tensor's rms times xi: the tensor's smallest elements change sign, as under an
accumulated rounding error) and, for the small workload, relative (each element times
1 + 0.012 xi: no sign changes).

Only oracle output is read: the clean trajectory (<workload>_<steps>_steps.npz) and the perturbed ones.

  python tests/golden/make_trajectory.py --workload W --grad-noise 0.012 --noise-seed 7 --noise-kind additive --out ADD.npz
  python tests/golden/make_trajectory.py --workload W --grad-noise 0.012 --noise-seed 7 --noise-kind relative --out REL.npz
  python tests/golden/make_noise_profile.py --workload W --additive ADD.npz [--relative REL.npz]
"""
from __future__ import annotations

import json
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))


def rel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.linalg.norm((a - b).ravel()) / max(np.linalg.norm(b.ravel()), 1e-30))


def profile(clean, noisy):
    names = sorted(k.split("/", 1)[1] for k in clean.files if k.startswith("offsets/"))
    out = {}
    for key in clean.files:
        if "@" not in key or key.startswith("offsets/"):
            continue
        head, name = (key.split("/", 1) + [""])[:2]
        q, step = head.split("@")
        if head.startswith("norm."):
            q = "|" + q[len("norm."):] + "|"
            a, b = float(noisy[key]), float(clean[key])
            e = abs(a - b) / b if b > 0 else None
        else:
            if np.linalg.norm(clean[key]) == 0:
                continue
            e = rel(noisy[key], clean[key])
        if e is None:
            continue
        out.setdefault(f"{q}@{step}", []).append(e)
    loss = np.abs(noisy["loss"] - clean["loss"]) / clean["loss_abs"]
    res = {k: {"median": float(np.median(v)), "max": float(np.max(v)), "n": len(v)} for k, v in sorted(out.items())}
    res["loss"] = {"median": float(np.median(loss)), "max": float(np.max(loss)), "n": int(loss.size)}
    return res


def main():
    import argparse
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", choices=("small", "mid"), default="small")
    ap.add_argument("--additive", required=True)
    ap.add_argument("--relative")
    args = ap.parse_args()
    name = {"small": "small_100", "mid": "mid_10"}[args.workload]
    clean = np.load(os.path.join(HERE, f"{name}_steps.npz"))
    rec = {"grad_noise": 0.012, "noise_seed": 7}
    for kind, path in (("relative", args.relative), ("additive", args.additive)):
        if not path:
            continue
        res = profile(clean, np.load(path))
        rec[kind] = res
        for k, v in res.items():
            print(f"{kind:8s} {k:14s} median {v['median']:.3e} max {v['max']:.3e} (n {v['n']})")
    path = os.path.join(HERE, f"{name}_noise_profile.json")
    with open(path, "w") as f:
        json.dump(rec, f, indent=1)
    print(f"wrote {path}")


if __name__ == "__main__":
    main()
