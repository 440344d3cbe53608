"""GPU parity at the workloads' full sizes against stored float64 oracle values (tests/golden/,
written by the scripts beside them, which call only the oracle and the seeded input generators).

* one-block stages at the full width of the mid workload (d_model 2048, heads of 128, SwiGLU 8192,
  seq 2048 x 4) and of the large one (d_model 4096, 32 query / 8 key-value heads, SwiGLU 14336,
  seq 4096 x 2, eight microbatches per step in a 1F1B order with 4 activation slots): step 0's
  output rows, the gradient handed upstream (dx_out) of every microbatch, the step's parameter
  gradient (seeded slices and whole-tensor norms), then the delayed updates of iterations 1 and 2
  (Error Feedback active at 2) in place on slices of the flat vector;
* the small workload (3 blocks, d_model 768, seq 1024 x 8, vocab-32000 embedding) free-running for
  100 iterations of Alg. 1 with Error Feedback: every step's surrogate loss, output rows, the
  gradient of steps 0, 1, 10, 50, 99 and the master weights, moments and EF buffer before
  iterations 2, 3, 10, 50 and 100 (slices and whole-tensor norms).
Tolerance: 2e-2 norm-wise relative (the bf16 bar), except where a comparison says otherwise."""
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


def test_small_workload_100_steps():
    import torch
    from paper_2606_30634_amd.stage import Stage
    z = _load("small_100_steps.npz")
    w = datagen.SMALL
    dev = torch.device("cuda:0")
    p0 = datagen.init_params(w)
    names = list(p0)
    offs = {n: int(z[f"offsets/{n}"]) for n in names}
    cnt = 512
    steps = len(z["loss"])
    x0 = {n: torch.from_numpy(p0[n].reshape(-1)).double() for n in names}
    st = Stage(shape_of(w), "cuda:0")
    st.load_master(p0)
    hp = hp_of(w)
    errs, tols = {}, {}
    y = torch.empty(w.micro_batch, w.seq_len, w.d_model, dtype=torch.bfloat16, device=dev)
    rows = [0, 1, 1023, 1024, 4095, 8191]
    log(f"golden small: {steps} iterations")

    def state_at(k):
        torch.cuda.synchronize()
        for n in names:
            x = st.view(n).double()
            errs[f"x@{k}.{n}"] = rel(x[offs[n]:offs[n] + cnt].cpu().numpy(), z[f"x@{k}/{n}"])
            # the displacement x_k - x_0 of the slice: what the updates moved
            d_ref = z[f"x@{k}/{n}"].astype(np.float64) - x0[n][offs[n]:offs[n] + cnt].numpy()
            d_gpu = x[offs[n]:offs[n] + cnt].cpu().numpy() - x0[n][offs[n]:offs[n] + cnt].numpy()
            if np.linalg.norm(d_ref) > 0:
                errs[f"dx@{k}.{n}"] = rel(d_gpu, d_ref)
            nd = float((x.cpu() - x0[n]).norm())
            ref = float(z[f"norm.dx@{k}/{n}"])
            if ref > 0:
                errs[f"|dx|@{k}.{n}"] = abs(nd - ref) / ref
            for pre, key in (("m", "m."), ("v", "v."), ("u_prev", "u_prev.")):
                full = st.view(key + n).double()
                ref_n = float(z[f"norm.{pre}@{k}/{n}"])
                if ref_n == 0:
                    continue
                errs[f"{pre}@{k}.{n}"] = rel(full[offs[n]:offs[n] + cnt].cpu().numpy(), z[f"{pre}@{k}/{n}"])
                errs[f"|{pre}|@{k}.{n}"] = abs(float(full.norm()) - ref_n) / ref_n

    for t in range(steps):
        if t in (2, 3, 10, 50):
            state_at(t)
        inp = to_device(datagen.step_inputs(w, t, 0), w, dev)
        st.forward(0, t, tokens=inp["tokens"], y_out=y)
        st.backward(0, dy=inp["dy"])
        if t in (0, 1, 10, 50, 99):
            torch.cuda.synchronize()
            for n in names:
                g = st.view(f"grad{t % 2}.{n}").double()[offs[n]:offs[n] + cnt].cpu().numpy()
                if np.linalg.norm(z[f"g@{t}/{n}"]) > 0:
                    errs[f"g@{t}.{n}"] = rel(g, z[f"g@{t}/{n}"])
            yr = y.float().reshape(-1, w.d_model)[rows].cpu().numpy()
            errs[f"y@{t}"] = rel(yr, z[f"y@{t}"])
        yv = y.double()
        dyv = inp["dy"].double()
        loss = float((yv * dyv).sum())
        errs[f"loss@{t}"] = abs(loss - float(z["loss"][t])) / float(z["loss_abs"][t])
        st.update(t, hp)
    state_at(steps)
    st.close()
    _report("golden small 100 steps", errs, tols)
