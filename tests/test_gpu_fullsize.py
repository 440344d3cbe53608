"""GPU parity at the workloads' full sizes, in the launch configuration the bench times.

* small workload (first stage, 3 blocks, d 768, seq 1024 x 8, vocab 32000): the whole step -
  output, every parameter gradient (float64 oracle at the same x_0), then the delayed update in
  place over the whole flat parameter vector.
* last-stage workload (3 blocks, d 768, seq 1024 x 8, untied head over vocab 49152): the whole
  step - loss, every parameter gradient (float64 oracle at the same x_0) - then the update in
  place over the whole flat vector.
* mid and large workloads: the last block's forward and backward recomputed by the oracle from the
  GPU's saved input of that block and the given upstream gradient (its output, all its weight
  gradients), and the update in place on sampled slices of the flat vector."""
import numpy as np
import pytest

import datagen
import oracle
from gpu_common import hp_of, log, rel, shape_of, to_device
from oracle import model
from oracle.update import HParams, flat_update

pytestmark = pytest.mark.gpu


def _host(t, shape=None):
    a = t.float().cpu().numpy()
    return a.reshape(shape) if shape is not None else a


def _update_in_place(st, w, hp_g, t, sample=None):
    """Capture the flat state before/after delayed_update(t) (all of it, or `sample` slices) and
    return the worst relative error against the oracle's elementwise rule."""
    import torch
    names = ["flat.master", "flat.m", "flat.v", "flat.u_prev", f"flat.grad{(t - 1) % 2}"]
    n = st.tensors["flat.master"][1]
    sl = sample if sample is not None else [(0, n)]
    pre = {k: [st.view(k)[a:a + c].float().cpu().numpy().astype(np.float64) for a, c in sl] for k in names}
    # the gradient buffer is clipped on the device by the global norm: the oracle needs that scale
    gnorm = float(np.sqrt(np.sum(np.square(st.view(names[4]).double().cpu().numpy()))))
    c = oracle.update.clip_coefficient(gnorm, w.clip_norm)
    st.update(t, hp_g)
    torch.cuda.synchronize()
    worst = 0.0
    hpo = HParams(lr=w.lr, beta1=w.beta1, beta2=w.beta2, eps=w.eps, weight_decay=w.weight_decay,
                  clip_norm=0.0, ef_lambda=w.ef_lambda, delay=1)
    for i, (a, cnt) in enumerate(sl):
        x, m, v, up = flat_update(pre["flat.master"][i], pre[names[4]][i] * c, pre["flat.m"][i],
                                  pre["flat.v"][i], pre["flat.u_prev"][i], t, hpo)
        for key, ref in (("flat.master", x), ("flat.m", m), ("flat.v", v), ("flat.u_prev", up)):
            worst = max(worst, rel(st.view(key)[a:a + cnt].float().cpu().numpy(), ref))
    return worst


def test_small_workload_full_step():
    import torch
    from paper_2606_30634_amd.stage import Stage
    w = datagen.SMALL
    dev = torch.device("cuda:0")
    log("fullsize small: GPU step 0")
    st = Stage(shape_of(w), "cuda:0")
    p0 = datagen.init_params(w)
    st.load_master(p0)
    inp = datagen.step_inputs(w, 0)
    d = to_device(inp, w, dev)
    y = torch.empty_like(d["dy"])
    st.forward(0, 0, tokens=d["tokens"], y_out=y)
    st.backward(0, dy=d["dy"])
    torch.cuda.synchronize()
    g = {n: _host(st.view(f"grad0.{n}"), p0[n].shape) for n in p0}
    yg = _host(y)
    log("fullsize small: oracle step 0 (float64)")
    ref, outs = model.stage_step_grads(p0, [inp], w, np.float64)
    errs = {"y": rel(yg, outs[0]["y"])}
    for n in p0:
        errs[f"grad.{n}"] = rel(g[n], ref[n])
    worst = max(errs, key=errs.get)
    log(f"fullsize small: {len(errs)} tensors, worst {worst} = {errs[worst]:.3e}")
    bad = {k: v for k, v in errs.items() if not v <= 2e-2}
    assert not bad, bad
    # step 1 and the first real update (consumes g_0), in place over all 52.9M parameters
    st.update(0, hp_of(w))
    d1 = to_device(datagen.step_inputs(w, 1), w, dev)
    st.forward(0, 1, tokens=d1["tokens"], y_out=y)
    st.backward(0, dy=d1["dy"])
    e = _update_in_place(st, w, hp_of(w), 1)
    log(f"fullsize small: update in place, worst rel {e:.3e}")
    assert e < 1e-5
    st.close()


def test_last_stage_full_step():
    import torch
    from paper_2606_30634_amd.stage import Stage
    w = datagen.LAST
    dev = torch.device("cuda:0")
    log("fullsize last: GPU step 0")
    st = Stage(shape_of(w), "cuda:0")
    p0 = datagen.init_params(w)
    st.load_master(p0)
    inp = datagen.step_inputs(w, 0)
    d = to_device(inp, w, dev)
    loss = torch.zeros(1, device=dev)
    st.forward(0, 0, x_in=d["x_in"], targets=d["targets"], loss=loss)
    st.backward(0)
    torch.cuda.synchronize()
    g = {n: _host(st.view(f"grad0.{n}"), p0[n].shape) for n in p0}
    lg = float(loss.item())
    log("fullsize last: oracle step 0 (float64)")
    ref, outs = model.stage_step_grads(p0, [inp], w, np.float64)
    errs = {"loss": abs(lg - float(outs[0]["loss"])) / abs(float(outs[0]["loss"]))}
    for n in p0:
        errs[f"grad.{n}"] = rel(g[n], ref[n])
    worst = max(errs, key=errs.get)
    log(f"fullsize last: {len(errs)} comparisons, loss {lg:.6f}, worst {worst} = {errs[worst]:.3e}")
    bad = {k: v for k, v in errs.items() if not v <= 2e-2}
    assert not bad, bad
    st.update(0, hp_of(w))
    d1 = to_device(datagen.step_inputs(w, 1), w, dev)
    st.forward(0, 1, x_in=d1["x_in"], targets=d1["targets"], loss=loss)
    st.backward(0)
    e = _update_in_place(st, w, hp_of(w), 1)
    log(f"fullsize last: update in place, worst rel {e:.3e}")
    assert e < 1e-5
    st.close()


@pytest.mark.parametrize("wname", ["mid", "large"])
def test_last_block_full_size(wname):
    import torch
    from paper_2606_30634_amd.stage import Stage
    w = datagen.WORKLOADS[wname].with_(microbatches_per_step=1, max_inflight=1)
    dt = np.float64 if wname == "mid" else np.float32
    dev = torch.device("cuda:0")
    log(f"fullsize {wname}: GPU forward + backward of one microbatch")
    st = Stage(shape_of(w), "cuda:0")
    p0 = datagen.init_params(w)
    st.load_master(p0)
    inp = datagen.step_inputs(w, 0)
    d = to_device(inp, w, dev)
    y = torch.empty_like(d["dy"])
    st.forward(0, 0, x_in=d["x_in"], y_out=y)
    st.backward(0, dy=d["dy"])
    torch.cuda.synchronize()
    L = w.n_blocks - 1
    B_, s, dm = w.micro_batch, w.seq_len, w.d_model
    x_last = _host(st.view(f"act0.blk{L}.x"), (B_, s, dm)).astype(dt)
    pre = f"blk{L}."
    names = [n for n in p0 if n.startswith(pre)]
    g = {n: _host(st.view(f"grad0.{n}"), p0[n].shape) for n in names}
    yg = _host(y, (B_, s, dm))
    log(f"fullsize {wname}: oracle block {L} forward + backward ({np.dtype(dt).name})")
    pb = {n[len(pre):]: p0[n].astype(dt) for n in names}
    y_ref, saves = model.block_fwd(pb, x_last, w, dt)
    _, gref = model.block_bwd(pb, saves, inp["dy"].astype(dt), w)
    errs = {"y": rel(yg, y_ref)}
    for k, v in gref.items():
        errs[f"grad.{pre}{k}"] = rel(g[pre + k], v)
    worst = max(errs, key=errs.get)
    log(f"fullsize {wname}: worst {worst} = {errs[worst]:.3e}")
    bad = {k: v for k, v in errs.items() if not v <= 2e-2}
    assert not bad, bad
    # one more step, then the first real update in place on 16 slices of the flat vector
    st.update(0, hp_of(w))
    d1 = to_device(datagen.step_inputs(w, 1), w, dev)
    st.forward(0, 1, x_in=d1["x_in"], y_out=y)
    st.backward(0, dy=d1["dy"])
    n = st.tensors["flat.master"][1]
    rng = np.random.default_rng(5)
    sample = [(int(a) // 64 * 64, 65536) for a in rng.integers(0, n - 65536, size=16)]
    e = _update_in_place(st, w, hp_of(w), 1, sample)
    log(f"fullsize {wname}: update in place on 16 slices, worst rel {e:.3e}")
    assert e < 1e-5
    st.close()
