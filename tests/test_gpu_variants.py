"""GPU parity of the elementwise update variants against the oracle, through the C ABI: Lion,
NAdam and Adan as the update function, and SAPipe weight prediction with the updated optimizer state (the
compute copy receives x_{t+1} - u_t(g_{t-1})).  The fused flat update on 1,000,003 elements
(ragged tail) at 1e-5 of the oracle's float64 rule; whole stages free-running at the usual bars
(fp32 1e-4, bf16 2e-2 with m, v at 5e-2).

Lion's sign is a discrete decision taken from floating point: where c = b1 m + (1 - b1) g is within
the rounding of its two terms (a few fp32 ulps; the kernel may contract it into one fma) either sign,
or zero, is a correct result, so Lion is checked in place, step by step, on the GPU's own state:
the unambiguous elements against the oracle's rule, the ambiguous ones for being one of the valid
steps, and losses of the free run."""
import numpy as np
import pytest

import datagen
import oracle
from gpu_common import hp_of, log, rel, run_gpu, run_oracle
from oracle.update import HParams, OptState, iteration_update
from test_gpu_stage import SMALL_R

pytestmark = pytest.mark.gpu

LION = dict(optimizer="lion", lr=5e-4, beta1=0.9, beta2=0.99, weight_decay=0.5)
# the ABI takes fp32 hyper-parameters: the oracle gets the same (fp32-representable) betas, else
# 1 - beta2 alone differs by 1.3e-5 relative at beta2 = 0.999
NADAM = dict(optimizer="nadam", beta1=float(np.float32(0.9)), beta2=float(np.float32(0.999)))
PREDICT = dict(predict="updated", ef_lambda=0.0)
# Adan with the betas of its authors' defaults (beta1 = 0.98 is the value the paper quotes), fp32-exact
ADAN = dict(optimizer="adan", beta1=float(np.float32(0.98)), beta2=float(np.float32(0.92)),
            beta3=float(np.float32(0.99)))


def _lion_check(x0, m0, g, u_prev0, x1, m1, u1, hp, c=1.0, ef=False):
    """One Lion update in place: worst relative error over the unambiguous elements, the number of
    ambiguous ones, and whether each of those took one of the valid steps."""
    x0, m0, g = (np.asarray(a, dtype=np.float64) for a in (x0, m0, g))
    gg = g * c
    a, b = hp.beta1 * m0, (1 - hp.beta1) * gg
    cc = a + b
    amb = np.abs(cc) <= 8 * 2.0 ** -24 * (np.abs(a) + np.abs(b))
    u = hp.lr * (np.sign(cc) + hp.weight_decay * x0)
    up0 = np.zeros_like(x0) if u_prev0 is None else np.asarray(u_prev0, dtype=np.float64)
    xr = x0 - u - (hp.ef_lambda * (u - up0) if ef else 0.0)
    mr = hp.beta2 * m0 + (1 - hp.beta2) * gg
    ok = ~amb
    errs = {"x": rel(np.asarray(x1)[ok], xr[ok]), "m": rel(m1, mr)}
    if u1 is not None:
        errs["u"] = rel(np.asarray(u1)[ok], u[ok])
    valid = True
    if amb.any():
        got = np.asarray(x1, dtype=np.float64)[amb]
        cand = [x0[amb] - hp.lr * (s + hp.weight_decay * x0[amb]) * (1 + (hp.ef_lambda if ef else 0.0))
                + (hp.ef_lambda * up0[amb] if ef else 0.0) for s in (-1.0, 0.0, 1.0)]
        dist = np.min([np.abs(got - cv) for cv in cand], axis=0)
        valid = bool(np.all(dist <= 1e-6 * np.maximum(np.abs(got), 1e-3)))
    return errs, int(amb.sum()), valid


def test_flat_update_lion_in_place():
    import torch
    from paper_2606_30634_amd import binding as B
    from paper_2606_30634_amd.stage import hparams
    n = 1_000_003
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream().cuda_stream
    for lam in (0.0, 1.0):
        kw = dict(dict(lr=1e-3, clip_norm=0.0, ef_lambda=lam, delay=1), **LION)
        hpg, hpo = hparams(**kw), HParams(**kw)
        x = torch.from_numpy(datagen.normal(19, "x", n, 0.02)).to(dev)
        m = torch.zeros(n, device=dev)
        v = torch.zeros(n, device=dev)
        up = torch.zeros(n, device=dev)
        sh = torch.zeros(n, device=dev, dtype=torch.bfloat16)
        for t in range(8):
            gv = datagen.normal(19, "g", n, 1e-3, step=max(t - 1, 0))
            gd = torch.from_numpy(gv).to(dev)
            pre = [a.cpu().numpy().copy() for a in (x, m, up)]
            B.delayed_update_flat(n, x.data_ptr(), gd.data_ptr(), False, m.data_ptr(), v.data_ptr(),
                                  up.data_ptr(), sh.data_ptr(), True, t, hpg, None, stream)
            torch.cuda.synchronize()
            if t == 0:
                continue
            errs, n_amb, valid = _lion_check(pre[0], pre[1], gv, pre[2], x.cpu().numpy(), m.cpu().numpy(),
                                             up.cpu().numpy() if lam else None, hpo, ef=bool(lam) and t >= 2)
            log(f"flat lion lambda={lam} t={t}: " + ", ".join(f"{k}={e:.2e}" for k, e in errs.items()) +
                f", {n_amb} ambiguous signs")
            assert max(errs.values()) < 1e-5 and valid, (t, errs, n_amb, valid)
        assert np.array_equal(sh.view(torch.int16).cpu().numpy().view(np.uint16), datagen.bf16_bits(x.cpu().numpy()))


@pytest.mark.parametrize("kind,lam", [("nadam", 0.0), ("nadam", 1.0), ("predict", 0.0)])
def test_flat_update_variants(kind, lam):
    import torch
    from paper_2606_30634_amd import binding as B
    from paper_2606_30634_amd.stage import hparams
    kw = {"nadam": NADAM, "predict": PREDICT}[kind]
    kw = dict(dict(lr=1e-3, clip_norm=0.0, ef_lambda=lam, delay=1), **kw)
    hpg, hpo = hparams(**kw), HParams(**kw)
    n = 1_000_003
    dev = torch.device("cuda:0")
    x0 = datagen.normal(17, "x", n, 0.02)
    x = torch.from_numpy(x0).to(dev)
    m = torch.zeros(n, device=dev)
    v = torch.zeros(n, device=dev)
    up = torch.zeros(n, device=dev)
    sh = torch.zeros(n, device=dev)   # fp32 compute copy: the predicted point unrounded
    st = OptState.create({"w": x0.astype(np.float64)})
    stream = torch.cuda.current_stream().cuda_stream
    log(f"flat {kind} lambda={lam}: {n} elements")
    for t in range(8):
        gv = datagen.normal(17, "g", n, 1e-3, step=max(t - 1, 0))   # g_{t-1}
        gd = torch.from_numpy(gv).to(dev)
        B.delayed_update_flat(n, x.data_ptr(), gd.data_ptr(), False, m.data_ptr(), v.data_ptr(),
                              up.data_ptr(), sh.data_ptr(), False, t, hpg, None, stream)
        # the oracle consumes at iteration t the gradient handed in at t - 1
        iteration_update(st, {"w": datagen.normal(17, "g", n, 1e-3, step=t).astype(np.float64)}, hpo)
    torch.cuda.synchronize()
    errs = {"x": rel(x.cpu().numpy(), st.x["w"]), "m": rel(m.cpu().numpy(), st.m["w"]),
            "v": rel(v.cpu().numpy(), st.v["w"])}
    if lam:
        errs["u_prev"] = rel(up.cpu().numpy(), st.u_prev["w"])
    xc = st.x_compute["w"] if st.x_compute is not None else st.x["w"]
    errs["compute copy"] = rel(sh.cpu().numpy(), xc)
    log(f"flat {kind} lambda={lam}: " + ", ".join(f"{k}={e:.2e}" for k, e in errs.items()))
    assert max(errs.values()) < 1e-5, errs


def _compare(w, g, o, tol, state_tol, label, compare_v=True):
    errs, tols = {}, {}
    for t, (lg, lo) in enumerate(zip(g["losses"], o["losses"])):
        for i, (a, b) in enumerate(zip(lg, lo)):
            scale = abs(b) if w.last_stage else o["loss_abs"][t][i]
            errs[f"loss[{t}][{i}]"] = abs(a - b) / max(scale, 1e-30)
    for pre in ("", "m.", "v.") if compare_v else ("", "m."):
        for n, ref in o["final"][pre].items():
            k = f"final.{pre}{n}"
            errs[k] = rel(g["final"][pre][n], ref)
            if pre:
                tols[k] = state_tol
    bad = {k: e for k, e in errs.items() if not e <= tols.get(k, tol)}
    worst = sorted(errs, key=lambda k: errs[k] / tols.get(k, tol), reverse=True)[:6]
    log(f"{label}: {len(errs)} comparisons; worst " + ", ".join(f"{k}={errs[k]:.2e}" for k in worst))
    assert not bad, f"{label}: {len(bad)} over tolerance: " + ", ".join(
        f"{k}={e:.2e}" for k, e in sorted(bad.items(), key=lambda kv: -kv[1])[:12])


@pytest.mark.parametrize("kind", ["nadam", "predict", "adan"])
def test_variant_tiny_fp32(kind):
    w = datagen.TINY
    kw = {"nadam": NADAM, "predict": PREDICT, "adan": ADAN}[kind]
    p0 = datagen.init_params(w)
    steps = 12
    log(f"{kind} tiny fp32: {steps} steps")
    g = run_gpu(w, steps, hp_of(w, **kw), p0)
    o = run_oracle(w, steps, oracle.hparams_of(w, **kw), p0)
    _compare(w, g, o, 1e-4, 1e-4, f"{kind} tiny")


def test_lion_tiny_fp32():
    # the update in place at four steps (the GPU's own state and clipped gradient), losses of the
    # free run at 1e-4
    w = datagen.TINY
    lam = 1.0
    p0 = datagen.init_params(w)
    steps = 12
    log(f"lion tiny fp32: {steps} steps")
    g = run_gpu(w, steps, hp_of(w, ef_lambda=lam, **LION), p0, upd_steps=(1, 2, 6, 11))
    o = run_oracle(w, steps, oracle.hparams_of(w, ef_lambda=lam, **LION), p0)
    hpo = oracle.hparams_of(w, ef_lambda=lam, **LION)
    errs = {}
    n_amb = 0
    for t, (pre, post) in g["upd"].items():
        gn = float(np.sqrt(sum(np.sum(np.square(a.astype(np.float64))) for a in pre["g"].values())))
        c = oracle.update.clip_coefficient(gn, hpo.clip_norm)
        for n in pre[""]:
            e, na, valid = _lion_check(pre[""][n], pre["m."][n], pre["g"][n], pre["u_prev."][n], post[""][n],
                                       post["m."][n], post["u_prev."][n], hpo, c=c, ef=t >= 2)
            assert valid, (t, n)
            n_amb += na
            for k, v in e.items():
                errs[f"update[{t}].{k}.{n}"] = v
    for t, (lg, lo) in enumerate(zip(g["losses"], o["losses"])):
        errs[f"loss[{t}]"] = abs(lg[0] - lo[0]) / abs(lo[0])
    worst = sorted(errs, key=errs.get, reverse=True)[:6]
    log(f"lion tiny: {len(errs)} comparisons, {n_amb} ambiguous signs; worst " +
        ", ".join(f"{k}={errs[k]:.2e}" for k in worst))
    assert max(errs.values()) <= 1e-4, {k: v for k, v in errs.items() if v > 1e-4}


@pytest.mark.parametrize("kind", ["nadam", "predict", "adan"])
def test_variant_reduced_bf16(kind):
    w = SMALL_R
    kw = {"nadam": NADAM, "predict": PREDICT, "adan": ADAN}[kind]
    p0 = datagen.init_params(w)
    steps = 8
    log(f"{kind} {w.name}: {steps} steps")
    g = run_gpu(w, steps, hp_of(w, **kw), p0)
    o = run_oracle(w, steps, oracle.hparams_of(w, **kw), p0)
    _compare(w, g, o, 2e-2, 5e-2, f"{kind} {w.name}")


@pytest.mark.parametrize("lam", [0.0, 1.0])
def test_flat_update_adan(lam):
    """delayed_update_flat_adan on 1,000,003 elements over 8 iterations (fp32 gradient, clip off,
    fp32 compute copy): x, m, n, the difference average d, the last clipped gradient, the EF buffer
    and the copy against the oracle's Adan at 1e-5."""
    import torch
    from paper_2606_30634_amd import binding as B
    from paper_2606_30634_amd.stage import hparams
    kw = dict(dict(lr=1e-3, clip_norm=0.0, ef_lambda=lam, delay=1), **ADAN)
    hpg, hpo = hparams(**kw), HParams(**kw)
    n = 1_000_003
    dev = torch.device("cuda:0")
    x0 = datagen.normal(27, "x", n, 0.02)
    x = torch.from_numpy(x0).to(dev)
    m, v, d, gl, up, sh = (torch.zeros(n, device=dev) for _ in range(6))
    st = OptState.create({"w": x0.astype(np.float64)})
    stream = torch.cuda.current_stream().cuda_stream
    log(f"flat adan lambda={lam}: {n} elements")
    for t in range(8):
        gd = torch.from_numpy(datagen.normal(27, "g", n, 1e-3, step=max(t - 1, 0))).to(dev)
        B.delayed_update_flat_adan(n, x.data_ptr(), gd.data_ptr(), False, m.data_ptr(), v.data_ptr(), d.data_ptr(),
                                   gl.data_ptr(), up.data_ptr(), sh.data_ptr(), False, t, hpg, None, stream)
        iteration_update(st, {"w": datagen.normal(27, "g", n, 1e-3, step=t).astype(np.float64)}, hpo)
    torch.cuda.synchronize()
    errs = {"x": rel(x.cpu().numpy(), st.x["w"]), "m": rel(m.cpu().numpy(), st.m["w"]),
            "n": rel(v.cpu().numpy(), st.v["w"]), "d": rel(d.cpu().numpy(), st.adan_d["w"]),
            "g_last": rel(gl.cpu().numpy(), st.adan_gprev["w"]), "copy": rel(sh.cpu().numpy(), st.x["w"])}
    if lam:
        errs["u_prev"] = rel(up.cpu().numpy(), st.u_prev["w"])
    log(f"flat adan lambda={lam}: " + ", ".join(f"{k}={e:.2e}" for k, e in errs.items()))
    assert max(errs.values()) < 1e-5, errs
