"""Oracle forward and backward of one pipeline stage: a stack of decoder blocks, with the token
embedding on a first stage and the LM head with next-token cross-entropy on a last stage (tied to
the embedding when the stage holds both ends, its own matrix otherwise).

TEST INFRASTRUCTURE: only the tests, the smoke check and the bench's CPU-baseline leg may use this
package.  It shares no code with the HIP path.

Block (App. E.2, Llama-style, pre-norm):
    h = x + Attn(RoPE(n1 Wq^T), RoPE(n1 Wk^T), n1 Wv^T) Wo^T,   n1 = RMSNorm(x; attn_norm)
    y = h + (silu(n2 Wg^T) * (n2 Wu^T)) Wd^T,                   n2 = RMSNorm(h; ffn_norm)
Head (last stage): logits = RMSNorm(x_L; final_norm) W^T with W the embedding E (tied) or the
stage's head matrix [vocab, d], loss = mean CE against the given next-token targets.
A stage without a head reports the surrogate loss sum(Y * dY) for the upstream gradient dY it is
handed, so that its backward is the gradient of that scalar.
"""
from __future__ import annotations

from typing import Dict, Tuple

import numpy as np

from . import ops


def _blk(params, i):
    p = f"blk{i}."
    return {k[len(p):]: v for k, v in params.items() if k.startswith(p)}


def block_fwd(p, x, w, dt):
    """One decoder block on x [B, s, d]; returns (y [B, s, d], saved tensors for backward)."""
    B, s, d = x.shape
    T = B * s
    Hq, Hkv, hd = w.n_heads, w.n_kv_heads, w.head_dim
    xf = x.reshape(T, d)
    n1, r1 = ops.rmsnorm_fwd(xf, p["attn_norm"], dt(w.rms_eps))
    q = ops.linear_fwd(n1, p["wq"]).reshape(B, s, Hq, hd)
    k = ops.linear_fwd(n1, p["wk"]).reshape(B, s, Hkv, hd)
    v = ops.linear_fwd(n1, p["wv"]).reshape(B, s, Hkv, hd)
    qr = ops.rope_apply(q, w.rope_theta)
    kr = ops.rope_apply(k, w.rope_theta)
    o, lse = ops.attention_fwd(qr, kr, v)
    of = o.reshape(T, Hq * hd)
    h = xf + ops.linear_fwd(of, p["wo"])
    n2, r2 = ops.rmsnorm_fwd(h, p["ffn_norm"], dt(w.rms_eps))
    a = ops.linear_fwd(n2, p["wgate"])
    b = ops.linear_fwd(n2, p["wup"])
    z = ops.swiglu_fwd(a, b)
    y = h + ops.linear_fwd(z, p["wdown"])
    saves = dict(x=xf, r1=r1, n1=n1, q=qr, k=kr, v=v, o=of, lse=lse, h=h, r2=r2, n2=n2,
                 a=a, b=b, z=z)
    return y.reshape(B, s, d), saves


def block_bwd(p, sv, dy, w):
    """Chain rule of block_fwd.  Returns (dx [B, s, d], dict of parameter gradients)."""
    B, s, d = dy.shape
    T = B * s
    Hq, Hkv, hd = w.n_heads, w.n_kv_heads, w.head_dim
    dyf = dy.reshape(T, d)
    g = {}
    dz, g["wdown"] = ops.linear_bwd(dyf, sv["z"], p["wdown"])
    da, db = ops.swiglu_bwd(dz, sv["a"], sv["b"])
    dn2a, g["wgate"] = ops.linear_bwd(da, sv["n2"], p["wgate"])
    dn2b, g["wup"] = ops.linear_bwd(db, sv["n2"], p["wup"])
    dhn, g["ffn_norm"] = ops.rmsnorm_bwd(dn2a + dn2b, sv["h"], sv["r2"], p["ffn_norm"])
    dh = dyf + dhn
    do, g["wo"] = ops.linear_bwd(dh, sv["o"], p["wo"])
    dqr, dkr, dv = ops.attention_bwd(do.reshape(B, s, Hq, hd), sv["q"], sv["k"], sv["v"])
    dq = ops.rope_apply(dqr, w.rope_theta, inverse=True)
    dk = ops.rope_apply(dkr, w.rope_theta, inverse=True)
    dn1q, g["wq"] = ops.linear_bwd(dq.reshape(T, Hq * hd), sv["n1"], p["wq"])
    dn1k, g["wk"] = ops.linear_bwd(dk.reshape(T, Hkv * hd), sv["n1"], p["wk"])
    dn1v, g["wv"] = ops.linear_bwd(dv.reshape(T, Hkv * hd), sv["n1"], p["wv"])
    dxn, g["attn_norm"] = ops.rmsnorm_bwd(dn1q + dn1k + dn1v, sv["x"], sv["r1"], p["attn_norm"])
    dx = dh + dxn
    return dx.reshape(B, s, d), g


def stage_forward(params: Dict[str, np.ndarray], inp: Dict[str, np.ndarray], w, dt=np.float64):
    """Forward of the stage on one microbatch.

    Returns (out, saves): out holds "y" (stage output, no head) or "logits" and "loss" (head); a
    stage without a head also gets the surrogate "loss" = sum(Y * dY) when dY is in inp."""
    P = {k: v.astype(dt) for k, v in params.items()}
    saves: Dict[str, object] = {}
    if w.first_stage:
        x = ops.embed_fwd(P["embed"], inp["tokens"])
    else:
        x = inp["x_in"].astype(dt)
    saves["x0"] = x
    blocks = []
    for i in range(w.n_blocks):
        x, sv = block_fwd(_blk(P, i), x, w, dt)
        blocks.append(sv)
    saves["blocks"] = blocks
    out: Dict[str, object] = {}
    if w.last_stage:
        B, s, d = x.shape
        xf = x.reshape(B * s, d)
        hf, rf = ops.rmsnorm_fwd(xf, P["final_norm"], dt(w.rms_eps))
        logits = ops.linear_fwd(hf, P["head"] if "head" in P else P["embed"])
        loss, lse = ops.ce_fwd(logits, inp["targets"].reshape(-1))
        saves.update(xL=xf, hf=hf, rf=rf, logits=logits, lse_ce=lse)
        out["logits"] = logits
        out["loss"] = loss
    else:
        out["y"] = x
        if "dy" in inp:
            prod = x.astype(np.float64) * inp["dy"].astype(np.float64)
            out["loss"] = float(np.sum(prod))
            out["loss_abs"] = float(np.sum(np.abs(prod)))  # condition of the sum, for comparisons
    return out, saves


def stage_backward(params, inp, saves, w, dt=np.float64, loss_scale: float = 1.0):
    """Backward of the stage on one microbatch.

    Head: gradient of loss_scale * mean CE.  No head: backward from inp["dy"].
    Returns (dict of parameter gradients, dx_in or None)."""
    P = {k: v.astype(dt) for k, v in params.items()}
    grads: Dict[str, np.ndarray] = {}
    if w.last_stage:
        logits, tg = saves["logits"], inp["targets"].reshape(-1)
        n = logits.shape[0]
        dlog = ops.ce_bwd(logits, tg, saves["lse_ce"], dt(loss_scale / n))
        untied = "head" in P
        dhf, dw = ops.linear_bwd(dlog, saves["hf"], P["head"] if untied else P["embed"])
        if untied:
            grads["head"], de_head = dw, None
        else:
            de_head = dw
        dxl, grads["final_norm"] = ops.rmsnorm_bwd(dhf, saves["xL"], saves["rf"], P["final_norm"])
        B, s = inp["targets"].shape
        dx = dxl.reshape(B, s, w.d_model)
    else:
        de_head = None
        dx = inp["dy"].astype(dt)
    for i in reversed(range(w.n_blocks)):
        dx, g = block_bwd(_blk(P, i), saves["blocks"][i], dx, w)
        for k, v in g.items():
            grads[f"blk{i}.{k}"] = v
    dx_in = None
    if w.first_stage:
        de, _, _ = ops.embed_bwd(dx, inp["tokens"], w.vocab)
        grads["embed"] = de if de_head is None else de + de_head
    else:
        dx_in = dx
    return grads, dx_in


def stage_step_grads(params, inputs_per_micro, w, dt=np.float64):
    """Forward and backward of all microbatches of one optimizer step at fixed weights.

    Gradients are summed over microbatches; a head's mean CE is divided by their number M.
    Returns (summed grads, list of per-microbatch outputs)."""
    M = len(inputs_per_micro)
    total = None
    outs = []
    for inp in inputs_per_micro:
        out, sv = stage_forward(params, inp, w, dt)
        g, _ = stage_backward(params, inp, sv, w, dt, loss_scale=1.0 / M)
        outs.append(out)
        if total is None:
            total = g
        else:
            for k in total:
                total[k] = total[k] + g[k]
    return total, outs
