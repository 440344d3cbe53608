"""Oracle primitive operations of one Llama-style decoder block (numpy, any float dtype).

TEST INFRASTRUCTURE: only the tests, the smoke check and the bench's CPU-baseline leg may use this
package.  It shares no code with the HIP path.

The paper names the block type (App. E.2, "Model architectures": Llama-style blocks with grouped
query attention, RMSNorm and SwiGLU) and trains it by next-token prediction (App. E, first
paragraph).  It fixes no constants, so the following readings are used throughout:
RMSNorm epsilon 1e-5 with statistics over the feature axis; RoPE in rotate-half form with base
10000 on positions 0..s-1 of each sequence; attention scale 1/sqrt(head_dim), causal mask that
keeps the diagonal, softmax in the working precision; query head h reads key/value head
floor(h * Hkv / Hq); SwiGLU z = silu(x Wg^T) * (x Wu^T); no biases anywhere.

Every function is a direct transcription of its textbook definition; backward functions are the
chain rule of the matching forward, pinned by finite differences in the tests.
"""
from __future__ import annotations

import numpy as np


# ---------------------------------------------------------------- RMSNorm
def rmsnorm_fwd(x, gamma, eps):
    """y = x * r * gamma with r = 1/sqrt(mean_j x_j^2 + eps); returns (y, r). x: [T, d]."""
    ms = np.mean(x * x, axis=-1)
    r = 1.0 / np.sqrt(ms + eps)
    return x * r[:, None] * gamma[None, :], r


def rmsnorm_bwd(dy, x, r, gamma):
    """Chain rule of rmsnorm_fwd: returns (dx, dgamma)."""
    xhat = x * r[:, None]
    dgamma = np.sum(dy * xhat, axis=0)
    g = dy * gamma[None, :]
    dx = r[:, None] * (g - xhat * np.mean(g * xhat, axis=-1, keepdims=True))
    return dx, dgamma


# ---------------------------------------------------------------- linear (no bias)
def linear_fwd(x, w):
    """y = x W^T; x [T, K], W [N, K] (output features by input features) -> [T, N]."""
    return x @ w.T


def linear_bwd(dy, x, w):
    """Returns (dx = dy W, dW = dy^T x)."""
    return dy @ w, dy.T @ x


# ---------------------------------------------------------------- RoPE
def rope_angles(seq_len, head_dim, theta, dtype):
    """angle[p, i] = p * theta^(-2i/head_dim) for i < head_dim/2."""
    half = head_dim // 2
    inv = theta ** (-(2.0 * np.arange(half, dtype=np.float64)) / head_dim)
    ang = np.arange(seq_len, dtype=np.float64)[:, None] * inv[None, :]
    return ang.astype(dtype)


def rope_apply(x, theta, inverse=False):
    """Rotate-half RoPE on x [B, s, H, hd]: pair (i, i+hd/2) turned by +angle (or -angle)."""
    B, s, H, hd = x.shape
    half = hd // 2
    ang = rope_angles(s, hd, theta, x.dtype)
    c = np.cos(ang)[None, :, None, :]
    sn = np.sin(ang)[None, :, None, :]
    if inverse:
        sn = -sn
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - b * sn, b * c + a * sn], axis=-1)


# ---------------------------------------------------------------- causal attention (GQA)
def attention_fwd(q, k, v):
    """Causal softmax attention.  q [B, s, Hq, hd], k, v [B, s, Hkv, hd].

    Returns (o [B, s, Hq, hd], lse [B, Hq, s]) where lse is the log-sum-exp of each scaled,
    masked score row."""
    B, s, Hq, hd = q.shape
    Hkv = k.shape[2]
    scale = 1.0 / np.sqrt(hd)
    mask = np.triu(np.ones((s, s), dtype=bool), k=1)  # True above the diagonal: masked
    o = np.zeros_like(q)
    lse = np.zeros((B, Hq, s), dtype=q.dtype)
    for b in range(B):
        for h in range(Hq):
            g = (h * Hkv) // Hq
            sc = (q[b, :, h, :] @ k[b, :, g, :].T) * scale
            sc = np.where(mask, -np.inf, sc)
            mx = np.max(sc, axis=-1, keepdims=True)
            e = np.exp(sc - mx)
            den = np.sum(e, axis=-1, keepdims=True)
            p = e / den
            o[b, :, h, :] = p @ v[b, :, g, :]
            lse[b, h, :] = (mx + np.log(den))[:, 0]
    return o, lse


def attention_bwd(do, q, k, v):
    """Chain rule of attention_fwd (probabilities recomputed): returns (dq, dk, dv).

    dP = dO V^T, dS = P * (dP - rowsum(dP * P)), dQ = dS K * scale, dK = dS^T Q * scale,
    dV = P^T dO; key/value gradients are summed over the query heads that share them."""
    B, s, Hq, hd = q.shape
    Hkv = k.shape[2]
    scale = 1.0 / np.sqrt(hd)
    mask = np.triu(np.ones((s, s), dtype=bool), k=1)
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    for b in range(B):
        for h in range(Hq):
            g = (h * Hkv) // Hq
            sc = (q[b, :, h, :] @ k[b, :, g, :].T) * scale
            sc = np.where(mask, -np.inf, sc)
            e = np.exp(sc - np.max(sc, axis=-1, keepdims=True))
            p = e / np.sum(e, axis=-1, keepdims=True)
            dp = do[b, :, h, :] @ v[b, :, g, :].T
            ds = p * (dp - np.sum(dp * p, axis=-1, keepdims=True))
            dq[b, :, h, :] = (ds @ k[b, :, g, :]) * scale
            dk[b, :, g, :] += (ds.T @ q[b, :, h, :]) * scale
            dv[b, :, g, :] += p.T @ do[b, :, h, :]
    return dq, dk, dv


# ---------------------------------------------------------------- SwiGLU
def sigmoid(a):
    return 1.0 / (1.0 + np.exp(-a))


def swiglu_fwd(a, b):
    """z = silu(a) * b, silu(a) = a * sigmoid(a)."""
    return a * sigmoid(a) * b


def swiglu_bwd(dz, a, b):
    """Returns (da, db): da = dz * b * sig(a) * (1 + a (1 - sig(a))), db = dz * silu(a)."""
    sg = sigmoid(a)
    return dz * b * sg * (1.0 + a * (1.0 - sg)), dz * a * sg


# ---------------------------------------------------------------- embedding
def embed_fwd(table, tokens):
    """x0[i] = E[tok[i]]; tokens int [...], table [V, d]."""
    return table[tokens]


def embed_bwd(dx0, tokens, vocab):
    """dE[v] = sum over positions i with tok[i] == v of dx0[i] (untouched rows exactly 0).

    Also returns the ascending unique ids and their counts."""
    flat_t = tokens.reshape(-1)
    flat_g = dx0.reshape(flat_t.shape[0], -1)
    de = np.zeros((vocab, flat_g.shape[1]), dtype=dx0.dtype)
    np.add.at(de, flat_t, flat_g)
    ids, counts = np.unique(flat_t, return_counts=True)
    return de, ids.astype(np.int32), counts.astype(np.int32)


# ---------------------------------------------------------------- tied head + cross-entropy
def logsumexp_rows(z):
    mx = np.max(z, axis=-1, keepdims=True)
    return (mx + np.log(np.sum(np.exp(z - mx), axis=-1, keepdims=True)))[:, 0]


def ce_fwd(logits, targets):
    """Mean next-token cross-entropy over rows: mean_i (lse(z_i) - z_i[t_i])."""
    n = logits.shape[0]
    lse = logsumexp_rows(logits)
    return np.mean(lse - logits[np.arange(n), targets]), lse


def ce_bwd(logits, targets, lse, scale):
    """d loss / d logits = (softmax - onehot) * scale  (scale = 1/N for the mean)."""
    n = logits.shape[0]
    p = np.exp(logits - lse[:, None])
    p[np.arange(n), targets] -= 1.0
    return p * scale
