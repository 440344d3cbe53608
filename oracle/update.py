"""Oracle of the delayed optimizer update (Alg. 1 of §2) with AdamW as the update function u,
the Error-Feedback correction of §3.2 and its lambda-scaled form (App. A.4).

TEST INFRASTRUCTURE: only the tests, the smoke check and the bench's CPU-baseline leg may use this
package.  It shares no code with the HIP path.

Alg. 1, one iteration t (g_{-1} = 0, u_{-1} = 0):
    compute g_t at x_t
    feed g_{t-1} to the optimizer statistics and form u_{t-1}(g_{t-1})
    standard async, or t <= 1:  x_{t+1} = x_t - u_{t-1}
    Error Feedback:             x_{t+1} = x_t - u_{t-1} - lambda (u_{t-1} - u_{t-2})
(lambda = 1 is the equation of §3.2; lambda = 0 is standard async.)  With delay 0 the same
update consumes g_t instead, which is plain synchronous AdamW.

Elementwise variants of u (the optimizer list of §3.3, on every parameter; same delay and EF):
    "lion"  (Chen et al., 2023):  u = lr (sign(b1 m + (1 - b1) g) + wd x_t),  m <- b2 m + (1 - b2) g
    "nadam" (Dozat, 2016, the momentum-decay schedule of torch.optim.NAdam): mu_k = b1 (1 - 0.5 0.96^(k psi)),
            m, v as AdamW, u = lr ((1 - mu_k) / (1 - P_k) g + mu_{k+1} / (1 - P_k mu_{k+1}) m) /
            (sqrt(v / (1 - b2^k)) + eps) + lr wd x_t,   P_k = mu_1 ... mu_k
    "adan"  (Xie et al., Adan, with the betas as averaging weights, (0.98, 0.92, 0.99) in its defaults):
            diff = g - g_prev (0 at the first update), g_prev the clipped gradient of the previous update,
            m <- b1 m + (1 - b1) g ;  d <- b2 d + (1 - b2) diff ;  n <- b3 n + (1 - b3) (g + b2 diff)^2
            u = lr ((m / (1 - b1^k) + b2 d / (1 - b2^k)) / (sqrt(n / (1 - b3^k)) + eps) + wd x_t)
            (n is kept in the v slot; d and g_prev are Adan's two extra state vectors; the decay is the
            decoupled one on x_t, as for the other rules)
and SAPipe weight prediction with the updated optimizer state (App. B.1, predict = "updated", AdamW):
the master follows the standard delayed update x_{t+1} = x_t - u_{t-1}(g_{t-1}), while the next
forward/backward runs at x~_{t+1} = x_{t+1} - u_t(g_{t-1}), the AdamW step from the state after the
real update fed g_{t-1} once more (bias correction k + 1, decay on x_{t+1}); the predicted state is
not kept.

Delay tau >= 2 (the delayed-gradient method of App. C with prev(k) = k - tau): iteration t consumes
g_{t-tau} (iterations t < tau change nothing), and Error Feedback takes the update formed tau
iterations earlier,
    x_{t+1} = x_t - u - lambda (u - u_{t-tau})
which is the appendix's x_{k+1} = x_k - (tau + 1) u_k + tau u_{k-tau} at lambda = tau (the
coefficients its convergence proof uses) and the printed algorithm's 2 / 1 at lambda = 1.  The step
is standard until tau earlier updates exist (the "t <= 1" rule of Alg. 1 for tau = 1).

u is decoupled AdamW (§2: beta = (0.9, 0.95); App. E.1: weight decay 0.1, clipping at 1.0):
    g <- c g,  c = min(1, clip / (||g||_2 + 1e-6))        (global norm over the stage)
    m <- b1 m + (1 - b1) g;   v <- b2 v + (1 - b2) g^2
    u  = lr ( (m / (1 - b1^k)) / (sqrt(v / (1 - b2^k)) + eps) + wd x_t )
with k the number of gradients consumed so far including this one, weight decay on the current
weights x_t (the form Alg. 2 of §4 writes, U = eta (O + lambda X_t)), and the following readings
where the paper is silent: eps = 1e-8; the clip epsilon 1e-6; weight decay on every parameter;
step t = 0 changes nothing (the zero gradient g_{-1} is not fed to the statistics, so the first
real update has k = 1); the EF buffer holds the whole previous update u_{t-2}, learning rate and
weight decay included.

A gradient whose global norm is not finite (a failure-detection reading; the paper is silent)
is consumed without effect: the iteration leaves x, m, v and every Error-Feedback
buffer as they are (x_{t+1} = x_t, the compute weights are x_{t+1}), but it still counts as an
iteration that consumed a gradient, so k - the bias-correction index, the count of consumed
gradients - advances, and Error Feedback starts once tau gradients have been consumed.  The EF
buffer the skipped iteration would have written keeps its contents (zero before its first write),
and a later iteration reads it as the update formed tau iterations earlier.  The skip is counted
in OptState.n_skipped.  k is therefore t - tau + 1 at every iteration of a delay-tau run, whether
or not earlier gradients were skipped.

With optimizer "muon", u of every 2-D weight matrix of a decoder block is the one of Alg. 2
(Delayed Muon, §4); the embedding and the RMSNorm gains keep AdamW:
    M <- mu M + (1 - mu) g              momentum (the EMA form §3 uses for mu = 0.95)
    O  = Newton-Schulz(M)                approximate orthogonalisation of M
    u  = lr ( s O + wd x_t )             s = rms sqrt(max(rows, cols)), rms = 0.2 (§3)
then the same standard or Error-Feedback step.  Readings where the paper is silent: Newton-Schulz
is the quintic iteration of the Muon write-up (Jordan et al., 2024) - X <- X / (||X||_F + 1e-7),
then 5 times X <- a X + (b A + c A A) X with A = X X^T on the wide orientation (rows <= cols) and
(a, b, c) = (3.4445, -4.7750, 2.0315); every matrix of the block (wq, wk, wv, wo, wgate, wup,
wdown) separately; the momentum takes the clipped gradient and has no bias correction (Newton-
Schulz is invariant to the scale of M); the "update RMS 0.2" scales O to RMS 0.2, the RMS of an
exactly orthogonal m x n matrix being 1 / sqrt(max(m, n)).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np


@dataclass
class HParams:
    lr: float = 1e-3
    beta1: float = 0.9
    beta2: float = 0.95
    eps: float = 1e-8
    weight_decay: float = 0.1
    clip_norm: float = 1.0       # <= 0 disables clipping
    ef_lambda: float = 0.0       # 0: standard async; 1: Error Feedback of §3.2
    delay: int = 1               # 1: Alg. 1; 0: synchronous; tau >= 2: g_{t-tau} with tau-step EF
    optimizer: str = "adamw"     # "adamw", or "muon": Alg. 2 on the blocks' weight matrices
    momentum: float = 0.95       # Muon momentum mu
    update_rms: float = 0.2      # Muon update RMS
    ns_steps: int = 5            # Newton-Schulz iterations
    nadam_psi: float = 0.004     # NAdam momentum decay
    beta3: float = 0.99          # Adan: weight of the second-moment average
    predict: str = "none"        # "updated": SAPipe-WP with the updated optimizer state (AdamW)


# quintic Newton-Schulz coefficients of the Muon write-up (Jordan et al., 2024)
NS_COEFFS = (3.4445, -4.7750, 2.0315)
NS_EPS = 1e-7
MUON_MATRICES = ("wq", "wk", "wv", "wo", "wgate", "wup", "wdown")


def is_muon_matrix(name: str) -> bool:
    """The 2-D weight matrices of a decoder block (names blk<i>.<matrix>)."""
    return name.startswith("blk") and name.split(".")[-1] in MUON_MATRICES


def newton_schulz(M: np.ndarray, steps: int = 5) -> np.ndarray:
    """O ~ U V^T for M = U S V^T (Alg. 2's Newton-Schulz step): normalise by the Frobenius norm,
    then iterate X <- a X + (b A + c A^2) X, A = X X^T, on the orientation with rows <= cols."""
    a, b, c = NS_COEFFS
    X = M / (np.linalg.norm(M) + NS_EPS)
    tall = X.shape[0] > X.shape[1]
    if tall:
        X = X.T
    for _ in range(steps):
        A = X @ X.T
        X = a * X + (b * A + c * (A @ A)) @ X
    return X.T if tall else X


def muon_scale(shape, rms: float) -> float:
    """s with RMS(s O) = rms for an exactly orthogonal O of this shape."""
    return rms * math.sqrt(max(shape))


def muon_u(x, g, M, hp: "HParams"):
    """One Muon evaluation (Alg. 2) on already-clipped g.  Returns (u, M_new)."""
    M1 = hp.momentum * M + (1.0 - hp.momentum) * g
    O = newton_schulz(M1, hp.ns_steps)
    u = hp.lr * (muon_scale(x.shape, hp.update_rms) * O + hp.weight_decay * x)
    return u, M1


def lion_u(x, g, m, hp: "HParams"):
    """One Lion evaluation on already-clipped g.  Returns (u, m_new)."""
    c = hp.beta1 * m + (1.0 - hp.beta1) * g
    u = hp.lr * (np.sign(c) + hp.weight_decay * x)
    return u, hp.beta2 * m + (1.0 - hp.beta2) * g


def nadam_mu(k: int, hp: "HParams") -> float:
    return hp.beta1 * (1.0 - 0.5 * 0.96 ** (k * hp.nadam_psi))


def nadam_u(x, g, m, v, k: int, hp: "HParams"):
    """One NAdam evaluation (k-th update) on already-clipped g.  Returns (u, m_new, v_new)."""
    prod = 1.0
    for j in range(1, k + 1):
        prod *= nadam_mu(j, hp)
    mu, mu_next = nadam_mu(k, hp), nadam_mu(k + 1, hp)
    m1 = hp.beta1 * m + (1.0 - hp.beta1) * g
    v1 = hp.beta2 * v + (1.0 - hp.beta2) * g * g
    denom = np.sqrt(v1 / (1.0 - hp.beta2 ** k)) + hp.eps
    u = hp.lr * ((1.0 - mu) / (1.0 - prod) * g + mu_next / (1.0 - prod * mu_next) * m1) / denom \
        + hp.lr * hp.weight_decay * x
    return u, m1, v1


def adan_u(x, g, m, n, d, g_prev, k: int, hp: "HParams"):
    """One Adan evaluation (k-th update) on already-clipped g.  g_prev is the clipped gradient of the
    previous update (ignored at k = 1, where the difference is zero).  Returns (u, m, n, d, g)."""
    diff = np.zeros_like(g) if k == 1 else g - g_prev
    m1 = hp.beta1 * m + (1.0 - hp.beta1) * g
    d1 = hp.beta2 * d + (1.0 - hp.beta2) * diff
    q = g + hp.beta2 * diff
    n1 = hp.beta3 * n + (1.0 - hp.beta3) * q * q
    denom = np.sqrt(n1 / (1.0 - hp.beta3 ** k)) + hp.eps
    u = hp.lr * ((m1 / (1.0 - hp.beta1 ** k) + hp.beta2 * d1 / (1.0 - hp.beta2 ** k)) / denom
                 + hp.weight_decay * x)
    return u, m1, n1, d1, g.copy()


def global_norm(grads: Dict[str, np.ndarray]) -> float:
    """||g||_2 over every tensor of the stage, accumulated in float64."""
    return math.sqrt(sum(float(np.sum(np.square(g.astype(np.float64)))) for g in grads.values()))


def clip_coefficient(norm: float, clip: float) -> float:
    """c = min(1, clip / (norm + 1e-6)); 1 when clipping is off."""
    if clip <= 0:
        return 1.0
    return min(1.0, clip / (norm + 1e-6))


def adamw_u(x, g, m, v, k: int, hp: HParams):
    """One AdamW evaluation on already-clipped g.  Returns (u, m_new, v_new)."""
    m1 = hp.beta1 * m + (1.0 - hp.beta1) * g
    v1 = hp.beta2 * v + (1.0 - hp.beta2) * g * g
    mhat = m1 / (1.0 - hp.beta1 ** k)
    vhat = v1 / (1.0 - hp.beta2 ** k)
    u = hp.lr * (mhat / (np.sqrt(vhat) + hp.eps) + hp.weight_decay * x)
    return u, m1, v1


def apply_update(x, u, u_prev, ef: bool, lam: float):
    """x_{t+1} from x_t: standard x - u, or the lambda-scaled EF form x - u - lam (u - u_prev)."""
    if ef:
        return x - u - lam * (u - u_prev)
    return x - u


@dataclass
class OptState:
    """Everything Alg. 1 carries from one iteration to the next."""
    x: Dict[str, np.ndarray]
    m: Dict[str, np.ndarray]
    v: Dict[str, np.ndarray]
    u_prev: Dict[str, np.ndarray]           # u_{t-2} at iteration t (zero before any update)
    pending: Optional[Dict[str, np.ndarray]] = None  # g_{t-1}, not yet consumed
    n_updates: int = 0                      # gradients consumed so far (applied or skipped)
    t: int = 0                              # next iteration index
    queue: List[Dict[str, np.ndarray]] = field(default_factory=list)   # delay >= 2: g_{t-tau} .. g_{t-1}
    x_compute: Optional[Dict[str, np.ndarray]] = None  # predict: the weights the next forward uses
    u_ring: List[Dict[str, np.ndarray]] = field(default_factory=list)  # delay >= 2: the last tau updates, oldest first
    n_skipped: int = 0                      # gradients skipped for a non-finite norm
    adan_d: Optional[Dict[str, np.ndarray]] = None      # Adan: average of gradient differences
    adan_gprev: Optional[Dict[str, np.ndarray]] = None  # Adan: clipped gradient of the previous update

    @staticmethod
    def create(x: Dict[str, np.ndarray], dt=np.float64) -> "OptState":
        xx = {k: np.array(v, dtype=dt) for k, v in x.items()}
        z = {k: np.zeros_like(v) for k, v in xx.items()}
        return OptState(xx, {k: v.copy() for k, v in z.items()}, {k: v.copy() for k, v in z.items()},
                        {k: v.copy() for k, v in z.items()})

    def copy(self) -> "OptState":
        cp = lambda d: None if d is None else {k: v.copy() for k, v in d.items()}
        return OptState(x=cp(self.x), m=cp(self.m), v=cp(self.v), u_prev=cp(self.u_prev),
                        pending=cp(self.pending), n_updates=self.n_updates, t=self.t,
                        queue=[cp(g) for g in self.queue], x_compute=cp(self.x_compute),
                        u_ring=[cp(u) for u in self.u_ring], n_skipped=self.n_skipped,
                        adan_d=cp(self.adan_d), adan_gprev=cp(self.adan_gprev))


def iteration_update(st: OptState, g_t: Dict[str, np.ndarray], hp: HParams) -> dict:
    """Second half of iteration t of Alg. 1, after g_t has been computed at x_t.

    Mutates st into the state at iteration t+1 and returns diagnostics (applied, norm, clip)."""
    if hp.delay < 0:
        raise ValueError("delay must be >= 0")
    if hp.delay == 0 and hp.ef_lambda != 0.0:
        raise ValueError("Error Feedback needs a delayed gradient (delay >= 1)")
    if hp.optimizer not in ("adamw", "muon", "lion", "nadam", "adan"):
        raise ValueError("optimizer must be adamw, muon, lion, nadam or adan")
    if hp.predict not in ("none", "updated"):
        raise ValueError("predict must be none or updated")
    if hp.predict == "updated" and (hp.optimizer != "adamw" or hp.ef_lambda != 0.0 or hp.delay != 1):
        raise ValueError("weight prediction is defined here for delay-1 AdamW without Error Feedback")
    if hp.delay >= 2:
        return _iteration_update_tau(st, g_t, hp)
    if hp.delay == 1:
        g_use = st.pending
    else:
        g_use = g_t
    info = dict(applied=False, skipped=False, norm=0.0, clip=1.0)
    if g_use is not None and not math.isfinite(global_norm(g_use)):
        # consumed without effect: x, m, v, u_prev kept; k advances (see the module docstring)
        st.n_updates += 1
        st.n_skipped += 1
        st.x_compute = {n: a.copy() for n, a in st.x.items()} if hp.predict == "updated" else None
        info.update(skipped=True, norm=float("nan"))
    elif g_use is not None:
        norm = global_norm(g_use)
        c = clip_coefficient(norm, hp.clip_norm)
        k = st.n_updates + 1
        ef = hp.ef_lambda != 0.0 and st.n_updates >= 1   # "t <= 1": the first update is standard
        pred = {} if hp.predict == "updated" else None
        for name in st.x:
            u = _u_of(st, name, g_use[name] * c, k, hp)
            st.x[name] = apply_update(st.x[name], u, st.u_prev[name], ef, hp.ef_lambda)
            st.u_prev[name] = u
            if pred is not None:   # the step from the updated state, not kept
                up, _, _ = adamw_u(st.x[name], g_use[name] * c, st.m[name], st.v[name], k + 1, hp)
                pred[name] = st.x[name] - up
        st.x_compute = pred
        st.n_updates = k
        info.update(applied=True, norm=norm, clip=c)
    st.pending = {k: v.copy() for k, v in g_t.items()} if hp.delay == 1 else None
    st.t += 1
    return info


def _u_of(st: OptState, name: str, g, k: int, hp: HParams):
    """u of one parameter from its clipped gradient; updates the optimizer statistics in st."""
    if hp.optimizer == "muon" and is_muon_matrix(name):
        u, st.m[name] = muon_u(st.x[name], g, st.m[name], hp)   # m holds Muon's momentum
    elif hp.optimizer == "lion":
        u, st.m[name] = lion_u(st.x[name], g, st.m[name], hp)
    elif hp.optimizer == "nadam":
        u, st.m[name], st.v[name] = nadam_u(st.x[name], g, st.m[name], st.v[name], k, hp)
    elif hp.optimizer == "adan":
        if st.adan_d is None:
            st.adan_d = {n: np.zeros_like(a) for n, a in st.x.items()}
            st.adan_gprev = {n: np.zeros_like(a) for n, a in st.x.items()}
        u, st.m[name], st.v[name], st.adan_d[name], st.adan_gprev[name] = adan_u(
            st.x[name], g, st.m[name], st.v[name], st.adan_d[name], st.adan_gprev[name], k, hp)
    else:
        u, st.m[name], st.v[name] = adamw_u(st.x[name], g, st.m[name], st.v[name], k, hp)
    return u


def _iteration_update_tau(st: OptState, g_t: Dict[str, np.ndarray], hp: HParams) -> dict:
    """Iteration t with delay tau = hp.delay >= 2: consume g_{t-tau} once tau gradients wait, EF
    against the update formed tau iterations earlier once tau updates exist."""
    tau = hp.delay
    info = dict(applied=False, skipped=False, norm=0.0, clip=1.0)
    if len(st.queue) == tau and not math.isfinite(global_norm(st.queue[0])):
        # consumed without effect; the EF buffer this iteration would write keeps what it holds:
        # the update of iteration t - tau once the ring is full, zero before its first write
        st.queue.pop(0)
        keep = st.u_ring[0] if len(st.u_ring) == tau else {n: np.zeros_like(a) for n, a in st.x.items()}
        st.u_ring.append({n: a.copy() for n, a in keep.items()})
        if len(st.u_ring) > tau:
            st.u_ring.pop(0)
        st.n_updates += 1
        st.n_skipped += 1
        info.update(skipped=True, norm=float("nan"))
    elif len(st.queue) == tau:
        g_use = st.queue.pop(0)
        norm = global_norm(g_use)
        c = clip_coefficient(norm, hp.clip_norm)
        k = st.n_updates + 1
        ef = hp.ef_lambda != 0.0 and len(st.u_ring) == tau
        new_u = {}
        for name in st.x:
            u = _u_of(st, name, g_use[name] * c, k, hp)
            old = st.u_ring[0][name] if ef else None
            st.x[name] = apply_update(st.x[name], u, old, ef, hp.ef_lambda)
            new_u[name] = u
        st.u_ring.append(new_u)
        if len(st.u_ring) > tau:
            st.u_ring.pop(0)
        st.n_updates = k
        info.update(applied=True, norm=norm, clip=c)
    st.queue.append({k: v.copy() for k, v in g_t.items()})
    st.t += 1
    return info


def flat_update(x, g, m, v, u_prev, t: int, hp: HParams, clip_scale: float = 1.0):
    """Elementwise form on flat arrays for a fixed-delay run (tau = hp.delay, at least 1): iteration
    t consumes g (= g_{t-tau}) and u_prev holds the update formed tau iterations earlier.

    t < tau is a no-op; the update is the k = (t - tau + 1)-th; EF applies once tau earlier updates
    exist (k > tau, i.e. t >= 2 tau).  Returns the new (x, m, v, u_prev)."""
    tau = max(hp.delay, 1)
    if t < tau:
        return x, m, v, u_prev
    k = t - tau + 1
    u, m1, v1 = adamw_u(x, g * clip_scale, m, v, k, hp)
    ef = hp.ef_lambda != 0.0 and k > tau
    return apply_update(x, u, u_prev, ef, hp.ef_lambda), m1, v1, u
