"""GPU parity of the whole stage step (forward, backward, delayed update) against the oracle, through
the C ABI.  Tolerances: fp32 workload 1e-4, bf16 workloads 2e-2, relative, norm-wise per tensor
(losses: scalar relative)."""
import numpy as np
import pytest

import datagen
import oracle
from gpu_common import hp_of, log, oracle_grads_at, rel, run_gpu, run_oracle, run_oracle_noisy

pytestmark = pytest.mark.gpu


def _compare(w, g, o, tol, grad_steps, label, lam=1.0, state_tol=None):
    """Free-running trajectories (each side its own x_t): per-step losses (a head's mean CE: scalar
    relative; a middle stage's surrogate sum(Y dY): error relative to sum |Y dY|, the condition of
    the sum), outputs Y and the final master weights at `tol`; final m, v and the EF buffer at
    `state_tol`.  Gradients teacher-forced: the GPU's g_t against the oracle's gradient at the GPU's
    own x_t, at `tol`.  All norm-wise relative; every failure is reported."""
    state_tol = tol if state_tol is None else state_tol
    errs, tols = {}, {}
    for t, (lg, lo) in enumerate(zip(g["losses"], o["losses"])):
        for i, (a, b) in enumerate(zip(lg, lo)):
            scale = abs(b) if w.last_stage else o["loss_abs"][t][i]
            errs[f"loss[{t}][{i}]"] = abs(a - b) / max(scale, 1e-30)
    for t in o["ys"]:
        for i, y in enumerate(o["ys"][t]):
            errs[f"y[{t}][{i}]"] = rel(g["ys"][t][i], y)
    for t in grad_steps:
        ref = oracle_grads_at(w, t, g["x_at"][t])
        for n in ref:
            errs[f"grad[{t}].{n}"] = rel(g["grads"][t][n], ref[n])
    for pre in ("", "m.", "v."):
        for n, ref in o["final"][pre].items():
            k = f"final.{pre}{n}"
            errs[k] = rel(g["final"][pre][n], ref)
            if pre:
                tols[k] = state_tol
    # the update in place: the oracle's rule applied to the GPU's own state before delayed_update(t)
    # and the gradient it consumed, against the GPU's state after it (fp32 vs float64 arithmetic)
    from oracle.update import OptState, iteration_update
    for t, (pre, post) in g.get("upd", {}).items():
        ost = OptState({n: v.astype(np.float64) for n, v in pre[""].items()},
                       {n: v.astype(np.float64) for n, v in pre["m."].items()},
                       {n: v.astype(np.float64) for n, v in pre["v."].items()},
                       {n: v.astype(np.float64) for n, v in pre["u_prev."].items()},
                       pending={n: v.astype(np.float64) for n, v in pre["g"].items()},
                       n_updates=max(t - 1, 0), t=t)
        iteration_update(ost, {n: np.zeros_like(v) for n, v in ost.x.items()}, oracle.hparams_of(w, ef_lambda=lam))
        for key, ref in (("", ost.x), ("m.", ost.m), ("v.", ost.v), ("u_prev.", ost.u_prev)):
            if key == "u_prev." and not lam:
                continue  # standard async keeps no EF buffer
            for n in ref:
                k = f"update[{t}].{key}{n}"
                errs[k] = rel(post[key][n], ref[n])
                tols[k] = 1e-5
    bad = {k: v for k, v in errs.items() if not v <= tols.get(k, tol)}
    worst = sorted(errs, key=errs.get, reverse=True)[:6]
    log(f"{label}: {len(errs)} comparisons; worst " + ", ".join(f"{k}={errs[k]:.2e}" for k in worst))
    assert not bad, f"{label}: {len(bad)} over tolerance: " + ", ".join(f"{k}={v:.2e}" for k, v in sorted(bad.items(), key=lambda kv: -kv[1])[:12])


@pytest.mark.parametrize("lam", [0.0, 1.0])
def test_tiny_fp32_20_steps(lam):
    w = datagen.TINY
    p0 = datagen.init_params(w)
    log(f"tiny fp32 20 steps lambda={lam}")
    g = run_gpu(w, 20, hp_of(w, ef_lambda=lam), p0, grad_steps=(0, 1, 19), upd_steps=(1, 2, 19))
    o = run_oracle(w, 20, oracle.hparams_of(w, ef_lambda=lam), p0, grad_steps=(0, 1, 19))
    _compare(w, g, o, 1e-4, (0, 1, 19), f"tiny lambda={lam}", lam)


@pytest.mark.parametrize("w", ["tiny", "large-reduced"])
def test_overlapped_early_update(w):
    # overlap mode with delayed_update(t) issued before step t's forwards and backwards: the same
    # trajectory (the update of iteration t reads only x_t and g_{t-1})
    w = datagen.TINY if w == "tiny" else LARGE_R
    tol = 1e-4 if w.dtype == "f32" else 2e-2
    steps = 10
    p0 = datagen.init_params(w)
    log(f"{w.name}: {steps} steps, update issued first, overlap mode")
    g = run_gpu(w, steps, hp_of(w), p0, grad_steps=(0, steps - 1), upd_steps=(1, 2, steps - 1), early_update=True)
    o = run_oracle(w, steps, oracle.hparams_of(w), p0, grad_steps=(0, steps - 1))
    _compare(w, g, o, tol, (0, steps - 1), f"{w.name} early update", w.ef_lambda,
             state_tol=None if w.dtype == "f32" else 5e-2)


@pytest.mark.parametrize("case", ["tiny", "tiny-delay2", "tiny-skip", "large-reduced"])
def test_deferred_update_pass_bit_identical(case):
    # overlap mode 2: the update's elementwise pass deferred in chunks launched beside the step's
    # attention backwards gives the trajectory of mode 1 bit for bit (the pass is elementwise), and
    # does run in chunks; with a delay of 2 as well (gradient and EF rings), and with an infinity
    # in the gradient of step 2, whose update every chunk skips
    import torch
    from paper_2606_30634_amd import binding as B
    w = LARGE_R if case == "large-reduced" else datagen.TINY
    hp = hp_of(w, delay=2, ef_lambda=2.0) if case == "tiny-delay2" else hp_of(w)
    steps = 6
    p0 = datagen.init_params(w)
    runs, launches = {}, {}
    for mode in (1, 2):
        def hook(t, st, mode=mode):
            if case == "tiny-skip" and t == 2:
                torch.cuda.synchronize()
                st.view(f"grad0.{next(iter(p0))}")[5] = float("inf")
                torch.cuda.synchronize()
            if t == 0:
                B.stage_profile_enable(st.handle, True)
            if t == steps - 2:
                launches[mode] = B.stage_profile_read(st.handle, B.PROF_UPDATE)[1]
        log(f"{w.name}: {steps} steps, update issued first, overlap mode {mode}")
        runs[mode] = run_gpu(w, steps, hp, p0, grad_steps=(0, steps - 1), y_steps=(0, steps - 1),
                             upd_steps=(2, 3, steps - 1), early_update=True, overlap_mode=mode, after_backward=hook)
    a, b = runs[1], runs[2]
    log(f"{w.name}: update launches over iterations 1..{steps - 2}: mode 1 {launches[1]}, mode 2 {launches[2]}")
    assert launches[1] == steps - 2 and launches[2] >= 2 * launches[1]
    assert a["skipped"] == b["skipped"] == (1 if case == "tiny-skip" else 0)
    assert a["losses"] == b["losses"]
    for t in a["ys"]:
        for ya, yb in zip(a["ys"][t], b["ys"][t]):
            assert np.array_equal(ya, yb), f"output of step {t}"
    for pre in ("", "m.", "v.", "u_prev."):
        for n in p0:
            assert np.array_equal(a["final"][pre][n], b["final"][pre][n]), f"final {pre}{n}"
    for t in a["upd"]:
        for k in a["upd"][t][1]:
            for n in p0:
                assert np.array_equal(a["upd"][t][1][k][n], b["upd"][t][1][k][n]), f"state {k}{n} after update {t}"


@pytest.mark.parametrize("lam", [0.0, 1.0])
def test_tiny_fp32_untied_last_stage(lam):
    # a last stage that is not the first: input activations, given targets, its own head matrix
    w = TINY_LAST
    p0 = datagen.init_params(w)
    log(f"{w.name} 12 steps lambda={lam}")
    g = run_gpu(w, 12, hp_of(w, ef_lambda=lam), p0, grad_steps=(0, 1, 11), upd_steps=(1, 2, 11))
    o = run_oracle(w, 12, oracle.hparams_of(w, ef_lambda=lam), p0, grad_steps=(0, 1, 11))
    _compare(w, g, o, 1e-4, (0, 1, 11), f"{w.name} lambda={lam}", lam)


TINY_LAST = datagen.TINY.with_(name="tiny-last-untied", first_stage=False, tie_embedding=False, seed=21)

# Reduced bf16 stages: the shapes of the bf16 workloads at sizes the oracle finishes in seconds,
# with ragged sequence lengths (not multiples of 64) and GQA.
SMALL_R = datagen.SMALL.with_(name="small-reduced", n_blocks=2, d_model=256, n_heads=4, n_kv_heads=4,
                              head_dim=64, d_ffn=512, vocab=1000, seq_len=96, micro_batch=2)
MID_R = datagen.MID.with_(name="mid-reduced", n_blocks=2, d_model=256, n_heads=2, n_kv_heads=2,
                          head_dim=128, d_ffn=640, seq_len=80, micro_batch=2)
LARGE_R = datagen.LARGE.with_(name="large-reduced", n_blocks=2, d_model=256, n_heads=4, n_kv_heads=2,
                              head_dim=64, d_ffn=384, seq_len=72, micro_batch=2,
                              microbatches_per_step=4, max_inflight=3)
# whole 128-token tiles (256 tokens per microbatch): the full-tile GEMM kernels with their fused
# epilogues (RoPE, SwiGLU forward and backward) at a size the oracle finishes in seconds
TILED_R = datagen.SMALL.with_(name="small-full-tiles", n_blocks=2, d_model=256, n_heads=4, n_kv_heads=4,
                              head_dim=64, d_ffn=512, vocab=1000, seq_len=128, micro_batch=2)


# the last stage with its own head: an odd vocabulary (scalar cross-entropy path, ragged head
# products), and whole tiles (vocab 4096, 256 tokens)
LAST_R = datagen.LAST.with_(name="last-reduced", n_blocks=2, d_model=256, n_heads=4, n_kv_heads=2,
                            head_dim=64, d_ffn=512, vocab=4001, seq_len=96, micro_batch=2)
LAST_TILED_R = datagen.LAST.with_(name="last-full-tiles", n_blocks=1, d_model=256, n_heads=4, n_kv_heads=4,
                                  head_dim=64, d_ffn=512, vocab=4096, seq_len=128, micro_batch=2)


# the mid and large widths (d 2048, 4096: the column-split RMSNorm backward) with a ragged token
# count (not a multiple of the 16 rows a block of the norm kernels covers)
WIDE_MID_R = datagen.MID.with_(name="mid-width-reduced", n_blocks=1, d_model=2048, n_heads=16, n_kv_heads=16,
                               head_dim=128, d_ffn=512, seq_len=45, micro_batch=2)
WIDE_LARGE_R = datagen.LARGE.with_(name="large-width-reduced", n_blocks=1, d_model=4096, n_heads=32, n_kv_heads=8,
                                   head_dim=128, d_ffn=512, seq_len=41, micro_batch=2,
                                   microbatches_per_step=2, max_inflight=2)


def _noise_envelope(w, steps, p0, g, o, label):
    # against the method's own sensitivity: the final weights, moments and EF buffer at most 1.5
    # times as far (median over the parameters) from the float64 run as the float64 run with
    # gradient noise of bf16 size ends up
    noisy = run_oracle_noisy(w, steps, oracle.hparams_of(w), p0)
    ratios = {}
    for pre in ("", "m.", "v.", "u_prev."):
        ge = [rel(g["final"][pre][n], o["final"][pre][n]) for n in p0]
        ne = [rel(noisy[pre][n], o["final"][pre][n]) for n in p0]
        ratios[pre or "x."] = float(np.median(ge)) / float(np.median(ne))
    log(f"{label}, final median error / noise-perturbed oracle's: " +
        ", ".join(f"{k[:-1]}={r:.2f}" for k, r in ratios.items()))
    assert all(r <= 1.5 for r in ratios.values()), ratios


@pytest.mark.parametrize("w", [SMALL_R, MID_R, LARGE_R, TILED_R, LAST_R, LAST_TILED_R, WIDE_MID_R, WIDE_LARGE_R],
                         ids=lambda w: w.name)
def test_reduced_bf16_stages(w):
    steps = 12
    p0 = datagen.init_params(w)
    log(f"{w.name}: {steps} steps")
    ys = (0, steps - 1) if not w.last_stage else ()
    g = run_gpu(w, steps, hp_of(w), p0, grad_steps=(0, 1, steps - 1), y_steps=ys, upd_steps=(1, 2, steps - 1))
    o = run_oracle(w, steps, oracle.hparams_of(w), p0, grad_steps=(0, 1, steps - 1), y_steps=ys)
    # bf16 free-running optimizer state: Adam turns noise-level gradient differences into lr-sized
    # differences of m / sqrt(v) wherever a gradient element is near zero, so m and v drift further
    # than the weights; they are held to 5e-2.  The EF buffer (the last update, sign-like wherever a
    # gradient is at noise level) is checked teacher-forced, and with the rest of the final state
    # against the noise-perturbed oracle run.
    _compare(w, g, o, 2e-2, (0, 1, steps - 1), w.name, state_tol=5e-2)
    _noise_envelope(w, steps, p0, g, o, f"{w.name} {steps} steps")


@pytest.mark.parametrize("w", [SMALL_R, MID_R, LARGE_R, LAST_R], ids=lambda w: w.name)
def test_reduced_bf16_100_steps(w):
    # the bf16 bar over 100 delay-1 steps with Error Feedback: every step's loss, the final weights
    # and the teacher-forced gradients of steps 0 and 99 at 2e-2; the update in place of steps 1
    # and 99 at 1e-5.  The free-running m, v are each side's average of its own recent gradients,
    # taken at weights that differ by up to 2e-2: over 100 steps the small attention-weight
    # gradients (a sum over tokens that largely cancels) differ by several percent there, so m, v
    # are held to 1e-1.
    steps = 100
    p0 = datagen.init_params(w)
    log(f"{w.name}: {steps} steps")
    g = run_gpu(w, steps, hp_of(w), p0, grad_steps=(0, steps - 1), upd_steps=(1, steps - 1))
    o = run_oracle(w, steps, oracle.hparams_of(w), p0, grad_steps=(0, steps - 1))
    _compare(w, g, o, 2e-2, (0, steps - 1), f"{w.name} 100 steps", state_tol=1e-1)
    _noise_envelope(w, steps, p0, g, o, f"{w.name} 100 steps")
