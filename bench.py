"""Stage throughput of the delay-1 training step on one MI355X.

One step = one pass of the whole hot path over one optimizer step's input: delayed_update(t)
(Alg. 1 with AdamW, Error Feedback lambda = 1, global-norm clipping at 1.0; it consumes g_{t-1}
and is issued first, in the stage's overlap mode, so that it runs beside the step's work), then
stage_forward and stage_backward of every microbatch of step t.  Default workload: the large bf16
stage (4 decoder blocks, d_model 4096, 32 query / 8 key-value heads of 128, SwiGLU 14336, seq 4096,
microbatch 2, eight microbatches per optimizer step in a 1F1B order with 4 activation slots:
65536 tokens per step), synthetic seeded inputs already resident in HBM.  Prints one JSON line.

  python bench.py [--steps K] [--warmup W] [--workload large|mid|small|tiny|last] [--no-cpu-baseline]
                  [--optimizer adamw|muon|lion|nadam|adan] [--predict] [--delay TAU] [--vocab V]

With --optimizer muon the blocks' weight matrices take delayed Muon (Alg. 2: momentum 0.95, five
quintic Newton-Schulz steps, update RMS 0.2) with Error Feedback lambda = 1, the embedding and gains
AdamW; the line then also reports the Newton-Schulz GEMMs as their own kernel class.  --delay TAU
(default 1) runs the fixed delay TAU of App. C (g_{t-TAU} consumed, Error Feedback lambda = TAU
against the update formed TAU iterations earlier).  --workload last is the last stage of the small
model's shape with its own LM head (vocab 49152; --vocab V sets another, e.g. 128256).  --optimizer
lion|nadam|adan and --predict (AdamW with SAPipe weight prediction from the updated state) select the
elementwise variants of the update, also for the update-only workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3    # MI355X fp32 vector
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def kernel_sources_sha256():
    """SHA-256 over the HIP sources of the library (file names and contents, in name order)."""
    import hashlib
    h = hashlib.sha256()
    d = os.path.join(ROOT, "paper_2606_30634_amd", "csrc")
    for name in sorted(os.listdir(d)):
        if name.endswith((".hip", ".h")):
            h.update(name.encode())
            with open(os.path.join(d, name), "rb") as f:
                h.update(f.read())
    return h.hexdigest()


def measured_traffic(workload, kernel_class):
    """HBM bytes per launch of a kernel class from the committed rocprofv3 --pmc summary of this
    workload (FETCH_SIZE and WRITE_SIZE, scaled by a plain copy's counters), or None when there is
    none or the kernel sources changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", f"hbm_traffic_{workload}.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    start = text.find("```json")
    if start < 0:
        return None
    end = text.find("```", start + 7)
    try:
        rec = json.loads(text[start + 7:end])
    except ValueError:
        return None
    if rec.get("sources_sha256") != kernel_sources_sha256():
        return None
    v = rec.get("bytes_per_launch", {}).get(kernel_class)
    return float(v) if v is not None else None


def measured_mfma(workload, kernel_class):
    """Counter-based matrix-core utilisation of a kernel class from the committed rocprofv3 --pmc summary of
    this workload (SQ_VALU_MFMA_BUSY_CYCLES over the dispatch's cycles at the measured clock), or None when
    there is none or the kernel sources changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", f"mfma_util_{workload}.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    start = text.find("```json")
    if start < 0:
        return None
    try:
        rec = json.loads(text[start + 7:text.find("```", start + 7)])
    except ValueError:
        return None
    if rec.get("sources_sha256") != kernel_sources_sha256():
        return None
    return rec.get("classes", {}).get(kernel_class)


def cpu_baseline(w, optimizer="adamw", predict=False):
    """The oracle (float32, numpy) timed on the machine's host cores.  A stage of width <= 1024: whole
    optimizer steps of the workload -- all sequences forward+backward, then the full delayed update --
    repeated until at least 10 s of CPU work (at most 4 steps).  A wider stage, whose step is hours of
    CPU work: one decoder block forward+backward on one sequence (the unit every block and sequence of
    the step repeats) and the delayed update on a 2^24-element slice of the flat vector (elementwise),
    each repeated until a few seconds, scaled to the step's blocks, sequences and parameters."""
    import numpy as np
    import datagen
    import oracle
    from oracle import model
    from oracle.update import OptState, iteration_update
    try:
        from threadpoolctl import threadpool_info
        cores = max(i.get("num_threads", 1) for i in threadpool_info()) or os.cpu_count()
    except Exception:
        cores = os.cpu_count()
    kw = update_rule(optimizer, predict)
    tokens_step = w.tokens_per_micro * w.microbatches_per_step
    n_params = sum(int(np.prod(s)) for _, s, _ in datagen.param_specs(w))
    if w.d_model > 1024:
        ws = w.with_(n_blocks=1, micro_batch=1, microbatches_per_step=1)
        p0 = {k: v.astype(np.float32) for k, v in datagen.init_params(ws).items()}
        inp = datagen.step_inputs(ws, 0)
        fb_s, reps = 0.0, 0
        while reps < 3 and (reps == 0 or fb_s < 8.0):
            t0 = time.perf_counter()
            model.stage_step_grads(p0, [inp], ws, np.float32)
            fb_s += time.perf_counter() - t0
            reps += 1
        n = 1 << 24
        rule = dict(kw, optimizer="adamw") if optimizer == "muon" else kw   # Muon's matrices: not elementwise
        hp = oracle.hparams_of(w, **(dict(rule, ef_lambda=0.0) if predict else rule))
        st = OptState.create({"flat": np.random.default_rng(0).standard_normal(n).astype(np.float32) * 0.02},
                             np.float32)
        g = {"flat": np.random.default_rng(1).standard_normal(n).astype(np.float32) * 1e-3}
        iteration_update(st, g, hp)
        upd_s, ureps = 0.0, 0
        while ureps < 8 and (ureps == 0 or upd_s < 2.0):
            t0 = time.perf_counter()
            iteration_update(st, g, hp)
            upd_s += time.perf_counter() - t0
            ureps += 1
        seqs = w.micro_batch * w.microbatches_per_step
        fb_step = fb_s / reps * w.n_blocks * seqs
        upd_step = upd_s / ureps * n_params / n
        step_s = fb_step + upd_step
        return {"value": tokens_step / step_s, "unit": "tokens/s", "cores": int(cores), "kind": "oracle",
                "sample": f"float32 numpy oracle: one decoder block forward+backward on one {w.seq_len}-token "
                          f"sequence ({fb_s / reps:.1f} s, {reps} reps) x {w.n_blocks} blocks x {seqs} sequences "
                          f"per step, plus the delayed update ({hp.optimizer} + Error Feedback) on a 2^24-element slice "
                          f"({upd_s / ureps:.2f} s, {ureps} reps) x {n_params / n:.1f} for {n_params} parameters; "
                          f"{step_s:.0f} s per step extrapolated",
                "measured_s": round(fb_s + upd_s, 2)}
    n_seq = w.micro_batch
    ws = w.with_(micro_batch=n_seq)
    p0 = datagen.init_params(ws)
    hp = oracle.hparams_of(ws, **(dict(kw, ef_lambda=0.0) if predict else kw))
    st = OptState.create(p0, np.float32)
    inp = datagen.step_inputs(ws, 0)
    g, _ = model.stage_step_grads(st.x, [inp], ws, np.float32)
    iteration_update(st, g, hp)   # t = 0: stashes g_0 (no arithmetic), untimed
    fb_s, upd_s, reps = 0.0, 0.0, 0
    while reps < 4 and (reps == 0 or fb_s + upd_s < 10.0):
        t0 = time.perf_counter()
        g, _ = model.stage_step_grads(st.x, [inp], ws, np.float32)
        t1 = time.perf_counter()
        iteration_update(st, g, hp)   # the full optimizer + clip + EF pass
        t2 = time.perf_counter()
        fb_s += t1 - t0
        upd_s += t2 - t1
        reps += 1
    fb_per_token = fb_s / reps / (n_seq * w.seq_len)
    step_s = fb_per_token * tokens_step + upd_s / reps
    whole = n_seq * w.seq_len == tokens_step
    how = (f"{reps} whole optimizer steps" if whole else
           f"{reps} steps, extrapolated linearly in tokens to {tokens_step} tokens per step")
    return {"value": tokens_step / step_s, "unit": "tokens/s", "cores": int(cores), "kind": "oracle",
            "sample": f"float32 numpy oracle: {n_seq} of the step's {w.micro_batch * w.microbatches_per_step} "
                      f"sequences forward+backward ({fb_s / reps:.1f} s per step) plus the full delayed update "
                      f"over {n_params} parameters ({upd_s / reps:.1f} s per step); {how}",
            "measured_s": round(fb_s + upd_s, 2)}


def update_rule(optimizer, predict):
    """Keyword arguments of the update rule (hparams) for the optimizer options of this script."""
    kw = {"lion": dict(optimizer="lion", beta1=0.9, beta2=0.99, weight_decay=0.5),
          "nadam": dict(optimizer="nadam", beta2=0.999),
          "adan": dict(optimizer="adan", beta1=0.98, beta2=0.92, beta3=0.99)}.get(optimizer, dict(optimizer=optimizer))
    if predict:
        kw.update(predict="updated")
    return kw


def update_workload(steps, optimizer="adamw", predict=False):
    """The update-only workload: delayed_update_flat over a flat 1.0e9-element fp32 vector (x, m, v,
    EF buffer), one bf16 gradient N(0, 1e-3), bf16 compute copy; `steps` iterations timed with HIP
    events on the stream, clipping off: 36 algorithmic bytes per element (Lion, which keeps no v: 28;
    the weight prediction, which has no EF buffer: 28).  Then the same with clipping at 1.0: the
    gradient's norm pass (grad_norm_flat, 2 more bytes per element) before every update.  The
    library's streaming copy (hbm_stream_copy, 16-byte non-temporal accesses) of x's 4.0e9 bytes is timed
    in the same process as the practical HBM ceiling."""
    import torch
    from paper_2606_30634_amd import binding as B
    from paper_2606_30634_amd.stage import hparams
    n = 1_000_000_000
    dev = torch.device("cuda:0")
    gen = torch.Generator(device=dev)
    gen.manual_seed(5)
    x = torch.randn(n, device=dev, generator=gen).mul_(0.02)
    g = torch.randn(n, device=dev, generator=gen).mul_(1e-3).to(torch.bfloat16)
    m = torch.zeros(n, device=dev)
    v = torch.zeros(n, device=dev)
    up = torch.zeros(n, device=dev)
    sh = torch.empty(n, device=dev, dtype=torch.bfloat16)
    kw = update_rule(optimizer, predict)
    lam = 0.0 if predict else 1.0
    hp = hparams(lr=1e-3, ef_lambda=lam, clip_norm=0.0, **kw)
    hp_clip = hparams(lr=1e-3, ef_lambda=lam, clip_norm=1.0, **kw)
    adan = optimizer == "adan"
    bpe = 2 + 2 + 8 + 8 + (0 if optimizer == "lion" else 8) + (8 if lam else 0) + (16 if adan else 0)
    d = torch.zeros(n, device=dev) if adan else None
    gl = torch.zeros(n, device=dev) if adan else None
    stream = torch.cuda.current_stream(dev)
    ws_bytes = B.grad_norm_flat_workspace_bytes()
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    norm_out = torch.zeros(2, device=dev)
    flag = torch.zeros(1, dtype=torch.int32, device=dev)
    if adan:
        call = lambda t, h, c: B.delayed_update_flat_adan(n, x.data_ptr(), g.data_ptr(), True, m.data_ptr(),
                                                          v.data_ptr(), d.data_ptr(), gl.data_ptr(), up.data_ptr(),
                                                          sh.data_ptr(), True, t, h, c, stream.cuda_stream)
    else:
        call = lambda t, h, c: B.delayed_update_flat(n, x.data_ptr(), g.data_ptr(), True, m.data_ptr(),
                                                     v.data_ptr(), up.data_ptr(), sh.data_ptr(), True, t, h, c,
                                                     stream.cuda_stream)
    norm = lambda: B.grad_norm_flat(n, g.data_ptr(), True, 1.0, norm_out.data_ptr(), flag.data_ptr(),
                                    ws.data_ptr(), ws_bytes, stream.cuda_stream)
    log(f"bench: update-only workload, {n} elements, {steps} iterations without and with the norm pass")
    call(1, hp, None)  # warm-up (t = 1: a real update)
    torch.cuda.synchronize(dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for t in range(2, 2 + steps):
        call(t, hp, None)
    e1.record(stream)
    torch.cuda.synchronize(dev)
    ms = e0.elapsed_time(e1) / steps
    gbs = bpe * n / (ms * 1e-3) / 1e9
    e0.record(stream)
    for t in range(2 + steps, 2 + 2 * steps):
        norm()
        call(t, hp_clip, norm_out.data_ptr() + 4)
    e1.record(stream)
    torch.cuda.synchronize(dev)
    ms_clip = e0.elapsed_time(e1) / steps
    gbs_clip = (bpe + 2) * n / (ms_clip * 1e-3) / 1e9
    del g, m, v, up, sh, d, gl
    src = x.view(torch.uint8)          # the 4.0e9 bytes of x
    nb = src.numel() // 16 * 16
    dst = torch.empty(nb, dtype=torch.uint8, device=dev)
    if src.numel() < nb or dst.numel() < nb:
        raise RuntimeError("copy ceiling: buffers smaller than the copy")
    log(f"bench: streaming-copy ceiling, {nb} bytes")
    B.hbm_stream_copy(dst.data_ptr(), src.data_ptr(), nb, stream.cuda_stream)
    torch.cuda.synchronize(dev)
    e0.record(stream)
    for _ in range(5):
        B.hbm_stream_copy(dst.data_ptr(), src.data_ptr(), nb, stream.cuda_stream)
    e1.record(stream)
    torch.cuda.synchronize(dev)
    copy_gbs = 2.0 * nb / (e0.elapsed_time(e1) / 5 * 1e-3) / 1e9
    return {"elements": n, "steps": steps, "rule": kw, "ef_lambda": lam, "bytes_per_element": bpe,
            "ms_per_step": round(ms, 4),
            "achieved_GBs": round(gbs, 1), "peak_GBs": PEAK_HBM_GBS, "frac": round(gbs / PEAK_HBM_GBS, 4),
            "stream_copy_GBs": round(copy_gbs, 1), "frac_of_copy": round(gbs / copy_gbs, 4),
            "with_clip_norm": {"bytes_per_element": bpe + 2, "ms_per_step": round(ms_clip, 4),
                               "achieved_GBs": round(gbs_clip, 1), "frac": round(gbs_clip / PEAK_HBM_GBS, 4),
                               "frac_of_copy": round(gbs_clip / copy_gbs, 4)}}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="large")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--optimizer", choices=("adamw", "muon", "lion", "nadam", "adan"), default="adamw")
    ap.add_argument("--predict", action="store_true",
                    help="AdamW with SAPipe weight prediction from the updated state (no Error Feedback)")
    ap.add_argument("--delay", type=int, default=1)
    ap.add_argument("--vocab", type=int, default=0, help="head vocabulary of a last-stage workload")
    ap.add_argument("--update-steps", type=int, default=50,
                    help="iterations of the update-only workload (1.0e9 fp32 elements); 0 skips it")
    ap.add_argument("--overlap-mode", type=int, choices=(1, 2), default=None,
                    help="update overlap mode (2: the update's elementwise pass in chunks beside the "
                         "attention backwards); default 2 for the large and mid workloads, else 1")
    ap.add_argument("--calib-copy", action="store_true",
                    help="run one plain 1 GiB device-to-device copy first (a known-size reference for "
                         "the FETCH_SIZE / WRITE_SIZE counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the library runs one pipeline stage's share on one MI355X "
              "and has no multi-GPU path; run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    import datagen
    from paper_2606_30634_amd import binding as B
    from paper_2606_30634_amd.stage import Stage, hparams, make_shape

    w = datagen.WORKLOADS[args.workload]
    if args.vocab:
        if not w.last_stage or w.first_stage:
            print("--vocab applies to a last-stage workload", file=sys.stderr)
            sys.exit(2)
        w = w.with_(vocab=args.vocab, name=w.name.replace(f"vocab{w.vocab}", f"vocab{args.vocab}"))
    muon = args.optimizer == "muon"
    dev = torch.device("cuda:0")
    bf = w.dtype == "bf16"
    st = Stage(make_shape(w.n_blocks, w.d_model, w.n_heads, w.n_kv_heads, w.head_dim, w.d_ffn, w.vocab,
                          w.first_stage, w.last_stage, w.tie_embedding, w.seq_len, w.micro_batch,
                          w.max_inflight, bf16=bf, rms_eps=w.rms_eps, rope_theta=w.rope_theta,
                          muon=muon, max_delay=args.delay, adan=args.optimizer == "adan"), "cuda:0")
    st.load_master(datagen.init_params(w))
    if args.predict and (args.optimizer != "adamw" or args.delay != 1):
        print("--predict applies to AdamW at delay 1", file=sys.stderr)
        sys.exit(2)
    lam = 0.0 if args.predict else float(args.delay)
    hp = hparams(**dict(dict(lr=w.lr, beta1=w.beta1, beta2=w.beta2, eps=w.eps, weight_decay=w.weight_decay,
                             clip_norm=w.clip_norm, ef_lambda=lam, delay=args.delay),
                        **update_rule(args.optimizer, args.predict)))
    M = w.microbatches_per_step
    cdt = torch.bfloat16 if bf else torch.float32
    # two distinct input sets per microbatch, resident in HBM, alternated across steps
    sets = []
    for k in range(2):
        per = []
        for i in range(M):
            inp = datagen.step_inputs(w, k, i)
            d = {}
            for name, v in inp.items():
                t = torch.from_numpy(v)
                d[name] = t.to(dev) if v.dtype == np.int32 else t.to(dev).to(cdt)
            if not w.last_stage:
                d["y"] = torch.empty(w.micro_batch, w.seq_len, w.d_model, dtype=cdt, device=dev)
            d["loss"] = torch.zeros(1, device=dev)
            per.append(d)
        sets.append(per)
    warm = max(0, min(w.max_inflight - 1, M))

    # overlap mode: delayed_update(t) - it reads x_t and g_{t-1} only - is issued before step t's
    # forwards and backwards and runs beside them on the stage's update stream.  Mode 2 runs its
    # elementwise pass in chunks beside the step's attention backwards instead of beside the first
    # forwards' products: measured 351-352 against 358-359 ms per step on the large workload and
    # 14.9-15.0 against 15.1 on the mid one, while the small workload's attention backwards (under
    # 0.2 ms) slow by more than the pass saves (2.89 against 2.83 ms).
    mode = args.overlap_mode or (2 if args.workload in ("large", "mid") and not muon else 1)
    st.set_update_overlap(mode)

    def step(t):
        st.update(t, hp)
        per = sets[t % 2]
        order, f, b = [], 0, 0
        for _ in range(warm):
            order.append(("F", f)); f += 1
        while b < M:
            if f < M:
                order.append(("F", f)); f += 1
            order.append(("B", b)); b += 1
        for kind, i in order:
            d = per[i]
            slot = i % w.max_inflight
            if kind == "F":
                st.forward(slot, t, tokens=d.get("tokens"), x_in=d.get("x_in"), targets=d.get("targets"),
                           y_out=d.get("y"), loss=d["loss"] if w.last_stage else None)
            else:
                st.backward(slot, dy=d.get("dy"), microbatches_per_step=M)

    if args.calib_copy:
        src = torch.ones(1 << 28, dtype=torch.float32, device=dev)   # 1 GiB
        dst = torch.empty_like(src)
        torch.cuda.synchronize(dev)
        dst.copy_(src)
        torch.cuda.synchronize(dev)
        del src, dst
    t = 0
    log(f"bench: {w.name}: warmup {args.warmup}")
    for _ in range(args.warmup):
        step(t); t += 1
    torch.cuda.synchronize(dev)
    stream = st.stream
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    log(f"bench: timing {args.steps} steps")
    wall0 = time.perf_counter()
    e0.record(stream)
    for _ in range(args.steps):
        step(t); t += 1
    st.join_update()   # the last update is part of the timed work
    e1.record(stream)
    torch.cuda.synchronize(dev)
    wall = time.perf_counter() - wall0
    ms = e0.elapsed_time(e1) / args.steps
    tokens = w.tokens_per_micro * M
    value = tokens / (ms * 1e-3)

    # kernel-class timing pass: HIP event pairs around every launch, on the stage's stream
    log("bench: kernel-class timing pass")
    B.stage_profile_enable(st.handle, True)
    for _ in range(args.steps):
        step(t); t += 1
    classes = {"gemm": B.PROF_GEMM, "attention_fwd": B.PROF_ATTN_FWD, "attention_bwd": B.PROF_ATTN_BWD,
               "delayed_update": B.PROF_UPDATE, "grad_norm": B.PROF_NORM, "newton_schulz": B.PROF_NS}
    kern = {}
    for name, c in classes.items():
        kms, n, work = B.stage_profile_read(st.handle, c)
        if n == 0:
            continue
        per_launch_ms = kms / n
        if c in (B.PROF_UPDATE, B.PROF_NORM):
            ach = work / (kms * 1e-3) / 1e9
            kern[name] = {"bound": "hbm", "ms_per_step": round(kms / args.steps, 4), "launches": n,
                          "avg_launch_ms": round(per_launch_ms, 4), "achieved": round(ach, 1),
                          "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(ach / PEAK_HBM_GBS, 4),
                          "work_per_launch": work / n}
        else:
            ach = work / (kms * 1e-3) / 1e12
            peak = PEAK_BF16_TFLOPS if bf else PEAK_FP32_TFLOPS
            kern[name] = {"bound": "mfma" if bf else "alu", "ms_per_step": round(kms / args.steps, 4),
                          "launches": n, "avg_launch_ms": round(per_launch_ms, 4), "achieved": round(ach, 1),
                          "peak": peak, "unit": "TFLOP/s", "frac": round(ach / peak, 4),
                          "work_per_launch": work / n}
    B.stage_profile_enable(st.handle, False)
    if mode == 2 and "delayed_update" in kern and kern["delayed_update"]["launches"] > args.steps:
        # its chunks share the chip with the attention backwards by design; the pass's own HBM
        # roofline is the update-only workload's
        kern["delayed_update"]["note"] = ("elementwise pass in chunks beside the attention backwards (overlap "
                                          "mode 2); the pass alone: update_workload")
    dom = max(kern, key=lambda k: kern[k]["ms_per_step"])
    kd = kern[dom]
    roofline = {"kernel": dom, "bound": kd["bound"], "achieved": kd["achieved"], "peak": kd["peak"],
                "unit": kd["unit"], "frac": kd["frac"],
                "traffic": None if args.vocab else measured_traffic(args.workload + ("-bf16" if bf else "-f32"), dom)}
    mc = None if args.vocab or args.optimizer != "adamw" else measured_mfma(args.workload + ("-bf16" if bf else "-f32"), dom)
    if mc:
        roofline["mfma_busy"] = mc.get("busy")
        roofline["mfma_busy_clock_GHz"] = mc.get("clock")
    rc, skipped = B.stage_poll_nonfinite(st.handle)
    st.close()

    upd = (update_workload(args.update_steps, args.optimizer, args.predict)
           if args.update_steps > 0 and not muon else None)

    cpu = None
    if not args.no_cpu_baseline:
        log("bench: CPU oracle baseline")
        cpu = cpu_baseline(w, args.optimizer, args.predict)

    out = {
        "metric": "stage tokens/sec (fwd+bwd+delayed update)",
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if bf else "f32",
        "data": "synthetic (seeded: uniform tokens / N(0,1) activations, N(0,1e-3) upstream gradients, N(0,0.02) weights)",
        "config": {"workload": w.name, "tokens_per_step": tokens, "microbatches_per_step": M,
                   "optimizer": ("Muon (momentum 0.95, 5 Newton-Schulz steps, update RMS 0.2) on the block "
                                 "matrices, AdamW elsewhere" if muon else
                                 {"adamw": "AdamW", "lion": "Lion (betas 0.9, 0.99; wd 0.5)",
                                  "nadam": "NAdam (betas 0.9, 0.999)",
                                  "adan": "Adan (betas 0.98, 0.92, 0.99)"}[args.optimizer]) +
                                (" with SAPipe weight prediction (updated state)" if args.predict else "") +
                                f", delay {args.delay}, Error Feedback lambda {lam:g}, clip 1.0",
                   "update_overlap_mode": mode,
                   "parallelism": "1 GPU, one stage"},
        "roofline": roofline,
        "kernels": kern,
        "update_workload": upd,
        "cpu_baseline": cpu,
        "wall_s_timed_region": round(wall, 3),
        "skipped_updates": skipped,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
