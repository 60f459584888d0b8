#!/usr/bin/env python3
"""Control steps/s of the Gated VLA-Cache hot path on one MI355X.

One control step (Alg. 1) on a Llama-2-7B-shaped VLA decoder with random
bf16 weights and seeded synthetic frames:
  margin gate on the previous step's margins  ->  Stage 1 static-patch
  selection  ->  prompt pass over the recomputed rows only  ->  7-token
  autoregressive action decode.
The workload keeps the cache at every step (the gate is evaluated and its
decision reported, but not applied), so every timed step reuses exactly the
128 static patches of 256 (50%).

Prints one JSON line.  --gpus N with N > 1 is refused: the path runs on one GPU.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
# sources of the dominant kernel; its stored traffic figure is used only while they are unchanged
KERNEL_SOURCES = ("paper_2608_10824_amd/csrc/k_decode.hip", "paper_2608_10824_amd/csrc/gvc_kernels.h",
                  "paper_2608_10824_amd/csrc/gvc_decode.h")
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA


def note(msg):
    """Progress of the run itself, on stderr (the JSON line stays alone on stdout)."""
    print("[bench] %s" % msg, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-c3", action="store_true", help="skip the C3 episode (recompute rate)")
    ap.add_argument("--no-c4", action="store_true", help="skip the C4 action-chunk queries")
    ap.add_argument("--no-vit", action="store_true", help="skip the steps with the ViT front end")
    ap.add_argument("--no-c5", action="store_true", help="skip the batch-16 prompt passes")
    ap.add_argument("--no-stage2", action="store_true",
                    help="skip the Stage 2 (top-k = 120) and Stage 2 + entropy Stage 3 steps")
    ap.add_argument("--no-fired", action="store_true", help="skip the C2 steps whose gate fires (full recompute)")
    ap.add_argument("--trace-jsonl", default="",
                    help="also write the C3 episode's per-step trace to this file, one JSON object per line")
    ap.add_argument("--c5-static", default="0,64,128,192,230",
                    help="static patches per episode of the C5 passes to time (comma-separated)")
    return ap.parse_args()


def layer_weight_bytes(cfg):
    d, F = cfg.d_model, cfg.ffn
    return (4 * d * d + 3 * d * F) * 2


def _blas_info():
    """BLAS library and thread count NumPy uses (threadpoolctl's view)."""
    try:
        from threadpoolctl import threadpool_info
        for i in threadpool_info():
            if i.get("user_api") == "blas":
                return {"blas": "%s %s" % (i.get("internal_api"), i.get("version")), "blas_threads": i.get("num_threads")}
    except Exception:   # pragma: no cover - threadpoolctl missing
        pass
    return {"blas": "unknown", "blas_threads": None}


def cpu_baseline(cfg, oracle, si):
    """The oracle timed over one whole C2 control step on the host cores:
    Stage 1, the 148-row partial prompt pass through all 32 layers, the 6
    single-token decode passes and the gate, after an untimed full step that
    fills its cache (its batched float64 mode, the one the 7B parity tests
    use).  Also the tiny C1 control step with BLAS on every core and on one
    thread, for scale."""
    import numpy as np
    from threadpoolctl import threadpool_limits
    from oracle.vla import OracleVLA
    import synth
    ft, fp, ids = si["frame_t"].numpy(), si["frame_prev"].numpy(), si["text_ids"].numpy()
    t0 = time.perf_counter()
    oracle.step_prefill(fp, ids)
    oracle.decode_actions()
    t_full = time.perf_counter() - t0
    t0 = time.perf_counter()
    oracle.margin_gate(force=[0])
    masks, _ = oracle.select_static(ft, fp)
    oracle.step_prefill(ft, ids, None, masks)
    oracle.decode_actions()
    t_step = time.perf_counter() - t0
    c1 = synth.config_c1()
    o1 = OracleVLA(c1, synth.model_weights(c1))
    s1 = synth.step_inputs(c1, 45)
    o1.step_prefill(s1["frame_prev"].numpy(), s1["text_ids"].numpy())
    o1.decode_actions()

    def c1_step():
        t = time.perf_counter()
        o1.margin_gate(force=[0])
        m1, _ = o1.select_static(s1["frame_t"].numpy(), s1["frame_prev"].numpy())
        o1.step_prefill(s1["frame_t"].numpy(), s1["text_ids"].numpy(), None, m1)
        o1.decode_actions()
        return time.perf_counter() - t

    c1_all = min(c1_step() for _ in range(3))
    with threadpool_limits(limits=1, user_api="blas"):
        c1_one = min(c1_step() for _ in range(3))
    cores = len(os.sched_getaffinity(0))
    info = _blas_info()
    return {"value": 1.0 / t_step, "unit": "control steps/s", "cores": cores, "kind": "oracle",
            "sample": "one whole C2 control step of the float64 oracle in its batched mode (Stage 1, the 148-row "
                      "partial prompt pass through 32 layers, 6 single-token decode passes, the gate; %.1f s) after "
                      "an untimed full step (%.1f s) that fills its cache" % (t_step, t_full),
            "seconds_per_step": t_step, "full_step_s": t_full, **info,
            "c1_ms_per_step_all_threads": c1_all * 1e3, "c1_ms_per_step_one_thread": c1_one * 1e3}


def c3_episode(dev):
    """The 50-frame moving-rectangle episode at the 7B shape with the gate
    applied (Alg. 1): per-layer reuse 80% -> 20%, tau = 249/250, theta = 0.1.
    Reports how often the gate fired (the recompute rate over steps 1..49;
    step 0 has no cache), the mean recomputed rows per layer, and the time
    per control step."""
    import torch
    import synth
    from paper_2608_10824_amd import gvc
    from paper_2608_10824_amd.session import Session
    cfg = synth.config_c3()
    w = synth.model_weights(cfg, device=dev)
    s = Session(cfg, w, device=dev)
    torch.cuda.synchronize()
    del w
    torch.cuda.empty_cache()
    note("C3 weights generated")
    frames = synth.c3_episode_frames(cfg).to(dev)
    ids = synth.text_ids(cfg).to(dev)
    s.step_prefill(frames[0:1], ids)
    s.decode_actions()
    n = frames.shape[0]
    stream = s.stream

    def run(trace):
        """Steps 1..n-1 with the gate applied; with trace, a record per step
        (and a synchronisation per step to read the static count and rows)."""
        fired, rows, out = [], [], []
        for t in range(1, n):
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)] if trace else None
            if ev:
                ev[0].record(stream)
            m, fire = s.margin_gate()
            fired.append(bool(fire[0]))
            mask, n_static = s.select_static(frames[t:t + 1], frames[t - 1:t])
            if ev:
                ev[1].record(stream)
            s.step_prefill(frames[t:t + 1], ids, None, mask)
            if ev:
                ev[2].record(stream)
            s.decode_actions()
            if ev:
                ev[3].record(stream)
                torch.cuda.synchronize()
                r = s.read(gvc.STATE_ROWS).cpu().tolist()
                rows.append(r)
                out.append({"step": t, "fired": bool(fire[0]), "margin_prev": round(float(m[0]), 6),
                            "static": int(n_static[0].item()), "rows_per_layer": r,
                            "us_gate_select": round(ev[0].elapsed_time(ev[1]) * 1e3, 1),
                            "us_prefill": round(ev[1].elapsed_time(ev[2]) * 1e3, 1),
                            "us_decode": round(ev[2].elapsed_time(ev[3]) * 1e3, 1)})
            if t % 10 == 0:
                note("C3 frame %d of %d%s" % (t, n - 1, " (trace)" if trace else ""))
        return fired, rows, out

    # timed episode (no per-step synchronisation), then the same episode traced
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    fired, _, _ = run(False)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    s.invalidate()
    s.step_prefill(frames[0:1], ids)
    s.decode_actions()
    fired2, rows, trace = run(True)
    s.close()
    L = cfg.n_layers
    return {"frames": n, "gated_steps": n - 1, "fired": sum(fired), "recompute_rate": sum(fired) / (n - 1),
            "traced_run_same_decisions": fired == fired2,
            "mean_recomputed_rows_per_layer": sum(sum(r) for r in rows) / (len(rows) * L),
            "prompt_len": cfg.prompt_len, "ms_per_step": dt * 1e3 / (n - 1),
            "reuse_permille": "%d -> %d over the layers" % (cfg.permille()[0], cfg.permille()[-1]),
            "tau": "%d/%d" % cfg.tau, "theta": cfg.theta, "trace": trace}


def c4_chunk(dev, steps, warmup):
    """The OFT-style action chunk at the 7B shape (two views, 512 visual + 20
    text tokens, a proprio row and 56 action-query rows, 307 static patches
    reused): one query is gate -> Stage 1 -> partial prompt pass -> the 56
    head rows, decoded in parallel with the action rows attending to each
    other both ways; executing the 8-step chunk means one query per 8
    control steps.  Reports the time per query, queries/s and the control
    steps/s that chunked execution gives."""
    import torch
    import synth
    from paper_2608_10824_amd import gvc
    from paper_2608_10824_amd.session import Session
    cfg = synth.config_c4().with_(action_bidir=True)
    w = synth.model_weights(cfg, device=dev)
    s = Session(cfg, w, device=dev)
    torch.cuda.synchronize()
    del w
    torch.cuda.empty_cache()
    note("C4 weights generated")
    si = synth.step_inputs(cfg, 307)
    fp, ft = si["frame_prev"].to(dev), si["frame_t"].to(dev)
    ids, ex = si["text_ids"].to(dev), si["extra_rows"].to(dev)
    s.step_prefill(fp, ids, ex)
    s.decode_actions()

    def query():
        s.margin_gate(force=[0])
        mask, _ = s.select_static(ft, fp)
        s.step_prefill(ft, ids, ex, mask)
        s.decode_actions()

    for _ in range(warmup):
        query()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        query()
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / steps
    rows = s.read(gvc.STATE_ROWS).cpu().tolist()
    s.close()
    chunk = cfg.n_action_q // 7
    return {"prompt_len": cfg.prompt_len, "action_rows": cfg.n_action_q, "action_bidir": True,
            "static_patches_reused": 307, "recomputed_rows_per_layer": rows[0], "ms_per_query": dt * 1e3,
            "queries_per_s": 1.0 / dt, "chunk_steps": chunk, "control_steps_per_s_chunked": chunk / dt,
            "steps": steps}


def c5_prefill(dev, reps, ks=(0, 64, 128, 192, 230)):
    """C5, 16 episodes batched: the prompt pass after a full step, for k of
    256 patches static in every episode (0, 25, 50, 75 and 90%).  With 16 x 148 = 2368 recomputed
    rows the projections are MFMA-bound, so this is where the prompt pass's
    MFMA utilisation is measured.  Reports per k the time of the partial
    prompt pass, its algorithmic TFLOP/s and the fraction of the dense bf16
    MFMA peak."""
    import torch
    import synth
    from paper_2608_10824_amd import gvc
    from paper_2608_10824_amd.session import Session
    cfg = synth.config_c5()
    w = synth.model_weights(cfg, device=dev)
    s = Session(cfg, w, device=dev)
    torch.cuda.synchronize()
    del w
    torch.cuda.empty_cache()
    note("C5 weights generated")
    d, F, V, L, P, B = cfg.d_model, cfg.ffn, cfg.vocab, cfg.n_layers, cfg.prompt_len, cfg.batch
    out = []
    for k in ks:
        note("C5 k=%d: full step, then %d timed partial passes" % (k, reps))
        si = synth.step_inputs(cfg, k, stream=k + 1)
        fp, ft = si["frame_prev"].to(dev), si["frame_t"].to(dev)
        ids = si["text_ids"].to(dev)
        s.invalidate()
        s.step_prefill(fp, ids)
        s.decode_actions()
        s.margin_gate(force=[0] * B)
        mask, _ = s.select_static(ft, fp)
        s.step_prefill(ft, ids, None, mask)       # warm-up of this row count
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            s.step_prefill(ft, ids, None, mask)   # the cache stays valid: the same partial pass each time
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        m = mask.cpu().numpy().astype(bool)
        flops = 2 * B * V * d
        for b in range(B):
            for l in range(L):
                qpos = [p for p in range(P) if not (1 <= p <= cfg.n_patches and m[b, l, p - 1])]
                flops += 2 * len(qpos) * (4 * d * d + 3 * d * F) + 2 * sum(2 * (p + 1) * d for p in qpos)
        tf = flops / (ms / 1e3) / 1e12
        rec = {"static_per_episode": k, "rows_per_layer": B * (P - k), "prefill_ms": ms, "tflops": tf,
               "mfma_util_pct": 100.0 * tf / BF16_PEAK_TFLOPS}
        if k == 128:   # the 16-episode action decode after the 50% reuse pass
            evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
            for ea, eb in evs:
                s.step_prefill(ft, ids, None, mask)
                ea.record()
                s.decode_actions()
                eb.record()
            torch.cuda.synchronize()
            dms = sum(ea.elapsed_time(eb) for ea, eb in evs) / reps
            # weights and LM head once per pass, plus every episode's K and V rows
            # 0..pos of every layer (pass j attends over P + j keys)
            dbytes = (cfg.n_decode - 1) * (L * layer_weight_bytes(cfg) + V * d * 2) + sum(
                L * B * 2 * (P + j) * d * 2 for j in range(1, cfg.n_decode))
            rec.update(decode_ms=dms, decode_gbs=dbytes / (dms / 1e3) / 1e9)
        out.append(rec)
        note("C5 k=%d: %.2f ms, %.0f TFLOP/s" % (k, ms, tf))
    s.close()
    return out


def vit_steps(dev, steps, warmup):
    """C2 with the ViT-L/14-shaped front end (24 blocks of width 1024, GELU
    projector to 4096) in place of the linear patch projection: every step
    runs the front end over all 256 patches, then the same partial prompt
    pass (128 static patches reused) and decode.  Reports the time per
    control step and the front end's GPU time per step."""
    import torch
    import synth
    from paper_2608_10824_amd import gvc
    from paper_2608_10824_amd.session import Session
    cfg = synth.config_c2v()
    w = synth.model_weights(cfg, device=dev)
    s = Session(cfg, w, device=dev)
    torch.cuda.synchronize()
    del w
    torch.cuda.empty_cache()
    note("C2 + ViT weights generated")
    si = synth.step_inputs(cfg, 128)
    fp, ft = si["frame_prev"].to(dev), si["frame_t"].to(dev)
    ids = si["text_ids"].to(dev)
    s.step_prefill(fp, ids)
    s.decode_actions()

    def step():
        s.margin_gate(force=[0])
        mask, _ = s.select_static(ft, fp)
        s.step_prefill(ft, ids, None, mask)
        s.decode_actions()

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / steps
    per_step = 2 + cfg.vit_layers * 7 + 2
    gvc.profile_begin(s.ctx, gvc.K_VIT, per_step + 8)
    step()
    torch.cuda.synchronize()
    vit_ms, vit_n = gvc.profile_end(s.ctx)
    s.close()
    return {"vit": "ViT-L/14 shape: 24 blocks, width 1024, 16 heads, MLP 4096; projector 1024 -> 4096 -> 4096",
            "ms_per_step": dt * 1e3, "control_steps_per_s": 1.0 / dt, "front_end_ms_per_step": vit_ms,
            "front_end_launches": vit_n, "steps": steps}


def staged_steps(cfg, w, si, dev, steps, warmup, entropy=False):
    """The C2 workload with Stage 2 on (the paper's top-k = 120): Stage 1's
    128 static patches minus those among the 120 that drew the most
    instruction attention in the previous pass; with entropy, Stage 3's
    per-layer proportions come from the previous pass's attention entropy.
    Reports the time per control step, the patches left static, the rows
    recomputed per layer and the signal kernel's time per layer."""
    import torch
    from paper_2608_10824_amd import gvc
    from paper_2608_10824_amd.session import Session
    cfg2 = cfg.with_(task_topk=120, entropy_reuse=entropy)
    s = Session(cfg2, w, device=dev)
    torch.cuda.synchronize()
    fp, ft = si["frame_prev"].to(dev), si["frame_t"].to(dev)
    ids = si["text_ids"].to(dev)
    s.step_prefill(fp, ids)
    s.decode_actions()

    def step():
        s.margin_gate(force=[0])
        mask, _ = s.select_static(ft, fp)
        s.step_prefill(ft, ids, None, mask)
        s.decode_actions()

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    n_static = int(s.n_static[0].item())
    rows = s.read(gvc.STATE_ROWS).cpu().tolist()
    layer_q = s.read(gvc.STATE_LAYER_Q)[0].cpu().tolist() if entropy else None
    gvc.profile_begin(s.ctx, gvc.K_STAGE2, cfg.n_layers * 2 + 8)
    step()
    torch.cuda.synchronize()
    sig_ms, sig_n = gvc.profile_end(s.ctx)
    s.close()
    out = {"task_topk": 120, "ms_per_step": dt * 1e3 / steps, "steps": steps, "static_patches": n_static,
           "recomputed_rows_per_layer": rows[0] if not entropy else rows,
           "signal_us_per_layer": sig_ms * 1e3 / max(sig_n, 1), "signal_launches_per_step": sig_n}
    if entropy:
        out["entropy_reuse"] = True
        out["layer_permille"] = layer_q
    return out


def fired_steps(s, cfg, si, dev, steps):
    """C2 control steps whose gate fires (Alg. 1, invalidate branch): the
    cache is invalidated, so the prompt pass recomputes all 276 rows, then
    the 7-token decode.  Reports the time per control step and the full
    prompt pass's time, TFLOP/s and MFMA utilisation."""
    import torch
    from paper_2608_10824_amd import gvc
    d, F, V, L, P = cfg.d_model, cfg.ffn, cfg.vocab, cfg.n_layers, cfg.prompt_len
    fp, ft, ids = si["frame_prev"].to(dev), si["frame_t"].to(dev), si["text_ids"].to(dev)
    stream = s.stream
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(steps)]

    def step(ev=None):
        s.margin_gate(force=[1])                # the gate fires: the next pass is full
        mask, _ = s.select_static(ft, fp)
        if ev:
            ev[0].record(stream)
        s.step_prefill(ft, ids, None, mask)
        if ev:
            ev[1].record(stream)
        s.decode_actions()

    step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        step(evs[i])
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / steps
    rows = s.read(gvc.STATE_ROWS).cpu().tolist()
    pms = sum(e[0].elapsed_time(e[1]) for e in evs) / steps
    flops = 2 * V * d + L * (2 * P * (4 * d * d + 3 * d * F) + 2 * sum(2 * (p + 1) * d for p in range(P)))
    tf = flops / (pms / 1e3) / 1e12
    return {"ms_per_step": dt * 1e3, "control_steps_per_s": 1.0 / dt, "recomputed_rows_per_layer": rows[0],
            "prefill_ms": pms, "prefill_tflops": tf, "prefill_mfma_util_pct": 100.0 * tf / BF16_PEAK_TFLOPS,
            "prefill_hbm_frac": (L * layer_weight_bytes(cfg) + V * d * 2) / (pms / 1e3) / 1e9 / HBM_PEAK_GBS,
            "steps": steps}


def stored_traffic(kernel_sources):
    """HBM bytes per launch of the dominant kernel from the committed rocprofv3
    counter summary, or None when the kernel sources changed since."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "traffic_decode_pass_c2.md")
    if not os.path.exists(path):
        return None
    h = hashlib.sha256()
    for f in kernel_sources:
        h.update(open(os.path.join(ROOT, f), "rb").read())
    rec = {}
    for line in open(path):
        if ":" in line and line.startswith("- "):
            k, v = line[2:].split(":", 1)
            rec[k.strip()] = v.strip().strip("`")
    if rec.get("kernel_sources_sha256") != h.hexdigest():
        return None
    try:
        return float(rec["fetch_bytes_per_launch"]) + float(rec["write_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py runs the hot path on one GPU; --gpus %d is not supported (multi-GPU sharding is "
              "described in DESIGN.md, not built)" % args.gpus, file=sys.stderr)
        return 2
    import torch
    import synth
    from paper_2608_10824_amd import gvc
    from paper_2608_10824_amd.session import Session

    cfg = synth.config_c2()
    n_static = 128
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = synth.model_weights(cfg, device=dev)
    si = synth.step_inputs(cfg, n_static)
    note("weights and inputs generated")
    w_stage2 = w if not args.no_stage2 else None
    # the oracle's float64 host copy (test infrastructure, for the CPU
    # baseline) is made after the GPU regions, so that building it does not
    # share the host with the timed launches
    w_oracle = w if not args.no_cpu_baseline else None
    s = Session(cfg, w, device=dev)
    torch.cuda.synchronize()
    del w
    torch.cuda.empty_cache()
    note("library context initialised (weights packed)")

    fp, ft = si["frame_prev"].to(dev), si["frame_t"].to(dev)
    ids = si["text_ids"].to(dev)
    stream = s.stream

    # first step: no cache yet, full pass
    s.step_prefill(fp, ids)
    s.decode_actions()

    fired = []

    def control_step(ev=None):
        m, fire = s.margin_gate(force=[0])      # Alg. 1 test on step t-1; the workload keeps the cache
        fired.append(bool(fire[0]))
        mask, _ = s.select_static(ft, fp)
        if ev:
            ev[0].record(stream)
        s.step_prefill(ft, ids, None, mask)
        if ev:
            ev[1].record(stream)
        s.decode_actions()
        if ev:
            ev[2].record(stream)

    for _ in range(args.warmup):
        control_step()
    torch.cuda.synchronize()
    note("warm-up done")

    # timed region: the steps/s value
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        control_step()
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    ms_step = dt * 1e3 / args.steps
    rows = s.read(gvc.STATE_ROWS).cpu().tolist()
    note("timed region done: %.2f ms per step" % ms_step)

    # second region, same steps: phase events and the dominant kernel's launches
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    launches_per_step = cfg.n_decode - 1
    gvc.profile_begin(s.ctx, gvc.K_DECODE_PASS, launches_per_step * args.steps + 8)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        control_step(evs[i])
    torch.cuda.synchronize()
    dt2 = time.perf_counter() - t0
    dk_ms, dk_n = gvc.profile_end(s.ctx)
    note("profiled region done")
    if dk_n == 0:
        raise SystemExit("bench: the single-launch decode pass did not run (GVC_DECODE=legacy or an ineligible shape)")
    prefill_ms = sum(e[0].elapsed_time(e[1]) for e in evs) / args.steps
    decode_ms = sum(e[1].elapsed_time(e[2]) for e in evs) / args.steps

    d, F, V, L, P = cfg.d_model, cfg.ffn, cfg.vocab, cfg.n_layers, cfg.prompt_len
    traffic = stored_traffic(KERNEL_SOURCES)
    # dominant kernel: the single-launch decode pass (all layers of one token),
    # one launch per decode pass; algorithmic bytes = every layer's weights
    # once + the K and V rows of positions 0..pos read by the attention,
    # averaged over the passes (pass j attends over P + j keys)
    n_pass = cfg.n_decode - 1
    dk_bytes = L * layer_weight_bytes(cfg) + sum(L * 2 * (P + j) * d * 2 for j in range(1, n_pass + 1)) / n_pass
    # the pass also runs the final norm, the LM head and the token choice
    # (unless GVC_DECODE_FLAGS masks the head bit): V x d head weights read,
    # V logits written
    head_fused = (int(os.environ.get("GVC_DECODE_FLAGS", "7")) & 4) != 0
    if head_fused:
        dk_bytes += V * d * 2 + V * 4
    dk_avg_s = dk_ms / 1e3 / max(dk_n, 1)
    dk_gbs = dk_bytes / dk_avg_s / 1e9
    # prompt pass algorithmic work: the recomputed rows of every layer, their
    # attention over the keys up to each row's position, and the head row
    mask = s.mask[0].cpu().numpy().astype(bool)              # [L][N]
    M = rows[0]
    prefill_flops = 2 * V * d
    for l in range(L):
        qpos = [p for p in range(P) if not (1 <= p <= cfg.n_patches and mask[l][p - 1])]
        prefill_flops += 2 * len(qpos) * (4 * d * d + 3 * d * F) + 2 * sum(2 * (p + 1) * d for p in qpos)
    prefill_bytes = L * layer_weight_bytes(cfg) + V * d * 2
    decode_bytes = (cfg.n_decode - 1) * (L * layer_weight_bytes(cfg) + V * d * 2
                                         + L * 2 * 2 * d * (P + cfg.n_decode))
    out = {
        "metric": "control steps/s at 7B, 256 visual tokens, 50% reuse; prefill MFMA util %",
        "value": args.steps / dt,
        "unit": "control steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "Llama-2-7B-shaped VLA decoder (32 layers, d=4096, 32 heads, FFN 11008, vocab "
                               "32000, 256 action bins), random bf16 weights; 224x224 frame = 256 visual + 20 text "
                               "tokens; 128 static patches reused (50%); 7-token autoregressive action decode",
                   "batch": 1, "prompt_len": P, "recomputed_rows_per_layer": M, "decode_tokens": cfg.n_decode},
        "prefill_ms": prefill_ms,
        "prefill_tflops": prefill_flops / (prefill_ms / 1e3) / 1e12,
        "prefill_mfma_util_pct": 100.0 * prefill_flops / (prefill_ms / 1e3) / 1e12 / BF16_PEAK_TFLOPS,
        "prefill_hbm_gbs": prefill_bytes / (prefill_ms / 1e3) / 1e9,
        "prefill_hbm_frac": prefill_bytes / (prefill_ms / 1e3) / 1e9 / HBM_PEAK_GBS,
        "decode_ms": decode_ms,
        "decode_gbs": decode_bytes / (decode_ms / 1e3) / 1e9,
        "decode_hbm_frac": decode_bytes / (decode_ms / 1e3) / 1e9 / HBM_PEAK_GBS,
        "gate_fired_steps": sum(fired),
        "roofline": {"bound": "hbm", "achieved": dk_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": dk_gbs / HBM_PEAK_GBS, "traffic": traffic,
                     "kernel": "k_decode_pass<128, 2> (one decode pass over all 32 layers%s, cooperative grid)"
                               % (", the final norm, the LM head and the token choice" if head_fused else ""),
                     "bytes_per_launch": dk_bytes, "avg_launch_us": dk_avg_s * 1e6, "launches": dk_n,
                     "region_ms_per_step": dt2 * 1e3 / args.steps},
    }
    if not args.no_fired:
        out["c2_fired"] = fired_steps(s, cfg, si, dev, min(args.steps, 10))
        note("C2 fired steps done: %.2f ms per step" % out["c2_fired"]["ms_per_step"])
    s.close()
    del s
    torch.cuda.empty_cache()
    if w_oracle is not None:
        from oracle.vla import OracleVLA
        oracle = OracleVLA(cfg, w_oracle, batched=True)
        del w_oracle
        note("oracle weights converted to float64 on the host")
        out["cpu_baseline"] = cpu_baseline(cfg, oracle, si)
        del oracle
        note("cpu baseline done")
    if w_stage2 is not None:
        out["stage2"] = staged_steps(cfg, w_stage2, si, dev, min(args.steps, 10), 2)
        note("Stage 2 steps done: %d static patches left" % out["stage2"]["static_patches"])
        out["stage3_entropy"] = staged_steps(cfg, w_stage2, si, dev, min(args.steps, 10), 2, entropy=True)
        note("Stage 2 + 3 steps done: layer proportions %s" % out["stage3_entropy"]["layer_permille"][:4])
        del w_stage2
        torch.cuda.empty_cache()
    if not args.no_c5:
        ks = tuple(int(k) for k in args.c5_static.split(",") if k.strip())
        out["c5_prefill"] = c5_prefill(dev, min(args.steps, 5), ks)
    if not args.no_vit:
        out["c2_vit"] = vit_steps(dev, min(args.steps, 10), 2)
        note("C2 + ViT steps done: %.2f ms per step" % out["c2_vit"]["ms_per_step"])
    if not args.no_c4:
        out["c4_chunk"] = c4_chunk(dev, min(args.steps, 10), 2)
        note("C4 chunk queries done: %.2f ms per query" % out["c4_chunk"]["ms_per_query"])
    if not args.no_c3:
        out["c3"] = c3_episode(dev)
        note("C3 episode done: recompute rate %.3f" % out["c3"]["recompute_rate"])
        if args.trace_jsonl:
            with open(args.trace_jsonl, "w") as f:
                for rec in out["c3"]["trace"]:
                    f.write(json.dumps(rec) + "\n")
            note("C3 trace written to %s" % args.trace_jsonl)
    # explicit teardown before the interpreter exits: every session is closed
    # above; wait for the device, then return the cached blocks
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    rc = main()
    if rc:
        sys.exit(rc)
