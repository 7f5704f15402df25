#!/usr/bin/env python3
"""Throughput of the generation-stage policy forward on one MI355X.

A step is one pass of the whole hot path over one batch of synthetic
observations: prefill (patch embedding, language embedding, every decoder
layer writing the paged KV cache) followed by the autoregressive action
decode (t0 from the prefix, six decode steps over the paged cache, 256-bin
argmax).  The default workload is the small bf16 VLA on 64 environments
(two 224x224 cameras, 32 language tokens, 12-layer d=1024 decoder); every
step yields one 7-dim action per environment.

Output: one JSON line with the throughput (actions/s), the roofline entry of
the dominant kernel (the prefill GEMMs, timed live with HIP events on the
policy's stream inside the timed region) and the CPU oracle timed on a
bounded sample on this host.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

WORKLOADS = {
    # name: (preset, n_envs, obs seed)
    "tiny-fp32": (1, 8, 1001),
    "small-bf16": (2, 64, 1002),
    "7b-bf16": (3, 32, 1003),
}
PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3      # MI355X fp32 vector
PEAK_HBM_GBS = 8000.0


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def cpu_baseline(preset: int, obs_seed: int, n_sample: int):
    """The oracle as it stands, on this host's cores, on n_sample envs."""
    import synth_inputs
    from oracle import model as M
    try:
        from threadpoolctl import threadpool_info
        cores = max([d.get("num_threads", 1) for d in threadpool_info()] + [1])
    except Exception:
        cores = os.cpu_count()
    cfg = M.PRESETS[preset]
    ids = list(range(n_sample))
    img = synth_inputs.pixels(obs_seed, ids, cfg.n_cams, cfg.img, cfg.img)
    lang = synth_inputs.lang_ids(obs_seed, ids, cfg.n_lang, cfg.vocab)
    t = time.perf_counter()
    pol = M.Policy(cfg, seed=0)
    for name in pol.shapes:          # weights generated up front, outside the timed sample
        pol.W(name)
    t_w = time.perf_counter() - t
    t = time.perf_counter()
    for i in ids:
        pol.decode(pol.prefill(img[i], lang[i]))
    dt = time.perf_counter() - t
    return {"value": round(n_sample / dt, 4), "unit": "actions/s", "cores": int(cores), "kind": "oracle",
            "sample": f"{n_sample} env(s) of the same workload: prefill + 6 decode steps in float64 "
                      f"(numpy/BLAS), {dt:.1f} s; weight generation ({t_w:.1f} s) excluded",
            "seconds": round(dt, 3)}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="small-bf16", choices=sorted(WORKLOADS))
    ap.add_argument("--cpu-sample", type=int, default=16, help="envs in the oracle sample (0 = skip)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU only (asked for --gpus {args.gpus}); environments "
              "are independent, so N GPUs would each run their own share (see DESIGN.md, sharding)",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import synth_inputs
    from paper_2609_27547_amd import ebrl as E

    preset, n, obs_seed = WORKLOADS[args.workload]
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    t = time.perf_counter()
    pol = E.Policy(preset, seed=0, stream=stream.cuda_stream)
    log(f"policy {args.workload} created in {time.perf_counter() - t:.1f} s")
    c = pol.cfg
    ids = list(range(n))
    img = synth_inputs.pixels(obs_seed, ids, c.n_cams, c.img, c.img)
    lang = synth_inputs.lang_ids(obs_seed, ids, c.n_lang, c.vocab)
    d_img = torch.from_numpy(img).cuda()
    d_lang = torch.from_numpy(lang).cuda()
    tok = torch.empty((n, c.n_action_tokens), dtype=torch.int32, device="cuda")
    act = torch.empty((n, c.n_action_tokens), dtype=torch.float32, device="cuda")

    def step():
        pol.prefill(ids, images=d_img, lang_ids=d_lang)
        pol.decode_actions(ids, tokens=tok, actions=act, margins=None, with_margin=False)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # ---- timed region: K steps; the dominant kernel class is timed live
    dominant = E.K_GEMM
    pol.profile_read(dominant, reset=True)
    pol.profile_enable([dominant])
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    pol.profile_enable([])
    gemm = pol.profile_read(dominant, reset=True)
    gpu_ms = ev0.elapsed_time(ev1)
    ms_per_step = 1000.0 * wall / args.steps
    actions_per_s = n * args.steps / wall

    # ---- breakdown pass (not part of the value): every kernel class, per phase
    classes = list(E.KERNEL_CLASSES)
    pol.profile_enable(classes)
    phase = {"prefill": 0.0, "decode": 0.0}
    pe = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    reps = max(3, min(args.steps, 10))
    for _ in range(reps):
        pe[0].record(stream)
        pol.prefill(ids, images=d_img, lang_ids=d_lang)
        pe[1].record(stream)
        pol.decode_actions(ids, tokens=tok, actions=act, margins=None, with_margin=False)
        pe[2].record(stream)
        torch.cuda.synchronize()
        phase["prefill"] += pe[0].elapsed_time(pe[1]) / reps
        phase["decode"] += pe[1].elapsed_time(pe[2]) / reps
    pol.profile_enable([])
    kernels = {}
    for cls, name in E.KERNEL_CLASSES.items():
        r = pol.profile_read(cls, reset=True)
        if r["launches"]:
            kernels[name] = {"launches_per_step": r["launches"] / reps, "ms_per_step": round(r["ms"] / reps, 4),
                             "tflops": round(r["flop"] / (r["ms"] * 1e9), 1) if r["ms"] else None,
                             "gbs": round(r["bytes"] / (r["ms"] * 1e6), 1) if r["ms"] else None}

    bf16 = pol.bf16
    peak = PEAK_BF16_TFLOPS if bf16 else PEAK_FP32_TFLOPS
    achieved = gemm["flop"] / (gemm["ms"] * 1e9) if gemm["ms"] else 0.0
    roofline = {"bound": "mfma", "achieved": round(achieved, 1), "peak": peak, "unit": "TFLOP/s",
                "frac": round(achieved / peak, 4), "traffic": None,
                "kernel": "gemm_bf16_big_kernel (prefill projections, M >= 256)",
                "launches": gemm["launches"], "avg_launch_us": round(1000 * gemm["ms"] / max(1, gemm["launches"]), 2),
                "flop_per_launch": round(gemm["flop"] / max(1, gemm["launches"])),
                "share_of_step": round(gemm["ms"] / gpu_ms, 3) if gpu_ms else None}

    base = None
    if args.cpu_sample > 0:
        log("timing the CPU oracle ...")
        base = cpu_baseline(preset, obs_seed, args.cpu_sample)

    out = {
        "metric": "policy actions/sec at 1 GPU",
        "value": round(actions_per_s, 2),
        "unit": "actions/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if bf16 else "f32",
        "data": "synthetic (seeded uniform pixels and token ids; random-init N(0, 0.02) weights)",
        "config": {"workload": f"{args.workload}: preset {preset}, {n} envs, prefix {c.max_seq} tokens, "
                               f"{c.layers}-layer d={c.d} decoder, prefill + {c.n_action_tokens - 1} decode steps",
                   "envs": n, "prefix_len": c.max_seq, "layers": c.layers, "d": c.d,
                   "action_tokens": c.n_action_tokens},
        "tokens_per_s": round(actions_per_s * c.n_action_tokens, 1),
        "gpu_ms_per_step": round(gpu_ms / args.steps, 3),
        "phases_ms": {k: round(v, 3) for k, v in phase.items()},
        "kernels": kernels,
        "roofline": roofline,
        "cpu_baseline": base,
    }
    print(json.dumps(out), flush=True)
    pol.close()


if __name__ == "__main__":
    main()
