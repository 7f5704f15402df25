#!/usr/bin/env python3
"""Throughput of the generation-stage policy forward on one MI355X.

A step is one pass of the whole hot path over one batch of synthetic
observations: prefill (patch embedding, language embedding, every decoder
layer writing the paged KV cache) followed by the autoregressive action
decode (t0 from the prefix, six decode steps over the paged cache, 256-bin
argmax).  The default workload is the 7B-class VLA on 32 environments (one
224x224 camera through a 24-layer ViT, 32 language tokens, 32-layer d=4096
decoder), the largest configuration that is timed as prefill + decode on one
GPU; every step yields one 7-dim action per environment.

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
    "flow-bf16": (4, 64, 1004),
    "wam-bf16": (5, 64, 1005),
    "ragged-7b": (3, 128, 1005),
}
# default oracle sample per workload: envs that take roughly 10-40 s on the host
CPU_SAMPLE = {"tiny-fp32": 8, "small-bf16": 32, "7b-bf16": 1, "flow-bf16": 3, "wam-bf16": 2, "ragged-7b": 1}
PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3      # MI355X fp32 vector
PEAK_HBM_GBS = 8000.0


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def stored_traffic(workload: str):
    """Per-launch HBM traffic of the large-M GEMM measured with hardware
    counters (pmc_traffic.py), if taken on the current GEMM sources."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    import pmc_traffic
    with open(path) as f:
        t = json.load(f)
    return t if t.get("sources_sha") == pmc_traffic.sources_hash() else None


def cpu_model() -> str:
    """The host CPU's model name (Linux /proc/cpuinfo), or "unknown"."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(workload: str, n_sample: int):
    """The oracle as it stands, on this host's cores, on n_sample envs of the
    same workload (envs are independent, so the rate scales per env)."""
    import synth_inputs
    from oracle import model as M
    try:
        from threadpoolctl import threadpool_info
        cores = max([d.get("num_threads", 1) for d in threadpool_info()] + [1])
    except Exception:
        cores = os.cpu_count()
    preset, pool, obs_seed = WORKLOADS[workload]
    cfg = M.PRESETS[preset]
    if workload == "ragged-7b":
        # decode-only calls on the env pool's language-only prefixes: the
        # first n_sample envs of the sequence's first call, each prefilled
        # outside the timed sample (as the GPU's pool is)
        T = synth_inputs.ragged_prefix_lengths(5, pool, 200, 320)
        ids = [int(e) for e in synth_inputs.ragged_calls(5, 1, pool, 128)[0][:n_sample]]
        lang = synth_inputs.lang_ids(obs_seed, list(range(pool)), 320, cfg.vocab)
    else:
        ids = list(range(n_sample))
        img = synth_inputs.pixels(obs_seed, ids, cfg.n_cams, cfg.img, cfg.img)
        lang = synth_inputs.lang_ids(obs_seed, ids, cfg.n_lang, cfg.vocab)
    t = time.perf_counter()
    pol = M.Policy(cfg, seed=0)
    for name in pol.shapes:          # weights generated up front, outside the timed sample
        pol.W(name)
    t_w = time.perf_counter() - t
    if workload == "ragged-7b":
        states = [pol.prefill(None, lang[e][:T[e]]) for e in ids]
        t = time.perf_counter()
        for st in states:
            pol.decode(st)
        dt = time.perf_counter() - t
        return {"value": round(len(ids) / dt, 4), "unit": "actions/s", "cores": int(cores), "cpu": cpu_model(), "kind": "oracle",
                "sample": f"{len(ids)} env(s) of the first ragged call (prefixes of "
                          f"{', '.join(str(int(T[e])) for e in ids)} tokens): 6 decode steps each in float64 "
                          f"(numpy/BLAS), {dt:.1f} s; weight generation ({t_w:.1f} s) and the pool's prefill excluded",
                "seconds": round(dt, 3)}
    t = time.perf_counter()
    per_env = cfg.chunk if cfg.exp_layers else 1
    for i in ids:
        st = pol.prefill(img[i], lang[i])
        if cfg.frame_tokens:
            pol.wam_denoise(st, synth_inputs.flow_noise(5, [i], cfg.frame_tokens, cfg.frame_dim)[0],
                            synth_inputs.flow_noise(4, [i], cfg.chunk, cfg.adim)[0])
        elif cfg.exp_layers:
            pol.flow_denoise(st, synth_inputs.flow_noise(4, [i], cfg.chunk, cfg.adim)[0])
        else:
            pol.decode(st)
    dt = time.perf_counter() - t
    what = "prefill + 10 Euler steps of the expert" if cfg.exp_layers else "prefill + 6 decode steps"
    return {"value": round(n_sample * per_env / dt, 4), "unit": "actions/s", "cores": int(cores), "cpu": cpu_model(), "kind": "oracle",
            "sample": f"{n_sample} env(s) of the same workload: {what} in float64 (numpy/BLAS), {dt:.1f} s; "
                      f"weight generation ({t_w:.1f} s) excluded",
            "seconds": round(dt, 3)}


def stream_read_gbs(E, torch, stream_ptr, nbytes: int = 1 << 30) -> float:
    """HBM read bandwidth of the library's streaming-read reference kernel on
    the given stream (so under that stream's CU mask): the ceiling the
    partitions' HBM-bound kernels are compared against."""
    x = torch.empty(nbytes // 4, dtype=torch.int32, device="cuda")
    x.fill_(1)
    o = torch.zeros(1, dtype=torch.int32, device="cuda")
    ext = torch.cuda.ExternalStream(stream_ptr)
    torch.cuda.synchronize()
    for _ in range(2):
        E.op_stream_read(x, o, stream_ptr)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(ext)
    for _ in range(5):
        E.op_stream_read(x, o, stream_ptr)
    e1.record(ext)
    torch.cuda.synchronize()
    gbs = 5 * nbytes / (e0.elapsed_time(e1) * 1e6)
    del x, o
    return round(gbs, 1)


def balanced_mask(quarters: int, n_cu: int = 256):
    """CU mask words for quarters/4 of the CUs: runs of 8 CUs spread so every
    XCD gets the same share whether CUs are numbered XCD by XCD or round-robin
    across XCDs."""
    words = [0] * (n_cu // 32)
    for i in range(n_cu):
        if (i // 8) % 4 < quarters:
            words[i // 32] |= 1 << (i % 32)
    return words


# The co-located training stand-in: one bf16 projection of a training step
# over 8192 tokens at the 7B-class width (M x N x K), run back to back.
LOAD_MNK = (8192, 4096, 4096)


def _events(torch, n):
    return [torch.cuda.Event(enable_timing=True) for _ in range(n)]


class _GemmLoad:
    """Keeps `depth` GEMMs queued on one stream from a host thread until
    stopped, with a timing event after each (their completion times)."""

    def __init__(self, E, torch, s_ptr, A, B, C, depth=4):
        import threading
        self.E, self.torch, self.s_ptr, self.A, self.B, self.C, self.depth = E, torch, s_ptr, A, B, C, depth
        self.events = []
        self.stop = threading.Event()
        self.started = threading.Event()
        self.error = None
        self.thread = threading.Thread(target=self._run, daemon=True)

    def _run(self):
        torch = self.torch
        try:
            torch.cuda.set_device(0)
            ext = torch.cuda.ExternalStream(self.s_ptr)
            k = 0
            while not self.stop.is_set():
                self.E.op_gemm(self.A, self.B, self.C, self.s_ptr)
                ev = torch.cuda.Event(enable_timing=True)
                ev.record(ext)
                self.events.append(ev)
                k += 1
                if k > self.depth:
                    self.events[k - 1 - self.depth].synchronize()
                    self.started.set()
        except Exception as e:  # reported by the caller
            self.error = e
            self.started.set()

    def __enter__(self):
        self.thread.start()
        self.started.wait(timeout=60)
        return self

    def __exit__(self, *exc):
        self.stop.set()
        self.thread.join(timeout=120)
        if self.error:
            raise self.error


def colocated(E, torch, w, args):
    """Generation on a CU-masked stream while the GEMM load runs on the
    complementary CUs (the paper's generation and training sharing one GPU
    under separate SM quotas), against each of the two alone on the same
    masks.  Generation is timed by events on its stream; the load's rate is
    taken from the completion events of its GEMMs inside the generation
    window."""
    Mg, Ng, Kg = LOAD_MNK
    flop = 2.0 * Mg * Ng * Kg
    A = torch.randn(Mg, Kg, device="cuda").to(torch.bfloat16)
    B = torch.randn(Ng, Kg, device="cuda").to(torch.bfloat16)
    C = torch.empty(Mg, Ng, device="cuda", dtype=torch.float32)
    res = {"load": f"bf16 GEMM {Mg} x {Ng} x {Kg} through ebrl_op_gemm, kept queued on the complementary CUs"}

    def gen_run(s_ptr):
        ext_g = torch.cuda.ExternalStream(s_ptr)
        if args.workload == "ragged-7b":
            w.call_i = 0
        g0, g1 = _events(torch, 2)
        g0.record(ext_g)
        n_act = 0
        for _ in range(args.steps):
            n_act += w.step()
        g1.record(ext_g)
        g1.synchronize()
        ms = g0.elapsed_time(g1)
        return n_act / (ms / 1000.0), ms, g0

    for q in (1, 2, 3):
        gmask = balanced_mask(q)
        lmask = [(~x) & 0xFFFFFFFF for x in gmask]
        s_gen = E.create_cu_masked_stream(0, gmask)
        s_load = E.create_cu_masked_stream(0, lmask)
        try:
            w.pol.bind_stream(s_gen)
            torch.cuda.synchronize()
            gen_iso, _, _ = gen_run(s_gen)
            torch.cuda.synchronize()
            with _GemmLoad(E, torch, s_load, A, B, C) as ld:
                t_ld = time.perf_counter()
                time.sleep(0.05)
                n0 = len(ld.events)
                gen_co, gen_ms, g0 = gen_run(s_gen)
            torch.cuda.synchronize()
            iso_ev = ld.events[max(1, n0 // 2):n0]          # the load alone, before generation started
            t_ev = [g0.elapsed_time(e) for e in ld.events[n0:]]
            inside = [t for t in t_ev if 0.0 <= t <= gen_ms]
            load_co = (len(inside) - 1) * flop / ((inside[-1] - inside[0]) * 1e9) if len(inside) >= 2 else None
            load_iso = ((len(iso_ev) - 1) * flop / (iso_ev[0].elapsed_time(iso_ev[-1]) * 1e9)
                        if len(iso_ev) >= 2 else None)
            res[f"{q / 4:.2f}"] = {
                "gen_isolated_actions_per_s": round(gen_iso, 2),
                "gen_colocated_actions_per_s": round(gen_co, 2),
                "gen_colocated_over_isolated": round(gen_co / gen_iso, 3),
                "load_isolated_tflops": round(load_iso, 1) if load_iso else None,
                "load_colocated_tflops": round(load_co, 1) if load_co else None,
                "load_gemms_during_gen": len(inside),
                "load_covered_gen": bool(t_ev) and t_ev[-1] > gen_ms,
            }
            log(f"colocated {q / 4:.2f}: {res[f'{q / 4:.2f}']} (load thread up {time.perf_counter() - t_ld:.2f} s)")
        finally:
            w.pol.bind_stream(torch.cuda.current_stream().cuda_stream)
            torch.cuda.synchronize()
            E.destroy_stream(s_gen)
            E.destroy_stream(s_load)
    del A, B, C
    return res


def gen_profile(E, torch, w, args, batches=(16, 32, 64, 128), quarters=(1, 2, 3, 4), calls=8):
    """P_gen(s, B) of Section 4.3.2 measured on this GPU: actions/s of decode
    calls of exactly B envs on a stream masked to s of the CUs (one action,
    i.e. one rollout chunk-step, per env per call)."""
    table = np.zeros((len(quarters), len(batches)))
    for i, q in enumerate(quarters):
        s_ptr = E.create_cu_masked_stream(0, balanced_mask(q))
        try:
            w.pol.bind_stream(s_ptr)
            ext = torch.cuda.ExternalStream(s_ptr)
            for j, b in enumerate(batches):
                ids = list(range(b))
                tok, act = w.tok[:b], w.act[:b]
                for _ in range(2):
                    w.pol.decode_actions(ids, tokens=tok, actions=act, margins=None, with_margin=False)
                e0, e1 = _events(torch, 2)
                e0.record(ext)
                for _ in range(calls):
                    w.pol.decode_actions(ids, tokens=tok, actions=act, margins=None, with_margin=False)
                e1.record(ext)
                e1.synchronize()
                table[i, j] = calls * b / (e0.elapsed_time(e1) / 1000.0)
        finally:
            w.pol.bind_stream(torch.cuda.current_stream().cuda_stream)
            torch.cuda.synchronize()
            E.destroy_stream(s_ptr)
    return [25 * q for q in quarters], list(batches), table


def load_profile(E, torch, quarters=(1, 2, 3, 4), reps=6):
    """TFLOP/s of the training stand-in GEMM alone on each CU share."""
    Mg, Ng, Kg = LOAD_MNK
    A = torch.randn(Mg, Kg, device="cuda").to(torch.bfloat16)
    B = torch.randn(Ng, Kg, device="cuda").to(torch.bfloat16)
    C = torch.empty(Mg, Ng, device="cuda", dtype=torch.float32)
    out = []
    for q in quarters:
        s_ptr = E.create_cu_masked_stream(0, balanced_mask(q))
        try:
            ext = torch.cuda.ExternalStream(s_ptr)
            for _ in range(2):
                E.op_gemm(A, B, C, s_ptr)
            e0, e1 = _events(torch, 2)
            e0.record(ext)
            for _ in range(reps):
                E.op_gemm(A, B, C, s_ptr)
            e1.record(ext)
            e1.synchronize()
            out.append(reps * 2.0 * Mg * Ng * Kg / (e0.elapsed_time(e1) * 1e9))
        finally:
            torch.cuda.synchronize()
            E.destroy_stream(s_ptr)
    del A, B, C
    return out


def allocation(E, torch, w, args):
    """Algorithm 1 of Section 4.3.2 on tables measured here (generation, and
    the GEMM stand-in for training) plus a modelled CPU simulator.  Model
    numbers, stated so the result can be read: a training chunk-step costs
    6 x 6.5e9 x 295 FLOP (forward and backward of the 7B-class decoder over
    one 288-token prefix plus its 7 action tokens) at the stand-in GEMM's
    measured rate; the simulator steps an environment in 40 ms on one core
    (the paper's average step time, Section 3.2) or 28 ms on two, with 64 host
    cores, and needs no GPU; device memory is 288 GB, of which generation
    holds its 14 GB of weights plus 168 MB of KV per env and training 120 GB
    (weights, gradients, Adam state) plus 2 GB per sample of its batch."""
    quotas, batches, gen = gen_profile(E, torch, w, args)
    tflops = load_profile(E, torch)
    flop_per_sample = 6 * 6.5e9 * 295
    train = np.array([[t * 1e12 / flop_per_sample] for t in tflops])
    P = dict(cenv=np.array([1, 2]), ssim=np.array([0]), sim=np.array([[64 / 0.040], [32 / 0.028]]),
             sgen=np.array(quotas), bgen=np.array(batches), gen=gen,
             gen_mem=np.array([14e9 + 168e6 * b for b in batches]),
             strain=np.array(quotas), btrain=np.array([32]), train=train,
             train_mem=np.array([120e9 + 2e9 * 32]))
    res = E.alloc_solve(P, cores=64, mem_bytes=288e9, sgen_min=10, strain_min=10)
    return {"gen_quota_pct": quotas, "gen_batch": batches,
            "P_gen_actions_per_s": [[round(x, 1) for x in row] for row in gen],
            "train_standin_tflops": [round(t, 1) for t in tflops],
            "P_train_chunk_steps_per_s": [round(x, 2) for x in train[:, 0]],
            "P_sim_chunk_steps_per_s": {"1 core/env": 1600.0, "2 cores/env": round(32 / 0.028, 1)},
            "result": {k: (round(v, 2) if isinstance(v, float) else v) for k, v in res.items()}}


def rollout(E, torch, w, args, groups=4, chunk=8, cores=16, horizon=20.0):
    """Section 4.2's rollout pipeline around the generation calls: the
    library's scheduler (group pipeline + Algorithm 2 core rebinding) over a
    discrete-event stand-in for the simulators (per-env step times with mean
    40 ms and P99 60 ms, Section 3.2), where each group's generation is the
    real call on this GPU -- prefill of the group's observations and flow
    denoising of its action chunk -- timed with HIP events.  chunk actions of
    each generated chunk are executed; time is simulated, generation time
    measured.  The same run with envs bound to fixed cores is reported next
    to it."""
    import synth_inputs
    from paper_2609_27547_amd import rollout as R
    n = w.n
    lat = synth_inputs.sim_step_latency(6, n, 40000)
    ext = torch.cuda.current_stream()

    def generate(ids):
        idx = torch.as_tensor(np.asarray(ids, dtype=np.int64), device="cuda")
        img, lang, noise = w.img.index_select(0, idx), w.lang.index_select(0, idx), w.noise.index_select(0, idx)
        e0, e1 = _events(torch, 2)
        e0.record(ext)
        w.pol.prefill(list(ids), images=img, lang_ids=lang)
        w.pol.flow_denoise(list(ids), noise)
        e1.record(ext)
        e1.synchronize()
        return e0.elapsed_time(e1) / 1000.0

    for g in range(groups):                     # capture the group-size graphs before timing
        generate(list(range(g * n // groups, (g + 1) * n // groups)))
    res = {"envs": n, "groups": groups, "chunk_actions_executed": chunk, "cores": cores,
           "simulated_horizon_s": horizon}
    for name, fixed in (("rebinding", False), ("fixed_binding", True)):
        out = R.run(n, groups, chunk, cores, lat, generate, horizon, fixed_binding=fixed)
        res[name] = {k: round(v, 4) if isinstance(v, float) else v for k, v in out.items()}
        log(f"rollout {name}: {res[name]}")
    return res


class Workload:
    """Sets up one workload's policy and resident inputs; step() enqueues
    one pass of the hot path and returns the actions it produces."""

    def __init__(self, name, E, torch, steps):
        import synth_inputs
        self.name = name
        preset, n, seed = WORKLOADS[name]
        self.torch = torch
        kw = {}
        if name == "ragged-7b":
            kw = dict(max_envs=128, max_seq=320)
        t = time.perf_counter()
        self.pol = E.Policy(preset, seed=0, stream=torch.cuda.current_stream().cuda_stream, **kw)
        log(f"policy {name} created in {time.perf_counter() - t:.1f} s")
        c = self.pol.cfg
        self.c = c
        self.n = n
        ids = list(range(n))
        self.ids = ids
        dev = lambda a: torch.from_numpy(a).cuda()
        if name == "ragged-7b":
            # env pool: language-only prefixes of length U[200, 320] (prefilled once)
            self.T = synth_inputs.ragged_prefix_lengths(5, n, 200, 320)
            lang = synth_inputs.lang_ids(seed, ids, 320, c.vocab)
            self.pol.prefill(ids, images=None, lang_ids=dev(lang), lang_len=self.T)
            # the seeded call sequence (n ~ U[1, 128] distinct ids per call);
            # timed regions always start at its first call
            self.calls = synth_inputs.ragged_calls(5, max(steps, 1), n, 128)
            self.call_i = 0
            self.tok = torch.empty((128, c.n_action_tokens), dtype=torch.int32, device="cuda")
            self.act = torch.empty((128, c.n_action_tokens), dtype=torch.float32, device="cuda")
            # set-up, untimed: one call per batch-size class, which captures
            # the decode graph of every class once (as a server would at start)
            t = time.perf_counter()
            sizes = sorted({k if k <= 4 else min(128, (k + 7) // 8 * 8) for k in range(1, 129)})
            for k in sizes:
                self.pol.decode_actions(ids[:k], tokens=self.tok[:k], actions=self.act[:k], margins=None,
                                        with_margin=False)
            torch.cuda.synchronize()
            log(f"ragged-7b: {len(sizes)} batch-size classes captured in {time.perf_counter() - t:.1f} s")
            return
        self.img = dev(synth_inputs.pixels(seed, ids, c.n_cams, c.img, c.img))
        self.lang = dev(synth_inputs.lang_ids(seed, ids, c.n_lang, c.vocab))
        if c.exp_layers:
            self.noise = dev(synth_inputs.flow_noise(4, ids, c.chunk, c.adim))
            self.out = torch.empty_like(self.noise)
            if c.frame_tokens:
                self.fnoise = dev(synth_inputs.flow_noise(5, ids, c.frame_tokens, c.frame_dim))
                self.fout = torch.empty_like(self.fnoise)
        else:
            self.tok = torch.empty((n, c.n_action_tokens), dtype=torch.int32, device="cuda")
            self.act = torch.empty((n, c.n_action_tokens), dtype=torch.float32, device="cuda")

    def prefill(self):
        self.pol.prefill(self.ids, images=self.img, lang_ids=self.lang)

    def head(self):
        if self.c.frame_tokens:
            self.pol.wam_denoise(self.ids, self.fnoise, self.noise, out_frames=self.fout, out_actions=self.out)
            return self.n * self.c.chunk
        if self.c.exp_layers:
            self.pol.flow_denoise(self.ids, self.noise, out=self.out)
            return self.n * self.c.chunk
        self.pol.decode_actions(self.ids, tokens=self.tok, actions=self.act, margins=None, with_margin=False)
        return self.n

    def step(self):
        if self.name == "ragged-7b":
            ids = self.calls[self.call_i % len(self.calls)]
            self.call_i += 1
            k = len(ids)
            self.pol.decode_actions(ids, tokens=self.tok[:k], actions=self.act[:k], margins=None,
                                    with_margin=False)
            return k
        self.prefill()
        return self.head()


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="7b-bf16", choices=sorted(WORKLOADS))
    ap.add_argument("--cpu-sample", type=int, default=None,
                    help="envs in the oracle sample (0 = skip; default: about 10-40 s of oracle work)")
    ap.add_argument("--partitions", action="store_true",
                    help="also time the steps on CU-masked streams of 25/50/75%% of the CUs")
    ap.add_argument("--allocate", action="store_true",
                    help="ragged-7b only: measure P_gen on CU shares and run the elastic allocator on it")
    ap.add_argument("--rollout", action="store_true",
                    help="flow-bf16 only: run the rollout scheduler with this GPU's generation calls")
    ap.add_argument("--colocate", action="store_true",
                    help="also time generation on 25/50/75%% of the CUs beside a GEMM load on the rest")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: measures one GPU only (asked for --gpus {args.gpus}); environments are "
              "independent, so N GPUs would each run their own share of them with replicated weights",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2609_27547_amd import ebrl as E

    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    w = Workload(args.workload, E, torch, args.steps)
    pol, c = w.pol, w.c
    for _ in range(args.warmup):
        w.step()
    torch.cuda.synchronize()

    # ---- untimed pre-pass: which kernel class dominates this workload
    classes = list(E.KERNEL_CLASSES)
    pol.profile_enable(classes)
    for _ in range(2):
        w.step()
    pol.profile_enable([])
    pre = {cls: pol.profile_read(cls, reset=True) for cls in classes}
    dominant = max(classes, key=lambda k: pre[k]["ms"])

    # ---- timed region: K steps; the dominant kernel class timed live with HIP
    # events.  Bracketing a class's launches with events makes the calls that
    # replay a HIP graph (decode, denoise) run eagerly; where the dominant
    # class runs inside such graphs (the ragged decode's GEMMs, the flow and
    # world-model experts' GEMMs) the value is therefore timed without events
    # and the dominant class in a second pass over the same steps.
    graphed = args.workload in ("ragged-7b", "flow-bf16", "wam-bf16") or dominant in (E.K_GEMM_SKINNY,
                                                                                       E.K_ATTN_DECODE)

    def timed(instrument):
        if args.workload == "ragged-7b":
            w.call_i = 0
        pol.profile_read(dominant, reset=True)
        if instrument:
            pol.profile_enable([dominant])
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        # per-step boundaries on the same stream (one event per step: the
        # difference of consecutive ones is that step's GPU latency)
        step_ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        ev0.record(stream)
        n_act = 0
        for k in range(args.steps):
            n_act += w.step()
            step_ev[k].record(stream)
        ev1.record(stream)
        torch.cuda.synchronize()
        wall_s = time.perf_counter() - t0
        pol.profile_enable([])
        d = pol.profile_read(dominant, reset=True)
        st = np.array([ev0.elapsed_time(step_ev[0])] +
                      [step_ev[k - 1].elapsed_time(step_ev[k]) for k in range(1, args.steps)])
        return n_act, wall_s, ev0.elapsed_time(ev1), st, d

    actions, wall, gpu_ms, step_ms, dom = timed(instrument=not graphed)
    if graphed:
        _, _, gpu_ms_instr, _, dom = timed(instrument=True)
    ms_per_step = 1000.0 * wall / args.steps
    actions_per_s = actions / wall

    # ---- breakdown pass (not part of the value): every kernel class, per phase
    pol.profile_enable(classes)
    phase = {"prefill": 0.0, "head": 0.0}
    pe = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    reps = max(3, min(args.steps, 10))
    for _ in range(reps):
        pe[0].record(stream)
        if args.workload != "ragged-7b":
            w.prefill()
        pe[1].record(stream)
        if args.workload != "ragged-7b":
            w.head()
        else:
            w.step()
        pe[2].record(stream)
        torch.cuda.synchronize()
        phase["prefill"] += pe[0].elapsed_time(pe[1]) / reps
        phase["head"] += pe[1].elapsed_time(pe[2]) / reps
    pol.profile_enable([])
    kernels = {}
    class_work = {}
    for cls, name in E.KERNEL_CLASSES.items():
        r = pol.profile_read(cls, reset=True)
        class_work[cls] = r
        if r["launches"]:
            kernels[name] = {"launches_per_step": r["launches"] / reps, "ms_per_step": round(r["ms"] / reps, 4),
                             "tflops": round(r["flop"] / (r["ms"] * 1e9), 1) if r["ms"] else None,
                             "gbs": round(r["bytes"] / (r["ms"] * 1e6), 1) if r["ms"] else None}

    # roofline fraction of every kernel class (breakdown pass, per-launch
    # events): the class's algorithmic flops and bytes give the time it
    # cannot beat, max(flop / peak flop rate, bytes / peak HBM rate); the
    # larger term names the bound, and frac is that time over the measured
    # one (prefill attention over a few hundred keys has an arithmetic
    # intensity well below the chip's balance point, so HBM bounds it)
    fractions = {}
    peak_flops = (PEAK_BF16_TFLOPS if pol.bf16 else PEAK_FP32_TFLOPS) * 1e12
    for cls, name in E.KERNEL_CLASSES.items():
        k, r = kernels.get(name), class_work[cls]
        if k is None or not r["ms"] or name == "other":
            continue
        t_flop, t_byte = r["flop"] / peak_flops, r["bytes"] / (PEAK_HBM_GBS * 1e9)
        t = r["ms"] / 1e3
        fractions[name] = {"bound": "mfma" if t_flop >= t_byte else "hbm", "achieved_tflops": k["tflops"],
                           "achieved_gbs": k["gbs"], "flop_per_byte": round(r["flop"] / r["bytes"], 1) if r["bytes"] else None,
                           "frac": round(max(t_flop, t_byte) / t, 4)}

    # ---- optional: the same steps on CU-masked partitions (the stand-in for SM quotas)
    partitions = None
    read_bw = {}
    if args.partitions:
        # every share, the whole chip included, timed the same way: the same
        # steps on a stream with that CU mask, no per-kernel events (so decode
        # and denoise calls replay their graphs)
        partitions = {}
        for q in (4, 1, 2, 3):
            s_ptr = E.create_cu_masked_stream(0, balanced_mask(q))
            try:
                pol.bind_stream(s_ptr)
                if args.workload == "ragged-7b":
                    w.call_i = 0
                torch.cuda.synchronize()
                t0 = time.perf_counter()
                n_act = 0
                for k in range(args.steps):
                    n_act += w.step()
                    if (k + 1) % 500 == 0:
                        log(f"partition {q / 4:.2f}: {k + 1} of {args.steps} steps enqueued")
                torch.cuda.synchronize()
                partitions[f"{q / 4:.2f}"] = round(n_act / (time.perf_counter() - t0), 2)
                read_bw[f"{q / 4:.2f}"] = stream_read_gbs(E, torch, s_ptr)
            finally:
                pol.bind_stream(stream.cuda_stream)
                torch.cuda.synchronize()
                E.destroy_stream(s_ptr)

    coloc = colocated(E, torch, w, args) if args.colocate else None
    alloc = allocation(E, torch, w, args) if args.allocate and args.workload == "ragged-7b" else None
    roll = rollout(E, torch, w, args) if args.rollout and args.workload == "flow-bf16" else None

    bf16 = pol.bf16
    if dominant in (E.K_GEMM, E.K_ATTN_PREFILL):
        peak = PEAK_BF16_TFLOPS if bf16 else PEAK_FP32_TFLOPS
        achieved = dom["flop"] / (dom["ms"] * 1e9) if dom["ms"] else 0.0
        roofline = {"bound": "mfma", "achieved": round(achieved, 1), "peak": peak, "unit": "TFLOP/s"}
        per_launch = {"flop_per_launch": round(dom["flop"] / max(1, dom["launches"]))}
    else:
        achieved = dom["bytes"] / (dom["ms"] * 1e6) if dom["ms"] else 0.0
        roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s"}
        per_launch = {"bytes_per_launch": round(dom["bytes"] / max(1, dom["launches"]))}
    traffic = stored_traffic(args.workload) if dominant == E.K_GEMM else None
    roofline.update({"frac": round(achieved / roofline["peak"], 4),
                     "traffic": traffic["traffic_bytes_per_launch"] if traffic else None,
                     "kernel": ({E.K_GEMM: "gemm_bf16_big_kernel (projections, M >= 256)",
                                 E.K_GEMM_SKINNY: "gemm_bf16_decode_kernel (decode projections, split-K reduced in-kernel)",
                                 E.K_ATTN_PREFILL: "attn_prefill_bf16_kernel",
                                 E.K_ATTN_DECODE: "attn_decode_bf16_kernel",
                                 E.K_OTHER: "row-wise kernels"} if bf16 else
                                {E.K_GEMM: "gemm_f32_kernel (projections)",
                                 E.K_GEMM_SKINNY: "gemm_f32_kernel (decode projections, split-K partials summed by "
                                                  "splitk_reduce_kernel)",
                                 E.K_ATTN_PREFILL: "attn_prefill_f32_kernel",
                                 E.K_ATTN_DECODE: "attn_decode_split_kernel + attn_decode_combine_kernel",
                                 E.K_OTHER: "row-wise kernels"})[dominant],
                     "launches": dom["launches"],
                     "avg_launch_us": round(1000 * dom["ms"] / max(1, dom["launches"]), 2),
                     "share_of_step": round(dom["ms"] / (gpu_ms_instr if graphed else gpu_ms), 3) if gpu_ms else None,
                     "timed": ("a second pass over the same steps, this class bracketed by HIP events launch by "
                               "launch (which runs the graphed calls eagerly)") if graphed else
                              "live in the timed region, HIP events around every launch of this class"})
    roofline.update(per_launch)
    roofline["algorithmic_bytes_per_launch"] = round(dom["bytes"] / max(1, dom["launches"]))
    if traffic:
        roofline["traffic_unit"] = "bytes per launch: rocprofv3 FETCH_SIZE + WRITE_SIZE, scaled by a 1 GiB copy"
        roofline["traffic_over_algorithmic"] = round(
            traffic["traffic_bytes_per_launch"] / max(1, roofline["algorithmic_bytes_per_launch"]), 3)

    base = None
    if args.cpu_sample is None:
        args.cpu_sample = CPU_SAMPLE[args.workload]
    if args.cpu_sample > 0:
        log("timing the CPU oracle ...")
        base = cpu_baseline(args.workload, args.cpu_sample)

    preset, n, _ = WORKLOADS[args.workload]
    if args.workload == "ragged-7b":
        desc = (f"ragged-7b: preset 3 (7B-class), pool of 128 language-only prefixes (T ~ U[200, 320]), "
                f"the first {args.steps} decode calls of the seeded sequence, n ~ U[1, 128] envs each")
    elif c.frame_tokens:
        desc = (f"{args.workload}: preset {preset}, {n} envs, prefix {c.max_seq} tokens, {c.layers}-layer "
                f"d={c.d} backbone + {c.n_steps} Euler steps of the {c.exp_layers}-layer diffusion transformer over "
                f"{c.frame_tokens} future-frame latents ({c.frame_dim} ch) + chunk {c.chunk}x{c.adim} per env")
    elif c.exp_layers:
        desc = (f"{args.workload}: preset {preset}, {n} envs, prefix {c.max_seq} tokens, {c.layers}-layer "
                f"d={c.d} backbone + {c.n_steps} Euler steps of the {c.exp_layers}-layer expert, chunk {c.chunk}x{c.adim}")
    else:
        desc = (f"{args.workload}: preset {preset}, {n} envs, prefix {c.max_seq} tokens, {c.layers}-layer "
                f"d={c.d} decoder, prefill + {c.n_action_tokens - 1} decode steps")
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
        "config": {"workload": desc, "envs": n, "prefix_len": c.max_seq, "layers": c.layers, "d": c.d},
        "gpu_ms_per_step": round(gpu_ms / args.steps, 3),
        "phases_ms": {k: round(v, 3) for k, v in phase.items()},
        "kernels": kernels,
        "class_roofline_fractions": fractions,
        "roofline": roofline,
        "cpu_baseline": base,
    }
    if c.exp_layers:
        out["chunks_per_s"] = round(actions_per_s / c.chunk, 2)
    else:
        out["action_tokens_per_s"] = round(actions_per_s * c.n_action_tokens, 2)
    out["step_latency_ms"] = {"p50": round(float(np.percentile(step_ms, 50)), 3),
                              "p90": round(float(np.percentile(step_ms, 90)), 3),
                              "p99": round(float(np.percentile(step_ms, 99)), 3),
                              "max": round(float(step_ms.max()), 3)}
    if partitions:
        out["partitions_actions_per_s"] = partitions
        out["partitions_stream_read_gbs"] = read_bw
    if coloc:
        out["colocated"] = coloc
    if alloc:
        out["allocation"] = alloc
    if roll:
        out["rollout"] = roll
    print(json.dumps(out), flush=True)
    pol.close()


if __name__ == "__main__":
    main()
