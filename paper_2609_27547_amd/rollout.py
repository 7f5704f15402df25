"""Discrete-event rollout around the library's scheduler (include/ebrl_sched.h).

Simulator workers are stood in for by a table of step durations (the
paper's simulators are out of scope); the generation stage is a callable
that takes a group's env ids and returns how long generating its next chunk
took -- with a GPU, the time of the real prefill + action-head calls for
that ragged group.  The event loop keeps one generation stage (groups served
in the order they finished) and `cores` CPU cores; after every event, each
free core asks the scheduler for work (Algorithm 2, or the fixed binding it
is compared with).  Time is simulated, so a run over a horizon of seconds
takes milliseconds of host time plus the generation calls.
"""
from __future__ import annotations

import heapq
import itertools
from typing import Callable, Sequence

from . import ebrl as E

GEN_DONE, STEP_DONE = 0, 1


def run(n_envs: int, n_groups: int, chunk_len: int, cores: int, step_latency, generate: Callable[[Sequence[int]], float],
        horizon: float, fixed_binding: bool = False, trace: list | None = None) -> dict:
    """Rolls out until simulated time `horizon` (seconds).  step_latency[e][k]
    is env e's k-th step duration.  Returns env steps, chunks delivered, core
    and generation busy time and the mean generation batch; `trace`, if
    given, receives (time, "gen", group) / ("step", core, env) /
    ("done", core, env) records."""
    sched = E.Sched(n_envs, n_groups, chunk_len)
    stride = cores if fixed_binding else 0
    order = itertools.count()
    heap: list = []
    core_busy = [False] * cores
    steps_taken = [0] * n_envs
    gen = {"busy": False}
    out = {"env_steps": 0, "chunks": 0, "core_busy_s": 0.0, "gen_busy_s": 0.0, "gen_calls": 0, "gen_envs": 0}
    rec = trace.append if trace is not None else (lambda _: None)

    def generation(now):
        if gen["busy"]:
            return
        group, ids = sched.next_group()
        if group < 0:
            return
        took = float(generate(ids))
        gen["busy"] = True
        out["gen_busy_s"] += took
        out["gen_calls"] += 1
        out["gen_envs"] += len(ids)
        rec((now, "gen", group))
        heapq.heappush(heap, (now + took, next(order), GEN_DONE, group, len(ids)))

    def cores_take_work(now):
        for c in range(cores):
            if core_busy[c]:
                continue
            e = sched.dispatch(c, stride)
            if e < 0:
                continue
            core_busy[c] = True
            d = float(step_latency[e][steps_taken[e]])
            steps_taken[e] += 1
            rec((now, "step", c, e))
            heapq.heappush(heap, (now + d, next(order), STEP_DONE, (c, e, d), 0))

    generation(0.0)
    cores_take_work(0.0)
    try:
        while heap:
            now, _, kind, what, size = heapq.heappop(heap)
            if now > horizon:
                break
            if kind == GEN_DONE:
                sched.deliver(what)
                gen["busy"] = False
                out["chunks"] += size
                generation(now)
            else:
                c, e, d = what
                finished_group = sched.complete(e, d)
                core_busy[c] = False
                out["env_steps"] += 1
                out["core_busy_s"] += d
                rec((now, "done", c, e))
                if finished_group:
                    generation(now)
            cores_take_work(now)
    finally:
        sched.close()
    out["env_steps_per_s"] = out["env_steps"] / horizon
    out["core_utilisation"] = out["core_busy_s"] / (cores * horizon)
    out["gen_utilisation"] = out["gen_busy_s"] / horizon
    out["mean_gen_batch"] = out["gen_envs"] / max(1, out["gen_calls"])
    return out
