"""Oracle of the rollout scheduler (Sections 4.2.2 and 4.2.3, Algorithm 2,
Eq. (1)) and of the discrete-event rollout the tests drive it with.

Test infrastructure only: plain Python, independent of the library (which
implements the same model in C++ behind include/ebrl_sched.h).  The model:
envs in contiguous groups; a group receives a chunk of K actions from
generation; each env steps through its chunk on whichever core frees up;
a group whose envs have all finished its chunk joins the generation queue
(FIFO); at the start every group is queued.  On a free core, Algorithm 2
builds the ready set of Eq. (1) and takes the env with the longest recorded
step duration, envs without a recorded step first, ties to the lowest id.
"""
from __future__ import annotations

import heapq


class Scheduler:
    def __init__(self, n_envs, n_groups, K):
        if not (1 <= n_groups <= n_envs) or K < 1:
            raise ValueError("bad scheduler shape")
        self.K = K
        self.groups = [list(range(g * n_envs // n_groups, (g + 1) * n_envs // n_groups)) for g in range(n_groups)]
        self.group_of = {e: g for g, envs in enumerate(self.groups) for e in envs}
        self.s = {e: 0 for e in range(n_envs)}            # actions done in the current chunk
        self.available = set()                            # envs holding a delivered chunk
        self.running = set()
        self.H = {}                                       # last recorded step duration
        self.queue = list(range(n_groups))
        self.generating = set()
        self.n_envs = n_envs

    def ready(self, allowed=None):
        """Eq. (1): unfinished chunk, no step in flight, next action available."""
        return [e for e in range(self.n_envs)
                if self.s[e] < self.K and e not in self.running and e in self.available
                and (allowed is None or allowed(e))]

    def dispatch(self, allowed=None):
        """Algorithm 2 on one free core; returns the env, or None if idle."""
        R = self.ready(allowed)
        if not R:
            return None
        no_hist = [e for e in R if e not in self.H]
        if no_hist:
            e_star = min(no_hist)
        else:
            longest = max(self.H[e] for e in R)
            e_star = min(e for e in R if self.H[e] == longest)
        self.running.add(e_star)
        return e_star

    def complete(self, e, duration):
        """Step done: advance the action index, record the duration, clear
        the running mark; returns True when this finished the group's chunk."""
        assert e in self.running
        self.running.discard(e)
        self.s[e] += 1
        self.H[e] = duration
        g = self.group_of[e]
        if all(self.s[x] == self.K for x in self.groups[g]):
            for x in self.groups[g]:
                self.available.discard(x)
            self.queue.append(g)
            return True
        return False

    def next_group(self):
        if not self.queue:
            return None, []
        g = self.queue.pop(0)
        self.generating.add(g)
        return g, list(self.groups[g])

    def deliver(self, g):
        assert g in self.generating
        self.generating.discard(g)
        for e in self.groups[g]:
            self.s[e] = 0
            self.available.add(e)


def simulate(n_envs, n_groups, K, cores, lat, gen_latency, horizon, fixed_binding=False):
    """Discrete-event rollout.  lat[e, k] is env e's k-th step duration;
    gen_latency(env_ids) the generation time of a group.  Events at equal
    times run in the order they were scheduled; after every event the free
    cores are offered work in core order.  Returns the trace of dispatches
    (time, core, env) and completions, and the totals."""
    S = Scheduler(n_envs, n_groups, K)
    events = []
    seq = [0]

    def push(t, kind, data):
        heapq.heappush(events, (t, seq[0], kind, data))
        seq[0] += 1

    free = [True] * cores
    k_of = [0] * n_envs
    gen_busy = [False]
    trace = []
    tot = dict(steps=0, busy=0.0, chunks=0, gen_time=0.0, gen_calls=0, gen_envs=0)

    def start_generation(t):
        if gen_busy[0]:
            return
        g, ids = S.next_group()
        if g is None:
            return
        d = float(gen_latency(ids))
        gen_busy[0] = True
        tot["gen_time"] += d
        tot["gen_calls"] += 1
        tot["gen_envs"] += len(ids)
        trace.append((t, "gen", g))
        push(t + d, "gen_done", g)

    def offer_cores(t):
        for c in range(cores):
            if not free[c]:
                continue
            allowed = (lambda e, c=c: e % cores == c) if fixed_binding else None
            e = S.dispatch(allowed)
            if e is None:
                continue
            free[c] = False
            d = float(lat[e, k_of[e]])
            k_of[e] += 1
            trace.append((t, "step", c, e))
            push(t + d, "step_done", (c, e, d))

    start_generation(0.0)
    offer_cores(0.0)
    while events:
        t, _, kind, data = heapq.heappop(events)
        if t > horizon:
            break
        if kind == "gen_done":
            S.deliver(data)
            gen_busy[0] = False
            tot["chunks"] += len(S.groups[data])
            start_generation(t)
        else:
            c, e, d = data
            done = S.complete(e, d)
            free[c] = True
            tot["steps"] += 1
            tot["busy"] += d
            trace.append((t, "done", c, e))
            if done:
                start_generation(t)
        offer_cores(t)
    return trace, tot
