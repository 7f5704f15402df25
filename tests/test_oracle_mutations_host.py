"""Planted mistakes in the allocator and scheduler oracles (no GPU).

As for the policy oracle: each mutant replaces one function or method of
oracle/alloc.py (Algorithm 1, Eq. (2), the runtime trigger, the table
refinement) or oracle/sched.py (Algorithm 2, Eq. (1), the group queue) with
a plausible slip, and the oracle pins of test_alloc.py / test_sched.py --
the `test_oracle_*` ones, which check the oracle against closed forms,
brute force and hand-worked schedules rather than against the library --
must fail on it.
"""
import itertools

import numpy as np
import pytest

from oracle import alloc as A
from oracle import sched as O
from tests import test_alloc as TA
from tests import test_sched as TS

# ------------------------------------------------------------ allocator --


def _rate_without_origin(quotas, column, s):
    xs = [float(q) for q in quotas]
    ys = [float(r) for r in column]
    if s <= xs[0]:
        return ys[0]
    if s >= xs[-1]:
        return ys[-1]
    return float(np.interp(s, xs, ys))


def _rate_dropping_past_the_table(quotas, column, s):
    if s > float(quotas[-1]):
        return 0.0
    return A.__dict__["_orig_rate"](quotas, column, s)


def _best_pair_ignoring_memory(P, mem, t_sim, s_g, s_t):
    return A.__dict__["_orig_best_pair"](P, float("inf"), t_sim, s_g, s_t)


def _solve(slip):
    def solve(P, cores, mem, sgen_min, strain_min, knee_tol=0.05):
        c_env, E, s_sim, T_s = A.simulator_first(P, cores, knee_tol)
        lo, hi = sgen_min, 100 - s_sim - strain_min
        if lo > hi:
            raise ValueError("minimum quotas exceed the GPU")
        if A.best_pair(P, mem, T_s, lo, 100 - s_sim - lo) is None:
            raise MemoryError("no batch-size pair fits the memory budget")
        rest = (lambda s_g: 100 - s_g) if slip == "quota_ignores_simulator" else (lambda s_g: 100 - s_sim - s_g)
        it = 0
        while hi - lo > 1:
            s_g = (lo + hi) // 2
            _, _, _, t_gen, t_train, t_r = A.best_pair(P, mem, T_s, s_g, rest(s_g))
            toward_training = t_r > t_train
            if slip == "bisection_reversed":
                toward_training = not toward_training
            if toward_training:
                hi = s_g
            else:
                lo = s_g
            it += 1
        cand = []
        for s_g in (lo, hi):
            th, bg, bt, t_gen, t_train, t_r = A.best_pair(P, mem, T_s, s_g, rest(s_g))
            cand.append((th, s_g, bg, bt, t_gen, t_train, t_r))
        pick = cand[0] if slip == "always_lower_end" else (cand[1] if cand[1][0] > cand[0][0] else cand[0])
        th, s_g, bg, bt, t_gen, t_train, t_r = pick
        return A.Allocation(c_env, E, s_sim, s_g, rest(s_g), bg, bt, it, T_s, t_gen, t_train, t_r, th)
    return solve


def _simulator_first(slip):
    def simulator_first(P, cores, knee_tol):
        cands = [c for c in range(len(P["cenv"])) if cores // int(P["cenv"][c]) >= 1]
        if not cands:
            raise ValueError("no per-environment core count fits the core budget")
        c_star = cands[0]
        for c in cands[1:]:
            if P["sim"][c, -1] > P["sim"][c_star, -1]:
                c_star = c
        row = P["sim"][c_star]
        best = max(row)
        tol = 0.0 if slip == "knee_at_the_maximum" else knee_tol
        j_knee = next(j for j in range(len(row)) if row[j] >= (1.0 - tol) * best)
        E = cores if slip == "one_core_per_env" else cores // int(P["cenv"][c_star])
        return int(P["cenv"][c_star]), E, int(P["ssim"][j_knee]), float(row[j_knee])
    return simulator_first


class _MonitorAgainstSlower(A.Monitor):
    def observe(self, rollout, train):
        self.hist.append((rollout, train))
        self.hist = self.hist[-self.window:]
        ar = sum(h[0] for h in self.hist) / len(self.hist)
        at = sum(h[1] for h in self.hist) / len(self.hist)
        if abs(ar - at) > self.gap * min(ar, at):
            self.streak += 1
        else:
            self.streak = 0
        if self.streak >= self.patience:
            self.streak = 0
            self.hist = []
            return True
        return False


class _MonitorOffByOne(A.Monitor):
    def observe(self, rollout, train):
        self.hist.append((rollout, train))
        self.hist = self.hist[-self.window:]
        ar = sum(h[0] for h in self.hist) / len(self.hist)
        at = sum(h[1] for h in self.hist) / len(self.hist)
        self.streak = self.streak + 1 if abs(ar - at) > self.gap * max(ar, at) else 0
        if self.streak > self.patience:
            self.streak = 0
            self.hist = []
            return True
        return False


def _refine_inverted(P, cur, observed_gen, observed_train):
    gen, train = P["gen"].copy(), P["train"].copy()
    jg = list(P["bgen"]).index(cur.bgen)
    jt = list(P["btrain"]).index(cur.btrain)
    if observed_gen > 0 and cur.t_gen > 0:
        gen[:, jg] = gen[:, jg] * (cur.t_gen / observed_gen)
    if observed_train > 0 and cur.t_train > 0:
        train[:, jt] = train[:, jt] * (cur.t_train / observed_train)
    return gen, train


ALLOC_MUTANTS = {
    "Eq. (2): rollout as the faster stage": ("theta", lambda s, g, t: (max(s, g), min(max(s, g), t))),
    "Eq. (2): end-to-end as the faster stage": ("theta", lambda s, g, t: (min(s, g), max(min(s, g), t))),
    "rates not anchored at zero quota": ("rate_at_quota", _rate_without_origin),
    "rates dropping past the profiled quotas": ("rate_at_quota", _rate_dropping_past_the_table),
    "batch pairs ignoring the memory budget": ("best_pair", _best_pair_ignoring_memory),
    "bisection moving the wrong way": ("solve", _solve("bisection_reversed")),
    "training quota ignoring the simulator's": ("solve", _solve("quota_ignores_simulator")),
    "always the lower bisection end": ("solve", _solve("always_lower_end")),
    "simulator knee at the maximum": ("simulator_first", _simulator_first("knee_at_the_maximum")),
    "one core per environment": ("simulator_first", _simulator_first("one_core_per_env")),
    "trigger gap against the slower rate": ("Monitor", _MonitorAgainstSlower),
    "trigger one step late": ("Monitor", _MonitorOffByOne),
    "refinement scaling inverted": ("refine", _refine_inverted),
}

# ------------------------------------------------------------ scheduler --


def _dispatch(slip):
    def dispatch(self, allowed=None):
        R = self.ready(allowed)
        if not R:
            return None
        no_hist = [e for e in R if e not in self.H]
        if no_hist and slip != "history_first":
            e_star = min(no_hist)
        else:
            hist = [e for e in R if e in self.H] or R
            pick = min if slip == "shortest_first" else max
            ext = pick(self.H.get(e, 0.0) for e in hist)
            tied = [e for e in hist if self.H.get(e, 0.0) == ext]
            e_star = max(tied) if slip == "ties_to_highest" else min(tied)
        self.running.add(e_star)
        return e_star
    return dispatch


def _ready_ignoring_running(self, allowed=None):
    return [e for e in range(self.n_envs)
            if self.s[e] < self.K and e in self.available and (allowed is None or allowed(e))]


def _complete(slip):
    def complete(self, e, duration):
        assert e in self.running
        self.running.discard(e)
        self.s[e] += 1
        self.H[e] = self.H.get(e, 0.0) + duration if slip == "cumulative_history" else duration
        g = self.group_of[e]
        test = any if slip == "any_env_finishes" else all
        if test(self.s[x] == self.K for x in self.groups[g]):
            for x in self.groups[g]:
                self.available.discard(x)
            self.queue.append(g)
            return True
        return False
    return complete


def _next_group_lifo(self):
    if not self.queue:
        return None, []
    g = self.queue.pop()
    self.generating.add(g)
    return g, list(self.groups[g])


SCHED_MUTANTS = {
    "Algorithm 2: shortest step first": ("dispatch", _dispatch("shortest_first")),
    "Algorithm 2: ties to the highest id": ("dispatch", _dispatch("ties_to_highest")),
    "Algorithm 2: envs with history first": ("dispatch", _dispatch("history_first")),
    "Eq. (1): running envs counted as ready": ("ready", _ready_ignoring_running),
    "step history accumulated": ("complete", _complete("cumulative_history")),
    "group queued when any env finishes": ("complete", _complete("any_env_finishes")),
    "generation queue last in, first out": ("next_group", _next_group_lifo),
}

# ------------------------------------------------------------------ runs --


def _calls(fn):
    """Every call of a pin: one per parameter combination of its
    parametrize marks (pins here take no fixtures)."""
    marks = [m for m in getattr(fn, "pytestmark", []) if m.name == "parametrize"]
    if not marks:
        return [{}]
    grids = []
    for m in marks:
        names = [n.strip() for n in m.args[0].split(",")] if isinstance(m.args[0], str) else list(m.args[0])
        vals = [v if len(names) > 1 else (v,) for v in m.args[1]]
        grids.append([dict(zip(names, v)) for v in vals])
    out = []
    for combo in itertools.product(*grids):
        d = {}
        for part in combo:
            d.update(part)
        out.append(d)
    return out


def _run(module):
    caught = []
    for name, fn in sorted(vars(module).items()):
        if not (name.startswith("test_oracle_") and callable(fn)):
            continue
        for kw in _calls(fn):
            try:
                with np.errstate(all="ignore"):
                    fn(**kw)
            except Exception:       # an assertion, or the mutant breaking the run
                caught.append(name)
                break
    return caught


def test_host_pins_pass_on_the_oracles_as_written():
    assert _run(TA) == [] and _run(TS) == []


@pytest.mark.parametrize("mutant", sorted(ALLOC_MUTANTS))
def test_allocator_pins_catch_planted_mistake(mutant, monkeypatch):
    target, repl = ALLOC_MUTANTS[mutant]
    monkeypatch.setitem(A.__dict__, "_orig_rate", A.rate_at_quota)
    monkeypatch.setitem(A.__dict__, "_orig_best_pair", A.best_pair)
    monkeypatch.setattr(A, target, repl)
    caught = _run(TA)
    print(f"{mutant}: caught by {caught}", flush=True)
    assert caught, f"no allocator pin fails when the oracle has: {mutant}"


@pytest.mark.parametrize("mutant", sorted(SCHED_MUTANTS))
def test_scheduler_pins_catch_planted_mistake(mutant, monkeypatch):
    target, repl = SCHED_MUTANTS[mutant]
    monkeypatch.setattr(O.Scheduler, target, repl)
    caught = _run(TS)
    print(f"{mutant}: caught by {caught}", flush=True)
    assert caught, f"no scheduler pin fails when the oracle has: {mutant}"
