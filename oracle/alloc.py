"""Oracle of the elastic resource allocator (Section 4.3.2).

Test infrastructure only: plain, slow Python that takes Algorithm 1's steps
in the paper's order, the end-to-end objective of Eq. (2), the runtime
trigger and the table refinement, under the readings that the allocator's
header lists for what the paper leaves open.  `exhaustive` is the brute force
the tests pin Algorithm 1 against.  It shares no code with the library.

Profiles are dicts of numpy arrays:
  cenv [C], ssim [S] (ascending percent), sim [C, S]
  sgen [G] (ascending percent), bgen [Bg], gen [G, Bg], gen_mem [Bg]
  strain [H], btrain [Bt], train [H, Bt], train_mem [Bt]
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


@dataclass
class Allocation:
    cenv: int
    envs: int
    ssim: int
    sgen: int
    strain: int
    bgen: int
    btrain: int
    iterations: int
    t_sim: float
    t_gen: float
    t_train: float
    t_rollout: float
    theta: float


def rate_at_quota(quotas, column, s):
    """A stage's rate at quota s (percent) from its profiled quotas: linear
    between profiled points, through rate 0 at quota 0, and held at the last
    profiled rate beyond the largest profiled quota."""
    xs = [0.0] + [float(q) for q in quotas]
    ys = [0.0] + [float(r) for r in column]
    if s <= 0:
        return 0.0
    if s >= xs[-1]:
        return ys[-1]
    for i in range(1, len(xs)):
        if s <= xs[i]:
            if s == xs[i]:
                return ys[i]
            t = (s - xs[i - 1]) / (xs[i] - xs[i - 1])
            return ys[i - 1] + t * (ys[i] - ys[i - 1])
    raise AssertionError("unreachable")


def theta(t_sim, t_gen, t_train):
    """Eq. (2): rollout is the slower of simulation and generation; the
    end-to-end rate is the slower of rollout and training."""
    t_r = min(t_sim, t_gen)
    return t_r, min(t_r, t_train)


def best_pair(P, mem, t_sim, s_g, s_t):
    """The batch-size pair of highest predicted Theta at (s_g, s_t) whose
    memory fits M_gpu; the first such pair in grid order on ties."""
    best = None
    for jg, bg in enumerate(P["bgen"]):
        t_gen = rate_at_quota(P["sgen"], P["gen"][:, jg], s_g)
        for jt, bt in enumerate(P["btrain"]):
            if P["gen_mem"][jg] + P["train_mem"][jt] > mem:
                continue
            t_train = rate_at_quota(P["strain"], P["train"][:, jt], s_t)
            t_r, th = theta(t_sim, t_gen, t_train)
            if best is None or th > best[0]:
                best = (th, int(bg), int(bt), t_gen, t_train, t_r)
    return best


def simulator_first(P, cores, knee_tol):
    """Algorithm 1's first four steps: cores per environment, concurrency,
    simulator knee quota, simulator capacity."""
    cands = [c for c in range(len(P["cenv"])) if cores // int(P["cenv"][c]) >= 1]
    if not cands:
        raise ValueError("no per-environment core count fits the core budget")
    c_star = cands[0]
    for c in cands[1:]:
        if P["sim"][c, -1] > P["sim"][c_star, -1]:
            c_star = c
    row = P["sim"][c_star]
    best = max(row)
    j_knee = next(j for j in range(len(row)) if row[j] >= (1.0 - knee_tol) * best)
    return int(P["cenv"][c_star]), cores // int(P["cenv"][c_star]), int(P["ssim"][j_knee]), float(row[j_knee])


def solve(P, cores, mem, sgen_min, strain_min, knee_tol=0.05):
    """Algorithm 1 (initial or updated profiles)."""
    c_env, E, s_sim, T_s = simulator_first(P, cores, knee_tol)
    lo, hi = sgen_min, 100 - s_sim - strain_min
    if lo > hi:
        raise ValueError("minimum quotas exceed the GPU")
    if best_pair(P, mem, T_s, lo, 100 - s_sim - lo) is None:
        raise MemoryError("no batch-size pair fits the memory budget")
    it = 0
    while hi - lo > 1:
        s_g = (lo + hi) // 2
        s_t = 100 - s_sim - s_g
        _, _, _, t_gen, t_train, t_r = best_pair(P, mem, T_s, s_g, s_t)
        if t_r > t_train:      # rollout faster: give training more compute units
            hi = s_g
        else:                  # otherwise toward a larger generation quota
            lo = s_g
        it += 1
    cand = []
    for s_g in (lo, hi):
        th, bg, bt, t_gen, t_train, t_r = best_pair(P, mem, T_s, s_g, 100 - s_sim - s_g)
        cand.append((th, s_g, bg, bt, t_gen, t_train, t_r))
    pick = cand[1] if cand[1][0] > cand[0][0] else cand[0]
    th, s_g, bg, bt, t_gen, t_train, t_r = pick
    return Allocation(c_env, E, s_sim, s_g, 100 - s_sim - s_g, bg, bt, it, T_s, t_gen, t_train, t_r, th)


def exhaustive(P, cores, mem, sgen_min, strain_min, knee_tol=0.05):
    """Brute force after the same simulator-first steps: the best Theta over
    every integer generation quota in range and every feasible batch pair."""
    c_env, E, s_sim, T_s = simulator_first(P, cores, knee_tol)
    best = None
    for s_g in range(sgen_min, 100 - s_sim - strain_min + 1):
        r = best_pair(P, mem, T_s, s_g, 100 - s_sim - s_g)
        if r is not None and (best is None or r[0] > best[0]):
            best = (r[0], s_g)
    return best


class Monitor:
    """Runtime adaptation: moving averages of the observed rollout and
    training rates over the last `window` steps; a trigger when their gap
    exceeds `gap` of the faster for `patience` consecutive steps."""

    def __init__(self, window=20, gap=0.15, patience=20):
        self.window, self.gap, self.patience = window, gap, patience
        self.hist = []
        self.streak = 0

    def observe(self, rollout, train):
        self.hist.append((rollout, train))
        self.hist = self.hist[-self.window:]
        ar = sum(h[0] for h in self.hist) / len(self.hist)
        at = sum(h[1] for h in self.hist) / len(self.hist)
        if abs(ar - at) > self.gap * max(ar, at):
            self.streak += 1
        else:
            self.streak = 0
        if self.streak >= self.patience:
            self.streak = 0
            self.hist = []
            return True
        return False


def refine(P, cur: Allocation, observed_gen, observed_train):
    """Tables updated from runtime measurements: the generation column of the
    running batch size scaled by observed / predicted, and likewise the
    training column."""
    gen = P["gen"].copy()
    train = P["train"].copy()
    jg = list(P["bgen"]).index(cur.bgen)
    jt = list(P["btrain"]).index(cur.btrain)
    if observed_gen > 0 and cur.t_gen > 0:
        gen[:, jg] = gen[:, jg] * (observed_gen / cur.t_gen)
    if observed_train > 0 and cur.t_train > 0:
        train[:, jt] = train[:, jt] * (observed_train / cur.t_train)
    return gen, train
