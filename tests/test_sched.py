"""The rollout scheduler (Sections 4.2.2-4.2.3, Algorithm 2, Eq. (1)): the
oracle pinned by hand-worked schedules, then the library's scheduler and its
event-driven rollout (paper_2609_27547_amd/rollout.py) checked against the
oracle's on seeded latency tables.  Host logic only; no GPU."""
import numpy as np
import pytest

import synth_inputs
from oracle import sched as O

E = pytest.importorskip("paper_2609_27547_amd.ebrl")
from paper_2609_27547_amd import rollout as R  # noqa: E402


# ------------------------------------------------------------- oracle pins --

def test_oracle_algorithm2_priority():
    S = O.Scheduler(4, 1, 3)
    assert S.dispatch() is None                          # no chunk delivered yet
    g, ids = S.next_group()
    assert (g, ids) == (0, [0, 1, 2, 3])
    S.deliver(0)
    # no recorded step: lowest id first
    assert [S.dispatch() for _ in range(4)] == [0, 1, 2, 3]
    assert S.dispatch() is None                          # all running
    for e, d in [(2, 0.05), (0, 0.03), (1, 0.07), (3, 0.01)]:
        assert not S.complete(e, d)
    # longest recorded step first
    assert [S.dispatch() for _ in range(4)] == [1, 2, 0, 3]


def test_oracle_algorithm2_ranks_by_the_last_recorded_step():
    # env 0 steps 5 then 1, env 1 steps 2: by the last recorded durations
    # (1 vs 2) env 1 goes next; by accumulated time (6 vs 2) env 0 would
    S = O.Scheduler(2, 1, 3)
    S.next_group()
    S.deliver(0)
    assert [S.dispatch(), S.dispatch()] == [0, 1]
    assert not S.complete(0, 5.0) and not S.complete(1, 2.0)
    assert S.dispatch() == 0                             # 5 > 2
    assert not S.complete(0, 1.0)
    assert S.dispatch() == 1                             # last steps: 2 > 1


def test_oracle_ready_set_and_group_queue():
    S = O.Scheduler(4, 2, 1)
    assert S.next_group() == (0, [0, 1]) and S.next_group() == (1, [2, 3])
    assert S.next_group() == (None, [])
    S.deliver(1)
    assert S.ready() == [2, 3]
    e = S.dispatch()
    assert e == 2 and S.ready() == [3]                   # running envs are not ready
    assert not S.complete(2, 0.1)
    assert S.ready() == [3]                              # chunk of length 1 finished
    e = S.dispatch()
    assert S.complete(e, 0.2)                            # last env of group 1: queued
    assert S.queue == [1] and S.ready() == []
    S.deliver(0)
    assert S.ready() == [0, 1]


def test_oracle_hand_worked_rollout():
    # 2 cores, groups {0, 1} and {2, 3}, chunks of 2 actions; per-env step
    # durations 1, 3, 2, 2 units and 0.5 units of generation per group (a
    # unit of 1/64 s keeps every sum exact, so equal times are real ties).
    # The schedule, worked by hand from Algorithm 2 and the group pipeline:
    u = 1.0 / 64
    lat = np.array([[1 * u] * 8, [3 * u] * 8, [2 * u] * 8, [2 * u] * 8])
    trace, tot = O.simulate(4, 2, 2, 2, lat, lambda ids: 0.5 * u, horizon=10 * u)
    want = [
        (0.0, "gen", 0),
        (0.5, "gen", 1), (0.5, "step", 0, 0), (0.5, "step", 1, 1),
        (1.5, "done", 0, 0), (1.5, "step", 0, 2),                  # no-history env 2 before env 0
        (3.5, "done", 1, 1), (3.5, "step", 1, 3),                  # no-history env 3 first
        (3.5, "done", 0, 2), (3.5, "step", 0, 1),                  # longest recorded: env 1 (3 units)
        (5.5, "done", 1, 3), (5.5, "step", 1, 2),                  # 2 and 3 tie at 2 units: lower id
        (6.5, "done", 0, 1), (6.5, "step", 0, 3),
        (7.5, "done", 1, 2), (7.5, "step", 1, 0),
        (8.5, "done", 0, 3), (8.5, "gen", 1),                      # group 1 finished its chunk
        (8.5, "done", 1, 0),                                       # group 0 queued behind it
        (9.0, "gen", 0), (9.0, "step", 0, 2), (9.0, "step", 1, 3),
    ]
    assert [(r[0] / u,) + tuple(r[1:]) for r in trace] == want
    assert tot["steps"] == 8 and tot["chunks"] == 8 and tot["gen_calls"] == 4


def test_oracle_fixed_binding_keeps_envs_on_their_core():
    lat = synth_inputs.sim_step_latency(3, 8, 400)
    trace, _ = O.simulate(8, 2, 5, 3, lat, lambda ids: 0.02, horizon=2.0, fixed_binding=True)
    assert all(r[3] % 3 == r[2] for r in trace if r[1] == "step")


def test_oracle_chunk_order_and_no_double_dispatch():
    lat = synth_inputs.sim_step_latency(4, 24, 2000)
    trace, tot = O.simulate(24, 4, 8, 6, lat, lambda ids: 0.01 + 0.001 * len(ids), horizon=5.0)
    running, per_chunk = set(), {}
    for r in trace:
        if r[1] == "step":
            assert r[3] not in running
            running.add(r[3])
            per_chunk[r[3]] = per_chunk.get(r[3], 0) + 1
            assert per_chunk[r[3]] <= 8                  # never past the chunk's actions
        elif r[1] == "done":
            running.discard(r[3])
        else:
            for e in range(r[2] * 6, r[2] * 6 + 6):      # a group goes to generation:
                assert per_chunk.get(e, 0) in (0, 8)    # all its envs finished their chunk
                per_chunk[e] = 0
    assert tot["steps"] > 0


# --------------------------------------------------- library against oracle --

def test_library_scheduler_matches_oracle_step_by_step():
    rng = np.random.default_rng(0)
    for _ in range(30):
        n = int(rng.integers(1, 20))
        G = int(rng.integers(1, n + 1))
        K = int(rng.integers(1, 5))
        S_o, S_l = O.Scheduler(n, G, K), E.Sched(n, G, K)
        for _ in range(300):
            op = rng.integers(0, 3)
            if op == 0:
                got = S_l.dispatch()
                want = S_o.dispatch()
                assert got == (-1 if want is None else want)
            elif op == 1 and S_o.running:
                e = int(rng.choice(sorted(S_o.running)))
                d = float(rng.choice([0.01, 0.02, rng.uniform(0, 0.1)]))
                assert S_l.complete(e, d) == S_o.complete(e, d)
            elif op == 2:
                g_o, ids_o = S_o.next_group()
                g_l, ids_l = S_l.next_group()
                assert g_l == (-1 if g_o is None else g_o) and list(ids_l) == ids_o
                if g_o is not None:
                    S_o.deliver(g_o)
                    S_l.deliver(g_l)
        S_l.close()


@pytest.mark.parametrize("fixed", [False, True])
def test_library_rollout_matches_oracle(fixed):
    for seed in range(4):
        n, G, K, C = [(32, 4, 8, 8), (64, 4, 5, 16), (17, 3, 3, 5), (48, 6, 1, 12)][seed]
        lat = synth_inputs.sim_step_latency(10 + seed, n, 4000)
        gen = lambda ids: 0.004 + 0.0007 * len(ids)
        tr_l = []
        out = R.run(n, G, K, C, lat, gen, horizon=6.0, fixed_binding=fixed, trace=tr_l)
        tr_o, tot = O.simulate(n, G, K, C, lat, gen, horizon=6.0, fixed_binding=fixed)
        assert tr_l == tr_o
        assert out["env_steps"] == tot["steps"] and out["chunks"] == tot["chunks"]


def test_library_scheduler_errors():
    with pytest.raises(E.EbrlError):
        E.Sched(4, 5, 1)
    with pytest.raises(E.EbrlError):
        E.Sched(4, 1, 0)
    S = E.Sched(4, 2, 2)
    with pytest.raises(E.EbrlError) as ex:
        S.complete(0, 0.01)                              # nothing in flight
    assert ex.value.code == -4
    with pytest.raises(E.EbrlError):
        S.deliver(0)                                     # not popped yet
    with pytest.raises(E.EbrlError):
        S.dispatch(3, 2)                                 # core outside the binding stride
    S.close()
