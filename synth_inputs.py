"""Seeded synthetic inputs shared by the tests, the smoke check and the benchmark.

This module produces *inputs only* -- observation pixels, language ids,
flow-matching noise and the ragged call sequence of the asynchronous-arrival
workload.  It holds none of the policy's arithmetic, and neither the CPU
oracle nor the GPU library imports the other through it.

The generator is Philox4x32-10 (Salmon et al., SC'11), written here with
numpy integer arithmetic so every value is exact and reproducible:

* pixel p (flat index into one env's ``[cams, H, W, 3]`` image) comes from
  draw ``q = p // 4`` with counter ``(lo32(q), hi32(q), env_id, 1)`` and
  key ``(lo32(obs_seed), hi32(obs_seed))``; word ``p % 4`` of the draw gives
  ``(u32 >> 8) * 2^-24``, an exact float32 in [0, 1).
* language id j of env e uses counter ``(lo32(q), hi32(q), e, 2)``; the id
  is ``u32 mod vocab``.
* flow noise element i of env e uses counter ``(lo32(i//2), hi32(i//2), e, 3)``;
  words 0 and 1 feed a Box-Muller pair (standard normal), rounded to float32.

The workloads stand in for the paper's simulated robot observations
(camera frames and task instructions, Section 2.1): uniform pixels in [0, 1)
and uniform token ids, shaped like the evaluated policies' inputs.
"""
from __future__ import annotations

import numpy as np

_M0 = np.uint64(0xD2511F53)
_M1 = np.uint64(0xCD9E8D57)
_W0 = np.uint32(0x9E3779B9)
_W1 = np.uint32(0xBB67AE85)
_MASK = np.uint64(0xFFFFFFFF)

STREAM_PIXELS = 1
STREAM_LANG = 2
STREAM_NOISE = 3
STREAM_FRAMES = 4


def philox4x32_10(c0, c1, c2, c3, seed: int):
    """Vectorised Philox4x32-10 over uint32 arrays; returns four uint32 arrays."""
    c0 = np.asarray(c0, dtype=np.uint32)
    c1 = np.broadcast_to(np.asarray(c1, dtype=np.uint32), c0.shape).copy()
    c2 = np.broadcast_to(np.asarray(c2, dtype=np.uint32), c0.shape).copy()
    c3 = np.broadcast_to(np.asarray(c3, dtype=np.uint32), c0.shape).copy()
    c0 = c0.copy()
    k0 = np.uint32(seed & 0xFFFFFFFF)
    k1 = np.uint32((seed >> 32) & 0xFFFFFFFF)
    with np.errstate(over="ignore"):
        for r in range(10):
            if r > 0:
                k0 = np.uint32(k0 + _W0)
                k1 = np.uint32(k1 + _W1)
            p0 = _M0 * c0.astype(np.uint64)
            p1 = _M1 * c2.astype(np.uint64)
            hi0 = (p0 >> np.uint64(32)).astype(np.uint32)
            lo0 = (p0 & _MASK).astype(np.uint32)
            hi1 = (p1 >> np.uint64(32)).astype(np.uint32)
            lo1 = (p1 & _MASK).astype(np.uint32)
            c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return c0, c1, c2, c3


def _words(seed: int, env_id: int, stream: int, count: int) -> np.ndarray:
    q = np.arange((count + 3) // 4, dtype=np.uint64)
    lo = (q & _MASK).astype(np.uint32)
    hi = (q >> np.uint64(32)).astype(np.uint32)
    w = philox4x32_10(lo, hi, np.uint32(env_id), np.uint32(stream), seed)
    return np.stack(w, axis=1).reshape(-1)[:count]


def pixels(obs_seed: int, env_ids, cams: int, h: int, w: int) -> np.ndarray:
    """float32 NHWC images ``[n, cams, h, w, 3]`` with exact values (u32>>8)*2^-24."""
    per = cams * h * w * 3
    out = np.empty((len(env_ids), per), dtype=np.float32)
    for i, e in enumerate(env_ids):
        u = _words(obs_seed, int(e), STREAM_PIXELS, per)
        out[i] = (u >> np.uint32(8)).astype(np.float32) * np.float32(2.0 ** -24)
    return out.reshape(len(env_ids), cams, h, w, 3)


def lang_ids(obs_seed: int, env_ids, count: int, vocab: int) -> np.ndarray:
    """int32 token ids ``[n, count]`` uniform in [0, vocab)."""
    out = np.empty((len(env_ids), count), dtype=np.int32)
    for i, e in enumerate(env_ids):
        u = _words(obs_seed, int(e), STREAM_LANG, count)
        out[i] = (u % np.uint32(vocab)).astype(np.int32)
    return out


def flow_noise(seed: int, env_ids, chunk: int, adim: int, call: int = 0, stream: int = STREAM_NOISE) -> np.ndarray:
    """float32 standard-normal noise ``[n, chunk, adim]`` (Box-Muller on Philox):
    env e's element pair j takes counter (j, call, e, stream) under key seed,
    the convention the library follows when it draws the noise itself
    (``call`` = the env's earlier such calls; frames use stream 4)."""
    count = chunk * adim
    out = np.empty((len(env_ids), count), dtype=np.float32)
    pairs = (count + 1) // 2
    assert pairs < 2 ** 32
    lo = np.arange(pairs, dtype=np.uint32)
    hi = np.full(pairs, call, dtype=np.uint32)
    for i, e in enumerate(env_ids):
        x0, x1, _, _ = philox4x32_10(lo, hi, np.uint32(int(e)), np.uint32(stream), seed)
        u1 = (x0.astype(np.float64) + 0.5) * 2.0 ** -32
        u2 = (x1.astype(np.float64) + 0.5) * 2.0 ** -32
        r = np.sqrt(-2.0 * np.log(u1))
        z = np.stack([r * np.cos(2 * np.pi * u2), r * np.sin(2 * np.pi * u2)], axis=1).reshape(-1)
        out[i] = z[:count].astype(np.float32)
    return out.reshape(len(env_ids), chunk, adim)


def ragged_calls(seed: int, n_calls: int, pool: int, max_batch: int):
    """The asynchronous-arrival call sequence: per call, n ~ U[1, max_batch]
    distinct env ids drawn from a pool of ``pool`` slots (sorted for
    readability; order does not matter to the policy)."""
    rng = np.random.Generator(np.random.Philox(seed))
    calls = []
    for _ in range(n_calls):
        n = int(rng.integers(1, max_batch + 1))
        ids = np.sort(rng.choice(pool, size=n, replace=False)).astype(np.int32)
        calls.append(ids)
    return calls


def ragged_prefix_lengths(seed: int, pool: int, lo: int, hi: int) -> np.ndarray:
    """Per-slot prefix lengths uniform in [lo, hi] for the env pool."""
    rng = np.random.Generator(np.random.Philox(seed + 1))
    return rng.integers(lo, hi + 1, size=pool).astype(np.int32)


def sim_step_latency(seed: int, n_envs: int, n_steps: int, mean: float = 0.040, p99: float = 0.060):
    """Simulator step durations (seconds) ``[n_envs, n_steps]``: entry
    [e, k] is env e's k-th step.  Log-normal with the given overall mean and
    99th percentile (the paper reports 40 ms and 60 ms for its simulators'
    step time, Section 3.2), the log-variance split evenly between a
    persistent per-env factor (some envs are slower) and per-step noise."""
    # log-normal: mean = exp(mu + s^2 / 2), p99 = exp(mu + 2.3263 s)
    z99 = 2.3263478740408408
    # solve z99 s - s^2 / 2 = ln(p99 / mean) for the smaller root
    c = np.log(p99 / mean)
    s = z99 - np.sqrt(z99 * z99 - 2.0 * c)
    mu = np.log(mean) - 0.5 * s * s
    rng = np.random.Generator(np.random.Philox(seed))
    env = rng.normal(0.0, s / np.sqrt(2.0), size=(n_envs, 1))
    step = rng.normal(0.0, s / np.sqrt(2.0), size=(n_envs, n_steps))
    return np.exp(mu + env + step)
