"""How far bf16 storage alone moves the exact oracle on the ragged workload
-- a diagnostic of the oracle, test infrastructure like the rest of oracle/.

For sampled envs of the ragged-decode workload (7B-class decoder,
language-only prefixes of U[200, 320] tokens; the same envs the full-size
GPU test samples) and for the 7B-class image prefix of that test, it runs the
oracle three ways on the same weights: exact (float64), with only the K/V
cache rounded to bf16, and with every activation storage point of a bf16
policy rounded (BF16_POINTS).  It prints, per env and variant, the
norm-relative deviation from the exact result of the last prefix row and of
the layer-0 / last-layer K and V rows, and the largest t0 logit deviation.
The bounds of the ragged GPU parity test are derived from this table.

    python3 -m oracle.bf16_storage_table [env ...]      (about 10 min per env)
"""
from __future__ import annotations

import json
import sys

import numpy as np

import synth_inputs
from oracle import model as M

RAGGED_SAMPLE = [0, 16, 32, 48, 64, 80, 96, 112]


def _rel(a, b):
    a = a.reshape(-1, b.shape[-1]) if a.ndim > 1 else a[None]
    b = b.reshape(a.shape)
    return float(np.max(np.linalg.norm(a - b, axis=-1) / np.linalg.norm(b, axis=-1)))


def main(envs):
    cfg = M.PRESETS[3]
    exact = M.Policy(cfg, seed=0)
    variants = {"exact": exact, "kv": M.Policy(cfg, seed=0, emulate_bf16={"kv"}),
                "all": M.Policy(cfg, seed=0, emulate_bf16=True)}
    for v in variants.values():
        v._raw = exact._raw                      # one copy of the generated weights
    T = synth_inputs.ragged_prefix_lengths(5, 128, 200, 320)
    lang = synth_inputs.lang_ids(1005, list(range(128)), 320, cfg.vocab)
    cases = [("ragged", e, None, lang[e][:T[e]]) for e in envs]
    ids = list(range(32))
    cases.append(("7b-image", 19, synth_inputs.pixels(1003, ids, 1, 224, 224)[19],
                  synth_inputs.lang_ids(1003, ids, cfg.n_lang, cfg.vocab)[19]))
    w = exact.W("W_act")
    for case, e, img, lg in cases:
        st = {k: p.prefill(img, lg) for k, p in variants.items()}
        ref = st["exact"]
        l_ref = w @ ref.h_last
        for k in ("kv", "all"):
            s = st[k]
            row = {"case": case, "env": int(e), "T": int(ref.T), "variant": k,
                   "h_last_pre": _rel(s.h_last_pre, ref.h_last_pre),
                   "k0": _rel(s.k[0].reshape(ref.T, -1), ref.k[0].reshape(ref.T, -1)),
                   "v0": _rel(s.v[0].reshape(ref.T, -1), ref.v[0].reshape(ref.T, -1)),
                   "k_last": _rel(s.k[-1].reshape(ref.T, -1), ref.k[-1].reshape(ref.T, -1)),
                   "v_last": _rel(s.v[-1].reshape(ref.T, -1), ref.v[-1].reshape(ref.T, -1)),
                   "t0_logit_dev": float(np.max(np.abs(w @ s.h_last - l_ref)))}
            print(json.dumps(row), flush=True)


if __name__ == "__main__":
    main([int(a) for a in sys.argv[1:]] or RAGGED_SAMPLE)
