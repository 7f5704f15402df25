"""Comparison helpers shared by the GPU parity tests (test infrastructure).

Agreement criteria for the policy forward:
* hidden states, KV rows and continuous outputs: per-row norm-relative
  error ||y - y_ref|| / ||y_ref||, maximum over rows, at most 2e-2 for bf16
  policies and 1e-4 for fp32 policies;
* action tokens, teacher-forced: the oracle re-runs decode feeding the GPU's
  own previous tokens; where the oracle's top-2 logit margin exceeds 1e-2 the
  GPU token must equal the oracle's argmax, otherwise the GPU token's oracle
  logit must be within 1e-2 of the oracle's maximum.
"""
import numpy as np

TOL_BF16 = 2e-2
TOL_FP32 = 1e-4
MARGIN = 1e-2


def bf16_to_f64(raw):
    return (np.asarray(raw).astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def row_rel_err(y, ref):
    y = np.asarray(y, dtype=np.float64).reshape(-1, np.asarray(ref).shape[-1])
    ref = np.asarray(ref, dtype=np.float64).reshape(y.shape)
    num = np.linalg.norm(y - ref, axis=-1)
    den = np.linalg.norm(ref, axis=-1)
    den = np.where(den == 0, 1.0, den)
    return float(np.max(num / den))


def check_tokens(gpu_tokens, oracle_result, n_bins=256):
    """Raises AssertionError on a violation; returns the number of steps
    decided by the margin rule (for reporting)."""
    close = 0
    for k, t in enumerate(gpu_tokens):
        lg = oracle_result.logits[k]
        if oracle_result.margins[k] > MARGIN:
            assert int(t) == int(oracle_result.tokens[k]), (
                f"step {k}: GPU token {t} vs oracle {oracle_result.tokens[k]} "
                f"(margin {oracle_result.margins[k]:.3g})")
        else:
            close += 1
            assert lg[int(t)] >= lg.max() - MARGIN, f"step {k}: token {t} not within margin"
    return close


def check_margins(gpu_margins, oracle_result, tol):
    """The GPU's top-2 margins against the teacher-forced oracle's.  A logit
    row within `tol` norm-relative of the oracle's moves each logit, and so
    the gap between two of them, by at most sqrt(2) * tol * ||logits||; the
    margin of every step is held to that.  Returns the largest deviation in
    units of that bound."""
    worst = 0.0
    for k, m in enumerate(gpu_margins):
        lg = oracle_result.logits[k]
        bound = np.sqrt(2.0) * tol * np.linalg.norm(lg)
        dev = abs(float(m) - float(oracle_result.margins[k]))
        assert dev <= bound, f"step {k}: margin {m} vs oracle {oracle_result.margins[k]} (bound {bound:.3g})"
        worst = max(worst, dev / bound)
    return worst


def margin_of(w_act, h_normed):
    """Top-1 minus top-2 of W_act . h (float64): the margin the action head
    must report for a final-normed row h."""
    s = np.sort(np.asarray(w_act, dtype=np.float64) @ np.asarray(h_normed, dtype=np.float64))
    return float(s[-1] - s[-2])
