"""Parity at the workloads' full sizes, in the launch configuration the
benchmark times, on outputs the oracle can compute env by env (envs are
independent, so a sampled env checks the whole batch's code path).

* 7B-class VLA (ViT + 32-layer decoder), 32 envs: sampled env against the
  oracle's teacher-forced single pass.
* flow-matching expert on the GQA backbone, 64 envs: sampled env's velocity
  at tau = 1 and its denoised chunk.
* world action model, 64 envs: sampled env's frames, actions and velocity.
* ragged asynchronous decode on the 7B-class model: a 128-slot pool of
  language-only prefixes (lengths U[200, 320]); calls of random size on the
  whole GPU and on a CU-masked stream give bitwise identical outputs, and
  eight sampled envs match the oracle.

Reference: the exact oracle (float64 throughout on the stored bf16 weights).
Bounds: 2e-2 norm-relative for rows, the 1e-2 top-2 margin rule for tokens,
and margins within what a logit row at the row bound implies -- except for
the ragged workload's language-only prefixes through the 32-layer decoder.
There, storing the K/V cache in bf16 (the format the workload fixes) already
moves the exact result 2.5-2.7e-2 on the last layer's K/V rows with every
other value kept in float64, and rounding every value a bf16 policy stores
5.1-5.5e-2 (python3 -m oracle.bf16_storage_table: the oracle alone, on the
same eight envs; RAGGED_TOL and RAGGED_MARGIN below are derived from it); no
implementation with a bf16 cache and bf16 GEMM operands meets 2e-2 on these
inputs.  The image prefixes of the
same model keep the plain bounds.
"""
import numpy as np
import pytest

import synth_inputs
from oracle import model as M
from tests import parity as P

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from paper_2609_27547_amd import ebrl as E  # noqa: E402

# Ragged workload (language-only prefixes, 32 layers): rows within 7e-2, 1.3 x
# the largest deviation (5.5e-2, layer-31 K/V) that storing the bf16
# policy's values in bf16 causes in the oracle alone on these eight envs
# (python3 -m oracle.bf16_storage_table); tokens decided by equality wherever
# the oracle's top-2 margin exceeds 0.2 (that table's largest t0 logit
# deviation is 0.19), otherwise within 0.2 of the oracle's maximum.
RAGGED_TOL = 7e-2
RAGGED_MARGIN = 0.2
RAGGED_SAMPLE = [0, 16, 32, 48, 64, 80, 96, 112]


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def report(name, value):
    print(f"PARITY {name} {value:.3e}", flush=True)


@pytest.fixture(scope="module")
def oracle_7b():
    return M.Policy(M.PRESETS[3], seed=0)


def _check_prefix(pol, e, st, layers, tag, tol=P.TOL_BF16):
    """Last prefix row (pre- and post-norm) and K/V rows of `layers` against
    the exact oracle; returns the largest deviation."""
    worst = 0.0
    checks = [("h_last_pre", pol.read_state(E.STATE_H_LAST_PRE, e), st.h_last_pre),
              ("h_last", pol.read_state(E.STATE_H_LAST, e), st.h_last)]
    for l in layers:
        for what, name, ref in [(E.STATE_K, "k", st.k[l]), (E.STATE_V, "v", st.v[l])]:
            g = P.bf16_to_f64(pol.read_state(what, e, l)).reshape(st.T, -1)
            checks.append((f"{name}{l}", g, ref.reshape(st.T, -1)))
    for name, got, ref in checks:
        err = P.row_rel_err(got, ref)
        report(f"{tag}.{name}", err)
        assert err < tol, (tag, name, err)
        worst = max(worst, err)
    return worst


def _check_tokens(tok, r, tag, thr=P.MARGIN):
    """Teacher-forced margin rule at threshold `thr`; returns how many steps
    the exact-equality branch decided."""
    strict = 0
    for k, t in enumerate(tok):
        if r.margins[k] > thr:
            assert int(t) == int(r.tokens[k]), (tag, k, int(t), int(r.tokens[k]), r.margins[k])
            strict += 1
        else:
            assert r.logits[k][int(t)] >= r.logits[k].max() - thr, (tag, k)
    report(f"{tag}.tokens_decided_exactly", strict)
    return strict


def _check_margins(pol, ref, e, mar, r, tag, tol=P.TOL_BF16):
    w = ref.W("W_act")
    hg = pol.read_state(E.STATE_H_LAST, e).astype(np.float64)
    assert abs(float(mar[0]) - P.margin_of(w, hg)) <= 1e-5 * np.linalg.norm(w @ hg)
    report(f"{tag}.margin_dev_over_bound", P.check_margins(mar, r, tol))


def test_7b_vla_full_batch_sampled_env(oracle_7b):
    cfg = M.PRESETS[3]
    ids = list(range(32))
    img = synth_inputs.pixels(1003, ids, cfg.n_cams, cfg.img, cfg.img)
    lang = synth_inputs.lang_ids(1003, ids, cfg.n_lang, cfg.vocab)
    pol = E.Policy(3, seed=0)
    pol.prefill(ids, images=_dev(img), lang_ids=_dev(lang))
    tok, act, mar = pol.decode_actions(ids)
    torch.cuda.synchronize()
    tok, mar = tok.cpu().numpy(), mar.cpu().numpy()
    e = 19
    st, r = oracle_7b.teacher_forced(img[e], lang[e], tok[e, :-1])
    _check_prefix(pol, e, st, [0, 31], "7b")
    _check_tokens(tok[e], r, "7b")
    _check_margins(pol, oracle_7b, e, mar[e], r, "7b")
    pol.close()


def test_flow_expert_full_batch_sampled_env():
    cfg = M.PRESETS[4]
    ids = list(range(64))
    img = synth_inputs.pixels(1004, ids, cfg.n_cams, cfg.img, cfg.img)
    lang = synth_inputs.lang_ids(1004, ids, cfg.n_lang, cfg.vocab)
    noise = synth_inputs.flow_noise(4, ids, cfg.chunk, cfg.adim)
    pol = E.Policy(4, seed=0)
    pol.prefill(ids, images=_dev(img), lang_ids=_dev(lang))
    out = pol.flow_denoise(ids, _dev(noise))
    torch.cuda.synchronize()
    out = out.cpu().numpy()
    ref = M.Policy(cfg, seed=0)
    e = 11
    st = ref.prefill(img[e], lang[e])
    _check_prefix(pol, e, st, [0, 17], "flow")
    x, v0 = ref.flow_denoise(st, noise[e], return_v0=True)
    gv0 = pol.read_state(E.STATE_FLOW_V0, e)
    ev, ex = P.row_rel_err(gv0, v0), P.row_rel_err(out[e], x)
    report("flow.v0", ev)
    report("flow.x10", ex)
    assert ev < P.TOL_BF16 and ex < P.TOL_BF16
    pol.close()


def test_world_action_model_full_batch_sampled_env():
    # preset 5: 64 envs, 98 frame-latent tokens + 50 action tokens each
    cfg = M.PRESETS[5]
    ids = list(range(64))
    img = synth_inputs.pixels(1005, ids, cfg.n_cams, cfg.img, cfg.img)
    lang = synth_inputs.lang_ids(1005, ids, cfg.n_lang, cfg.vocab)
    nf = synth_inputs.flow_noise(5, ids, cfg.frame_tokens, cfg.frame_dim)
    na = synth_inputs.flow_noise(6, ids, cfg.chunk, cfg.adim)
    pol = E.Policy(5, seed=0)
    pol.prefill(ids, images=_dev(img), lang_ids=_dev(lang))
    f, a = pol.wam_denoise(ids, _dev(nf), _dev(na))
    torch.cuda.synchronize()
    f, a = f.cpu().numpy(), a.cpu().numpy()
    ref = M.Policy(cfg, seed=0)
    e = 42
    st = ref.prefill(img[e], lang[e])
    xf, xa, v0 = ref.wam_denoise(st, nf[e], na[e], return_v0=True)
    ef, ea = P.row_rel_err(f[e], xf), P.row_rel_err(a[e], xa)
    ev = P.row_rel_err(pol.read_state(E.STATE_FLOW_V0, e), v0)
    report("wam.frames", ef)
    report("wam.actions", ea)
    report("wam.v0", ev)
    assert ef < P.TOL_BF16 and ea < P.TOL_BF16 and ev < P.TOL_BF16
    pol.close()


def balanced_mask(frac_quarters: int, n_cu: int = 256):
    """CU mask words selecting frac_quarters/4 of the CUs, 8-CU runs spread so
    that every XCD gets the same share whether the runtime numbers CUs XCD by
    XCD or round-robin across XCDs."""
    words = [0] * (n_cu // 32)
    for i in range(n_cu):
        if (i // 8) % 4 < frac_quarters:
            words[i // 32] |= 1 << (i % 32)
    return words


@pytest.fixture(scope="module")
def ragged(oracle_7b):
    """The ragged workload on the GPU (the seeded calls on the whole chip and
    on a quarter of it, one env alone, the eight sampled envs together) and
    the exact oracle's teacher-forced pass for each sampled env."""
    cfg = M.PRESETS[3]
    pool = 128
    T = synth_inputs.ragged_prefix_lengths(5, pool, 200, 320)
    lang = synth_inputs.lang_ids(1005, list(range(pool)), 320, cfg.vocab)
    pol = E.Policy(3, seed=0, max_envs=pool, max_seq=320)
    pol.prefill(list(range(pool)), images=None, lang_ids=_dev(lang), lang_len=T)
    calls = synth_inputs.ragged_calls(5, 3, pool, 128)
    full = []
    for ids in calls:
        tok, _, mar = pol.decode_actions(ids)
        full.append((tok.clone(), mar.clone()))
    torch.cuda.synchronize()
    masked = []
    s25 = E.create_cu_masked_stream(0, balanced_mask(1))
    try:
        pol.bind_stream(s25)
        for ids in calls:
            tok, _, mar = pol.decode_actions(ids)
            torch.cuda.synchronize()
            masked.append((tok.clone(), mar.clone()))
        pol.bind_stream(torch.cuda.current_stream().cuda_stream)
    finally:
        torch.cuda.synchronize()
        E.destroy_stream(s25)
    ids0 = calls[0]
    e = int(ids0[len(ids0) // 2])
    tok_solo, _, mar_solo = pol.decode_actions([e])
    tok_s, _, mar_s = pol.decode_actions(RAGGED_SAMPLE)
    torch.cuda.synchronize()
    sampled = []
    for i, env in enumerate(RAGGED_SAMPLE):
        st, r = oracle_7b.teacher_forced(None, lang[env][:T[env]], tok_s[i, :-1].cpu().numpy())
        sampled.append((env, st, r))
    yield dict(pol=pol, calls=calls, full=full, masked=masked, solo=(e, tok_solo, mar_solo),
               tok_s=tok_s, mar_s=mar_s, sampled=sampled)
    pol.close()


@pytest.mark.timeout(1200)
def test_ragged_decode_partitions_bitwise_and_sampled_parity(ragged, oracle_7b):
    """Bitwise: every call's tokens and margins on a quarter of the CUs equal
    the whole chip's, and an env decoded alone equals the same env inside a
    call.  Parity of the eight sampled envs at the bounds the oracle's own
    bf16 storage table gives (RAGGED_TOL, RAGGED_MARGIN)."""
    pol, calls, full = ragged["pol"], ragged["calls"], ragged["full"]
    for (tok, mar), (tok_f, mar_f) in zip(ragged["masked"], full):
        assert torch.equal(tok, tok_f) and torch.equal(mar, mar_f)
    e, tok_solo, mar_solo = ragged["solo"]
    j = list(calls[0]).index(e)
    assert torch.equal(tok_solo[0], full[0][0][j]) and torch.equal(mar_solo[0], full[0][1][j])
    tok_s, mar_s = ragged["tok_s"], ragged["mar_s"]
    if e in RAGGED_SAMPLE:
        assert torch.equal(tok_s[RAGGED_SAMPLE.index(e)], full[0][0][j])
    tok_s, mar_s = tok_s.cpu().numpy(), mar_s.cpu().numpy()
    strict, rows_within_plain = 0, 0
    for i, (env, st, r) in enumerate(ragged["sampled"]):
        worst = _check_prefix(pol, env, st, [0, 31], f"ragged{env}", tol=RAGGED_TOL)
        rows_within_plain += worst < P.TOL_BF16
        strict += _check_tokens(tok_s[i], r, f"ragged{env}", thr=RAGGED_MARGIN)
        _check_margins(pol, oracle_7b, env, mar_s[i], r, f"ragged{env}", tol=RAGGED_TOL)
    print(f"RAGGED tokens decided exactly: {strict} of {7 * len(RAGGED_SAMPLE)}; "
          f"envs with every row within 2e-2: {rows_within_plain} of {len(RAGGED_SAMPLE)}", flush=True)


@pytest.mark.xfail(reason="bf16 storage alone moves these language-only 32-layer prefixes past 2e-2 "
                          "(python3 -m oracle.bf16_storage_table: 2.5-2.7e-2 from the K/V cache alone, "
                          "5.1-5.5e-2 from every bf16 storage point)", strict=False)
def test_ragged_sampled_envs_at_the_plain_bounds(ragged):
    """The same eight sampled envs held to the plain bounds (2e-2 rows, the
    1e-2 margin rule): expected to fail for the reason the oracle's storage
    table gives, kept so that the gap stays visible."""
    pol = ragged["pol"]
    tok_s = ragged["tok_s"].cpu().numpy()
    for i, (env, st, r) in enumerate(ragged["sampled"]):
        _check_prefix(pol, env, st, [0, 31], f"ragged_plain{env}", tol=P.TOL_BF16)
        _check_tokens(tok_s[i], r, f"ragged_plain{env}", thr=P.MARGIN)
