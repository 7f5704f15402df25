"""Pins of the CPU oracle against facts fixed by mathematics and by the
published algorithms it follows (no GPU).

Each test checks the oracle against something other than itself: closed
forms, special cases that reduce to a textbook result, brute force on tiny
integer inputs, invariants, or a second independent implementation of a
published algorithm.  The paper prints no worked example of the policy
forward, so there is no golden tensor from the paper to compare against;
the one stored fixture (tests/golden) holds the published known-answer
vectors of the Philox generator.
"""
import dataclasses
import math

import numpy as np
import pytest

import synth_inputs
from oracle import model as M

TINY = M.PRESETS[1]


def tiny_cfg(**kw):
    base = dict(name="pin", bf16=False, n_cams=1, img=32, patch=16, layers=2, d=32,
                q_heads=4, kv_heads=4, head_dim=8, mlp=48, vocab=50, n_lang=5)
    base.update(kw)
    return M.Config(**base)


# ---------------------------------------------------------------- RNG ----


def _philox_kat():
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "philox4x32_10_kat.txt")
    rows = []
    for line in open(path):
        line = line.split("#")[0].split()
        if line:
            v = [int(x, 16) for x in line]
            rows.append((v[0:4], v[4] | (v[5] << 32), v[6:10]))
    return rows


def test_philox_published_known_answers():
    # Published known-answer vectors of Philox4x32-10 (tests/golden): pins
    # both implementations to the algorithm itself, not just to each other.
    rows = _philox_kat()
    assert len(rows) == 3
    for ctr, seed, want in rows:
        assert [int(x) for x in M.philox_words(seed, ctr)] == want
        got = synth_inputs.philox4x32_10(np.array(ctr[0:1], np.uint32), np.array(ctr[1:2], np.uint32),
                                         np.array(ctr[2:3], np.uint32), np.array(ctr[3:4], np.uint32), seed)
        assert [int(w[0]) for w in got] == want


def test_philox_two_independent_implementations_agree():
    # The oracle's C Philox and the input generator's numpy Philox are
    # written separately from the published definition; a typo in either
    # (a constant, the word permutation, the key schedule) breaks agreement.
    rng = np.random.default_rng(123)
    for _ in range(50):
        ctr = rng.integers(0, 2 ** 32, size=4, dtype=np.uint64).astype(np.uint32)
        seed = int(rng.integers(0, 2 ** 63))
        a = M.philox_words(seed, ctr)
        b = synth_inputs.philox4x32_10(ctr[0:1], ctr[1:2], ctr[2:3], ctr[3:4], seed)
        assert [int(x[0]) for x in b] == [int(x) for x in a]


def test_philox_words_uniform_and_counter_sensitive():
    seed = 7
    q = np.arange(1 << 16, dtype=np.uint32)
    w = synth_inputs.philox4x32_10(q, 0, 0, 0, seed)
    words = np.concatenate(w)
    # top byte histogram: chi-square with 255 dof, mean 255, sd ~22.6
    h = np.bincount(words >> np.uint32(24), minlength=256)
    e = len(words) / 256
    chi2 = float(((h - e) ** 2 / e).sum())
    assert chi2 < 255 + 6 * 22.6
    # a one-bit counter change flips about half of the 128 output bits
    a = np.stack(synth_inputs.philox4x32_10(q[:1000], 0, 0, 0, seed), 1)
    b = np.stack(synth_inputs.philox4x32_10(q[:1000] ^ np.uint32(1), 0, 0, 0, seed), 1)
    flips = np.unpackbits((a ^ b).view(np.uint8)).reshape(1000, -1).sum(1)
    assert abs(flips.mean() - 64) < 2


def test_normal_weights_moments():
    n = 4_000_000
    z = M.gen_tensor(11, 99, (n,), 1.0, bf16=False).astype(np.float64)
    assert abs(z.mean()) < 4 / math.sqrt(n)
    assert abs(z.var() - 1) < 4 * math.sqrt(2 / n)
    # fourth moment of a Gaussian is 3 (catches a uniform or triangular slip)
    assert abs((z ** 4).mean() - 3) < 0.05
    w = M.gen_tensor(11, 99, (1000,), 0.02, bf16=False)
    # same draws scaled by the std (z above was rounded to fp32 once already)
    assert np.allclose(w, z[:1000] * 0.02, rtol=2e-7, atol=0)


def test_bf16_weights_are_nearest_even_rounding_of_fp32():
    f = M.gen_tensor(3, 17, (100_000,), 0.02, bf16=False).astype(np.float64)
    b = M.bf16_bits_to_f64(M.gen_tensor(3, 17, (100_000,), 0.02, bf16=True))
    assert np.array_equal(b, M.f64_to_bf16_value(f))
    # ties: 1 + 2^-8 is halfway between 1 and 1 + 2^-7 -> even (1)
    assert M.f64_to_bf16_value(np.array([1 + 2 ** -8]))[0] == 1.0
    assert M.f64_to_bf16_value(np.array([1 + 3 * 2 ** -8]))[0] == 1 + 2 ** -6
    assert np.max(np.abs(b - f) / np.abs(f)) <= 2 ** -8


# ------------------------------------------------------- elementary ops ----


def test_linear_brute_force_integer_and_one_hot():
    rng = np.random.default_rng(0)
    x = rng.integers(-5, 6, size=(3, 4)).astype(np.float64)
    w = rng.integers(-5, 6, size=(5, 4)).astype(np.float64)   # [out, in]
    y = M.linear(x, w)
    for i in range(3):
        for o in range(5):
            assert y[i, o] == sum(x[i, k] * w[o, k] for k in range(4))
    one_hot = np.zeros((5, 4))
    one_hot[2, 3] = 1.0
    y = M.linear(x, one_hot)
    assert np.array_equal(y[:, 2], x[:, 3]) and not y[:, [0, 1, 3, 4]].any()


def test_softmax_sums_to_one_and_shift_invariant():
    rng = np.random.default_rng(1)
    s = rng.normal(size=(7, 33)) * 10
    p = M.softmax(s)
    assert np.all(np.abs(p.sum(-1) - 1) <= 1e-12)
    assert np.allclose(M.softmax(s + 123.0), p, rtol=1e-12, atol=0)
    two = M.softmax(np.array([[0.0, math.log(3.0)]]))
    assert np.allclose(two, [[0.25, 0.75]], atol=1e-15)


def test_attention_single_key_mean_scale_and_causal():
    rng = np.random.default_rng(2)
    q = rng.normal(size=(3, 8))
    k1 = rng.normal(size=(1, 8))
    v1 = rng.normal(size=(1, 8))
    pos = np.arange(3)
    out = M.attention(q, k1, v1, pos + 5, np.array([0]), causal=True)
    assert np.array_equal(out, np.repeat(v1, 3, axis=0))
    K = np.repeat(k1, 4, axis=0)
    V = rng.normal(size=(4, 8))
    out = M.attention(q, K, V, pos + 5, np.arange(4), causal=False)
    assert np.allclose(out, V.mean(0)[None].repeat(3, 0), atol=1e-14)
    # scale 1/sqrt(hd): with q.k = a, b the weights are softmax([a, b]/sqrt(8))
    qq = np.zeros((1, 8)); qq[0, 0] = 1.0
    KK = np.zeros((2, 8)); KK[0, 0] = 2.0; KK[1, 0] = -1.0
    VV = np.array([[1.0] + [0] * 7, [0.0, 1.0] + [0] * 6])
    out = M.attention(qq, KK, VV, np.array([9]), np.arange(2), causal=True)
    w = np.exp(np.array([2.0, -1.0]) / math.sqrt(8))
    w /= w.sum()
    assert np.allclose(out[0, :2], w, atol=1e-15)
    # causal: query at position 0 sees key 0 only
    Kc = rng.normal(size=(3, 8))
    Vc = rng.normal(size=(3, 8))
    out = M.attention(q, Kc, Vc, pos, pos, causal=True)
    assert np.allclose(out[0], Vc[0], atol=1e-15)
    # and query 1 does not depend on key/value 2
    Kc2, Vc2 = Kc.copy(), Vc.copy()
    Kc2[2] += 5
    Vc2[2] -= 3
    out2 = M.attention(q, Kc2, Vc2, pos, pos, causal=True)
    assert np.array_equal(out[:2], out2[:2])


def test_grouped_kv_heads_map_h_to_h_over_group():
    rng = np.random.default_rng(3)
    q = rng.normal(size=(4, 6, 8))
    k = rng.normal(size=(5, 2, 8))
    v = rng.normal(size=(5, 2, 8))
    pos = np.arange(4) + 1
    kp = np.arange(5)
    g = M.multihead_attention(q, k, v, pos, kp, True)
    # the equivalent MHA repeats each KV head for its group of 3 query heads
    full = M.multihead_attention(q, np.repeat(k, 3, axis=1), np.repeat(v, 3, axis=1), pos, kp, True)
    assert np.array_equal(g, full)
    assert np.allclose(g[:, 2], M.attention(q[:, 2], k[:, 0], v[:, 0], pos, kp, True))
    assert np.allclose(g[:, 3], M.attention(q[:, 3], k[:, 1], v[:, 1], pos, kp, True))


def test_rope_rotate_half_pairs_angles_and_relative_position():
    # hd = 4: pairs (0, 2) rotate by p * 1 and (1, 3) by p * 10000^(-1/2)
    e0 = np.array([[[1.0, 0, 0, 0]]])
    e1 = np.array([[[0, 1.0, 0, 0]]])
    for p in [0, 1, 7]:
        r0 = M.rope(e0, np.array([p]))[0, 0]
        r1 = M.rope(e1, np.array([p]))[0, 0]
        assert np.allclose(r0, [math.cos(p), 0, math.sin(p), 0], atol=1e-15)
        a = p * 0.01
        assert np.allclose(r1, [0, math.cos(a), 0, math.sin(a)], atol=1e-15)
    rng = np.random.default_rng(4)
    x = rng.normal(size=(3, 2, 16))
    assert np.array_equal(M.rope(x, np.zeros(3, dtype=int)), x)
    r = M.rope(x, np.array([3, 50, 900]))
    assert np.allclose(np.linalg.norm(r, axis=-1), np.linalg.norm(x, axis=-1), atol=1e-12)
    q = rng.normal(size=(1, 1, 16))
    k = rng.normal(size=(1, 1, 16))
    dots = [float(np.sum(M.rope(q, np.array([m])) * M.rope(k, np.array([m - 4]))))
            for m in [4, 10, 333]]
    assert np.allclose(dots, dots[0], atol=1e-12)


def test_rmsnorm_closed_form_scale_invariance_unit_rms():
    x = np.array([3.0, 4.0])
    assert np.allclose(M.rmsnorm(x), x / math.sqrt(12.5 + 1e-6), atol=0, rtol=1e-15)
    rng = np.random.default_rng(5)
    y = rng.normal(size=(4, 64)) * 10
    assert np.allclose(M.rmsnorm(y * 7.5), M.rmsnorm(y), atol=1e-14)
    rms = np.sqrt(np.mean(M.rmsnorm(y) ** 2, axis=-1))
    assert np.allclose(rms, 1.0, atol=1e-7)


def test_silu_properties():
    x = np.linspace(-30, 30, 121)
    s = M.silu(x)
    assert M.silu(np.array([0.0]))[0] == 0.0
    assert np.allclose(s - M.silu(-x), x, atol=1e-12)           # silu(x) - silu(-x) = x
    assert abs(M.silu(np.array([1.0]))[0] - 1 / (1 + math.exp(-1))) < 1e-16


def test_patchify_raster_order_and_inner_index():
    cams, H, W, P = 2, 4, 6, 2
    img = np.zeros((cams, H, W, 3))
    for c in range(cams):
        for y in range(H):
            for x in range(W):
                for ch in range(3):
                    img[c, y, x, ch] = c * 10000 + y * 100 + x * 10 + ch
    p = M.patchify(img, P)
    assert p.shape == (cams * (H // P) * (W // P), P * P * 3)
    # patch index = cam * 6 + py * 3 + px ; element (dy * P + dx) * 3 + ch
    cam, py, px, dy, dx, ch = 1, 1, 2, 1, 0, 2
    row = cam * 6 + py * 3 + px
    col = (dy * P + dx) * 3 + ch
    assert p[row, col] == cam * 10000 + (py * P + dy) * 100 + (px * P + dx) * 10 + ch


def test_argmax_ties_lowest_and_detokenize_endpoints():
    assert M.argmax_lowest(np.array([0.0, 2.0, 2.0, 1.0])) == 1
    assert M.argmax_lowest(np.zeros(256)) == 0
    oh = np.zeros(256); oh[200] = 1.0
    assert M.argmax_lowest(oh) == 200
    assert M.top2_margin(np.array([1.0, 3.5, 2.0])) == 1.5
    assert M.detokenize(0) == -1 + 1 / 256
    assert M.detokenize(255) == 1 - 1 / 256
    assert M.detokenize(127) + M.detokenize(128) == 0


def test_time_embedding_and_euler_closed_forms():
    te = M.time_embedding(0.0, 16)
    assert np.array_equal(te, np.r_[np.zeros(8), np.ones(8)])
    te = M.time_embedding(0.3, 16)
    assert abs(te[0] - math.sin(300.0)) < 1e-12 and abs(te[8] - math.cos(300.0)) < 1e-12
    assert abs(te[7] - math.sin(300.0 * 10000 ** (-7 / 8))) < 1e-12
    rng = np.random.default_rng(6)
    eps = rng.normal(size=(50, 7))
    c = rng.normal(size=(50, 7))
    assert np.allclose(M.euler_integrate(eps, lambda x, t: c, 10), eps - c, atol=1e-14)
    a = 0.7
    assert np.allclose(M.euler_integrate(eps, lambda x, t: a * x, 10),
                       (1 - a / 10) ** 10 * eps, atol=1e-14)
    # tau schedule 1, 0.9, ..., 0.1: sum / 10 = 0.55
    assert np.allclose(M.euler_integrate(eps, lambda x, t: np.full_like(x, t), 10),
                       eps - 0.55, atol=1e-14)


# ------------------------------------------------------------ the model ----


def _obs(cfg, env_ids, seed=1001):
    img = synth_inputs.pixels(seed, env_ids, cfg.n_cams, cfg.img, cfg.img)
    lang = synth_inputs.lang_ids(seed, env_ids, cfg.n_lang, cfg.vocab)
    return img, lang


def _zero_blocks(cfg, kinds=("dec",), which=("o", "down")):
    ov = {}
    for name, (tid, shape) in M.tensor_shapes(cfg).items():
        parts = name.split(".")
        if len(parts) == 3 and parts[0] in kinds and parts[2] in which:
            ov[name] = np.zeros(shape)
    return ov


def test_single_token_block_closed_forms():
    cfg = tiny_cfg()
    pol = M.Policy(cfg, seed=0)
    Wl = pol.layer("dec", 0)
    x = np.random.default_rng(7).normal(size=(1, cfg.d))
    pos = np.array([3])
    # with the MLP output zeroed a single token sees only itself:
    # x + rmsnorm(x) Wv^T Wo^T (the query/key values and RoPE drop out)
    W1 = dict(Wl); W1["down"] = np.zeros_like(Wl["down"])
    out, _, _ = pol.block(x, W1, cfg.q_heads, cfg.kv_heads, cfg.head_dim, pos)
    h = M.rmsnorm(x)
    assert np.allclose(out, x + h @ Wl["v"].T @ Wl["o"].T, atol=1e-13)
    # with the attention output zeroed only the SwiGLU branch remains
    W2 = dict(Wl); W2["o"] = np.zeros_like(Wl["o"])
    out, _, _ = pol.block(x, W2, cfg.q_heads, cfg.kv_heads, cfg.head_dim, pos)
    g = h @ Wl["gate"].T
    u = h @ Wl["up"].T
    assert np.allclose(out, x + (g / (1 + np.exp(-g)) * u) @ Wl["down"].T, atol=1e-13)
    # both branches: the MLP reads the norm of the stream after the
    # attention residual, x1 = x + rmsnorm(x) Wv^T Wo^T
    out, _, _ = pol.block(x, Wl, cfg.q_heads, cfg.kv_heads, cfg.head_dim, pos)
    x1 = x + h @ Wl["v"].T @ Wl["o"].T
    h1 = M.rmsnorm(x1)
    g1 = h1 @ Wl["gate"].T
    u1 = h1 @ Wl["up"].T
    assert np.allclose(out, x1 + (g1 / (1 + np.exp(-g1)) * u1) @ Wl["down"].T, atol=1e-13)


def test_block_output_invariant_to_a_common_position_shift():
    # rotary scores depend on positions only through their differences and
    # the causal mask only on their order, so shifting every position of a
    # sequence by the same amount leaves a block's output unchanged (as long
    # as queries and keys are rotated alike)
    cfg = tiny_cfg()
    pol = M.Policy(cfg, seed=0)
    Wl = pol.layer("dec", 0)
    x = np.random.default_rng(8).normal(size=(5, cfg.d))
    outs = [pol.block(x, Wl, cfg.q_heads, cfg.kv_heads, cfg.head_dim, np.arange(5) + p)[0]
            for p in (0, 7, 100)]
    assert np.allclose(outs[1], outs[0], atol=1e-12) and np.allclose(outs[2], outs[0], atol=1e-12)
    # while the positions do matter: a different spacing changes the output
    spread = pol.block(x, Wl, cfg.q_heads, cfg.kv_heads, cfg.head_dim, 3 * np.arange(5))[0]
    assert not np.allclose(spread, outs[0], atol=1e-9)


def test_prefix_order_embeddings_and_action_head_closed_form():
    cfg = tiny_cfg()
    pol = M.Policy(cfg, seed=0, overrides=_zero_blocks(cfg))
    img, lang = _obs(cfg, [0])
    st = pol.prefill(img[0], lang[0])
    assert st.T == cfg.n_img_tokens + cfg.n_lang
    # zeroed residual branches: the last row is the last language embedding
    assert np.array_equal(st.h_last_pre, pol.W("E_lang")[lang[0][-1]])
    # without language the last row is the last patch through W_pe
    st2 = pol.prefill(img[0], [])
    patches = M.patchify(img[0].astype(np.float64), cfg.patch)
    assert np.allclose(st2.h_last_pre, patches[-1] @ pol.W("W_pe").T, atol=1e-14)
    # decode chain: each step's hidden is rmsnorm(E_act[t_prev])
    r = pol.decode(st)
    t = M.argmax_lowest(pol.W("W_act") @ M.rmsnorm(st.h_last_pre))
    assert r.tokens[0] == t
    for k in range(1, 7):
        t = M.argmax_lowest(pol.W("W_act") @ M.rmsnorm(pol.W("E_act")[t]))
        assert r.tokens[k] == t
    assert np.array_equal(r.actions, -1 + (2 * r.tokens + 1) / 256)


def test_causal_prefix_perturbing_later_tokens_leaves_earlier_rows_bitwise():
    cfg = tiny_cfg()
    pol = M.Policy(cfg, seed=0)
    img, lang = _obs(cfg, [0])
    a = pol.prefill(img[0], lang[0])
    l2 = lang[0].copy()
    l2[-1] = (l2[-1] + 1) % cfg.vocab
    b = pol.prefill(img[0], l2)
    T = a.T
    for l in range(cfg.layers):
        assert np.array_equal(a.k[l][:T - 1], b.k[l][:T - 1])
        assert np.array_equal(a.v[l][:T - 1], b.v[l][:T - 1])
        assert not np.array_equal(a.k[l][T - 1], b.k[l][T - 1])


def test_incremental_decode_equals_full_prefill():
    cfg = tiny_cfg(kv_heads=2)   # grouped KV heads too
    pol = M.Policy(cfg, seed=0)
    img, lang = _obs(cfg, [0])
    st = pol.prefill(img[0], lang[0])
    r = pol.decode(st)
    rows = pol.embed_prefix(img[0], lang[0])
    seq = np.concatenate([rows, pol.W("E_act")[r.tokens[:-1]]], axis=0)
    hn = pol.run_sequence(seq)
    for k in range(7):
        lg = pol.W("W_act") @ hn[st.T - 1 + k]
        assert np.allclose(lg, r.logits[k], rtol=0, atol=1e-12)


def test_teacher_forcing_feeds_given_tokens():
    cfg = tiny_cfg()
    pol = M.Policy(cfg, seed=0)
    img, lang = _obs(cfg, [1])
    st = pol.prefill(img[0], lang[0])
    forced = [5, 9, 250, 0, 17, 3]
    r = pol.decode(st, forced=forced)
    rows = pol.embed_prefix(img[0], lang[0])
    seq = np.concatenate([rows, pol.W("E_act")[forced]], axis=0)
    hn = pol.run_sequence(seq)
    for k in range(7):
        assert np.allclose(pol.W("W_act") @ hn[st.T - 1 + k], r.logits[k], atol=1e-12)


def test_vit_path_closed_form_with_zeroed_blocks():
    cfg = tiny_cfg(vit_layers=2, vit_d=24, vit_heads=3, vit_mlp=40, n_cams=1)
    ov = _zero_blocks(cfg, kinds=("dec", "vit"))
    pol = M.Policy(cfg, seed=0, overrides=ov)
    img, _ = _obs(cfg, [0])
    st = pol.prefill(img[0], [])
    patches = M.patchify(img[0].astype(np.float64), cfg.patch)
    v = patches @ pol.W("W_pe").T + pol.W("vit_pos")
    expect = M.rmsnorm(v) @ pol.W("W_proj").T
    assert np.allclose(st.h_last_pre, expect[-1], atol=1e-13)


def _permute_patches(img, p, perm):
    """Image whose patch at raster index perm[j] is the input's patch j."""
    cams, H, W, C = img.shape
    gw = W // p
    out = np.empty_like(img)
    for j, dst in enumerate(perm):
        sy, sx = divmod(j, gw)
        dy, dx = divmod(int(dst), gw)
        out[:, dy * p:(dy + 1) * p, dx * p:(dx + 1) * p] = img[:, sy * p:(sy + 1) * p, sx * p:(sx + 1) * p]
    return out


def test_vit_blocks_permutation_equivariant_without_position_embedding():
    # With the learned position embedding zeroed nothing in a non-causal,
    # rotary-free encoder depends on where a patch sits: moving the patches
    # moves the output rows the same way.  A causal mask or rotary
    # embeddings in the ViT blocks would break this (checked below on the
    # same data, so the pin has the power to catch either slip).
    cfg = tiny_cfg(img=64, vit_layers=2, vit_d=24, vit_heads=3, vit_mlp=40, n_cams=1)
    pol = M.Policy(cfg, seed=0, overrides={"vit_pos": np.zeros((16, 24))})
    img, _ = _obs(cfg, [0])
    perm = np.random.default_rng(5).permutation(16)
    a = pol.embed_prefix(img[0], [])
    b = pol.embed_prefix(_permute_patches(img[0], cfg.patch, perm), [])
    assert np.allclose(b[perm], a, rtol=0, atol=1e-12)
    # the same check fails for blocks that are causal or rotary
    patches = M.patchify(img[0].astype(np.float64), cfg.patch)
    v0 = patches @ pol.W("W_pe").T
    pos = np.arange(16)
    for causal, use_rope in [(True, False), (False, True)]:
        ya, _, _ = pol.block(v0, pol.layer("vit", 0), 3, 3, 8, pos, causal=causal, use_rope=use_rope)
        yb, _, _ = pol.block(v0[np.argsort(perm)], pol.layer("vit", 0), 3, 3, 8, pos, causal=causal,
                             use_rope=use_rope)
        assert not np.allclose(yb[perm], ya, rtol=0, atol=1e-6)


def _tiny_flow_cfg(**kw):
    return tiny_cfg(kv_heads=2, q_heads=4, action_logits=False, exp_layers=2, exp_d=16,
                    exp_heads=2, exp_mlp=24, chunk=5, adim=3, n_steps=10, **kw)


def test_flow_zero_output_projection_returns_noise_exactly():
    cfg = _tiny_flow_cfg()
    pol = M.Policy(cfg, seed=0, overrides={"W_aout": np.zeros((cfg.adim, cfg.exp_d))})
    img, lang = _obs(cfg, [0])
    st = pol.prefill(img[0], lang[0])
    eps = synth_inputs.flow_noise(9, [0], cfg.chunk, cfg.adim)[0]
    assert np.array_equal(pol.flow_denoise(st, eps), eps.astype(np.float64))


def test_flow_zeroed_expert_blocks_closed_form():
    cfg = _tiny_flow_cfg()
    pol = M.Policy(cfg, seed=0, overrides=_zero_blocks(cfg, kinds=("exp",)))
    img, lang = _obs(cfg, [0])
    st = pol.prefill(img[0], lang[0])
    x = synth_inputs.flow_noise(9, [0], cfg.chunk, cfg.adim)[0].astype(np.float64)
    out = pol.flow_denoise(st, x)
    for k in range(10):
        tau = 1 - k / 10
        te = M.time_embedding(tau, cfg.exp_d)
        pre = pol.W("W_t1") @ te
        tv = pol.W("W_t2") @ (pre / (1 + np.exp(-pre)))
        h = x @ pol.W("W_ain").T + tv
        x = x - (M.rmsnorm(h) @ pol.W("W_aout").T) / 10
    assert np.allclose(out, x, atol=1e-13)


def test_flow_prefix_kv_is_read_per_layer():
    # The expert's layer l reads the backbone's layer-l cache: perturbing the
    # cache of a layer the expert does not have (l >= exp_layers) changes
    # nothing, perturbing layer 0's cache changes the result.
    cfg = _tiny_flow_cfg(layers=3)
    pol = M.Policy(cfg, seed=0)
    img, lang = _obs(cfg, [0])
    st = pol.prefill(img[0], lang[0])
    eps = synth_inputs.flow_noise(9, [0], cfg.chunk, cfg.adim)[0]
    base = pol.flow_denoise(st, eps)
    st2 = dataclasses.replace(st, k=list(st.k), v=list(st.v))
    st2.k[2] = st.k[2] + 1.0
    assert np.array_equal(pol.flow_denoise(st2, eps), base)
    st3 = dataclasses.replace(st, k=list(st.k), v=list(st.v))
    st3.v[0] = st.v[0] * 2.0
    assert not np.allclose(pol.flow_denoise(st3, eps), base)


def test_expert_action_tokens_attend_without_a_mask():
    # Non-causal among the chunk: changing only the last action token's input
    # changes the first token's velocity (a causal expert would leave it
    # bitwise unchanged), and every token's velocity changes.
    cfg = _tiny_flow_cfg()
    pol = M.Policy(cfg, seed=0)
    img, lang = _obs(cfg, [0])
    st = pol.prefill(img[0], lang[0])
    x = synth_inputs.flow_noise(9, [0], cfg.chunk, cfg.adim)[0].astype(np.float64)
    x2 = x.copy()
    x2[-1] += 0.5
    v, v2 = pol.velocity(st, x, 0.7), pol.velocity(st, x2, 0.7)
    assert np.all(np.linalg.norm(v2 - v, axis=-1) > 1e-6 * np.linalg.norm(v, axis=-1))


def test_expert_single_action_token_is_the_decoder_continued_one_position():
    # With a chunk of one token the expert's mask does not matter, and with
    # the expert given the decoder's own blocks (same widths, heads and
    # weights) its layer l -- attending to the backbone's layer-l prefix K/V
    # plus itself at rotary position T -- is exactly the decoder's layer l on
    # the sequence [prefix ; h0] at position T.  So v is W_aout applied to
    # the final-normed last row of a plain causal pass over that sequence.
    # This pins the action tokens' positions (T onwards, not 0) and the
    # layer pairing against the independently pinned causal decoder.
    cfg = tiny_cfg(q_heads=2, kv_heads=2, action_logits=False, exp_layers=2, exp_d=32, exp_heads=2,
                   exp_mlp=48, chunk=1, adim=3, n_steps=10)
    base = M.Policy(cfg, seed=0)
    ov = {f"exp.{l}.{s}": base.W(f"dec.{l}.{s}") for l in range(2) for s in M.SLOT}
    pol = M.Policy(cfg, seed=0, overrides=ov)
    img, lang = _obs(cfg, [0])
    st = pol.prefill(img[0], lang[0])
    x = synth_inputs.flow_noise(9, [0], 1, cfg.adim)[0].astype(np.float64)
    tau = 0.6
    h0 = x @ pol.W("W_ain").T + pol.time_vector(tau)
    seq = np.concatenate([pol.embed_prefix(img[0], lang[0]), h0], axis=0)
    expect = pol.run_sequence(seq)[-1] @ pol.W("W_aout").T
    assert np.allclose(pol.velocity(st, x, tau)[0], expect, rtol=0, atol=1e-12)


def _tiny_wam_cfg(**kw):
    return _tiny_flow_cfg(frame_tokens=4, frame_dim=6, **kw)


def _wam_noise(cfg, seed=9):
    nf = synth_inputs.flow_noise(seed, [0], cfg.frame_tokens, cfg.frame_dim)[0]
    na = synth_inputs.flow_noise(seed + 1, [0], cfg.chunk, cfg.adim)[0]
    return nf, na


def test_wam_zero_output_projections_return_noise_exactly():
    cfg = _tiny_wam_cfg()
    pol = M.Policy(cfg, seed=0, overrides={"W_aout": np.zeros((cfg.adim, cfg.exp_d)),
                                           "W_fout": np.zeros((cfg.frame_dim, cfg.exp_d))})
    img, lang = _obs(cfg, [0])
    st = pol.prefill(img[0], lang[0])
    nf, na = _wam_noise(cfg)
    f, a = pol.wam_denoise(st, nf, na)
    assert np.array_equal(f, nf.astype(np.float64)) and np.array_equal(a, na.astype(np.float64))


def test_wam_without_frame_tokens_is_the_action_expert():
    # no frame tokens: the joint velocity is the action-only expert's
    cfg = _tiny_wam_cfg()
    pol = M.Policy(cfg, seed=0)
    img, lang = _obs(cfg, [0])
    st = pol.prefill(img[0], lang[0])
    _, na = _wam_noise(cfg)
    vf, va = pol.joint_velocity(st, np.zeros((0, cfg.frame_dim)), na.astype(np.float64), 0.7)
    assert vf.shape == (0, cfg.frame_dim)
    assert np.array_equal(va, pol.velocity(st, na.astype(np.float64), 0.7))


def test_wam_actions_depend_on_frames_only_through_the_blocks():
    # with the expert blocks zeroed every token sees only itself: the action
    # chunk is the action-only expert's exactly, whatever the frame latents;
    # with the blocks in place the frames steer the actions
    cfg = _tiny_wam_cfg()
    img, lang = _obs(cfg, [0])
    nf, na = _wam_noise(cfg)
    zero = M.Policy(cfg, seed=0, overrides=_zero_blocks(cfg, kinds=("exp",)))
    st = zero.prefill(img[0], lang[0])
    _, a0 = zero.wam_denoise(st, nf, na)
    _, a1 = zero.wam_denoise(st, 3.0 * nf, na)
    assert np.array_equal(a0, a1) and np.array_equal(a0, zero.flow_denoise(st, na))
    pol = M.Policy(cfg, seed=0)
    st = pol.prefill(img[0], lang[0])
    _, b0 = pol.wam_denoise(st, nf, na)
    _, b1 = pol.wam_denoise(st, 3.0 * nf, na)
    assert not np.allclose(b0, b1)


def test_wam_frames_zeroed_blocks_closed_form():
    # zeroed blocks: frame token i's velocity is rmsnorm(x_i W_fin^T + t(tau)) W_fout^T
    cfg = _tiny_wam_cfg()
    pol = M.Policy(cfg, seed=0, overrides=_zero_blocks(cfg, kinds=("exp",)))
    img, lang = _obs(cfg, [0])
    st = pol.prefill(img[0], lang[0])
    nf, na = _wam_noise(cfg)
    f, _ = pol.wam_denoise(st, nf, na)
    x = nf.astype(np.float64)
    for k in range(10):
        tau = 1 - k / 10
        pre = pol.W("W_t1") @ M.time_embedding(tau, cfg.exp_d)
        tv = pol.W("W_t2") @ (pre / (1 + np.exp(-pre)))
        h = x @ pol.W("W_fin").T + tv
        x = x - (M.rmsnorm(h) @ pol.W("W_fout").T) / 10
    assert np.allclose(f, x, atol=1e-13)


def test_wam_preset_shapes():
    cfg = M.PRESETS[5]
    sh = M.tensor_shapes(cfg)
    assert sh["W_fin"] == (M.TID_FIN, (1024, 32)) and sh["W_fout"] == (M.TID_FOUT, (32, 1024))
    assert cfg.frame_tokens + cfg.chunk == 148


def test_tiny_preset_shapes_and_determinism():
    cfg = M.PRESETS[1]
    assert cfg.prefix_len == 24 and cfg.patch_dim == 768
    pol = M.Policy(cfg, seed=0)
    img, lang = _obs(cfg, [3])
    a = pol.decode(pol.prefill(img[0], lang[0]))
    pol2 = M.Policy(cfg, seed=0)
    b = pol2.decode(pol2.prefill(img[0], lang[0]))
    assert np.array_equal(a.logits, b.logits)
    assert a.tokens.shape == (7,) and np.all((a.tokens >= 0) & (a.tokens < 256))


def test_preset_parameter_counts():
    def count(cfg, prefix):
        return sum(int(np.prod(sh)) for n, (_, sh) in M.tensor_shapes(cfg).items()
                   if n.startswith(prefix))
    c4 = M.PRESETS[4]
    expert = count(c4, "exp.") + sum(int(np.prod(M.tensor_shapes(c4)[n][1]))
                                     for n in ["W_ain", "W_t1", "W_t2", "W_aout"])
    assert 300e6 < expert < 310e6           # "300M-param" expert
    c3 = M.PRESETS[3]
    total = sum(int(np.prod(sh)) for _, sh in M.tensor_shapes(c3).values())
    assert 6.5e9 < total < 7.5e9            # "7B-class"


def test_teacher_forced_single_pass_equals_prefill_then_forced_decode():
    cfg = tiny_cfg(kv_heads=2)
    pol = M.Policy(cfg, seed=0)
    img, lang = _obs(cfg, [2])
    forced = [7, 200, 31, 31, 0, 255]
    st_ref = pol.prefill(img[0], lang[0])
    r_ref = pol.decode(st_ref, forced=forced)
    st, r = pol.teacher_forced(img[0], lang[0], forced)
    assert st.T == st_ref.T
    assert np.allclose(st.h_last_pre, st_ref.h_last_pre, rtol=0, atol=1e-12)
    for l in range(cfg.layers):
        assert np.allclose(st.k[l], st_ref.k[l], atol=1e-12) and np.allclose(st.v[l], st_ref.v[l], atol=1e-12)
    assert np.allclose(r.logits, r_ref.logits, rtol=0, atol=1e-12)
    assert np.array_equal(r.tokens, r_ref.tokens)


def test_bf16_emulation_rounds_only_at_storage_points():
    # fp32 policies ignore the flag; with it a bf16 policy stays close to the
    # exact one and every stored K/V element is a bf16 value
    cfg = tiny_cfg()
    img, lang = _obs(cfg, [0])
    a = M.Policy(cfg, seed=0).prefill(img[0], lang[0])
    b = M.Policy(cfg, seed=0, emulate_bf16=True).prefill(img[0], lang[0])
    assert np.array_equal(a.h_last_pre, b.h_last_pre)
    cfg16 = tiny_cfg(bf16=True)
    a = M.Policy(cfg16, seed=0).prefill(img[0], lang[0])
    e = M.Policy(cfg16, seed=0, emulate_bf16=True)
    b = e.prefill(img[0], lang[0])
    for l in range(cfg16.layers):
        assert np.array_equal(M.f64_to_bf16_value(b.k[l]), b.k[l])
        assert np.array_equal(M.f64_to_bf16_value(b.v[l]), b.v[l])
    err = np.linalg.norm(a.h_last_pre - b.h_last_pre) / np.linalg.norm(a.h_last_pre)
    assert 1e-5 < err < 3e-2
    # the bf16 attention differs from the exact one only by rounding P
    rng = np.random.default_rng(8)
    q = rng.normal(size=(5, 2, 16)); k = rng.normal(size=(7, 1, 16)); v = rng.normal(size=(7, 1, 16))
    qp = np.arange(5) + 2; kp = np.arange(7)
    ex = M.multihead_attention(q, k, v, qp, kp, True)
    em = M.Policy._attention_bf16(q, k, v, qp, kp, True)
    assert np.allclose(ex, em, rtol=0, atol=2e-2) and not np.array_equal(ex, em)
    # single key: the numerator exp(0) = 1 is a bf16 value, so the output is V
    one = M.Policy._attention_bf16(q[:, :1], k[:1], v[:1], qp, kp[:1], True)
    assert np.array_equal(one, np.repeat(v[:1], 5, axis=0)[:, :1])
    # equal scores: every numerator is exactly 1 -> the mean of V
    same = M.Policy._attention_bf16(np.zeros((3, 1, 16)), k[:4], v[:4], np.arange(3) + 9, kp[:4], True)
    assert np.allclose(same, np.repeat(v[:4].mean(0, keepdims=True), 3, axis=0), atol=1e-15)
    # storage points one at a time: with only the cache rounded, layer 0's
    # K and V are the exact ones rounded (its inputs are exact) and Q-only
    # rounding leaves layer 0's K/V untouched
    kv_only = M.Policy(cfg16, seed=0, emulate_bf16={"kv"}).prefill(img[0], lang[0])
    q_only = M.Policy(cfg16, seed=0, emulate_bf16={"q"}).prefill(img[0], lang[0])
    assert np.array_equal(kv_only.k[0], M.f64_to_bf16_value(a.k[0]))
    assert np.array_equal(kv_only.v[0], M.f64_to_bf16_value(a.v[0]))
    assert np.array_equal(q_only.k[0], a.k[0]) and not np.array_equal(q_only.k[1], a.k[1])
    with pytest.raises(ValueError):
        M.Policy(cfg16, seed=0, emulate_bf16={"weights"})
    # a whole emulated decode stays within rounding of the exact one
    ex = M.Policy(cfg16, seed=0)
    ra = ex.decode(a)
    re = e.decode(b, forced=ra.tokens[:-1])
    assert np.max(np.abs(re.logits - ra.logits)) < 5e-2 * np.max(np.abs(ra.logits))
