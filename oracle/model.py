"""CPU oracle of the generation-stage policy forward -- TEST INFRASTRUCTURE.

This is the plain, slow, obviously-correct reference that the GPU library is
checked against.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
benchmark's ``cpu_baseline`` leg may import it; the product path never does,
and it imports nothing from the GPU library.

What it computes.  The paper's generation stage takes each environment's
observation (camera frames plus a task instruction) and produces the next
action (Section 2.1, "Embodied Models"; Section 2.2, generation stage): a
vision-language backbone fuses the inputs into a KV cache that an action head
consumes.  The paper fixes the family but no architecture, so the concrete
policy below is a *reading* of the paper (one choice among many it allows):

* patchify + linear patch embedding; for the 7B-class model a 24-layer
  non-causal ViT with learned position embeddings and a projector;
* a pre-norm decoder (RMSNorm, rotary embeddings, causal softmax attention
  with optional grouped KV heads, SwiGLU MLP, residual adds);
* an autoregressive action head: 256-bin logits from the final-normed last
  prefix row give token t0, then six decode steps feed the action-token
  embedding of the previous token and emit t1..t6; bins map to [-1, 1];
* a flow-matching action expert (config 4): 10 Euler steps from Gaussian
  noise, each running an 18-layer expert whose layer l attends to the
  backbone's layer-l prefix K/V plus its own 50 action tokens.

Precision: float64 arithmetic on the exact stored weights (bf16 or fp32
values) and the exact float32 inputs.  Library primitives used as steps:
numpy's matmul, exp, sqrt, sin, cos.  No blocking, fusion or reordering.

Parity pins for every function live in ``tests/test_oracle_pins.py``.
The architectural readings themselves (which layers exist, in which order)
have nothing in the paper to compare against: parity unpinned for the
architecture choice; only its internal consistency is pinned.  One such
reading no invariant can tell from its alternative: the world action
model's token order (frame tokens before the action chunk, hence their
rotary positions) -- parity unpinned.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import Dict, List, Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))

# --------------------------------------------------------------------------
# Policy configurations (the five workloads' model shapes)
# --------------------------------------------------------------------------


@dataclasses.dataclass(frozen=True)
class Config:
    name: str
    bf16: bool
    n_cams: int
    img: int
    patch: int
    layers: int
    d: int
    q_heads: int
    kv_heads: int
    head_dim: int
    mlp: int
    vocab: int
    n_lang: int
    vit_layers: int = 0
    vit_d: int = 0
    vit_heads: int = 0
    vit_mlp: int = 0
    action_logits: bool = True
    n_action_tokens: int = 7
    n_bins: int = 256
    exp_layers: int = 0
    exp_d: int = 0
    exp_heads: int = 0
    exp_mlp: int = 0
    chunk: int = 0
    adim: int = 0
    n_steps: int = 0
    frame_tokens: int = 0        # world action model: latent future-frame tokens per env
    frame_dim: int = 0           # channels of a frame-latent token
    std: float = 0.02
    eps: float = 1e-6
    rope_base: float = 10000.0

    @property
    def patches_per_cam(self) -> int:
        return (self.img // self.patch) ** 2

    @property
    def n_img_tokens(self) -> int:
        return self.n_cams * self.patches_per_cam

    @property
    def patch_dim(self) -> int:
        return self.patch * self.patch * 3

    @property
    def prefix_len(self) -> int:
        return self.n_img_tokens + self.n_lang


PRESETS: Dict[int, Config] = {
    # tiny fp32 VLA: one 64x64 camera, 16x16 patches, 8 language tokens
    1: Config("tiny-fp32", bf16=False, n_cams=1, img=64, patch=16, layers=2, d=256,
              q_heads=4, kv_heads=4, head_dim=64, mlp=1024, vocab=1024, n_lang=8),
    # small bf16 VLA: two 224x224 cameras, patch 16, 32 language tokens
    2: Config("small-bf16", bf16=True, n_cams=2, img=224, patch=16, layers=12, d=1024,
              q_heads=16, kv_heads=16, head_dim=64, mlp=4096, vocab=32000, n_lang=32),
    # 7B-class VLA: ViT (d 1024, patch 14, 24 layers) + 32-layer d=4096 decoder
    3: Config("7b-bf16", bf16=True, n_cams=1, img=224, patch=14, layers=32, d=4096,
              q_heads=32, kv_heads=32, head_dim=128, mlp=11008, vocab=32000, n_lang=32,
              vit_layers=24, vit_d=1024, vit_heads=16, vit_mlp=4096),
    # flow-matching expert on an 18-layer d=2048 GQA backbone
    4: Config("flow-bf16", bf16=True, n_cams=3, img=224, patch=16, layers=18, d=2048,
              q_heads=16, kv_heads=8, head_dim=128, mlp=8192, vocab=32000, n_lang=12,
              action_logits=False, exp_layers=18, exp_d=1024, exp_heads=8, exp_mlp=4096,
              chunk=50, adim=7, n_steps=10),
    # world action model: preset 4's backbone and expert, which also denoises
    # two future frames of 7 x 7 latent tokens (32 channels each)
    5: Config("wam-bf16", bf16=True, n_cams=3, img=224, patch=16, layers=18, d=2048,
              q_heads=16, kv_heads=8, head_dim=128, mlp=8192, vocab=32000, n_lang=12,
              action_logits=False, exp_layers=18, exp_d=1024, exp_heads=8, exp_mlp=4096,
              chunk=50, adim=7, n_steps=10, frame_tokens=98, frame_dim=32),
}

# Tensor enumeration used to key the weight generator (counter word 2).
TID_PATCH, TID_ELANG, TID_EACT, TID_WACT = 1, 2, 3, 4
TID_VITPOS, TID_PROJ, TID_AIN, TID_T1, TID_T2, TID_AOUT = 5, 6, 7, 8, 9, 10
TID_FIN, TID_FOUT = 11, 12
STACK_BASE = {"dec": 1000, "vit": 2000, "exp": 3000}
SLOT = {"q": 0, "k": 1, "v": 2, "o": 3, "gate": 4, "up": 5, "down": 6}


def tensor_shapes(cfg: Config) -> Dict[str, tuple]:
    """Logical [out, in] shape and generator id of every weight tensor."""
    s: Dict[str, tuple] = {}
    pe_out = cfg.vit_d if cfg.vit_layers else cfg.d
    s["W_pe"] = (TID_PATCH, (pe_out, cfg.patch_dim))
    s["E_lang"] = (TID_ELANG, (cfg.vocab, cfg.d))
    if cfg.action_logits:
        s["E_act"] = (TID_EACT, (cfg.n_bins, cfg.d))
        s["W_act"] = (TID_WACT, (cfg.n_bins, cfg.d))
    if cfg.vit_layers:
        s["vit_pos"] = (TID_VITPOS, (cfg.patches_per_cam * cfg.n_cams, cfg.vit_d))
        s["W_proj"] = (TID_PROJ, (cfg.d, cfg.vit_d))
    if cfg.exp_layers:
        s["W_ain"] = (TID_AIN, (cfg.exp_d, cfg.adim))
        s["W_t1"] = (TID_T1, (cfg.exp_d, cfg.exp_d))
        s["W_t2"] = (TID_T2, (cfg.exp_d, cfg.exp_d))
        s["W_aout"] = (TID_AOUT, (cfg.adim, cfg.exp_d))
        if cfg.frame_tokens:
            s["W_fin"] = (TID_FIN, (cfg.exp_d, cfg.frame_dim))
            s["W_fout"] = (TID_FOUT, (cfg.frame_dim, cfg.exp_d))

    def stack(kind, n, d, hq, hkv, hd, mlp):
        for l in range(n):
            b = STACK_BASE[kind] + 16 * l
            s[f"{kind}.{l}.q"] = (b + 0, (hq * hd, d))
            s[f"{kind}.{l}.k"] = (b + 1, (hkv * hd, d))
            s[f"{kind}.{l}.v"] = (b + 2, (hkv * hd, d))
            s[f"{kind}.{l}.o"] = (b + 3, (d, hq * hd))
            s[f"{kind}.{l}.gate"] = (b + 4, (mlp, d))
            s[f"{kind}.{l}.up"] = (b + 5, (mlp, d))
            s[f"{kind}.{l}.down"] = (b + 6, (d, mlp))

    stack("dec", cfg.layers, cfg.d, cfg.q_heads, cfg.kv_heads, cfg.head_dim, cfg.mlp)
    if cfg.vit_layers:
        hd = cfg.vit_d // cfg.vit_heads
        stack("vit", cfg.vit_layers, cfg.vit_d, cfg.vit_heads, cfg.vit_heads, hd, cfg.vit_mlp)
    if cfg.exp_layers:
        # the expert's K/V heads equal the backbone's KV heads so that it can
        # attend to the backbone cache head for head
        stack("exp", cfg.exp_layers, cfg.exp_d, cfg.exp_heads, cfg.exp_heads, cfg.head_dim,
              cfg.exp_mlp)
    return s


# --------------------------------------------------------------------------
# Weight generator (C, glibc libm) -- see orc_rng.c
# --------------------------------------------------------------------------

_LIB = None


def _lib():
    global _LIB
    if _LIB is None:
        path = os.path.join(HERE, "liborc_rng.so")
        if not os.path.exists(path):
            from . import build_oracle
            build_oracle.build()
        lib = ctypes.CDLL(path)
        lib.orc_normal_f32.argtypes = [ctypes.c_uint64, ctypes.c_uint32, ctypes.c_int64,
                                       ctypes.c_double, ctypes.c_void_p]
        lib.orc_normal_bf16.argtypes = [ctypes.c_uint64, ctypes.c_uint32, ctypes.c_int64,
                                        ctypes.c_double, ctypes.c_void_p]
        lib.orc_philox.argtypes = [ctypes.c_uint64, ctypes.c_void_p, ctypes.c_void_p]
        _LIB = lib
    return _LIB


def philox_words(seed: int, ctr: Sequence[int]) -> np.ndarray:
    c = np.asarray(ctr, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    _lib().orc_philox(ctypes.c_uint64(seed), c.ctypes.data, out.ctypes.data)
    return out


def gen_tensor(seed: int, tid: int, shape, std: float, bf16: bool) -> np.ndarray:
    """Raw stored weights: uint16 bf16 patterns (bf16) or float32."""
    count = int(np.prod(shape))
    if bf16:
        out = np.empty(count, dtype=np.uint16)
        _lib().orc_normal_bf16(seed, tid, count, std, out.ctypes.data)
    else:
        out = np.empty(count, dtype=np.float32)
        _lib().orc_normal_f32(seed, tid, count, std, out.ctypes.data)
    return out.reshape(shape)


def bf16_bits_to_f64(raw: np.ndarray) -> np.ndarray:
    return (raw.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def f64_to_bf16_value(x: np.ndarray) -> np.ndarray:
    """Round to the nearest bf16 value (ties to even), returned as float64."""
    f = np.asarray(x, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    u = (u + np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)
    return bf16_bits_to_f64(u.astype(np.uint16))


# --------------------------------------------------------------------------
# Elementary operations (each pinned in tests/test_oracle_pins.py)
# --------------------------------------------------------------------------


def linear(x: np.ndarray, w: np.ndarray) -> np.ndarray:
    """y = x W^T with W stored [out, in]."""
    return x @ w.T


def rmsnorm(x: np.ndarray, eps: float = 1e-6) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps); gains are 1 (not learned at init)."""
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def softmax(s: np.ndarray) -> np.ndarray:
    m = np.max(s, axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=-1, keepdims=True)


def rope(x: np.ndarray, pos: np.ndarray, base: float = 10000.0) -> np.ndarray:
    """Rotary embedding, rotate-half pairing (i, i + hd/2), theta_i = base^(-2i/hd).

    x: [T, H, hd]; pos: [T] absolute positions."""
    hd = x.shape[-1]
    half = hd // 2
    i = np.arange(half, dtype=np.float64)
    theta = base ** (-2.0 * i / hd)
    ang = pos.astype(np.float64)[:, None] * theta[None, :]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    x1 = x[..., :half]
    x2 = x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, q_pos: np.ndarray,
              k_pos: np.ndarray, causal: bool) -> np.ndarray:
    """softmax(Q K^T / sqrt(hd) + mask) V for one head.

    q: [Tq, hd]; k, v: [Tk, hd].  Causal: key j visible to query i iff
    k_pos[j] <= q_pos[i]."""
    hd = q.shape[-1]
    s = (q @ k.T) / np.sqrt(hd)
    if causal:
        mask = k_pos[None, :] <= q_pos[:, None]
        s = np.where(mask, s, -np.inf)
    return softmax(s) @ v


def multihead_attention(q, k, v, q_pos, k_pos, causal):
    """q: [Tq, Hq, hd]; k, v: [Tk, Hkv, hd]; query head h reads kv head
    h // (Hq / Hkv) (grouped KV heads)."""
    hq = q.shape[1]
    hkv = k.shape[1]
    group = hq // hkv
    out = np.empty_like(q)
    for h in range(hq):
        g = h // group
        out[:, h, :] = attention(q[:, h, :], k[:, g, :], v[:, g, :], q_pos, k_pos, causal)
    return out


def patchify(image: np.ndarray, p: int) -> np.ndarray:
    """[cams, H, W, 3] -> [cams * (H/p) * (W/p), p*p*3]; patches in raster
    order per camera, flat index (dy * p + dx) * 3 + c inside a patch."""
    cams, h, w, c = image.shape
    out = []
    for cam in range(cams):
        for py in range(h // p):
            for px in range(w // p):
                out.append(image[cam, py * p:(py + 1) * p, px * p:(px + 1) * p, :].reshape(-1))
    return np.asarray(out, dtype=np.float64)


def argmax_lowest(logits: np.ndarray) -> int:
    """Index of the maximum; ties go to the lowest index."""
    best = 0
    for i in range(1, len(logits)):
        if logits[i] > logits[best]:
            best = i
    return best


def top2_margin(logits: np.ndarray) -> float:
    s = np.sort(logits)
    return float(s[-1] - s[-2])


def detokenize(b, n_bins: int = 256):
    """Bin b in [0, n_bins) -> its centre in [-1, 1]: -1 + (2b + 1) / n_bins."""
    return -1.0 + (2.0 * np.asarray(b, dtype=np.float64) + 1.0) / n_bins


def time_embedding(tau: float, dim: int) -> np.ndarray:
    """[sin(1000 tau w_j), cos(1000 tau w_j)], w_j = 10000^(-j/(dim/2)), j < dim/2."""
    half = dim // 2
    j = np.arange(half, dtype=np.float64)
    w = 10000.0 ** (-j / half)
    a = 1000.0 * tau * w
    return np.concatenate([np.sin(a), np.cos(a)])


def euler_integrate(x0: np.ndarray, velocity, n_steps: int) -> np.ndarray:
    """tau_k = 1 - k/n; x_{k+1} = x_k - v(x_k, tau_k) / n, k = 0..n-1.

    Convention x_tau = tau * eps + (1 - tau) * a, v = eps - a: integrating
    from tau = 1 (noise) to tau = 0 (action)."""
    x = x0
    for k in range(n_steps):
        tau = 1.0 - k / n_steps
        x = x - velocity(x, tau) / n_steps
    return x


# --------------------------------------------------------------------------
# The policy
# --------------------------------------------------------------------------


@dataclasses.dataclass
class PrefixState:
    """What prefill leaves for one environment."""
    T: int
    k: List[np.ndarray]          # per decoder layer, [T, Hkv, hd], post-rotary
    v: List[np.ndarray]          # per decoder layer, [T, Hkv, hd]
    h_last_pre: np.ndarray       # last prefix row before the final norm, [d]
    h_last: np.ndarray           # after the final norm, [d]


@dataclasses.dataclass
class DecodeResult:
    tokens: np.ndarray           # [7] int
    logits: np.ndarray           # [7, 256]
    margins: np.ndarray          # [7]
    actions: np.ndarray          # [7]


# Where a bf16 policy stores activations in bf16 (diagnostic emulation):
# normalised rows and patches entering a GEMM, rotated Q, the K/V cache,
# softmax numerators before the P.V product, attention and SwiGLU outputs.
BF16_POINTS = ("gemm_in", "q", "kv", "p", "attn_out", "swiglu_out")


class Policy:
    """Seeded random-init policy evaluated in float64."""

    def __init__(self, cfg: Config, seed: int = 0, overrides: Optional[Dict[str, np.ndarray]] = None,
                 cache_limit_params: int = 600_000_000, emulate_bf16=False):
        self.cfg = cfg
        self.seed = seed
        # Optional diagnostic: round to bf16 where a bf16 policy stores
        # activations in bf16; all arithmetic between those points stays
        # float64.  emulate_bf16 is True (every point) or a collection of
        # point names from BF16_POINTS.  Off by default; parity is always
        # judged against the exact mode, never against this one.
        if emulate_bf16 is True:
            points = set(BF16_POINTS)
        else:
            points = set(emulate_bf16 or ())
            if not points <= set(BF16_POINTS):
                raise ValueError(f"unknown bf16 storage points {points - set(BF16_POINTS)}")
        self.bf16_points = points if cfg.bf16 else set()
        self.emulate_bf16 = bool(self.bf16_points)
        self.shapes = tensor_shapes(cfg)
        self.overrides = dict(overrides or {})
        total = sum(int(np.prod(sh)) for _, sh in self.shapes.values())
        self._cache_f64 = total <= cache_limit_params
        self._raw: Dict[str, np.ndarray] = {}
        self._f64: Dict[str, np.ndarray] = {}

    # weights ---------------------------------------------------------------
    def raw(self, name: str) -> np.ndarray:
        if name not in self._raw:
            tid, shape = self.shapes[name]
            self._raw[name] = gen_tensor(self.seed, tid, shape, self.cfg.std, self.cfg.bf16)
        return self._raw[name]

    def W(self, name: str) -> np.ndarray:
        if name in self.overrides:
            return np.asarray(self.overrides[name], dtype=np.float64)
        if name in self._f64:
            return self._f64[name]
        r = self.raw(name)
        w = bf16_bits_to_f64(r) if self.cfg.bf16 else r.astype(np.float64)
        if self._cache_f64:
            self._f64[name] = w
        return w

    def layer(self, kind: str, l: int) -> Dict[str, np.ndarray]:
        return {s: self.W(f"{kind}.{l}.{s}") for s in SLOT}

    # blocks ----------------------------------------------------------------
    def _prenorm(self, x):
        """Operand of the projection after a pre-norm: the normalised row
        (rounded to bf16 when emulating bf16 storage)."""
        return self._r(rmsnorm(x, self.cfg.eps), "gemm_in")

    def block(self, x, Wl, n_heads, n_kv, hd, pos, past_k=None, past_v=None, past_pos=None,
              causal=True, use_rope=True):
        """Pre-norm transformer block.  Returns (x_out, k_new, v_new)."""
        t = x.shape[0]
        R = self._r
        h = self._prenorm(x)
        q = linear(h, Wl["q"]).reshape(t, n_heads, hd)
        k = linear(h, Wl["k"]).reshape(t, n_kv, hd)
        v = linear(h, Wl["v"]).reshape(t, n_kv, hd)
        if use_rope:
            q = rope(q, pos, self.cfg.rope_base)
            k = rope(k, pos, self.cfg.rope_base)
        q, k, v = R(q, "q"), R(k, "kv"), R(v, "kv")
        if past_k is not None:
            K = np.concatenate([past_k, k], axis=0)
            V = np.concatenate([past_v, v], axis=0)
            kpos = np.concatenate([past_pos, pos])
        else:
            K, V, kpos = k, v, pos
        if "p" in self.bf16_points:
            o = self._attention_bf16(q, K, V, pos, kpos, causal)
        else:
            o = multihead_attention(q, K, V, pos, kpos, causal)
        o = R(o.reshape(t, n_heads * hd), "attn_out")
        x = x + linear(o, Wl["o"])
        h = self._prenorm(x)
        x = x + linear(R(silu(linear(h, Wl["gate"])) * linear(h, Wl["up"]), "swiglu_out"), Wl["down"])
        return x, k, v

    def _r(self, a, point):
        return f64_to_bf16_value(a) if point in self.bf16_points else a

    @staticmethod
    def _attention_bf16(q, k, v, q_pos, k_pos, causal):
        """Softmax attention whose numerators exp(s - max s) enter the P.V
        product rounded to bf16 while the denominator sums the unrounded
        ones (bf16 storage of P).  Without rounding this is `attention`."""
        hq, hkv, hd = q.shape[1], k.shape[1], q.shape[-1]
        out = np.empty_like(q)
        for h in range(hq):
            g = h // (hq // hkv)
            s = (q[:, h, :] @ k[:, g, :].T) / np.sqrt(hd)
            if causal:
                s = np.where(k_pos[None, :] <= q_pos[:, None], s, -np.inf)
            e = np.exp(s - np.max(s, axis=-1, keepdims=True))
            out[:, h, :] = (f64_to_bf16_value(e) @ v[:, g, :]) / np.sum(e, axis=-1, keepdims=True)
        return out

    # prefill ---------------------------------------------------------------
    def embed_prefix(self, image: Optional[np.ndarray], lang: Sequence[int]) -> np.ndarray:
        """Token rows [cam0 patches, cam1, ..., language] in the decoder width."""
        cfg = self.cfg
        rows = []
        if image is not None:
            patches = self._r(patchify(np.asarray(image, dtype=np.float64), cfg.patch), "gemm_in")
            if cfg.vit_layers:
                v = linear(patches, self.W("W_pe")) + self.W("vit_pos")
                hd = cfg.vit_d // cfg.vit_heads
                pos = np.arange(v.shape[0])
                for l in range(cfg.vit_layers):
                    v, _, _ = self.block(v, self.layer("vit", l), cfg.vit_heads, cfg.vit_heads, hd,
                                         pos, causal=False, use_rope=False)
                rows.append(linear(self._r(rmsnorm(v, cfg.eps), "gemm_in"), self.W("W_proj")))
            else:
                rows.append(linear(patches, self.W("W_pe")))
        E = self.W("E_lang")
        if len(lang):
            rows.append(E[np.asarray(lang, dtype=np.int64)])
        return np.concatenate(rows, axis=0)

    def prefill(self, image: Optional[np.ndarray], lang: Sequence[int]) -> PrefixState:
        cfg = self.cfg
        x = self.embed_prefix(image, lang)
        T = x.shape[0]
        pos = np.arange(T)
        ks, vs = [], []
        for l in range(cfg.layers):
            x, k, v = self.block(x, self.layer("dec", l), cfg.q_heads, cfg.kv_heads,
                                 cfg.head_dim, pos)
            ks.append(k)
            vs.append(v)
        return PrefixState(T, ks, vs, x[-1].copy(), rmsnorm(x[-1], cfg.eps))

    def teacher_forced(self, image: Optional[np.ndarray], lang: Sequence[int],
                       forced: Sequence[int]):
        """Prefill and teacher-forced action decode in one causal pass over
        [prefix rows ; E_act[forced[0..5]]]: by causality the prefix rows
        (and their K/V) are those of prefill alone, and the logits at
        positions T-1 .. T+5 are those of the incremental decode fed the
        forced tokens.  Returns (PrefixState, DecodeResult)."""
        cfg = self.cfg
        rows = self.embed_prefix(image, lang)
        T = rows.shape[0]
        x = np.concatenate([rows, self.W("E_act")[np.asarray(forced, dtype=np.int64)]], axis=0)
        pos = np.arange(x.shape[0])
        ks, vs = [], []
        for l in range(cfg.layers):
            x, k, v = self.block(x, self.layer("dec", l), cfg.q_heads, cfg.kv_heads, cfg.head_dim, pos)
            ks.append(k[:T])
            vs.append(v[:T])
        hn = rmsnorm(x, cfg.eps)
        st = PrefixState(T, ks, vs, x[T - 1].copy(), hn[T - 1].copy())
        L = np.stack([self.logits(hn[T - 1 + k]) for k in range(cfg.n_action_tokens)])
        toks = np.asarray([argmax_lowest(r) for r in L], dtype=np.int64)
        return st, DecodeResult(toks, L, np.array([top2_margin(r) for r in L]),
                                detokenize(toks, cfg.n_bins))

    def run_sequence(self, x: np.ndarray) -> np.ndarray:
        """Decoder over explicit input rows at positions 0..len-1 (causal);
        returns the final-normed rows.  Used to pin incremental decode."""
        cfg = self.cfg
        pos = np.arange(x.shape[0])
        for l in range(cfg.layers):
            x, _, _ = self.block(x, self.layer("dec", l), cfg.q_heads, cfg.kv_heads,
                                 cfg.head_dim, pos)
        return rmsnorm(x, cfg.eps)

    # autoregressive action decode -------------------------------------------
    def logits(self, h_normed: np.ndarray) -> np.ndarray:
        return linear(h_normed[None, :], self.W("W_act"))[0]

    def decode(self, st: PrefixState, forced: Optional[Sequence[int]] = None) -> DecodeResult:
        """t0 from the prefix; step k = 1..6 feeds E_act[t_{k-1}] at position
        T + k - 1 and emits t_k.  With ``forced`` the inputs are forced[k-1]
        (teacher forcing) while the emitted tokens are still this policy's
        own argmax."""
        cfg = self.cfg
        n_tok = cfg.n_action_tokens
        logits = [self.logits(st.h_last)]
        tokens = [argmax_lowest(logits[0])]
        ks = list(st.k)
        vs = list(st.v)
        kpos = np.arange(st.T)
        E = self.W("E_act")
        for step in range(1, n_tok):
            t_in = tokens[-1] if forced is None else int(forced[step - 1])
            x = E[t_in][None, :]
            pos = np.array([st.T + step - 1])
            for l in range(cfg.layers):
                x, k, v = self.block(x, self.layer("dec", l), cfg.q_heads, cfg.kv_heads,
                                     cfg.head_dim, pos, ks[l], vs[l], kpos)
                ks[l] = np.concatenate([ks[l], k], axis=0)
                vs[l] = np.concatenate([vs[l], v], axis=0)
            kpos = np.concatenate([kpos, pos])
            lg = self.logits(rmsnorm(x[0], cfg.eps))
            logits.append(lg)
            tokens.append(argmax_lowest(lg))
        L = np.stack(logits)
        toks = np.asarray(tokens, dtype=np.int64)
        return DecodeResult(toks, L, np.array([top2_margin(r) for r in L]),
                            detokenize(toks, cfg.n_bins))

    # flow-matching action expert -------------------------------------------
    def time_vector(self, tau: float) -> np.ndarray:
        te = time_embedding(tau, self.cfg.exp_d)
        return linear(silu(linear(te[None, :], self.W("W_t1"))), self.W("W_t2"))[0]

    def velocity(self, st: PrefixState, x: np.ndarray, tau: float) -> np.ndarray:
        """v(x, tau) for one env: x [chunk, adim] -> [chunk, adim]."""
        cfg = self.cfg
        h = linear(x, self.W("W_ain")) + self.time_vector(tau)[None, :]
        pos = st.T + np.arange(cfg.chunk)
        ppos = np.arange(st.T)
        for l in range(cfg.exp_layers):
            h, _, _ = self.block(h, self.layer("exp", l), cfg.exp_heads, cfg.exp_heads,
                                 cfg.head_dim, pos, st.k[l], st.v[l], ppos, causal=False)
        return linear(rmsnorm(h, cfg.eps), self.W("W_aout"))

    def flow_denoise(self, st: PrefixState, noise: np.ndarray, return_v0: bool = False):
        v0 = []

        def vel(x, tau):
            v = self.velocity(st, x, tau)
            if not v0:
                v0.append(v)
            return v

        x = euler_integrate(np.asarray(noise, dtype=np.float64), vel, self.cfg.n_steps)
        return (x, v0[0]) if return_v0 else x


    # world action model ------------------------------------------------------
    def joint_velocity(self, st: PrefixState, xf: np.ndarray, xa: np.ndarray, tau: float):
        """The diffusion transformer's velocity for one env's frame latents
        xf [F, frame_dim] and action chunk xa [chunk, adim]: each modality
        enters through its own input projection (plus the shared time
        vector), all F + chunk tokens run through the expert blocks together
        -- frames at positions T .. T+F-1, actions after them, no mask among
        them, the backbone cache of the same layer as context -- and leave
        through the final norm and each modality's own output projection."""
        cfg = self.cfg
        F = xf.shape[0]
        t = self.time_vector(tau)[None, :]
        h = np.concatenate([linear(xf, self.W("W_fin")) + t, linear(xa, self.W("W_ain")) + t], axis=0)
        pos = st.T + np.arange(F + cfg.chunk)
        ppos = np.arange(st.T)
        for l in range(cfg.exp_layers):
            h, _, _ = self.block(h, self.layer("exp", l), cfg.exp_heads, cfg.exp_heads,
                                 cfg.head_dim, pos, st.k[l], st.v[l], ppos, causal=False)
        y = rmsnorm(h, cfg.eps)
        return linear(y[:F], self.W("W_fout")), linear(y[F:], self.W("W_aout"))

    def wam_denoise(self, st: PrefixState, frame_noise: np.ndarray, action_noise: np.ndarray,
                    return_v0: bool = False):
        """Both modalities integrated by the same Euler schedule as the
        action-only expert, from their noises at tau = 1."""
        F = frame_noise.shape[0]
        x0 = np.concatenate([np.asarray(frame_noise, dtype=np.float64).reshape(F, -1),
                             np.asarray(action_noise, dtype=np.float64).reshape(self.cfg.chunk, -1)], axis=None)
        nf = frame_noise.size
        v0 = []

        def vel(x, tau):
            vf, va = self.joint_velocity(st, x[:nf].reshape(F, -1), x[nf:].reshape(self.cfg.chunk, -1), tau)
            v = np.concatenate([vf.reshape(-1), va.reshape(-1)])
            if not v0:
                v0.append(v)
            return v

        x = euler_integrate(x0, vel, self.cfg.n_steps)
        out = (x[:nf].reshape(frame_noise.shape), x[nf:].reshape(action_noise.shape))
        if return_v0:
            return out + (v0[0][nf:].reshape(action_noise.shape),)
        return out


def load_config(preset: int) -> Config:
    return PRESETS[preset]
