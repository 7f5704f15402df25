"""Thin Python binding of the C ABI in include/*.h (argument marshalling only).

Every step of the policy forward runs in libebrl.so's HIP kernels; this
module only passes device pointers (from torch tensors), host id arrays and
the stream handle.  PyTorch supplies device memory and streams.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libebrl.so")

EBRL_OK = 0
ERRORS = {-1: "EBRL_E_INVALID", -2: "EBRL_E_OOM", -3: "EBRL_E_HIP", -4: "EBRL_E_STATE",
          -5: "EBRL_E_UNSUPPORTED"}
DTYPE_FP32, DTYPE_BF16 = 0, 1
STATE_H_LAST_PRE, STATE_H_LAST, STATE_K, STATE_V, STATE_FLOW_V0, STATE_PREFIX_LEN, STATE_GRAPHS = range(7)
K_GEMM, K_GEMM_SKINNY, K_ATTN_PREFILL, K_ATTN_DECODE, K_OTHER = range(5)
KERNEL_CLASSES = {K_GEMM: "gemm", K_GEMM_SKINNY: "gemm_skinny", K_ATTN_PREFILL: "attn_prefill",
                  K_ATTN_DECODE: "attn_decode", K_OTHER: "other"}

_I32 = ctypes.c_int32


class Config(ctypes.Structure):
    _fields_ = [(n, _I32) for n in (
        "dtype", "n_cams", "img", "patch", "vit_layers", "vit_d", "vit_heads", "vit_mlp",
        "layers", "d", "q_heads", "kv_heads", "head_dim", "mlp", "vocab", "n_lang",
        "action_logits", "n_action_tokens", "n_bins",
        "exp_layers", "exp_d", "exp_heads", "exp_mlp", "chunk", "adim", "n_steps",
        "max_envs", "max_seq")] + [("kv_budget_bytes", ctypes.c_int64), ("init_std", ctypes.c_double),
                                   ("frame_tokens", _I32), ("frame_dim", _I32)]

    def as_dict(self):
        return {n: getattr(self, n) for n, _ in self._fields_}


class ObsBatch(ctypes.Structure):
    _fields_ = [("images", ctypes.c_void_p), ("lang_ids", ctypes.c_void_p),
                ("lang_len", ctypes.c_void_p), ("lang_stride", _I32)]


_PI32, _PF64 = ctypes.POINTER(_I32), ctypes.POINTER(ctypes.c_double)


class AllocProfiles(ctypes.Structure):
    _fields_ = [("n_cenv", _I32), ("cenv", _PI32), ("n_ssim", _I32), ("ssim", _PI32), ("sim_rate", _PF64),
                ("n_sgen", _I32), ("sgen", _PI32), ("n_bgen", _I32), ("bgen", _PI32), ("gen_rate", _PF64),
                ("gen_mem", _PF64),
                ("n_strain", _I32), ("strain", _PI32), ("n_btrain", _I32), ("btrain", _PI32),
                ("train_rate", _PF64), ("train_mem", _PF64)]


class AllocLimits(ctypes.Structure):
    _fields_ = [("cores", _I32), ("mem_bytes", ctypes.c_double), ("sgen_min", _I32), ("strain_min", _I32),
                ("knee_tol", ctypes.c_double)]


class AllocResult(ctypes.Structure):
    _fields_ = [(n, _I32) for n in ("cenv", "envs", "ssim", "sgen", "strain", "bgen", "btrain", "iterations")] + \
               [(n, ctypes.c_double) for n in ("t_sim", "t_gen", "t_train", "t_rollout", "theta")]

    def as_dict(self):
        return {n: getattr(self, n) for n, _ in self._fields_}


class EbrlError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"{ERRORS.get(code, code)}: {msg}")
        self.code = code


_LIB = None

EXPORTED = [
    "ebrl_config_preset", "ebrl_policy_create", "ebrl_policy_destroy",
    "ebrl_stream_create_cu_masked", "ebrl_stream_destroy", "ebrl_policy_bind_stream",
    "ebrl_prefill", "ebrl_decode_actions", "ebrl_flow_denoise", "ebrl_wam_denoise", "ebrl_last_error",
    "ebrl_read_state", "ebrl_generate_weight_host", "ebrl_read_weight", "ebrl_write_weight",
    "ebrl_profile_enable", "ebrl_profile_read", "ebrl_op_gemm", "ebrl_op_gemm_noalloc", "ebrl_op_stream_read",
    "ebrl_alloc_solve", "ebrl_alloc_objective", "ebrl_alloc_monitor_create", "ebrl_alloc_monitor_observe",
    "ebrl_alloc_monitor_destroy", "ebrl_alloc_refine",
    "ebrl_sched_create", "ebrl_sched_destroy", "ebrl_sched_dispatch", "ebrl_sched_complete",
    "ebrl_sched_next_group", "ebrl_sched_deliver", "ebrl_sched_env_state",
]


def lib():
    """Load libebrl.so; raises if it has not been built (there is no fallback)."""
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with "
                          "`python -c 'import __graft_entry__ as g; g.build()'`")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, u32, u64 = ctypes.c_void_p, _I32, ctypes.c_int64, ctypes.c_uint32, ctypes.c_uint64
    pI32 = ctypes.POINTER(_I32)
    sig = {
        "ebrl_config_preset": (i32, [i32, ctypes.POINTER(Config)]),
        "ebrl_policy_create": (i32, [ctypes.POINTER(Config), u64, ctypes.POINTER(vp)]),
        "ebrl_policy_destroy": (None, [vp]),
        "ebrl_stream_create_cu_masked": (i32, [i32, ctypes.POINTER(u32), u32, ctypes.POINTER(vp)]),
        "ebrl_stream_destroy": (i32, [vp]),
        "ebrl_policy_bind_stream": (i32, [vp, vp]),
        "ebrl_prefill": (i32, [vp, ctypes.POINTER(ObsBatch), pI32, i32]),
        "ebrl_decode_actions": (i32, [vp, pI32, i32, vp, vp, vp]),
        "ebrl_flow_denoise": (i32, [vp, pI32, i32, vp, vp]),
        "ebrl_wam_denoise": (i32, [vp, pI32, i32, vp, vp, vp, vp]),
        "ebrl_last_error": (ctypes.c_char_p, [vp]),
        "ebrl_read_state": (i32, [vp, i32, i32, i32, vp, i64]),
        "ebrl_generate_weight_host": (i32, [u64, u32, i64, ctypes.c_double, i32, vp]),
        "ebrl_read_weight": (i32, [vp, u32, vp, i64]),
        "ebrl_write_weight": (i32, [vp, u32, vp, i64]),
        "ebrl_profile_enable": (i32, [vp, i32]),
        "ebrl_profile_read": (i32, [vp, i32, ctypes.POINTER(i64), ctypes.POINTER(ctypes.c_double),
                                    ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double), i32]),
        "ebrl_op_gemm": (i32, [i32, vp, vp, vp, i32, i32, i32, vp]),
        "ebrl_op_gemm_noalloc": (i32, [i32, vp, vp, vp, i32, i32, i32, vp]),
        "ebrl_op_stream_read": (i32, [vp, i64, vp, vp]),
        "ebrl_alloc_solve": (i32, [ctypes.POINTER(AllocProfiles), ctypes.POINTER(AllocLimits),
                                   ctypes.POINTER(AllocResult)]),
        "ebrl_alloc_objective": (i32, [ctypes.POINTER(AllocProfiles), ctypes.POINTER(AllocResult)]),
        "ebrl_alloc_monitor_create": (i32, [i32, ctypes.c_double, i32, ctypes.POINTER(vp)]),
        "ebrl_alloc_monitor_observe": (i32, [vp, ctypes.c_double, ctypes.c_double, pI32]),
        "ebrl_alloc_monitor_destroy": (None, [vp]),
        "ebrl_alloc_refine": (i32, [ctypes.POINTER(AllocProfiles), ctypes.POINTER(AllocResult), ctypes.c_double,
                                    ctypes.c_double, _PF64, _PF64]),
        "ebrl_sched_create": (i32, [i32, i32, i32, ctypes.POINTER(vp)]),
        "ebrl_sched_destroy": (None, [vp]),
        "ebrl_sched_dispatch": (i32, [vp, i32, i32, pI32]),
        "ebrl_sched_complete": (i32, [vp, i32, ctypes.c_double, pI32]),
        "ebrl_sched_next_group": (i32, [vp, pI32, pI32, i32, pI32]),
        "ebrl_sched_deliver": (i32, [vp, i32]),
        "ebrl_sched_env_state": (i32, [vp, i32, pI32, pI32, pI32, _PF64]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    _LIB = L
    return L


def preset(n: int) -> Config:
    c = Config()
    rc = lib().ebrl_config_preset(n, ctypes.byref(c))
    if rc != EBRL_OK:
        raise EbrlError(rc, f"unknown preset {n}")
    return c


def _ids(env_ids) -> ctypes.Array:
    a = np.ascontiguousarray(np.asarray(env_ids, dtype=np.int32))
    return a, a.ctypes.data_as(ctypes.POINTER(_I32))


def _ptr(t) -> Optional[int]:
    return None if t is None else int(t.data_ptr())


# ---------------------------------------------------- resource allocator --

def _alloc_profiles(P: dict):
    """Marshals a profile dict (cenv, ssim, sim[C, S], sgen, bgen, gen[G, Bg],
    gen_mem, strain, btrain, train[H, Bt], train_mem) into the C struct;
    returns the struct and the arrays it points into (kept alive by the
    caller)."""
    keep = {}

    def i32(k):
        keep[k] = np.ascontiguousarray(np.asarray(P[k], dtype=np.int32))
        return len(keep[k]), keep[k].ctypes.data_as(_PI32)

    def f64(k):
        keep[k] = np.ascontiguousarray(np.asarray(P[k], dtype=np.float64))
        return keep[k].ctypes.data_as(_PF64)

    pr = AllocProfiles()
    pr.n_cenv, pr.cenv = i32("cenv")
    pr.n_ssim, pr.ssim = i32("ssim")
    pr.sim_rate = f64("sim")
    pr.n_sgen, pr.sgen = i32("sgen")
    pr.n_bgen, pr.bgen = i32("bgen")
    pr.gen_rate, pr.gen_mem = f64("gen"), f64("gen_mem")
    pr.n_strain, pr.strain = i32("strain")
    pr.n_btrain, pr.btrain = i32("btrain")
    pr.train_rate, pr.train_mem = f64("train"), f64("train_mem")
    for k, shape in (("sim", (pr.n_cenv, pr.n_ssim)), ("gen", (pr.n_sgen, pr.n_bgen)),
                     ("train", (pr.n_strain, pr.n_btrain))):
        if keep[k].shape != shape:
            raise EbrlError(-1, f"profile table {k} has shape {keep[k].shape}, expected {shape}")
    for k, n in (("gen_mem", pr.n_bgen), ("train_mem", pr.n_btrain)):
        if keep[k].shape != (n,):
            raise EbrlError(-1, f"{k} has shape {keep[k].shape}, expected ({n},)")
    return pr, keep


def alloc_solve(P: dict, cores: int, mem_bytes: float, sgen_min: int, strain_min: int,
                knee_tol: float = 0.05) -> dict:
    """Algorithm 1 through the library (include/ebrl_alloc.h)."""
    pr, keep = _alloc_profiles(P)
    lim = AllocLimits(cores, mem_bytes, sgen_min, strain_min, knee_tol)
    out = AllocResult()
    rc = lib().ebrl_alloc_solve(ctypes.byref(pr), ctypes.byref(lim), ctypes.byref(out))
    if rc != EBRL_OK:
        raise EbrlError(rc, "ebrl_alloc_solve")
    return out.as_dict()


def alloc_objective(P: dict, cfg: dict) -> dict:
    pr, keep = _alloc_profiles(P)
    out = AllocResult(**{k: cfg[k] for k in ("sgen", "strain", "bgen", "btrain", "t_sim")})
    rc = lib().ebrl_alloc_objective(ctypes.byref(pr), ctypes.byref(out))
    if rc != EBRL_OK:
        raise EbrlError(rc, "ebrl_alloc_objective")
    return out.as_dict()


def alloc_refine(P: dict, cur: dict, observed_gen: float, observed_train: float):
    pr, keep = _alloc_profiles(P)
    res = AllocResult(**{k: cur[k] for k in ("bgen", "btrain", "t_gen", "t_train")})
    gen = np.empty_like(keep["gen"])
    train = np.empty_like(keep["train"])
    rc = lib().ebrl_alloc_refine(ctypes.byref(pr), ctypes.byref(res), observed_gen, observed_train,
                                 gen.ctypes.data_as(_PF64), train.ctypes.data_as(_PF64))
    if rc != EBRL_OK:
        raise EbrlError(rc, "ebrl_alloc_refine")
    return gen, train


class AllocMonitor:
    """The runtime adaptation trigger (ebrl_alloc_monitor_*)."""

    def __init__(self, window: int = 20, gap: float = 0.15, patience: int = 20):
        h = ctypes.c_void_p()
        rc = lib().ebrl_alloc_monitor_create(window, gap, patience, ctypes.byref(h))
        if rc != EBRL_OK:
            raise EbrlError(rc, "ebrl_alloc_monitor_create")
        self.h = h.value

    def observe(self, rollout_rate: float, train_rate: float) -> bool:
        t = _I32()
        rc = lib().ebrl_alloc_monitor_observe(self.h, rollout_rate, train_rate, ctypes.byref(t))
        if rc != EBRL_OK:
            raise EbrlError(rc, "ebrl_alloc_monitor_observe")
        return bool(t.value)

    def close(self):
        if self.h:
            lib().ebrl_alloc_monitor_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# ------------------------------------------------------ rollout scheduler --

class Sched:
    """The group pipeline and Algorithm 2 dispatcher (include/ebrl_sched.h)."""

    def __init__(self, n_envs: int, n_groups: int, chunk_len: int):
        h = ctypes.c_void_p()
        rc = lib().ebrl_sched_create(n_envs, n_groups, chunk_len, ctypes.byref(h))
        if rc != EBRL_OK:
            raise EbrlError(rc, "ebrl_sched_create")
        self.h = h.value
        self.n_envs = n_envs
        self._ids = np.empty(n_envs, dtype=np.int32)

    def _check(self, rc, what):
        if rc != EBRL_OK:
            raise EbrlError(rc, what)

    def dispatch(self, core: int = 0, bind_stride: int = 0) -> int:
        e = _I32()
        self._check(lib().ebrl_sched_dispatch(self.h, core, bind_stride, ctypes.byref(e)), "ebrl_sched_dispatch")
        return e.value

    def complete(self, env: int, duration: float) -> bool:
        d = _I32()
        self._check(lib().ebrl_sched_complete(self.h, env, duration, ctypes.byref(d)), "ebrl_sched_complete")
        return bool(d.value)

    def next_group(self):
        g, n = _I32(), _I32()
        self._check(lib().ebrl_sched_next_group(self.h, ctypes.byref(g), self._ids.ctypes.data_as(_PI32),
                                                self.n_envs, ctypes.byref(n)), "ebrl_sched_next_group")
        return g.value, self._ids[:n.value].copy()

    def deliver(self, group: int) -> None:
        self._check(lib().ebrl_sched_deliver(self.h, group), "ebrl_sched_deliver")

    def env_state(self, env: int):
        a, b, c, d = _I32(), _I32(), _I32(), ctypes.c_double()
        self._check(lib().ebrl_sched_env_state(self.h, env, ctypes.byref(a), ctypes.byref(b), ctypes.byref(c),
                                               ctypes.byref(d)), "ebrl_sched_env_state")
        return a.value, bool(b.value), bool(c.value), d.value

    def close(self):
        if self.h:
            lib().ebrl_sched_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def generate_weight_host(seed: int, tensor_id: int, count: int, std: float, bf16: bool) -> np.ndarray:
    out = np.empty(count, dtype=np.uint16 if bf16 else np.float32)
    rc = lib().ebrl_generate_weight_host(seed, tensor_id, count, std, int(bf16), out.ctypes.data)
    if rc != EBRL_OK:
        raise EbrlError(rc, "generate_weight_host")
    return out


def op_gemm(A, B, C, stream=None, noalloc=False) -> None:
    """C = A B^T through the library's GEMM kernel (torch device tensors);
    noalloc: the entry point that allocates nothing (fixed device scratch)."""
    import torch
    dt = DTYPE_BF16 if A.dtype == torch.bfloat16 else DTYPE_FP32
    M, K = A.shape
    N = B.shape[0]
    s = stream if stream is not None else torch.cuda.current_stream().cuda_stream
    fn = lib().ebrl_op_gemm_noalloc if noalloc else lib().ebrl_op_gemm
    rc = fn(dt, A.data_ptr(), B.data_ptr(), C.data_ptr(), M, N, K, s)
    if rc != EBRL_OK:
        raise EbrlError(rc, "ebrl_op_gemm_noalloc" if noalloc else "ebrl_op_gemm")


def op_stream_read(buf, out, stream=None) -> None:
    """Streaming read of a device tensor's bytes (the HBM read reference)."""
    import torch
    s = stream if stream is not None else torch.cuda.current_stream().cuda_stream
    rc = lib().ebrl_op_stream_read(buf.data_ptr(), buf.numel() * buf.element_size(), out.data_ptr(), s)
    if rc != EBRL_OK:
        raise EbrlError(rc, "ebrl_op_stream_read")


def create_cu_masked_stream(device: int, mask_words: Sequence[int]) -> int:
    arr = (ctypes.c_uint32 * len(mask_words))(*[int(w) & 0xFFFFFFFF for w in mask_words])
    out = ctypes.c_void_p()
    rc = lib().ebrl_stream_create_cu_masked(device, arr, len(mask_words), ctypes.byref(out))
    if rc != EBRL_OK:
        raise EbrlError(rc, lib().ebrl_last_error(None).decode())
    return out.value


def destroy_stream(s: int) -> None:
    lib().ebrl_stream_destroy(s)


class Policy:
    """One policy on the current device; calls enqueue on the bound stream."""

    def __init__(self, config, seed: int = 0, stream=None, **overrides):
        import torch
        cfg = preset(config) if isinstance(config, int) else config
        for k, v in overrides.items():
            setattr(cfg, k, v)
        self.cfg = cfg
        self.seed = seed
        h = ctypes.c_void_p()
        rc = lib().ebrl_policy_create(ctypes.byref(cfg), seed, ctypes.byref(h))
        if rc != EBRL_OK:
            raise EbrlError(rc, lib().ebrl_last_error(None).decode())
        self.h = h.value
        self.torch = torch
        self.bind_stream(stream if stream is not None else torch.cuda.current_stream().cuda_stream)

    # lifecycle -------------------------------------------------------------
    def close(self):
        if getattr(self, "h", None):
            lib().ebrl_policy_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _check(self, rc, what):
        if rc != EBRL_OK:
            raise EbrlError(rc, f"{what}: {lib().ebrl_last_error(self.h).decode()}")

    def bind_stream(self, stream) -> None:
        self.stream = int(stream or 0)
        self._check(lib().ebrl_policy_bind_stream(self.h, self.stream or None), "bind_stream")

    @property
    def bf16(self) -> bool:
        return self.cfg.dtype == DTYPE_BF16

    # calls -----------------------------------------------------------------
    def prefill(self, env_ids, images=None, lang_ids=None, lang_len=None) -> None:
        ids, pids = _ids(env_ids)
        ob = ObsBatch()
        ob.images = _ptr(images)
        ob.lang_ids = _ptr(lang_ids)
        ob.lang_stride = int(lang_ids.shape[1]) if lang_ids is not None else 0
        ll = None
        if lang_len is not None:
            ll = np.ascontiguousarray(np.asarray(lang_len, dtype=np.int32))
            ob.lang_len = ll.ctypes.data
        self._keep = (ids, ll, images, lang_ids)
        self._check(lib().ebrl_prefill(self.h, ctypes.byref(ob), pids, len(ids)), "prefill")

    def decode_actions(self, env_ids, tokens=None, actions=None, margins=None, with_margin=True):
        torch = self.torch
        ids, pids = _ids(env_ids)
        n, nt = len(ids), self.cfg.n_action_tokens
        dev = torch.device("cuda", torch.cuda.current_device())
        if tokens is None:
            tokens = torch.empty((n, nt), dtype=torch.int32, device=dev)
        if actions is None:
            actions = torch.empty((n, nt), dtype=torch.float32, device=dev)
        if margins is None and with_margin:
            margins = torch.empty((n, nt), dtype=torch.float32, device=dev)
        self._check(lib().ebrl_decode_actions(self.h, pids, n, _ptr(tokens), _ptr(actions), _ptr(margins)),
                    "decode_actions")
        return tokens, actions, margins

    def _chunk_out(self, n, rows, cols):
        return self.torch.empty((n, rows, cols), dtype=self.torch.float32, device="cuda")

    def flow_denoise(self, env_ids, noise=None, out=None):
        """noise None: the library draws it (seeded, per-env call count)."""
        ids, pids = _ids(env_ids)
        if out is None:
            out = self._chunk_out(len(ids), self.cfg.chunk, self.cfg.adim) if noise is None else \
                self.torch.empty_like(noise)
        self._check(lib().ebrl_flow_denoise(self.h, pids, len(ids), _ptr(noise), _ptr(out)), "flow_denoise")
        return out

    def wam_denoise(self, env_ids, frame_noise=None, action_noise=None, out_frames=None, out_actions=None):
        """Joint denoising of future-frame latents and the action chunk;
        a noise of None is drawn by the library."""
        ids, pids = _ids(env_ids)
        c = self.cfg
        if out_frames is None:
            out_frames = self._chunk_out(len(ids), c.frame_tokens, c.frame_dim) if frame_noise is None else \
                self.torch.empty_like(frame_noise)
        if out_actions is None:
            out_actions = self._chunk_out(len(ids), c.chunk, c.adim) if action_noise is None else \
                self.torch.empty_like(action_noise)
        self._check(lib().ebrl_wam_denoise(self.h, pids, len(ids), _ptr(frame_noise), _ptr(action_noise),
                                           _ptr(out_frames), _ptr(out_actions)), "wam_denoise")
        return out_frames, out_actions

    # inspection ------------------------------------------------------------
    def read_state(self, what: int, env_id: int, layer: int = 0) -> np.ndarray:
        c = self.cfg
        if what in (STATE_H_LAST_PRE, STATE_H_LAST):
            out = np.empty(c.d, dtype=np.float32)
        elif what in (STATE_PREFIX_LEN, STATE_GRAPHS):
            out = np.empty(1, dtype=np.int32)
        elif what == STATE_FLOW_V0:
            out = np.empty((c.chunk, c.adim), dtype=np.float32)
        else:
            T = int(self.read_state(STATE_PREFIX_LEN, env_id)[0])
            out = np.empty((T, c.kv_heads, c.head_dim), dtype=np.uint16 if self.bf16 else np.float32)
        self._check(lib().ebrl_read_state(self.h, what, env_id, layer, out.ctypes.data, out.nbytes), "read_state")
        return out

    def read_weight(self, tensor_id: int, shape) -> np.ndarray:
        out = np.empty(shape, dtype=np.uint16 if self.bf16 else np.float32)
        self._check(lib().ebrl_read_weight(self.h, tensor_id, out.ctypes.data, out.nbytes), "read_weight")
        return out

    def write_weight(self, tensor_id: int, values: np.ndarray) -> None:
        a = np.ascontiguousarray(values, dtype=np.uint16 if self.bf16 else np.float32)
        self._check(lib().ebrl_write_weight(self.h, tensor_id, a.ctypes.data, a.nbytes), "write_weight")

    def profile_enable(self, classes=(K_GEMM, K_GEMM_SKINNY, K_ATTN_PREFILL, K_ATTN_DECODE, K_OTHER)) -> None:
        mask = 0
        for c in classes:
            mask |= 1 << c
        self._check(lib().ebrl_profile_enable(self.h, mask), "profile_enable")

    def profile_read(self, cls: int, reset: bool = False) -> dict:
        n = ctypes.c_int64()
        ms, fl, by = ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
        self._check(lib().ebrl_profile_read(self.h, cls, ctypes.byref(n), ctypes.byref(ms), ctypes.byref(fl),
                                            ctypes.byref(by), int(reset)), "profile_read")
        return {"launches": n.value, "ms": ms.value, "flop": fl.value, "bytes": by.value}
