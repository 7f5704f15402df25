"""Host-side checks of the GPU library (no GPU): it loads, exports every
symbol its headers declare, its presets match the oracle's model table, and
its host weight generator reproduces the oracle's weights bit for bit
(two independent implementations of Philox4x32-10 + Box-Muller)."""
import os
import re

import numpy as np
import pytest

from oracle import model as M
from paper_2609_27547_amd import ebrl as E

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    names = set()
    for h in sorted(os.listdir(os.path.join(ROOT, "include"))):
        if not h.endswith(".h"):
            continue
        src = open(os.path.join(ROOT, "include", h)).read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        names |= set(re.findall(r"\b(ebrl_[a-z0-9_]+)\s*\(", src))
    return names


def test_library_exports_every_declared_symbol():
    L = E.lib()
    names = _declared()
    assert "ebrl_prefill" in names and "ebrl_flow_denoise" in names
    for n in sorted(names):
        assert hasattr(L, n), f"{n} not exported"
    assert set(E.EXPORTED) == names


@pytest.mark.parametrize("n", [1, 2, 3, 4, 5])
def test_presets_match_oracle_model_table(n):
    c = E.preset(n)
    o = M.PRESETS[n]
    assert c.dtype == (E.DTYPE_BF16 if o.bf16 else E.DTYPE_FP32)
    for f in ["n_cams", "img", "patch", "layers", "d", "q_heads", "kv_heads", "head_dim", "mlp",
              "vocab", "n_lang", "vit_layers", "vit_d", "vit_heads", "vit_mlp", "n_action_tokens",
              "n_bins", "exp_layers", "exp_d", "exp_heads", "exp_mlp", "chunk", "adim", "n_steps",
              "frame_tokens", "frame_dim"]:
        assert getattr(c, f) == getattr(o, f), f
    assert bool(c.action_logits) == o.action_logits
    assert c.max_seq == o.prefix_len
    assert abs(c.init_std - o.std) < 1e-9


def test_preset_rejects_unknown():
    with pytest.raises(E.EbrlError):
        E.preset(7)


@pytest.mark.parametrize("bf16", [False, True])
def test_host_weight_generator_bitwise_equals_oracle(bf16):
    for tid, count in [(1, 768 * 256), (1003, 4097), (3016 + 5, 1001), (7, 1)]:
        a = E.generate_weight_host(0, tid, count, 0.02, bf16)
        b = M.gen_tensor(0, tid, (count,), 0.02, bf16)
        assert a.dtype == b.dtype
        assert np.array_equal(a.view(np.uint8), b.view(np.uint8)), tid
    a = E.generate_weight_host(123456789012345, 2, 5000, 0.02, bf16)
    b = M.gen_tensor(123456789012345, 2, (5000,), 0.02, bf16)
    assert np.array_equal(a.view(np.uint8), b.view(np.uint8))
