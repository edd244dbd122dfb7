"""Planted mistakes in the CPU oracle: each one must fail a pin.

The pins in test_oracle_pins.py hold for the oracle as written.  Here a
plausible mistake is planted in oracle/llama_ref.py, one per test and only for
that test (monkeypatch), and the pin meant to catch it is checked to fail:

* the whole-model forward against the brute-force pure-Python forward, which
  shares no code with the oracle beyond the weight matrices;
* incremental KV-cache decode against full causal recompute, for mistakes in
  the decode path (``attend``, ``kv_head_of``), which the full recompute does
  not use.
"""
import math

import numpy as np
import pytest

from oracle import llama_ref as R
from tests.test_oracle_pins import TOY, TOY_EXACT_KV, _py_forward_toy


def forward_pin_holds(shape=TOY_EXACT_KV, seed=11):
    w = R.Weights(shape, seed)
    toks = [3, 17, 0, shape.vocab - 1, 8, 8]
    got = R.forward_causal(w, toks)
    return bool(np.allclose(got, _py_forward_toy(w, toks), rtol=1e-10, atol=1e-12))


def incremental_pin_holds():
    w = R.Weights(TOY, seed=12)
    rng = np.random.default_rng(8)
    prompts = [rng.integers(0, TOY.vocab, size=n).tolist() for n in (5, 1, 9)]
    toks, logits = R.greedy_decode(w, prompts, [6, 3, 1])
    for i in range(3):
        full = R.forward_causal(w, prompts[i] + toks[i][:-1])
        n = len(prompts[i])
        if not np.allclose(logits[i], full[n - 1:], rtol=1e-10, atol=1e-10):
            return False
    return True


def test_pins_hold_without_a_planted_mistake():
    assert forward_pin_holds() and incremental_pin_holds()


# ---------------------------------------------------------------- mistakes in the forward

_apply_rope, _rope_angles, _causal, _rmsnorm, _embed = (R.apply_rope, R.rope_angles, R.causal_attention, R.rmsnorm,
                                                        R.embed_rows)


def rope_negated(x, positions, base):
    return _apply_rope(x, [-p for p in positions], base)


def rope_half_split_pairs(x, positions, base):
    """Pairs (i, i + hd/2) instead of adjacent (2i, 2i+1)."""
    T, nh, hd = x.shape
    ang = _rope_angles(positions, hd, base)
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    a, b = x[..., :hd // 2], x[..., hd // 2:]
    return np.concatenate([a * c - b * s, a * s + b * c], axis=-1)


def rope_angles_single_i(positions, head_dim, base):
    """theta_i = base^(-i/hd): the factor 2 dropped."""
    i = np.arange(head_dim // 2, dtype=np.float64)
    return np.asarray(positions, dtype=np.float64)[:, None] * (base ** (-i / head_dim))[None, :]


def attention_unscaled(q, k, v):
    return _causal(q * math.sqrt(q.shape[-1]), k, v)


def attention_unmasked(q, k, v):
    T, H, hd = q.shape
    group = H // k.shape[1]
    kh = np.repeat(k, group, axis=1).transpose(1, 2, 0)
    vh = np.repeat(v, group, axis=1).transpose(1, 0, 2)
    s = np.matmul(q.transpose(1, 0, 2), kh) / math.sqrt(hd)
    return np.matmul(R.softmax(s), vh).transpose(1, 0, 2)


def attention_heads_tiled(q, k, v):
    """KV heads assigned round-robin (h % Hkv) instead of in consecutive groups."""
    return _causal(q, np.tile(k, (1, q.shape[1] // k.shape[1], 1)), np.tile(v, (1, q.shape[1] // k.shape[1], 1)))


def swiglu_silu_on_up(m, w1, w3, w2):
    return ((m @ w1.T) * R.silu(m @ w3.T)) @ w2.T


def swiglu_without_gate(m, w1, w3, w2):
    return (R.silu(m @ w1.T) + (m @ w3.T)) @ w2.T


def rmsnorm_without_eps(x, g, eps):
    return _rmsnorm(x, g, 0.0)


def rmsnorm_without_sqrt(x, g, eps):
    x = np.asarray(x, dtype=np.float64)
    return x / (np.mean(x * x, axis=-1, keepdims=True) + eps) * g


def embed_next_row(w, tokens):
    return _embed(w, [(int(t) + 1) % w.shape.vocab for t in tokens])


FORWARD_MISTAKES = {
    "rope_negated": ("apply_rope", rope_negated),
    "rope_half_split_pairs": ("apply_rope", rope_half_split_pairs),
    "rope_angles_single_i": ("rope_angles", rope_angles_single_i),
    "attention_unscaled": ("causal_attention", attention_unscaled),
    "attention_unmasked": ("causal_attention", attention_unmasked),
    "attention_heads_tiled": ("causal_attention", attention_heads_tiled),
    "swiglu_silu_on_up": ("swiglu", swiglu_silu_on_up),
    "swiglu_without_gate": ("swiglu", swiglu_without_gate),
    "rmsnorm_without_eps": ("rmsnorm", rmsnorm_without_eps),
    "rmsnorm_without_sqrt": ("rmsnorm", rmsnorm_without_sqrt),
    "embed_next_row": ("embed_rows", embed_next_row),
}


@pytest.mark.parametrize("mistake", sorted(FORWARD_MISTAKES))
def test_forward_mistake_fails_the_brute_force_pin(mistake, monkeypatch):
    attr, bad = FORWARD_MISTAKES[mistake]
    monkeypatch.setattr(R, attr, bad)
    assert not forward_pin_holds()


def test_transposed_output_projection_fails_the_brute_force_pin(monkeypatch):
    """x + o Wo instead of x + o Wo^T (the toy shape's Wo is square, so the mistake runs)."""
    assert TOY_EXACT_KV.d_model == TOY_EXACT_KV.n_heads * TOY_EXACT_KV.head_dim
    layer = R.Weights.layer

    def transposed(self, i):
        d = dict(layer(self, i))
        d["wo"] = d["wo"].T
        return d

    monkeypatch.setattr(R.Weights, "layer", transposed)
    assert not forward_pin_holds()


# ---------------------------------------------------------------- mistakes in the decode path

_attend = R.attend


def attend_unscaled(q, K, V):
    return _attend(q * math.sqrt(q.shape[-1]), K, V)


def kv_head_round_robin(h, n_heads, n_kv_heads):
    return h % n_kv_heads


DECODE_MISTAKES = {
    "attend_unscaled": ("attend", attend_unscaled),
    "kv_head_round_robin": ("kv_head_of", kv_head_round_robin),
}


@pytest.mark.parametrize("mistake", sorted(DECODE_MISTAKES))
def test_decode_mistake_fails_the_recompute_pin(mistake, monkeypatch):
    attr, bad = DECODE_MISTAKES[mistake]
    monkeypatch.setattr(R, attr, bad)
    assert forward_pin_holds()          # the full forward does not use the decode path
    assert not incremental_pin_holds()
