"""How far the logits move when cached keys/values land on the other side of a storage rounding boundary.

A helper of the CPU tests (it imports only the oracle).  Two implementations
that both follow the KV-cache reading -- compute a key or value, round it to
the cache format, attend to the rounded values -- can still round a few
elements differently, because each computes the value before rounding with
its own arithmetic.  This module runs the oracle's forward pass (Section II-A:
every position attends to the cached keys/values of its prefix) several times
in lockstep over the same weights, each run with its own key/value arithmetic
and cache format, and reports the logit differences between runs: the floor
below which no parity gate between two such implementations can be set.

Runs (cache format / arithmetic of the cached values):
  bf16_f64      the oracle's own: keys/values in fp64, rounded to bf16
  bf16_f32      keys/values from fp32 operands with fp32 accumulation and
                fp32 rotary embedding (what a fp32-accumulating device does),
                rounded to bf16
  bf16_f64_ulp  the fp64 values moved up by one fp32 ulp, then rounded to bf16
  bf16_hilo     as bf16_f32, but the projection input carried as two bf16
                parts (hi = bf16(a), lo = bf16(a - hi): 16 significant bits)
  f32_f64       fp64 values rounded to fp32
  f32_f32       fp32 arithmetic as in bf16_f32, kept in fp32
Everything else (norms, projections, attention, MLP, LM head) is the oracle's
fp64 arithmetic in every run.  The runs share each layer's weights, so their
projections are done as one stacked product per matrix.
"""
from __future__ import annotations

from typing import Dict, Sequence

import numpy as np

from oracle import llama_ref as R

RUNS = ("bf16_f64", "bf16_f32", "bf16_f64_ulp", "bf16_hilo", "f32_f64", "f32_f32")


def _rope_f32(x32: np.ndarray, positions: Sequence[int], base: float) -> np.ndarray:
    """RoPE in fp32 arithmetic: cos/sin of the fp64 angles rounded to fp32, products and sums in fp32."""
    T, nh, hd = x32.shape
    ang = R.rope_angles(positions, hd, base)
    c = np.cos(ang).astype(np.float32)[:, None, :]
    s = np.sin(ang).astype(np.float32)[:, None, :]
    even, odd = x32[..., 0::2], x32[..., 1::2]
    out = np.empty_like(x32)
    out[..., 0::2] = even * c - odd * s
    out[..., 1::2] = even * s + odd * c
    return out


def _to_bf16(f32: np.ndarray) -> np.ndarray:
    u = f32.astype(np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


def _hi_lo(a32: np.ndarray) -> np.ndarray:
    """fp32 values as the sum of their two bf16 parts hi = bf16(a), lo = bf16(a - hi) (exact in fp32)."""
    hi = _to_bf16(a32)
    lo = _to_bf16((a32.astype(np.float64) - hi).astype(np.float32))
    return (hi + lo).astype(np.float32)


def _cached(run: str, kv64: np.ndarray, kv32: np.ndarray) -> np.ndarray:
    if run == "bf16_f64":
        return R.round_to_storage(kv64, bf16=True)
    if run in ("bf16_f32", "bf16_hilo"):
        return _to_bf16(kv32)
    if run == "bf16_f64_ulp":
        return _to_bf16(np.nextafter(kv64.astype(np.float32), np.float32(np.inf)))
    if run == "f32_f64":
        return R.round_to_storage(kv64, bf16=False)
    if run == "f32_f32":
        return kv32.astype(np.float64)
    raise ValueError(run)


def lockstep_logits(shape: R.Shape, seed: int, tokens: Sequence[int], runs: Sequence[str] = RUNS,
                    progress=None) -> Dict[str, np.ndarray]:
    """Logits [T, V] at every position of `tokens` for each run."""
    sh = shape
    w = R.Weights(sh, seed, resident=False)
    tokens = np.asarray(tokens, dtype=np.int64)
    T = len(tokens)
    pos = list(range(T))
    g = w.gain()
    x0 = R.embed_rows(w, tokens)
    xs = {r: x0.copy() for r in runs}
    nr = len(runs)
    for layer in range(sh.n_layers):
        W = w.layer(layer)
        A = np.concatenate([R.rmsnorm(xs[r], g, sh.rms_eps) for r in runs])      # [nr*T, d]
        q = (A @ W["wq"].T).reshape(nr, T, sh.n_heads, sh.head_dim)
        k64 = (A @ W["wk"].T).reshape(nr, T, sh.n_kv_heads, sh.head_dim)
        v64 = (A @ W["wv"].T).reshape(nr, T, sh.n_kv_heads, sh.head_dim)
        A32 = A.astype(np.float32)
        for i, r in enumerate(runs):
            if r == "bf16_hilo":
                A32[i * T:(i + 1) * T] = _hi_lo(A32[i * T:(i + 1) * T])
        k32 = (A32 @ W["wk"].astype(np.float32).T).reshape(nr, T, sh.n_kv_heads, sh.head_dim)
        v32 = (A32 @ W["wv"].astype(np.float32).T).reshape(nr, T, sh.n_kv_heads, sh.head_dim)
        O = np.empty((nr, T, sh.n_heads * sh.head_dim))
        for i, r in enumerate(runs):
            qi = R.apply_rope(q[i], pos, sh.rope_base)
            ki = _cached(r, R.apply_rope(k64[i], pos, sh.rope_base), _rope_f32(k32[i], pos, sh.rope_base))
            vi = _cached(r, v64[i], v32[i])
            O[i] = R.causal_attention(qi, ki, vi).reshape(T, -1)
        O = O.reshape(nr * T, -1)
        Xo = np.concatenate([xs[r] for r in runs]) + O @ W["wo"].T
        M = R.rmsnorm(Xo, g, sh.rms_eps)
        Xo = Xo + R.swiglu(M, W["w1"], W["w3"], W["w2"])
        for i, r in enumerate(runs):
            xs[r] = Xo[i * T:(i + 1) * T]
        del W
        if progress is not None:
            progress(layer)
    lm = w.matrix("lm_head")
    return {r: R.rmsnorm(xs[r], g, sh.rms_eps) @ lm.T for r in runs}


def floors(z: Dict[str, np.ndarray]) -> Dict[str, Dict[str, float]]:
    """Worst (over positions) max-abs and relative-L2 logit differences between the runs that share
    a cache format, and the mean over positions of each position's relative L2 difference."""
    out = {}
    for a, b in (("bf16_f64", "bf16_f32"), ("bf16_f64", "bf16_f64_ulp"), ("bf16_f64", "bf16_hilo"),
                 ("f32_f64", "f32_f32")):
        if a in z and b in z:
            d = z[a] - z[b]
            rel = np.linalg.norm(d, axis=1) / np.linalg.norm(z[a], axis=1)
            out[f"{a}~{b}"] = {"max_abs": float(np.abs(d).max()), "rel_l2": float(rel.max()),
                               "mean_rel_l2": float(rel.mean())}
    return out
