"""Seeded synthetic decode workloads (inputs only; none of the model's arithmetic).

Both the device path and the CPU oracle consume what this module draws, so it
imports neither.  A request is: directive prefix of its level ++ user prompt
(the directive goes first, as a system prompt placed before the user's text,
Section III-E), plus a stop length L = number of tokens it generates.  Token
ids are uniform over the vocabulary; the paper's prompt corpora (Table 1) are
not available, so lognormal lengths stand in for them.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List

import numpy as np

from .configs import DecodeConfig


@dataclasses.dataclass
class Workload:
    tokens: List[np.ndarray]      # per request: prefix ++ prompt (int32)
    levels: np.ndarray            # directive level per request
    prefix_lens: np.ndarray
    prompt_lens: np.ndarray       # user prompt only
    stop_lens: np.ndarray         # tokens generated per request, >= 1
    directive_ids: List[np.ndarray]

    @property
    def batch(self) -> int:
        return len(self.tokens)

    @property
    def seq_lens(self) -> np.ndarray:
        return np.array([len(t) for t in self.tokens], dtype=np.int64)

    def decode_tokens(self) -> int:
        """Tokens produced by decode steps (the prefill emits the first one)."""
        return int(np.sum(self.stop_lens - 1))

    def subset(self, idx) -> "Workload":
        idx = list(idx)
        return Workload([self.tokens[i] for i in idx], self.levels[idx], self.prefix_lens[idx],
                        self.prompt_lens[idx], self.stop_lens[idx], self.directive_ids)


def _lognormal_lengths(rng: np.random.Generator, median: float, sigma: float, n: int, lo: int, hi: int) -> np.ndarray:
    x = rng.lognormal(mean=math.log(median), sigma=sigma, size=n)
    return np.clip(np.rint(x), lo, hi).astype(np.int64)


def make_workload(cfg: DecodeConfig, seed: int = None) -> Workload:
    rec = cfg.workload
    V = cfg.model.vocab
    rng = np.random.default_rng(cfg.workload_seed if seed is None else seed)
    # One fixed id sequence per directive level (a level is a pre-defined text, Definition 1).
    directive_ids = [rng.integers(0, V, size=p).astype(np.int32) for p in rec.prefix_lens]
    B = rec.batch
    if len(rec.prefix_lens) == 1:
        levels = np.zeros(B, dtype=np.int64)
    else:
        levels = rng.integers(0, len(rec.prefix_lens), size=B)
    if rec.prompt_lens is not None:
        prompt_lens = np.array(rec.prompt_lens, dtype=np.int64)
    else:
        prompt_lens = _lognormal_lengths(rng, rec.prompt_median, rec.sigma, B, *rec.prompt_clip)
    if rec.stop_lens is not None:
        stop_lens = np.array(rec.stop_lens, dtype=np.int64)
    else:
        stop_lens = np.array([_lognormal_lengths(rng, rec.stop_medians[l], rec.sigma, 1, *rec.stop_clip)[0]
                              for l in levels], dtype=np.int64)
    tokens = []
    for i in range(B):
        prompt = rng.integers(0, V, size=int(prompt_lens[i])).astype(np.int32)
        tokens.append(np.concatenate([directive_ids[levels[i]], prompt]).astype(np.int32))
    prefix_lens = np.array([rec.prefix_lens[l] for l in levels], dtype=np.int64)
    return Workload(tokens, levels, prefix_lens, prompt_lens, stop_lens, directive_ids)


def workload_stats(cfg: DecodeConfig, w: Workload) -> dict:
    """Algorithmic decode bytes and tokens of the whole closed batch."""
    m = cfg.model
    wbytes = m.weight_elements_per_step() * m.weight_bytes
    kvtok = m.kv_bytes_per_token()
    n = w.seq_lens
    L = w.stop_lens
    steps = int(L.max()) - 1 if len(L) else 0
    total_bytes = 0
    active_sum = 0
    for s in range(1, steps + 1):
        act = L > s
        ctx = n[act] + s            # positions attended to, the new one included
        total_bytes += wbytes + int(np.sum(ctx - 1)) * kvtok + int(act.sum()) * (kvtok + m.d_model * m.weight_bytes)
        active_sum += int(act.sum())
    return {"steps": steps, "decode_tokens": int(np.sum(L - 1)), "bytes": total_bytes,
            "avg_active": active_sum / max(steps, 1), "weight_bytes_per_step": wbytes}
