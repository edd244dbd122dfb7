"""Shared helpers of the GPU parity tests: run the device decode, compare with the oracle."""
from __future__ import annotations

import sys
from typing import Dict, List, Optional, Sequence

import numpy as np

from oracle import llama_ref as R
from paper_2403_12900_amd.configs import ModelConfig


def oracle_shape(m: ModelConfig) -> R.Shape:
    return R.Shape(m.n_layers, m.d_model, m.n_heads, m.n_kv_heads, m.head_dim, m.d_ff, m.vocab,
                   m.rope_base, m.rms_eps, m.bf16, kv_bf16=m.kv_is_bf16)


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


class DeviceRun:
    """Free-running greedy decode of a closed batch on the device.

    tokens[i] = [g_0 .. g_{L_i - 1}]; logits[i][s] = fp32 logits that produced
    g_s (s = 0 is the prefill) for the recorded steps (of the requests in
    `keep`, default all); active[s] = slots fed at decode step s.
    """

    def __init__(self, model: ModelConfig, seed: int, prompts: Sequence[Sequence[int]], stops: Sequence[int],
                 record: str | set = "all", max_ctx: Optional[int] = None, kv_blocks: Optional[int] = None,
                 keep: Optional[set] = None):
        import torch
        from paper_2403_12900_amd.binding import DecodeModel
        B = len(prompts)
        seq = [len(p) for p in prompts]
        need = max(s + L - 1 for s, L in zip(seq, stops))
        max_ctx = max_ctx or need
        blocks = sum((s + L - 1 + 15) // 16 for s, L in zip(seq, stops))
        self.m = DecodeModel(model, seed, max_slots=B, max_ctx=max_ctx, kv_blocks=kv_blocks or blocks)
        tok = self.m.new_token_buffer()

        def kept(rows, lg):
            """The logits rows of the requests in `keep` (sliced on the device)."""
            if lg is None or keep is None:
                return list(rows), lg
            ks = [k for k, i in enumerate(rows) if i in keep]
            return [rows[k] for k in ks], (lg[ks] if ks else None)

        want0 = record == "all" or 0 in record
        l0, retired = self.m.prefill(list(range(B)), prompts, stops, tok, want_logits=want0)
        snaps = [tok.clone()]
        fed = [list(range(B))]
        logs = [kept(list(range(B)), l0)]
        lens = list(seq)
        active = [i for i in range(B) if not retired[i]]
        self.active: List[List[int]] = []
        s = 1
        while active:
            want = record == "all" or s in record
            lg, retired = self.m.decode_step(active, [lens[i] for i in active], tok, want_logits=want)
            self.active.append(list(active))
            snaps.append(tok.clone())
            fed.append(list(active))
            logs.append(kept(active, lg))
            for i in active:
                lens[i] += 1
            active = [i for k, i in enumerate(active) if not retired[k]]
            s += 1
        torch.cuda.synchronize()
        self.tokens: List[List[int]] = [[] for _ in range(B)]
        self.logits: List[Dict[int, np.ndarray]] = [dict() for _ in range(B)]
        for s, (rows, lg) in enumerate(logs):
            t = snaps[s].cpu().numpy()
            for i in fed[s]:
                self.tokens[i].append(int(t[i]))
            if lg is not None:
                L = lg.cpu().numpy()
                for k, i in enumerate(rows):
                    self.logits[i][s] = L[k]
        self.lens = lens

    def close(self):
        import torch
        self.m.close()
        torch.cuda.empty_cache()


def compare_logits(dev: np.ndarray, ref: np.ndarray, dev_tok: int, abs_tol: float, rel_tol: float, tag: str):
    """One (request, step) row: tolerance gates and the greedy-token rules.

    (i) the device token is the argmax of the device's own logits, lowest index
    on ties -- always exact;  (ii) it equals the oracle's argmax unless the
    oracle's top-2 margin is within 2 max|dz| (a provable near tie), in which
    case it must lie within 2 max|dz| of the oracle's maximum.
    Returns (max abs error, relative L2 error, near_tie).
    """
    dz = np.abs(dev.astype(np.float64) - ref)
    mx = float(dz.max())
    rel = float(np.linalg.norm(dev.astype(np.float64) - ref) / np.linalg.norm(ref))
    assert mx <= abs_tol, f"{tag}: max abs {mx:.3e} > {abs_tol}"
    assert rel <= rel_tol, f"{tag}: rel L2 {rel:.3e} > {rel_tol}"
    assert dev_tok == int(np.argmax(dev)), f"{tag}: token {dev_tok} is not the argmax of its own logits"
    o = int(np.argmax(ref))
    near = False
    if dev_tok != o:
        top2 = np.sort(ref)[-2:]
        margin = top2[1] - top2[0]
        assert margin <= 2 * mx, f"{tag}: token {dev_tok} != oracle {o} with margin {margin:.3e} > 2*{mx:.3e}"
        assert ref[o] - ref[dev_tok] <= 2 * mx, f"{tag}: device token too far below the oracle max"
        near = True
    return mx, rel, near


def check_against_oracle(run: DeviceRun, w: R.Weights, prompts, stops, requests, abs_tol, rel_tol,
                         steps_of=None):
    """Teacher-forced oracle logits for the given requests at their recorded steps, all requests in
    one pass over the layers (each layer's weights drawn once).  Returns the worst errors, the rows
    compared, the near ties, and the largest context (cached positions) compared."""
    worst_abs = worst_rel = 0.0
    n_rows = n_near = 0
    max_ctx = 0
    todo = []
    for i in requests:
        steps = sorted(run.logits[i]) if steps_of is None else steps_of(i)
        steps = [s for s in steps if s in run.logits[i]]
        if steps:
            todo.append((i, steps))
    if not todo:
        return {"rows": 0, "near_ties": 0, "max_abs": 0.0, "max_rel": 0.0, "max_context": 0}
    every = max(1, w.shape.n_layers // 8)
    refs = R.teacher_forced_logits_requests(
        w, [prompts[i] for i, _ in todo], [run.tokens[i] for i, _ in todo], [st for _, st in todo],
        progress=lambda l: say(f"  oracle requests {[i for i, _ in todo]}: layer {l + 1}/{w.shape.n_layers}")
        if (l + 1) % every == 0 else None)
    for (i, steps), ref in zip(todo, refs):
        for r, s in enumerate(steps):
            mx, rel, near = compare_logits(run.logits[i][s], ref[r], run.tokens[i][s], abs_tol, rel_tol,
                                           f"request {i} step {s}")
            worst_abs, worst_rel = max(worst_abs, mx), max(worst_rel, rel)
            n_rows += 1
            n_near += near
            max_ctx = max(max_ctx, len(prompts[i]) + s)
    return {"rows": n_rows, "near_ties": n_near, "max_abs": worst_abs, "max_rel": worst_rel,
            "max_context": max_ctx}
