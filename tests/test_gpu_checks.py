"""Greedy tie rule and device-side input checks, on the device through the C ABI (needs an MI355X).

Section II-A's loop picks the next token from the model's output at every
step; the greedy choice takes the largest logit and, among equal largest
logits, the lowest token id.  Random logits never tie, so these tests plant
exact ties: LM-head row m (the step's argmax) is copied over another row t, so
both rows give the same logit bit for bit, and the token must become
min(m, t).  The copies cover every level of the device's reduction: the four
rows one lane holds, the four lane groups of one 16-row tile, and the
candidates of different tiles merged by the final argmax kernel.  The oracle
gets the same row copy and must pick the same token (numpy's argmax returns
the first maximum).
"""
import math

import numpy as np
import pytest

from oracle import llama_ref as R
from paper_2403_12900_amd.configs import ModelConfig

from ._harness import oracle_shape, say

pytestmark = pytest.mark.gpu

TIE_MODEL = ModelConfig(n_layers=2, d_model=128, n_heads=4, n_kv_heads=2, head_dim=64, d_ff=176, vocab=1000)
SEED = 4321


def _forced_step(dm, prompt, forced):
    """Prefill one request, force its next input token, run one decode step; returns (logits, token)."""
    import torch
    tok = dm.new_token_buffer()
    dm.prefill([0], [prompt], [4], tok)
    tok.fill_(int(forced))
    z, _ = dm.decode_step([0], [len(prompt)], tok, want_logits=True)
    torch.cuda.synchronize()
    return z[0].cpu().numpy(), int(tok[0].item())


def _case():
    """A prompt whose step argmax m admits all five planted-tie targets (deterministic search)."""
    from paper_2403_12900_amd.binding import DecodeModel
    for k in range(64):
        rng = np.random.default_rng(1000 + k)
        prompt = rng.integers(0, TIE_MODEL.vocab, size=int(rng.integers(5, 40))).astype(np.int32)
        forced = int(rng.integers(0, TIE_MODEL.vocab))
        dm = DecodeModel(TIE_MODEL, SEED, max_slots=1, max_ctx=64)
        z, m = _forced_step(dm, prompt, forced)
        dm.close()
        assert m == int(np.argmax(z))
        r = m % 16
        if m >= 16 and m + 16 < TIE_MODEL.vocab and 4 <= r <= 14 and r % 4 != 0:
            return prompt, forced, m
    pytest.fail("no prompt in the search gave an argmax admitting every planted-tie target")


def test_planted_ties_pick_the_lowest_index():
    from paper_2403_12900_amd.binding import DecodeModel
    prompt, forced, m = _case()
    targets = {
        "lower, another tile": m - 16,
        "lower, same lane": m - 1,
        "lower, another lane group of the tile": m - 4,
        "higher, same tile": m + 1,
        "higher, another tile": m + 16,
    }
    say(f"planted ties: argmax {m}, targets {targets}")
    for what, t in targets.items():
        dm = DecodeModel(TIE_MODEL, SEED, max_slots=1, max_ctx=64)
        dm.test_write_lm_head_row(t, m)
        z, got = _forced_step(dm, prompt, forced)
        dm.close()
        want = min(m, t)
        assert z[t] == z[m], f"{what}: copied rows give logits {z[t]!r} and {z[m]!r}"
        assert float(z.max()) == z[m], what
        assert got == want, f"{what}: token {got}, expected {want} (tie between {m} and {t})"
        w = R.Weights(oracle_shape(TIE_MODEL), SEED)
        lm = w.matrix("lm_head")
        lm[t] = lm[m]
        ref = R.forward_causal(w, list(prompt) + [forced], [len(prompt)])[0]
        assert ref[t] == ref[m] and int(R.argmax_first(ref)) == want, what
        say(f"  {what}: t={t}, token {got}")


def test_out_of_range_forced_token_fails_the_next_call():
    import torch
    from paper_2403_12900_amd.binding import DecodeModel, SproutError, SPR_ERR_DEVICE_CHECK
    rng = np.random.default_rng(11)
    prompt = rng.integers(0, TIE_MODEL.vocab, size=9).astype(np.int32)
    for bad in (TIE_MODEL.vocab, -1):
        dm = DecodeModel(TIE_MODEL, SEED, max_slots=1, max_ctx=64)
        tok = dm.new_token_buffer()
        dm.prefill([0], [prompt], [6], tok)
        dm.decode_step([0], [9], tok)                       # healthy
        tok.fill_(bad)
        dm.decode_step([0], [10], tok)                      # enqueued: its embedding sees the bad id
        torch.cuda.synchronize()
        for _ in range(2):                                  # the next call fails, and every later one
            with pytest.raises(SproutError) as e:
                dm.decode_step([0], [11], tok)
            assert e.value.status == SPR_ERR_DEVICE_CHECK and "token id" in str(e.value)
        dm.close()


def test_nan_logits_fail_the_next_call():
    import torch
    from paper_2403_12900_amd.binding import DecodeModel, SproutError, SPR_ERR_DEVICE_CHECK
    rng = np.random.default_rng(12)
    prompt = rng.integers(0, TIE_MODEL.vocab, size=9).astype(np.int32)
    dm = DecodeModel(TIE_MODEL, SEED, max_slots=1, max_ctx=64)
    tok = dm.new_token_buffer()
    dm.prefill([0], [prompt], [6], tok)
    dm.test_write_lm_head_row(517, -1, math.nan)            # row 517's logit is NaN from now on
    z, _ = dm.decode_step([0], [9], tok, want_logits=True)
    torch.cuda.synchronize()
    assert np.isnan(z[0, 517].item()) and int(tok[0].item()) == 0
    with pytest.raises(SproutError) as e:
        dm.decode_step([0], [10], tok)
    assert e.value.status == SPR_ERR_DEVICE_CHECK and "logits" in str(e.value)
    dm.close()


def test_write_lm_head_row_checks_its_arguments():
    from paper_2403_12900_amd.binding import DecodeModel, SproutError, SPR_ERR_INVALID_ARG
    dm = DecodeModel(TIE_MODEL, SEED, max_slots=1, max_ctx=16)
    for dst, src in ((TIE_MODEL.vocab, 0), (-1, 0), (3, TIE_MODEL.vocab)):
        with pytest.raises(SproutError) as e:
            dm.test_write_lm_head_row(dst, src)
        assert e.value.status == SPR_ERR_INVALID_ARG
    dm.close()
