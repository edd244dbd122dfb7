"""spr_decode_step_static_scratch against spr_decode_step, through the C ABI (needs an MI355X).

The static-scratch variant is for callers that cannot allocate: its split
partials (attention's, and past 8 rows the projections' split-K slices),
arrival counters and greedy candidates live in the library's fixed
per-device array instead of the model's workspace.  It must give the
same tokens and the same logits as spr_decode_step on the same inputs, on
consecutive calls that share the array, the second with a smaller batch (the
array keeps the first call's contents).
"""
import numpy as np
import pytest

from paper_2403_12900_amd.configs import CONFIGS, ModelConfig

from ._harness import say

pytestmark = pytest.mark.gpu

CASES = {
    # Contexts of 300-700 positions at hd64: several KV splits per row, merged through the scratch.
    "toy_gqa2_hd64": (ModelConfig(n_layers=2, d_model=128, n_heads=4, n_kv_heads=2, head_dim=64, d_ff=176,
                                  vocab=1000), [700, 301, 455, 16, 640, 333]),
    # The benchmarked model's shape: 2000 LM-head tiles of greedy candidates in the scratch.
    "llama2_7b": (CONFIGS["c3"].model, [517, 140, 1033, 64]),
    # 24 and then 12 rows: the projections' split-K partials and counters in the scratch too.
    "llama2_7b_24_rows": (CONFIGS["c3"].model, [517, 140, 1033, 64, 300, 17, 250, 96, 401, 33, 129, 77,
                                                 610, 45, 160, 288, 71, 512, 20, 199, 345, 88, 131, 256]),
}


@pytest.mark.parametrize("case", sorted(CASES))
def test_static_scratch_step_equals_the_workspace_step(case):
    import torch
    from paper_2403_12900_amd.binding import DecodeModel
    m, plens = CASES[case]
    say(f"static scratch: {case}")
    rng = np.random.default_rng(77)
    prompts = [rng.integers(0, m.vocab, size=n).astype(np.int32) for n in plens]
    B = len(prompts)
    dm = DecodeModel(m, 5, max_slots=B, max_ctx=max(plens) + 8)
    tok = dm.new_token_buffer()
    dm.prefill(list(range(B)), prompts, [6] * B, tok)
    torch.cuda.synchronize()
    for n in (B, B // 2):                                   # two calls in a row, the second smaller
        slots = list(range(n))
        lens = [len(prompts[i]) for i in slots]
        tok0 = tok.clone()
        za, _ = dm.decode_step(slots, lens, tok, want_logits=True)
        ta = tok.clone()
        for i in slots:
            dm.rewind(i, lens[i], 1)
        tok.copy_(tok0)
        zb, _ = dm.decode_step_static_scratch(slots, lens, tok, want_logits=True)
        tb = tok.clone()
        torch.cuda.synchronize()
        za, zb = za.cpu().numpy(), zb.cpu().numpy()
        assert np.array_equal(ta.cpu().numpy(), tb.cpu().numpy()), f"{case}, {n} rows: tokens differ"
        d = float(np.abs(za - zb).max())
        assert np.array_equal(za, zb), f"{case}, {n} rows: logits differ by up to {d}"
        assert [dm.slot_info(i)[1] for i in slots] == [2] * n
        for i in slots:                                     # back to the prefilled state for the next call
            dm.rewind(i, lens[i], 1)
        tok.copy_(tok0)
        say(f"  {n} rows: tokens and logits identical")
    dm.close()
