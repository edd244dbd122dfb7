"""Device decode vs the CPU oracle, through the C ABI (needs an MI355X).

Every case runs the device free-running (greedy) and feeds the device's own
tokens to the oracle (teacher forcing), so both see the same inputs at every
step.  Gates per (request, step) logits row:
  * fp32 models: max abs error <= 1e-4 and relative L2 <= 1e-5;
  * bf16 models: max abs error <= 5e-2 and relative L2 <= 1e-2;
  * greedy tokens: the argmax of the device's own logits exactly, and the
    oracle's argmax unless the oracle's top-2 margin is within 2 max|dz|;
  * retirement bookkeeping: bit-exact against the closed form.
"""
import zlib

import numpy as np
import pytest

from oracle import _clib
from oracle import llama_ref as R
from paper_2403_12900_amd.configs import CONFIGS, LLAMA2_7B, ModelConfig
from paper_2403_12900_amd.workload import make_workload

from ._harness import DeviceRun, check_against_oracle, oracle_shape, say

pytestmark = pytest.mark.gpu

FP32_TOL = (1e-4, 1e-5)
BF16_TOL = (5e-2, 1e-2)


def _tol(m: ModelConfig):
    return BF16_TOL if m.bf16 else FP32_TOL


def _prompts(rng, V, lens):
    return [rng.integers(0, V, size=n).astype(np.int32) for n in lens]


# ------------------------------------------------------------------ weights

@pytest.mark.parametrize("bf16", [False, True])
def test_weight_generator_bit_exact(bf16):
    m = ModelConfig(n_layers=2, d_model=48, n_heads=4, n_kv_heads=2, head_dim=64, d_ff=40, vocab=70, bf16=bf16)
    say(f"weights bit-exact bf16={bf16}")
    from paper_2403_12900_amd.binding import DecodeModel
    dm = DecodeModel(m, seed=424242, max_slots=2, max_ctx=32)
    sh = oracle_shape(m)
    for name in ("embed", "wq", "wk", "wv", "wo", "w1", "w3", "w2", "lm_head"):
        rows, cols = sh.matrix_dims(name)
        for layer in ((0, 1) if name not in ("embed", "lm_head") else (0,)):
            got = dm.export_weight_rows(name, layer, 0, rows, cols).cpu().numpy()
            want = _clib.wgen_rows(424242, R.TENSOR_IDS[name], layer, cols, 0, rows, bf16, dtype=np.float32)
            assert np.array_equal(got.view(np.uint32), want.view(np.uint32)), (name, layer)
    dm.close()


def test_weight_generator_bit_exact_7b_rows():
    """Sampled rows of every Llama-2-7B matrix, including the fused QKV and interleaved gate/up layouts."""
    say("weights bit-exact 7B sampled rows")
    from paper_2403_12900_amd.binding import DecodeModel
    m = LLAMA2_7B
    dm = DecodeModel(m, seed=1003, max_slots=1, max_ctx=16)
    sh = oracle_shape(m)
    for name in ("embed", "wq", "wk", "wv", "wo", "w1", "w3", "w2", "lm_head"):
        rows, cols = sh.matrix_dims(name)
        layers = (0,) if name in ("embed", "lm_head") else (0, 31)
        for layer in layers:
            for r0 in (0, rows // 2 + 3, rows - 2):
                got = dm.export_weight_rows(name, layer, r0, 2, cols).cpu().numpy()
                want = _clib.wgen_rows(1003, R.TENSOR_IDS[name], layer, cols, r0, 2, True, dtype=np.float32)
                assert np.array_equal(got.view(np.uint32), want.view(np.uint32)), (name, layer, r0)
    dm.close()


# ------------------------------------------------------------------ tiny configuration (fp32)

def test_tiny_config_all_steps():
    """The tiny fp32 configuration end to end: every request, every step."""
    cfg = CONFIGS["c1"]
    wl = make_workload(cfg)
    say("tiny config c1")
    run = DeviceRun(cfg.model, cfg.weight_seed, wl.tokens, wl.stop_lens.tolist())
    assert run.active == R.active_schedule(wl.stop_lens.tolist())
    assert [len(t) for t in run.tokens] == wl.stop_lens.tolist()
    w = R.Weights(oracle_shape(cfg.model), cfg.weight_seed)
    st = check_against_oracle(run, w, wl.tokens, wl.stop_lens, range(wl.batch), *FP32_TOL)
    say("c1", st)
    assert st["rows"] == int(wl.stop_lens.sum())
    run.close()


# ------------------------------------------------------------------ toy shapes: tails and paths

TOY_CASES = {
    # name: (model, prompt lengths, stop lengths)
    "bf16_mha_hd64_ragged": (
        ModelConfig(n_layers=2, d_model=128, n_heads=2, n_kv_heads=2, head_dim=64, d_ff=200, vocab=1000),
        [15, 16, 17, 1, 31, 32, 33, 47], [3, 5, 2, 9, 1, 4, 6, 2]),
    "bf16_gqa4_hd128_wide_o": (
        ModelConfig(n_layers=2, d_model=256, n_heads=8, n_kv_heads=2, head_dim=128, d_ff=344, vocab=777),
        [5, 64, 100, 3, 18, 77, 19, 2, 40, 9, 12, 33, 1, 60, 8, 16, 17, 90, 4, 25], [4] * 10 + [2, 7] * 5),
    "fp32_gqa2_hd128": (
        ModelConfig(n_layers=1, d_model=64, n_heads=2, n_kv_heads=1, head_dim=128, d_ff=100, vocab=50,
                    bf16=False),
        [3, 20, 16, 1, 45], [6, 2, 3, 4, 5]),
    "bf16_batch40_jt4": (
        ModelConfig(n_layers=1, d_model=64, n_heads=1, n_kv_heads=1, head_dim=64, d_ff=64, vocab=300),
        list(range(1, 41)), [3] * 40),
    "bf16_weights_fp32_kv_gqa8": (
        ModelConfig(n_layers=2, d_model=256, n_heads=8, n_kv_heads=1, head_dim=128, d_ff=344, vocab=500,
                    kv_bf16=False),
        [40, 3, 17, 90, 1], [5, 9, 2, 4, 6]),
    # One row of ~1700 positions at hd128 with 4 query heads per KV head: 107 blocks would be 27
    # one-block-per-wave splits, past the 16 one merge round takes, so the run per wave grows.
    "bf16_gqa4_hd128_long_context": (
        ModelConfig(n_layers=2, d_model=256, n_heads=8, n_kv_heads=2, head_dim=128, d_ff=344, vocab=500),
        [1690, 30, 5], [12, 4, 2]),
    "bf16_long_context_splits": (
        ModelConfig(n_layers=2, d_model=128, n_heads=4, n_kv_heads=4, head_dim=64, d_ff=128, vocab=500),
        [700, 300], [20, 3]),
    # 32 KV heads x 24 rows of 141-147 positions: two splits per row would be 1536 attention
    # work-groups, more than the 1024 resident on MI355X, so the pass takes three-block runs per wave
    # and one split per row.
    "bf16_mha32_splits_fit_resident": (
        ModelConfig(n_layers=1, d_model=256, n_heads=32, n_kv_heads=32, head_dim=64, d_ff=128, vocab=300),
        [140 + (i % 5) for i in range(24)], [3] * 24),
    # Split-K past 8 rows with slices of unequal length: d = 4160 (130 K-blocks: QKV and O slices
    # of 32 and 33) and d_ff = 6208 (194: down slices of 48 and 49).  At 17-20 rows QKV, O, gate/up
    # and down split; at 9-16 QKV and down; at 1-8 none.  13 query heads per KV head.
    "bf16_split_k_uneven_slices": (
        ModelConfig(n_layers=1, d_model=4160, n_heads=65, n_kv_heads=5, head_dim=64, d_ff=6208, vocab=600),
        [(5 * i) % 23 + 1 for i in range(20)], [2] * 4 + [3] * 4 + [5, 6] * 6),
    # The slot limit: 64 requests, so the first decode pass has 64 rows (four row tiles); later
    # passes shrink through two and one row tiles as requests retire.
    "bf16_batch64_max_slots": (
        ModelConfig(n_layers=1, d_model=128, n_heads=4, n_kv_heads=2, head_dim=64, d_ff=176, vocab=300),
        [(7 * i) % 50 + 1 for i in range(64)], [(i % 6) + 2 for i in range(64)]),
    # A prompt spanning prefill chunks: 7347 rows run as chunks of 4096 and 3251 rows, and the
    # 2500-row prompt crosses the boundary at its row 1089.
    "bf16_prompts_across_chunks": (
        ModelConfig(n_layers=2, d_model=128, n_heads=4, n_kv_heads=2, head_dim=64, d_ff=176, vocab=400),
        [3000, 7, 2500, 40, 1800], [3, 4, 2, 5, 3]),
    # The first chunk (4096 rows) ends exactly at the 96-row prompt's last row; the next chunk
    # starts with a prompt at position 0.
    "bf16_chunk_ends_at_prompt_end": (
        ModelConfig(n_layers=2, d_model=128, n_heads=4, n_kv_heads=2, head_dim=64, d_ff=176, vocab=400),
        [4000, 96, 300, 5], [2, 3, 4, 2]),
    # One prompt longer than a chunk: its first 4096 rows fill a chunk and its last 404 rows, with
    # the next prompt, attend to them from the second.
    "bf16_prompt_longer_than_a_chunk": (
        ModelConfig(n_layers=2, d_model=128, n_heads=4, n_kv_heads=2, head_dim=64, d_ff=176, vocab=400),
        [4500, 12], [3, 2]),
}


@pytest.mark.parametrize("case", sorted(TOY_CASES))
def test_toy_shapes(case):
    m, plens, stops = TOY_CASES[case]
    say(f"toy {case}")
    rng = np.random.default_rng(zlib.crc32(case.encode()))
    prompts = _prompts(rng, m.vocab, plens)
    run = DeviceRun(m, 77, prompts, stops)
    assert run.active == R.active_schedule(stops)
    w = R.Weights(oracle_shape(m), 77)
    st = check_against_oracle(run, w, prompts, stops, range(len(prompts)), *_tol(m))
    say(case, st)
    run.close()


def test_fragmented_kv_reservation():
    """Paged KV with a fragmented reservation: slots 0-2 reserve blocks [0,1], [2,3], [4,5]; slot 1 is
    freed and refilled with a longer prompt, which reserves [2,3,6,7].  Teacher-forced logits of all three
    rows match the oracle."""
    import torch
    from paper_2403_12900_amd.binding import DecodeModel
    m, _, _ = TOY_CASES["bf16_mha_hd64_ragged"]
    say("fragmented KV reservation")
    rng = np.random.default_rng(9)
    dm = DecodeModel(m, 78, max_slots=3, max_ctx=96, kv_blocks=12)
    tok = dm.new_token_buffer()
    first = _prompts(rng, m.vocab, [20, 20, 20])
    dm.prefill([0, 1, 2], first, [4, 4, 4], tok)
    dm.free_slot(1)
    longer = _prompts(rng, m.vocab, [50])[0]
    dm.prefill([1], [longer], [4], tok)
    assert dm.lib.spr_free_blocks(dm.h) == 12 - 8
    prompts = [first[0], longer, first[2]]
    forced = rng.integers(0, m.vocab, size=(3, 3)).astype(np.int32)
    lens = [20, 50, 20]
    got = []
    for s in range(3):
        tok.copy_(torch.from_numpy(forced[s]).to(tok.device))
        lg, _ = dm.decode_step([0, 1, 2], lens, tok, want_logits=True)
        got.append(lg.cpu().numpy())
        lens = [l + 1 for l in lens]
    w = R.Weights(oracle_shape(m), 78)
    for i in range(3):
        ref = R.forward_causal(w, list(prompts[i]) + forced[:, i].tolist(), [len(prompts[i]) + s for s in range(3)])
        for s in range(3):
            d = np.abs(got[s][i] - ref[s]).max()
            assert d <= BF16_TOL[0], (i, s, d)
    dm.close()


def test_forced_tokens_and_in_place_buffer():
    """Teacher forcing through the device token buffer equals the oracle fed the same tokens."""
    m, plens, stops = TOY_CASES["bf16_mha_hd64_ragged"]
    say("forced tokens")
    import torch
    from paper_2403_12900_amd.binding import DecodeModel
    rng = np.random.default_rng(5)
    prompts = _prompts(rng, m.vocab, [9, 20])
    dm = DecodeModel(m, 78, max_slots=2, max_ctx=64)
    tok = dm.new_token_buffer()
    dm.prefill([0, 1], prompts, [5, 5], tok)
    forced = rng.integers(0, m.vocab, size=(4, 2)).astype(np.int32)
    lens = [9, 20]
    got = []
    for s in range(4):
        tok.copy_(torch.from_numpy(forced[s]).to(tok.device))
        lg, _ = dm.decode_step([0, 1], lens, tok, want_logits=True)
        got.append(lg.cpu().numpy())
        lens = [l + 1 for l in lens]
    w = R.Weights(oracle_shape(m), 78)
    for i in range(2):
        ref = R.forward_causal(w, list(prompts[i]) + forced[:, i].tolist(),
                               [len(prompts[i]) + s for s in range(4)])
        for s in range(4):
            d = np.abs(got[s][i] - ref[s]).max()
            assert d <= BF16_TOL[0], (i, s, d)
    dm.close()


def test_read_ceiling_streams_every_weight_matrix():
    """The read-ceiling probe reads every projection and the LM head once per pass, and checks its arguments."""
    m, _, _ = TOY_CASES["bf16_mha_hd64_ragged"]
    from paper_2403_12900_amd.binding import DecodeModel, SproutError
    dm = DecodeModel(m, 78, max_slots=2, max_ctx=64)
    gbps, nbytes = dm.read_ceiling(3)
    e = 2 if m.bf16 else 4
    raw = e * (m.n_layers * ((m.n_heads + 2 * m.n_kv_heads) * m.head_dim * m.d_model
                             + m.d_model * m.n_heads * m.head_dim + 3 * m.d_ff * m.d_model) + m.vocab * m.d_model)
    say("read ceiling", gbps, nbytes, raw)
    assert raw <= nbytes <= 1.25 * raw + 4096 * (4 * m.n_layers + 1)   # tile padding and 256-byte alignment only
    assert gbps > 0
    with pytest.raises(SproutError):
        dm.read_ceiling(0)
    dm.close()


def test_rewind_regenerates_identically():
    m, _, _ = TOY_CASES["bf16_gqa4_hd128_wide_o"]
    say("rewind")
    import torch
    from paper_2403_12900_amd.binding import DecodeModel
    rng = np.random.default_rng(6)
    prompts = _prompts(rng, m.vocab, [30, 7])
    dm = DecodeModel(m, 79, max_slots=2, max_ctx=64)
    tok = dm.new_token_buffer()
    dm.prefill([0, 1], prompts, [6, 6], tok)
    first = tok.clone()

    def run():
        out = []
        lens = [30, 7]
        for _ in range(5):
            dm.decode_step([0, 1], lens, tok)
            out.append(tok.cpu().numpy().copy())
            lens = [l + 1 for l in lens]
        return np.stack(out)

    a = run()
    dm.rewind(0, 30, 1)
    dm.rewind(1, 7, 1)
    tok.copy_(first)
    b = run()
    assert np.array_equal(a, b)
    dm.close()


@pytest.mark.parametrize("case", ["bf16_gqa4_hd128_wide_o", "bf16_gqa4_hd128_long_context",
                                  "bf16_split_k_uneven_slices"])
def test_repeat_runs_are_bitwise_identical(case):
    """Two runs of the same batch give bitwise equal tokens and logits at every step: cross-wave and
    cross-split reductions have a fixed order (the split merges count arrivals with an atomic, but the
    last split reads every partial in split order).  The first case passes through 20, 15 and 5 rows
    (two-tile, one-tile and packed-row projections), the second through attention splits over a
    1690-position context, the third through the projections' split-K slices."""
    m, plens, stops = TOY_CASES[case]
    say(f"repeat runs {case}")
    rng = np.random.default_rng(11)
    prompts = _prompts(rng, m.vocab, plens)
    a = DeviceRun(m, 80, prompts, stops)
    b = DeviceRun(m, 80, prompts, stops)
    for i in range(len(prompts)):
        assert a.tokens[i] == b.tokens[i], (case, i)
        for s_, z in a.logits[i].items():
            assert np.array_equal(z.view(np.uint32), b.logits[i][s_].view(np.uint32)), (case, i, s_)
    a.close()
    b.close()


def test_batch_invariance():
    """A request decoded alone or inside a batch gives the same tokens and logits within tolerance."""
    m, plens, stops = TOY_CASES["bf16_gqa4_hd128_wide_o"]
    say("batch invariance")
    rng = np.random.default_rng(7)
    prompts = _prompts(rng, m.vocab, plens)
    full = DeviceRun(m, 80, prompts, stops)
    for i in (1, 13):
        alone = DeviceRun(m, 80, [prompts[i]], [stops[i]])
        for s, z in alone.logits[0].items():
            assert np.abs(z - full.logits[i][s]).max() <= BF16_TOL[0]
        alone.close()
    full.close()


# ------------------------------------------------------------------ full-size configurations

def _full_size(key, pick):
    """The configuration's whole closed batch decodes on the device, free-running, to every request's
    stop length; the requests `pick(context lengths)` names are compared with the oracle at every step
    (prefill included), all of them in one oracle pass over the layers."""
    cfg = CONFIGS[key]
    wl = make_workload(cfg)
    seq, stops = wl.seq_lens, wl.stop_lens
    ctx = seq + stops - 1
    sampled = sorted(set(int(i) for i in pick(ctx)))
    record = set(range(int(max(stops[i] for i in sampled))))
    say(f"{cfg.name}: checking requests {sampled} (contexts {[int(ctx[i]) for i in sampled]}) at every step")
    run = DeviceRun(cfg.model, cfg.weight_seed, wl.tokens, stops.tolist(), record=record, keep=set(sampled))
    assert run.active == R.active_schedule(stops.tolist())
    assert [len(t) for t in run.tokens] == stops.tolist()
    say(f"{cfg.name}: device decode done; oracle")
    w = R.Weights(oracle_shape(cfg.model), cfg.weight_seed, resident=False)
    st = check_against_oracle(run, w, wl.tokens, stops, sampled, *BF16_TOL)
    say(cfg.name, st)
    assert st["rows"] == int(sum(stops[i] for i in sampled))
    assert st["max_context"] == int(max(ctx[i] for i in sampled))   # positions attended at the last step
    run.close()
    return st


def _shortest(ctx, n):
    return [int(i) for i in np.argsort(ctx, kind="stable")[:n]]


def _longest(ctx, n):
    return [int(i) for i in np.argsort(ctx, kind="stable")[::-1][:n]]


def _nearest(ctx, target):
    return int(np.argmin(np.abs(ctx - target)))


def _at_ranks(ctx, taken, quantiles):
    """One request per quantile of the context lengths (the request at that rank of the sorted
    contexts, or the next longer one not already in `taken`)."""
    order = [int(i) for i in np.argsort(ctx, kind="stable")]
    out = list(taken)
    for q in quantiles:
        r = int(round(q * (len(order) - 1)))
        while order[r] in out:
            r += 1
        out.append(order[r])
    return out


def test_llama2_7b_ragged_batch32():
    """The benchmarked workload at full size: all 32 requests decode to their stop lengths.  Checked at
    every step: the three longest contexts (1635, 1234 and 1107 positions at the last step; the
    longest, a 616-token prompt with 1020 generated, decodes alone for half of the batch's steps), the
    one nearest the median context (307) and the two shortest (132, 149): every directive level."""
    _full_size("c3", lambda ctx: _shortest(ctx, 2) + _longest(ctx, 3) + [_nearest(ctx, np.median(ctx))])


def test_llama2_7b_batch1_256_tokens():
    """The latency case: one request, prompt 128, 256 generated tokens, every step checked."""
    _full_size("c2", lambda ctx: [0])


def test_llama2_13b_ragged_batch64():
    """13B shape, 64 ragged requests in 16-position KV pages, eight of them checked at every step: the
    longest context (1353 positions), the two shortest (127, 144) and one at each of the 20th, 40th,
    50th, 60th and 80th percentiles of the contexts (234 to 580 positions): every directive level."""
    _full_size("c4", lambda ctx: _at_ranks(ctx, _shortest(ctx, 2) + _longest(ctx, 1), (0.2, 0.4, 0.5, 0.6, 0.8)))


def test_llama2_70b_gqa_ragged_batch16():
    """70B shape with grouped-query attention (8 query heads per KV head), ~138 GB of weights on one
    GPU: four requests, the one nearest the median context (884 positions) and the three shortest
    (177, 292, 381), are checked at every step against the oracle, which streams the weights layer by
    layer."""
    _full_size("c5", lambda ctx: _shortest(ctx, 3) + [_nearest(ctx, np.median(ctx))])
