"""Pins of the CPU oracle against facts that do not come from the oracle itself.

Each test checks the oracle against a closed form, an invariant, a special
case that reduces to a textbook result or library routine, a published test
vector, or a brute-force pure-Python computation on tiny inputs.  Together
they are chosen so that a dropped term, a wrong sign or index, or a
transposed operand anywhere in oracle/llama_ref.py or oracle/wgen.c fails at
least one of them.
"""
import dataclasses
import math
import os

import numpy as np
import pytest
from scipy.special import expit

from oracle import _clib
from oracle import llama_ref as R

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

TOY = R.Shape(n_layers=2, d_model=32, n_heads=4, n_kv_heads=2, head_dim=8, d_ff=40, vocab=50, bf16=True)
TOY_MHA = R.Shape(n_layers=1, d_model=16, n_heads=2, n_kv_heads=2, head_dim=8, d_ff=24, vocab=20, bf16=False)
# The brute-force forward below keeps cached keys/values exact.
TOY_EXACT_KV = dataclasses.replace(TOY, kv_round=False)
TOY_MHA_EXACT_KV = dataclasses.replace(TOY_MHA, kv_round=False)


# ---------------------------------------------------------------- generator

def test_splitmix64_published_vector():
    lines = [l for l in open(os.path.join(GOLDEN, "splitmix64_seed1234567.txt")) if not l.startswith("#")]
    want = [int(l) for l in lines if l.strip()]
    got = [_clib.splitmix_output(1234567, n) for n in range(1, 6)]
    assert got == want


def _py_mix(z):
    M = 2**64 - 1
    z ^= z >> 30
    z = (z * 0xBF58476D1CE4E5B9) & M
    z ^= z >> 27
    z = (z * 0x94D049BB133111EB) & M
    z ^= z >> 31
    return z


def test_wgen_elements_follow_the_definition():
    """A few elements recomputed in pure Python from the generator's definition."""
    G = 0x9E3779B97F4A7C15
    M = 2**64 - 1
    seed, tensor, layer, cols = 77, 5, 3, 40
    key = _py_mix((seed + (1 + 256 * tensor + layer) * G) & M)
    rows = _clib.wgen_rows(seed, tensor, layer, cols, 2, 3, bf16=False, dtype=np.float32)
    for (r, c) in [(0, 0), (1, 17), (2, 39)]:
        e = (2 + r) * cols + c
        r0 = _py_mix((key + (2 * e + 1) * G) & M)
        r1 = _py_mix((key + (2 * e + 2) * G) & M)
        S = sum((r0 >> (16 * i)) & 0xFFFF for i in range(4)) + sum((r1 >> (16 * i)) & 0xFFFF for i in range(4))
        val = np.float32(S - 262140) * np.float32(float.fromhex("0x1.91530cp-22"))
        assert rows[r, c] == val


def test_wgen_moments_and_bounds():
    n_cols = 1000
    w = _clib.wgen_rows(1234, 1, 0, n_cols, 0, 1000, bf16=False)   # 10^6 draws
    assert abs(w.mean()) < 3 * 0.02 / 1000
    assert abs(w.std() / 0.02 - 1.0) < 0.01
    # Irwin-Hall(8) support is bounded: |S - mean| <= 262140.
    assert np.abs(w).max() <= 262140 * float.fromhex("0x1.91530cp-22") * (1 + 1e-7)
    # Kurtosis of a sum of 8 uniforms: 3 - 1.2/8 = 2.85.
    k = np.mean((w - w.mean()) ** 4) / w.var() ** 2
    assert abs(k - 2.85) < 0.02


def test_wgen_bf16_is_rne_of_fp32():
    f32 = _clib.wgen_rows(9, 2, 1, 256, 0, 64, bf16=False, dtype=np.float32)
    b16 = _clib.wgen_rows(9, 2, 1, 256, 0, 64, bf16=True, dtype=np.float32)
    u = b16.view(np.uint32)
    assert np.all((u & 0xFFFF) == 0)
    # Round-to-nearest-even onto the bf16 grid: error at most half an ulp, and ties go to even.
    err = np.abs(b16.astype(np.float64) - f32.astype(np.float64))
    ulp = np.abs(np.spacing(b16.astype(np.float32)).astype(np.float64)) * 2**16
    assert np.all(err <= ulp / 2 + 1e-30)


def test_wgen_rows_are_slices_of_one_matrix():
    full = _clib.wgen_rows(5, 7, 2, 33, 0, 10, bf16=True)
    part = _clib.wgen_rows(5, 7, 2, 33, 4, 3, bf16=True)
    assert np.array_equal(full[4:7], part)
    other_layer = _clib.wgen_rows(5, 7, 3, 33, 0, 10, bf16=True)
    other_tensor = _clib.wgen_rows(5, 6, 2, 33, 0, 10, bf16=True)
    assert not np.array_equal(full, other_layer) and not np.array_equal(full, other_tensor)


# ---------------------------------------------------------------- RMSNorm

def test_rmsnorm_unit_rms_and_scale_invariance():
    rng = np.random.default_rng(0)
    x = rng.normal(size=(5, 64)) * 3
    y = R.rmsnorm(x, np.ones(64), 0.0)
    assert np.allclose(np.sqrt(np.mean(y * y, axis=-1)), 1.0, atol=1e-12)
    assert np.allclose(R.rmsnorm(7.5 * x, np.ones(64), 0.0), y, atol=1e-12)
    # A gain of 2 doubles the output RMS.
    y2 = R.rmsnorm(x, 2 * np.ones(64), 0.0)
    assert np.allclose(np.sqrt(np.mean(y2 * y2, axis=-1)), 2.0, atol=1e-12)


def test_rmsnorm_constant_vector_and_eps():
    # RMSNorm(c * 1) = sign(c) when eps << c^2; with eps = c^2 it is sign(c)/sqrt(2).
    for c in (-3.0, 0.5, 10.0):
        y = R.rmsnorm(np.full((1, 8), c), np.ones(8), 1e-12)
        assert np.allclose(y, np.sign(c), atol=1e-9)
        y = R.rmsnorm(np.full((1, 8), c), np.ones(8), c * c)
        assert np.allclose(y, np.sign(c) / math.sqrt(2), atol=1e-12)
    # The textbook example x = (3, 4): mean square 12.5.
    y = R.rmsnorm(np.array([[3.0, 4.0]]), np.ones(2), 0.0)
    assert np.allclose(y, [[3 / math.sqrt(12.5), 4 / math.sqrt(12.5)]])


# ---------------------------------------------------------------- RoPE

def test_rope_textbook_rotation():
    # head_dim 2: one pair with theta_0 = 1, so position p rotates (1, 0) to (cos p, sin p).
    for p in (0, 1, 3, 100):
        y = R.apply_rope(np.array([[[1.0, 0.0]]]), [p], 10000.0)
        assert np.allclose(y[0, 0], [math.cos(p), math.sin(p)], atol=1e-12)
    # head_dim 4, base 10000: pair 1 has theta = 10000^(-1/2) = 0.01, so position 100 turns it by 1 rad.
    y = R.apply_rope(np.array([[[0.0, 0.0, 1.0, 0.0]]]), [100], 10000.0)
    assert np.allclose(y[0, 0], [0.0, 0.0, math.cos(1.0), math.sin(1.0)], atol=1e-12)


def test_rope_pairs_are_adjacent_and_norm_preserving():
    rng = np.random.default_rng(1)
    x = rng.normal(size=(6, 3, 16))
    pos = [0, 1, 7, 50, 999, 3083]
    y = R.apply_rope(x, pos, 10000.0)
    assert np.allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), atol=1e-12)
    # Each pair keeps its own norm (rotation acts inside the pair (2i, 2i+1) only).
    pn = lambda v: np.sqrt(v[..., 0::2] ** 2 + v[..., 1::2] ** 2)
    assert np.allclose(pn(y), pn(x), atol=1e-12)
    assert np.allclose(R.apply_rope(x, [0] * 6, 10000.0), x, atol=0)


def test_rope_relative_position():
    rng = np.random.default_rng(2)
    q = rng.normal(size=(1, 1, 32))
    k = rng.normal(size=(1, 1, 32))
    for m, n in [(5, 2), (100, 37), (3000, 11)]:
        lhs = np.sum(R.apply_rope(q, [m], 1e4) * R.apply_rope(k, [n], 1e4))
        rhs = np.sum(R.apply_rope(q, [m - n], 1e4) * k)
        assert abs(lhs - rhs) < 1e-9 * (1 + abs(rhs))


# ---------------------------------------------------------------- softmax / attention

def test_softmax_sums_to_one_and_shift_invariance():
    rng = np.random.default_rng(3)
    s = rng.normal(size=(7, 33)) * 20
    p = R.softmax(s)
    assert np.all(np.abs(p.sum(-1) - 1) <= 1e-12)
    assert np.allclose(R.softmax(s + 123.0), p, atol=1e-15)
    row = [1.0, 2.0, -1.0]
    e = [math.exp(v) for v in row]
    assert np.allclose(R.softmax(np.array(row)), [v / sum(e) for v in e], atol=1e-15)


def test_attention_special_cases():
    rng = np.random.default_rng(4)
    H, Hkv, hd = 4, 2, 8
    K = rng.normal(size=(1, Hkv, hd))
    V = rng.normal(size=(1, Hkv, hd))
    q = rng.normal(size=(H, hd))
    o = R.attend(q, K, V)          # one cached position: the output is that value
    for h in range(H):
        assert np.allclose(o[h], V[0, h // 2])
    K = rng.normal(size=(9, Hkv, hd))
    V = rng.normal(size=(9, Hkv, hd))
    o = R.attend(np.zeros((H, hd)), K, V)   # q = 0: uniform weights, the mean of the values
    for h in range(H):
        assert np.allclose(o[h], V[:, h // 2].mean(0))


def test_gqa_equals_mha_with_repeated_kv():
    rng = np.random.default_rng(5)
    H, Hkv, hd, ctx = 8, 2, 16, 13
    q = rng.normal(size=(H, hd))
    K = rng.normal(size=(ctx, Hkv, hd))
    V = rng.normal(size=(ctx, Hkv, hd))
    Kr = np.repeat(K, H // Hkv, axis=1)    # head h uses kv head h // 4
    Vr = np.repeat(V, H // Hkv, axis=1)
    assert np.allclose(R.attend(q, K, V), R.attend(q, Kr, Vr), atol=1e-12)


def test_attention_brute_force_loops():
    rng = np.random.default_rng(6)
    T, H, Hkv, hd = 5, 4, 2, 4
    q = rng.normal(size=(T, H, hd))
    k = rng.normal(size=(T, Hkv, hd))
    v = rng.normal(size=(T, Hkv, hd))
    got = R.causal_attention(q, k, v)
    for t in range(T):
        for h in range(H):
            g = h // (H // Hkv)
            sc = [sum(q[t, h, i] * k[j, g, i] for i in range(hd)) / math.sqrt(hd) for j in range(t + 1)]
            mx = max(sc)
            ex = [math.exp(s - mx) for s in sc]
            z = sum(ex)
            ref = [sum(ex[j] / z * v[j, g, i] for j in range(t + 1)) for i in range(hd)]
            assert np.allclose(got[t, h], ref, atol=1e-12)


# ---------------------------------------------------------------- MLP / argmax

def test_silu_and_swiglu():
    x = np.linspace(-30, 30, 61)
    assert R.silu(np.array([0.0]))[0] == 0.0
    assert np.allclose(R.silu(x), x * expit(x), atol=1e-12)
    rng = np.random.default_rng(7)
    d, f = 3, 5
    m = rng.normal(size=(2, d))
    w1, w3, w2 = rng.normal(size=(f, d)), rng.normal(size=(f, d)), rng.normal(size=(d, f))
    got = R.swiglu(m, w1, w3, w2)
    for r in range(2):
        hid = []
        for j in range(f):
            g = sum(m[r, i] * w1[j, i] for i in range(d))
            u = sum(m[r, i] * w3[j, i] for i in range(d))
            hid.append(g / (1 + math.exp(-g)) * u)
        ref = [sum(hid[j] * w2[o, j] for j in range(f)) for o in range(d)]
        assert np.allclose(got[r], ref, atol=1e-12)


def test_argmax_lowest_index_on_ties():
    z = np.array([[1.0, 3.0, 3.0, 2.0], [5.0, 5.0, 5.0, 5.0], [-1.0, -2.0, -1.0, -3.0]])
    assert R.argmax_first(z).tolist() == [1, 0, 0]


# ---------------------------------------------------------------- whole model

def _py_forward_toy(w: R.Weights, tokens):
    """Brute-force pure-Python Llama-2 forward (lists and math only) for tiny shapes."""
    sh = w.shape
    d, H, Hkv, hd, f = sh.d_model, sh.n_heads, sh.n_kv_heads, sh.head_dim, sh.d_ff
    E = w.matrix("embed").tolist()
    xs = [list(E[t]) for t in tokens]
    T = len(tokens)

    def norm(v):
        ms = sum(a * a for a in v) / len(v)
        return [a / math.sqrt(ms + sh.rms_eps) for a in v]

    def mv(W, v):
        return [sum(W[o][i] * v[i] for i in range(len(v))) for o in range(len(W))]

    def rot(vec, p):
        out = list(vec)
        for i in range(hd // 2):
            th = p * sh.rope_base ** (-2.0 * i / hd)
            a, b = vec[2 * i], vec[2 * i + 1]
            out[2 * i] = a * math.cos(th) - b * math.sin(th)
            out[2 * i + 1] = a * math.sin(th) + b * math.cos(th)
        return out

    for layer in range(sh.n_layers):
        Wd = {n: w.matrix(n, layer).tolist() for n in R.Weights.LAYER_MATS}
        qs, ks, vs = [], [], []
        for t in range(T):
            a = norm(xs[t])
            q, k, v = mv(Wd["wq"], a), mv(Wd["wk"], a), mv(Wd["wv"], a)
            qs.append([rot(q[h * hd:(h + 1) * hd], t) for h in range(H)])
            ks.append([rot(k[g * hd:(g + 1) * hd], t) for g in range(Hkv)])
            vs.append([v[g * hd:(g + 1) * hd] for g in range(Hkv)])
        new = []
        for t in range(T):
            o = []
            for h in range(H):
                g = h * Hkv // H
                sc = [sum(qs[t][h][i] * ks[j][g][i] for i in range(hd)) / math.sqrt(hd) for j in range(t + 1)]
                mx = max(sc)
                ex = [math.exp(s - mx) for s in sc]
                z = sum(ex)
                o += [sum(ex[j] / z * vs[j][g][i] for j in range(t + 1)) for i in range(hd)]
            x = [a + b for a, b in zip(xs[t], mv(Wd["wo"], o))]
            m = norm(x)
            g1, u = mv(Wd["w1"], m), mv(Wd["w3"], m)
            hdn = [a / (1 + math.exp(-a)) * b for a, b in zip(g1, u)]
            new.append([a + b for a, b in zip(x, mv(Wd["w2"], hdn))])
        xs = new
    lm = w.matrix("lm_head").tolist()
    return np.array([mv(lm, norm(x)) for x in xs])


@pytest.mark.parametrize("shape", [TOY_EXACT_KV, TOY_MHA_EXACT_KV], ids=["gqa_bf16", "mha_fp32"])
def test_forward_matches_brute_force(shape):
    w = R.Weights(shape, seed=11)
    toks = [3, 17, 0, shape.vocab - 1, 8, 8]
    got = R.forward_causal(w, toks)
    ref = _py_forward_toy(w, toks)
    assert np.allclose(got, ref, rtol=1e-10, atol=1e-12)


def test_round_to_storage():
    # Near 1 the bf16 grid spacing is 2^-7.  1 + 2^-8 is a tie and goes to the
    # even neighbour 1.0; 1 + 3 * 2^-8 is a tie between 1 + 2^-7 (odd) and
    # 1 + 2^-6 (even) and goes to 1 + 2^-6.
    x = np.array([1.0, 1 + 2**-8, 1 + 3 * 2**-8, -2.5, 1e-3, 0.0])
    b = R.round_to_storage(x, True)
    assert b.tolist()[:4] == [1.0, 1.0, 1 + 2**-6, -2.5]
    assert np.all((b.astype(np.float32).view(np.uint32) & 0xFFFF) == 0)
    assert abs(b[4] - 1e-3) <= 1e-3 * 2**-8
    f = R.round_to_storage(np.array([1 + 2**-30]), False)
    assert f[0] == 1.0                      # fp32 rounding


def test_kv_cache_storage_rounding_is_small_and_consistent():
    """Rounded and exact caches give close logits; incremental == recompute holds for both."""
    w_r = R.Weights(TOY, seed=21)
    w_e = R.Weights(TOY_EXACT_KV, seed=21)
    toks = [3, 9, 27, 4, 4, 11, 2]
    a = R.forward_causal(w_r, toks)
    b = R.forward_causal(w_e, toks)
    assert 0 < np.abs(a - b).max() < 1e-2 * np.abs(b).max()
    # The cache the incremental decoder holds is on the bf16 grid.
    dec = R.KVCacheDecoder(w_r)
    dec.prefill(0, toks, capacity=len(toks))
    K = dec.K[0][1][: len(toks)]
    assert np.all((K.astype(np.float32).view(np.uint32) & 0xFFFF) == 0)


def test_layer_streaming_matches_resident():
    toks = [1, 2, 3, 4, 40, 2]
    a = R.forward_causal(R.Weights(TOY, 3, resident=True), toks)
    b = R.forward_causal(R.Weights(TOY, 3, resident=False), toks)
    assert np.array_equal(a, b)


def test_incremental_kv_cache_equals_full_recompute():
    """Section II-A: cached keys/values are reused, not recomputed -- the result must not change."""
    w = R.Weights(TOY, seed=12)
    rng = np.random.default_rng(8)
    prompts = [rng.integers(0, TOY.vocab, size=n).tolist() for n in (5, 1, 9)]
    stops = [6, 3, 1]
    toks, logits = R.greedy_decode(w, prompts, stops)
    for i in range(3):
        assert len(toks[i]) == stops[i]
        seq = prompts[i] + toks[i][:-1]
        full = R.forward_causal(w, seq)
        n = len(prompts[i])
        assert np.allclose(logits[i], full[n - 1:], rtol=1e-10, atol=1e-10)
        assert toks[i] == R.argmax_first(full[n - 1:]).tolist()
        tf = R.teacher_forced_logits(w, prompts[i], toks[i])
        assert np.allclose(tf, logits[i], rtol=1e-10, atol=1e-10)


def test_batch_independence_exact():
    w = R.Weights(TOY, seed=13)
    rng = np.random.default_rng(9)
    prompts = [rng.integers(0, TOY.vocab, size=n).tolist() for n in (4, 7, 2)]
    stops = [5, 2, 4]
    toks, logits = R.greedy_decode(w, prompts, stops)
    for i in range(3):
        t1, l1 = R.greedy_decode(w, [prompts[i]], [stops[i]])
        assert t1[0] == toks[i]
        assert np.allclose(l1[0], logits[i], rtol=1e-12, atol=1e-12)


def test_teacher_forcing_feeds_given_tokens():
    w = R.Weights(TOY, seed=14)
    prompts = [[1, 2, 3], [4, 5]]
    stops = [4, 3]
    forced = [[7, 7, 7, 7], [9, 9, 9]]
    _, logits = R.greedy_decode(w, prompts, stops, forced=forced)
    for i in range(2):
        ref = R.teacher_forced_logits(w, prompts[i], forced[i])
        assert np.allclose(logits[i], ref, rtol=1e-10, atol=1e-10)


def test_directive_prefix_changes_the_continuation():
    """The directive is ordinary context (Section II-B: its tokens sit in the KV cache)."""
    w = R.Weights(TOY, seed=15)
    prompt = [5, 6, 7]
    a = R.forward_causal(w, prompt)[-1]
    b = R.forward_causal(w, [30, 31] + prompt)[-1]
    assert not np.allclose(a, b)


# ---------------------------------------------------------------- retirement

def test_retirement_closed_form():
    stops = [32, 8, 16, 4, 1, 8]
    sched = R.active_schedule(stops)
    assert len(sched) == max(stops) - 1
    for s, act in enumerate(sched, start=1):
        assert act == sorted(i for i in range(len(stops)) if stops[i] > s)
    assert sum(len(a) for a in sched) == sum(L - 1 for L in stops)
    assert R.active_schedule([1, 1]) == []


def test_requests_share_layers_without_mixing():
    """forward_causal_requests gives each request what forward_causal gives it alone (requests stacked
    into one product per matrix must not see each other's positions)."""
    w = R.Weights(TOY, 21)
    rng = np.random.default_rng(31)
    seqs = [rng.integers(0, TOY.vocab, size=n).tolist() for n in (7, 1, 12)]
    want = [[0, 6], None, [3, 11]]
    got = R.forward_causal_requests(w, seqs, want)
    for s, wp, g in zip(seqs, want, got):
        assert np.allclose(g, R.forward_causal(w, s, wp), rtol=1e-12, atol=1e-12)
