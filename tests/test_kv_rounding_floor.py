"""The KV-cache rounding floor, measured with the oracle alone (no GPU).

Section II-A: the KV cache stores the key and value vectors of processed
tokens and later tokens attend to them.  The served model's cache holds them
in its own storage format (the paper's server manages the cache with vLLM,
Section III-E), so a key or value is rounded when cached.  Two implementations
that both do this, but compute the value before rounding in different valid
arithmetic, store a few elements on opposite sides of a rounding boundary.
tests/kv_floor.py runs the oracle in lockstep with fp64 and with fp32
key/value arithmetic (and with fp64 values moved by one fp32 ulp) and reports
how far the logits then differ: no parity gate between two such
implementations can be tighter than that floor.

* Llama-2-7B shape (the benchmarked model): with a bf16 cache the floor is well
  inside the 5e-2 / 1e-2 gate, and bf16 boundary flips dominate it (the fp32
  cache floor is orders of magnitude lower).
* Llama-2-70B GQA shape (slow; SPROUT_SLOW_TESTS=1): with a bf16 cache the
  floor exceeds the 5e-2 gate on a 16-token request, so that configuration is
  checked with an fp32 cache (paper_2403_12900_amd/configs.py, LLAMA2_70B).
* The precision of the projection input matters on top of that: keys and values
  computed from an input carried as two bf16 parts (16 significant bits) cross
  rounding boundaries far more often than fp32-computed ones.  At the 13B shape
  over a 212-position request (slow) that raises the distance to the oracle at
  every position by about a third, and the worst row by 14-75%, which is why
  the device's QKV input carries all 24 bits of the residual (hi + mid + lo).
"""
import os

import numpy as np
import pytest

from oracle import llama_ref as R
from paper_2403_12900_amd.configs import CONFIGS

from .kv_floor import floors, lockstep_logits

RUNS = ("bf16_f64", "bf16_f32", "bf16_hilo", "f32_f64", "f32_f32")
GATE_ABS, GATE_REL = 5e-2, 1e-2


def _shape(key):
    m = CONFIGS[key].model
    return R.Shape(m.n_layers, m.d_model, m.n_heads, m.n_kv_heads, m.head_dim, m.d_ff, m.vocab, m.rope_base,
                   m.rms_eps, m.bf16)


def _measure(key, T, runs=RUNS, prompt=()):
    cfg = CONFIGS[key]
    toks = list(prompt) + np.random.default_rng(7).integers(0, cfg.model.vocab, size=T).tolist()
    z = lockstep_logits(_shape(key), cfg.weight_seed, toks, runs)
    P = max(len(prompt) - 1, 0)                       # positions from the last prompt row on
    f = floors({r: v[P:] for r, v in z.items()})
    print(key, T, f, flush=True)
    return f


@pytest.mark.slow
def test_kv_rounding_floor_7b_shape():
    f = _measure("c3", 8)
    bf, fp = f["bf16_f64~bf16_f32"], f["f32_f64~f32_f32"]
    assert fp["max_abs"] < 1e-3 and fp["rel_l2"] < 1e-4
    assert bf["max_abs"] > 20 * fp["max_abs"]              # the bf16 boundary flips set the floor
    assert bf["max_abs"] < GATE_ABS / 2 and bf["rel_l2"] < GATE_REL / 2
    # 16-bit projection inputs move the logits further
    assert f["bf16_f64~bf16_hilo"]["mean_rel_l2"] > bf["mean_rel_l2"]


@pytest.mark.slow
@pytest.mark.skipif(os.environ.get("SPROUT_SLOW_TESTS") != "1",
                    reason="about 4 minutes on 8 cores (40 layers, 212 positions, three runs); set SPROUT_SLOW_TESTS=1")
def test_two_part_qkv_input_moves_the_logits_further_at_13b():
    """The 13B request whose bf16 logits once missed the gate on the device with a two-part QKV input
    (c4 request 39: 152-token prompt), followed by 60 positions: the fp32-arithmetic floor stays near
    half the gate, and a 16-bit input raises the distance over every position (mean relative L2
    3.3e-3 -> 4.3e-3; worst max abs 0.027 -> 0.030 here, 0.024 -> 0.041 with another 60 tokens)."""
    from paper_2403_12900_amd.workload import make_workload
    prompt = make_workload(CONFIGS["c4"]).tokens[39]
    f = _measure("c4", 60, ("bf16_f64", "bf16_f32", "bf16_hilo"), prompt=prompt)
    bf, hl = f["bf16_f64~bf16_f32"], f["bf16_f64~bf16_hilo"]
    assert bf["max_abs"] < 0.6 * GATE_ABS and bf["rel_l2"] < GATE_REL / 2
    assert hl["mean_rel_l2"] > 1.2 * bf["mean_rel_l2"]


@pytest.mark.slow
@pytest.mark.skipif(os.environ.get("SPROUT_SLOW_TESTS") != "1",
                    reason="about 5 minutes on 8 cores (80 layers x 0.86 G weights); set SPROUT_SLOW_TESTS=1")
def test_kv_rounding_floor_70b_shape_exceeds_the_gate_with_a_bf16_cache():
    f = _measure("c5", 16, RUNS + ("bf16_f64_ulp",))
    bf, fp = f["bf16_f64~bf16_f32"], f["f32_f64~f32_f32"]
    assert bf["max_abs"] > GATE_ABS                        # measured 0.061 (one-ulp move alone: 0.021)
    assert fp["max_abs"] < 1e-3 and fp["rel_l2"] < 1e-4   # measured 1.1e-4 / 1.2e-5
    assert not CONFIGS["c5"].model.kv_is_bf16
