"""Workload generator: determinism, directive order (Section III-E), length recipe."""
import math

import numpy as np

from paper_2403_12900_amd.configs import CONFIGS, DecodeConfig, WorkloadRecipe, LLAMA2_7B
from paper_2403_12900_amd.workload import make_workload, workload_stats


def test_deterministic():
    for k in CONFIGS:
        a, b = make_workload(CONFIGS[k]), make_workload(CONFIGS[k])
        assert all(np.array_equal(x, y) for x, y in zip(a.tokens, b.tokens))
        assert np.array_equal(a.stop_lens, b.stop_lens)


def test_directive_precedes_prompt():
    for k in ("c1", "c3", "c5"):
        w = make_workload(CONFIGS[k])
        for i, t in enumerate(w.tokens):
            p = w.prefix_lens[i]
            assert np.array_equal(t[:p], w.directive_ids[w.levels[i]])
            assert len(t) == p + w.prompt_lens[i]


def test_tiny_config_fixed_lengths():
    w = make_workload(CONFIGS["c1"])
    assert w.seq_lens.tolist() == [22, 30, 38, 14]
    assert w.stop_lens.tolist() == [32, 8, 16, 4]
    assert w.decode_tokens() == 31 + 7 + 15 + 3


def test_length_distribution_recipe():
    """Medians within 10 % over 10^4 draws, clip bounds hold, level mix near uniform."""
    rec = WorkloadRecipe(batch=10000, prompt_median=200.0, prompt_clip=(16, 1024), prefix_lens=(0, 8, 12),
                         stop_medians=(400.0, 120.0, 40.0), stop_clip=(1, 1024))
    cfg = DecodeConfig("probe", LLAMA2_7B, rec, 1, 7)
    w = make_workload(cfg)
    assert abs(np.median(w.prompt_lens) / 200 - 1) < 0.1
    assert w.prompt_lens.min() >= 16 and w.prompt_lens.max() <= 1024
    for lvl, med in enumerate((400, 120, 40)):
        L = w.stop_lens[w.levels == lvl]
        assert abs(np.median(L) / med - 1) < 0.1
        assert abs(len(L) / 10000 - 1 / 3) < 0.03
    assert w.stop_lens.min() >= 1 and w.stop_lens.max() <= 1024
    # Log-space spread of the unclipped middle matches sigma = 0.6.
    L0 = np.log(w.stop_lens[(w.levels == 1)])
    assert abs(np.std(L0) - 0.6) < 0.05


def test_stats_sum_of_steps():
    cfg = CONFIGS["c1"]
    st = workload_stats(cfg, make_workload(cfg))
    assert st["steps"] == 31 and st["decode_tokens"] == 56
