"""Continuous (iteration-level) batching scheduler, on the host alone.

The scheduler behind spr_serve (csrc/host_state.cpp, `serve`) refills slots
that retire with waiting requests, in the manner of the iteration-level
batching and paged KV cache the paper's inference server relies on
(Section IV, inference server; related work on Orca and vLLM).  Here it runs
over a device stand-in that only records which call produced which token, so
its invariants can be checked exactly without a GPU.
"""
import ctypes
import os

import numpy as np
import pytest

from oracle import llama_ref as R
from paper_2403_12900_amd import binding
from paper_2403_12900_amd.configs import TINY

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
# SPROUT_HOST_LIB selects another build of the same sources (the sanitizer build).
HOST_LIB = os.environ.get("SPROUT_HOST_LIB", os.path.join(ROOT, "paper_2403_12900_amd", "libsprout_host.so"))
I32 = ctypes.POINTER(ctypes.c_int32)


class Sched:
    def __init__(self, max_slots=4, max_ctx=256, kv_blocks=64):
        L = ctypes.CDLL(HOST_LIB)
        L.sprh_new.restype = ctypes.c_void_p
        L.sprh_new.argtypes = [ctypes.POINTER(binding.SprConfig)]
        L.sprh_delete.argtypes = [ctypes.c_void_p]
        L.sprh_serve.argtypes = [ctypes.c_void_p, ctypes.c_int, I32, I32, I32, ctypes.c_int, ctypes.c_int, I32, I32,
                                 I32, I32, I32, I32, ctypes.c_int, I32, ctypes.POINTER(ctypes.c_int64)]
        L.sprh_prefill.argtypes = [ctypes.c_void_p, ctypes.c_int, I32, I32, I32, I32]
        L.sprh_free_blocks.argtypes = [ctypes.c_void_p]
        L.sprh_last_error.restype = ctypes.c_char_p
        self.L = L
        self.cfg = binding.make_config(TINY, max_slots, max_ctx, kv_blocks)
        self.h = L.sprh_new(ctypes.byref(self.cfg))
        assert self.h

    def close(self):
        self.L.sprh_delete(self.h)

    def run(self, n_tokens, stop, arrival=None, max_active=None, eos=()):
        """eos: (request, token index) pairs whose token is the EOS id."""
        n = len(stop)
        arrival = [0] * n if arrival is None else arrival
        max_active = self.cfg.max_slots if max_active is None else max_active
        a = [np.ascontiguousarray(np.asarray(x, dtype=np.int32)) for x in (n_tokens, stop, arrival)]
        er = np.ascontiguousarray(np.asarray([e[0] for e in eos] or [0], dtype=np.int32))
        ei = np.ascontiguousarray(np.asarray([e[1] for e in eos] or [0], dtype=np.int32))
        lengths = np.full(max(n, 1), -1, dtype=np.int32)
        tot = int(sum(stop))
        it, sl, call = (np.full(tot, -1, dtype=np.int32) for _ in range(3))
        batch = np.full(4096, -1, dtype=np.int32)
        cnt = np.zeros(5, dtype=np.int64)
        p = lambda x: x.ctypes.data_as(I32)
        st = self.L.sprh_serve(self.h, n, p(a[0]), p(a[1]), p(a[2]), max_active, len(eos), p(er), p(ei), p(it), p(sl),
                               p(call), p(batch), len(batch), p(lengths),
                               cnt.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)))
        self.lengths = lengths[:n].tolist()
        off = np.concatenate([[0], np.cumsum(stop)]).astype(int)
        per = [(it[off[i]:off[i + 1]], sl[off[i]:off[i + 1]], call[off[i]:off[i + 1]]) for i in range(n)]
        steps = int(cnt[1])
        return st, per, batch[:steps].tolist(), dict(zip(["iterations", "decode_steps", "prefill_calls",
                                                          "decode_tokens", "max_batch"], cnt.tolist()))


def check_invariants(per, stop, arrival, max_active, n_slots):
    n = len(stop)
    for i in range(n):
        its, slots, calls = per[i]
        assert len(its) == stop[i] and (calls >= 0).all(), i              # every token produced once
        assert np.all(np.diff(calls) > 0), i                                 # in order, one per call
        # Admission iteration: prefill emits token 0 and that iteration's decode step token 1;
        # afterwards one token per iteration.
        assert np.all(np.diff(its[1:]) == 1) and (len(its) < 2 or its[1] == its[0]), i
        assert its[0] >= arrival[i], i                                       # admitted after arrival
        assert len(set(slots.tolist())) == 1 and 0 <= slots[0] < n_slots, i  # one slot for life
    firsts = [per[i][0][0] for i in range(n)]
    assert all(a <= b for a, b in zip(firsts, firsts[1:]))                   # first come, first served
    # Slot exclusivity and the in-flight bound, iteration by iteration.
    last = max(p[0][-1] for p in per)
    for t in range(last + 1):
        live = [i for i in range(n) if per[i][0][0] <= t <= per[i][0][-1]]
        assert len(live) <= max_active, t
        assert len({int(per[i][1][0]) for i in live}) == len(live), t


def test_no_contention_matches_the_closed_batch_schedule():
    """All requests admitted at once: one prefill, then the closed-batch active set per step."""
    s = Sched(max_slots=8, kv_blocks=256)
    stop = [5, 1, 9, 3, 9, 2, 7, 4]
    st, per, batch, c = s.run([10] * 8, stop)
    assert st == 0
    assert c["prefill_calls"] == 1
    assert batch == [len(a) for a in R.active_schedule(stop)]
    assert c["decode_tokens"] == sum(x - 1 for x in stop)
    check_invariants(per, stop, [0] * 8, 8, 8)
    s.close()


def test_empty_request_list_is_a_no_op():
    """No requests: success, no prefill or decode call, and every KV block still free."""
    s = Sched(max_slots=4, kv_blocks=64)
    free0 = s.L.sprh_free_blocks(s.h)
    st, per, batch, c = s.run([], [])
    assert st == 0, s.L.sprh_last_error()
    assert per == [] and batch == []
    assert c == {"iterations": 0, "decode_steps": 0, "prefill_calls": 0, "decode_tokens": 0, "max_batch": 0}
    assert s.L.sprh_free_blocks(s.h) == free0
    s.close()


def test_refills_retired_slots_in_order():
    rng = np.random.default_rng(7)
    stop = rng.integers(1, 30, size=40).tolist()
    n_tok = rng.integers(1, 60, size=40).tolist()
    s = Sched(max_slots=6, max_ctx=128, kv_blocks=64)
    st, per, batch, c = s.run(n_tok, stop, max_active=5)
    assert st == 0, s.L.sprh_last_error()
    check_invariants(per, stop, [0] * 40, 5, 6)
    assert max(batch) <= 5 and c["decode_tokens"] == sum(x - 1 for x in stop)
    assert s.L.sprh_free_blocks(s.h) == 64                                   # every block returned
    s.close()


def test_one_slot_serves_requests_back_to_back():
    stop = [3, 1, 4, 2]
    s = Sched(max_slots=2)
    st, per, batch, c = s.run([5, 6, 7, 8], stop, max_active=1)
    assert st == 0
    assert batch == [1] * sum(x - 1 for x in stop)
    ends = [p[0][-1] for p in per]
    starts = [p[0][0] for p in per]
    assert all(starts[i + 1] > ends[i] for i in range(3))                    # strictly sequential
    s.close()


def test_arrivals_and_idle_gaps():
    stop = [4, 3, 5, 2]
    arrival = [0, 2, 40, 41]
    s = Sched(max_slots=4)
    st, per, batch, c = s.run([8, 8, 8, 8], stop, arrival)
    assert st == 0
    check_invariants(per, stop, arrival, 4, 4)
    assert per[2][0][0] == 40                          # idle iterations are skipped, not spun
    assert c["iterations"] < 50
    s.close()


def test_kv_pool_bounds_admission():
    """Each request needs 4 of the 8 blocks: at most two in flight even with four slots."""
    stop = [10] * 6
    s = Sched(max_slots=4, max_ctx=64, kv_blocks=8)
    st, per, batch, c = s.run([55] * 6, stop, max_active=4)   # 55 + 10 - 1 = 64 positions = 4 blocks
    assert st == 0
    assert max(batch) == 2
    check_invariants(per, stop, [0] * 6, 2, 4)
    s.close()


def test_rejects_what_can_never_run():
    s = Sched(max_slots=2, max_ctx=64, kv_blocks=2)
    st, *_ = s.run([60], [10])                          # 69 positions > max_ctx
    assert st == binding.SPR_ERR_INVALID_ARG
    st, *_ = s.run([40], [1])                           # 3 blocks > pool of 2
    assert st == binding.SPR_ERR_INVALID_ARG
    st, *_ = s.run([4], [2], max_active=3)              # max_active > slots
    assert st == binding.SPR_ERR_INVALID_ARG
    s.close()


def test_needs_an_idle_model():
    s = Sched(max_slots=2)
    one = np.ones(1, dtype=np.int32)
    r = np.zeros(1, dtype=np.int32)
    p = lambda x: x.ctypes.data_as(I32)
    assert s.L.sprh_prefill(s.h, 1, p(np.zeros(1, dtype=np.int32)), p(one * 3), p(one * 4), p(r)) == 0
    st, *_ = s.run([4], [2])
    assert st == binding.SPR_ERR_STATE
    s.close()


def test_eos_retires_one_iteration_late():
    """Generation ends at EOS or at the limit (Section II-A).  The device reports EOS one iteration
    late, so a request runs at most one more decode row (two if EOS was the prefill's token, whose
    iteration already decoded), its length ends at the first EOS, and its slot is reused no earlier
    than two iterations after the EOS iteration."""
    stop = [12, 12, 12, 12, 12, 5]
    eos = [(0, 3), (1, 0), (2, 11), (3, 6), (3, 8)]          # request 3: only the first EOS counts
    s = Sched(max_slots=2)
    st, per, batch, c = s.run([9] * 6, stop, max_active=2, eos=eos)
    assert st == 0
    assert s.lengths == [4, 1, 12, 7, 12, 5]
    for r, k in [(0, 3), (1, 0), (3, 6)]:
        its, slots, _ = per[r]
        produced = int((its >= 0).sum())
        extra = produced - (k + 1)
        assert 0 <= extra <= (2 if k == 0 else 1), (r, produced)
        t_eos = its[k]
        later = [q for q in range(len(stop)) if q > r and per[q][1][0] == slots[0] and per[q][0][0] > t_eos]
        assert all(per[q][0][0] >= t_eos + 2 for q in later), r
    assert s.L.sprh_free_blocks(s.h) == s.cfg.kv_blocks
    s.close()


def test_eos_on_the_last_token_changes_nothing():
    stop = [4, 6]
    s = Sched(max_slots=2)
    st, per, batch, c = s.run([5, 5], stop, eos=[(0, 3), (1, 5)])
    assert st == 0 and s.lengths == [4, 6]
    assert batch == [len(a) for a in R.active_schedule(stop)]
    s.close()
