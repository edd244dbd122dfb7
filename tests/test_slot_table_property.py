"""Random call sequences against the host slot table and KV-block pool (no GPU).

Every entry point validates against the host slot table before any device
work, and the table alone decides KV-block reservation and retirement.  A
plain Python model of the documented rules predicts each call's outcome; after
every call of a random sequence (valid calls mixed with invalid ones) the
library's slots, free-block count and block rows must match it:

* a rejected call changes nothing;
* a request reserves ceil((seq_len + stop_len - 1) / 16) blocks at prefill and
  keeps them until freed; no block is held twice;
* decode advances each listed slot by one position and retires it when it
  has produced its stop length; rewind keeps the prompt and sets the count.
"""
import numpy as np
from hypothesis import given, settings
from hypothesis import strategies as st

from tests.test_abi_host import Host

FREE, ACTIVE, FINISHED = 0, 1, 2
S, MAX_CTX, KV_BLOCKS = 4, 64, 10


def blocks_for(seq, stop):
    return (seq + stop - 1 + 15) // 16


class Model:
    def __init__(self):
        self.slots = [None] * S     # None or dict(len, produced, stop, need)

    def free_blocks(self):
        return KV_BLOCKS - sum(s["need"] for s in self.slots if s is not None)

    def state(self, i):
        s = self.slots[i]
        if s is None:
            return FREE
        return FINISHED if s["produced"] >= s["stop"] else ACTIVE


def check(h: Host, m: Model):
    held = []
    for i in range(S):
        length, produced, stop, state = h.slot(i)
        assert state == m.state(i), (i, h.slot(i))
        s = m.slots[i]
        if s is None:
            continue
        assert (length, produced, stop) == (s["len"], s["produced"], s["stop"]), (i, h.slot(i), s)
        held += h.row(i)[:s["need"]].tolist()
    assert h.free_blocks() == m.free_blocks()
    assert len(set(held)) == len(held) and all(0 <= b < KV_BLOCKS for b in held), held


def step(h: Host, m: Model, rng):
    op = rng.choice(["prefill", "decode", "rewind", "free"], p=[0.3, 0.4, 0.15, 0.15])
    if op == "prefill":
        n = int(rng.integers(1, 4))
        slots = [int(x) for x in rng.integers(0, S, size=n)]
        seq = [int(x) for x in rng.integers(0, 50, size=n)]
        stop = [int(x) for x in rng.integers(0, 30, size=n)]
        valid = (len(set(slots)) == n and all(m.state(s) == FREE for s in slots)
                 and all(q >= 1 and t >= 1 and q + t - 1 <= MAX_CTX for q, t in zip(seq, stop))
                 and sum(blocks_for(q, t) for q, t in zip(seq, stop)) <= m.free_blocks())
        st_, retired = h.prefill(slots, seq, stop)
        assert (st_ == 0) == valid, (op, slots, seq, stop, st_)
        if valid:
            for s, q, t in zip(slots, seq, stop):
                m.slots[s] = {"len": q, "produced": 1, "stop": t, "need": blocks_for(q, t)}
            assert retired.tolist() == [int(t == 1) for t in stop]
    elif op == "decode":
        active = [i for i in range(S) if m.state(i) == ACTIVE]
        pool = active if active and rng.random() < 0.8 else list(range(S))
        n = int(rng.integers(1, len(pool) + 1))
        slots = [int(x) for x in rng.choice(pool, size=n, replace=bool(rng.random() < 0.1))]   # duplicates now and then
        lens = [m.slots[s]["len"] if m.slots[s] is not None else 0 for s in slots]
        if rng.random() < 0.1:
            lens[0] += 1
        valid = (len(set(slots)) == n and all(m.state(s) == ACTIVE for s in slots)
                 and all(m.slots[s]["len"] == l for s, l in zip(slots, lens)))
        st_, retired = h.decode(slots, lens)
        assert (st_ == 0) == valid, (op, slots, lens, st_)
        if valid:
            for k, s in enumerate(slots):
                m.slots[s]["len"] += 1
                m.slots[s]["produced"] += 1
                assert retired[k] == int(m.slots[s]["produced"] == m.slots[s]["stop"])
    elif op == "rewind":
        s = int(rng.integers(0, S))
        cur = m.slots[s]
        prompt = cur["len"] - cur["produced"] + 1 if cur is not None else 1
        produced = int(rng.integers(0, (cur["produced"] if cur is not None else 1) + 2))
        length = prompt + produced - 1 + (1 if rng.random() < 0.2 else 0)
        valid = cur is not None and 1 <= produced <= cur["produced"] and length == prompt + produced - 1
        st_ = h.L.sprh_rewind(h.h, s, length, produced)
        assert (st_ == 0) == valid, (op, s, length, produced, st_)
        if valid:
            cur["len"], cur["produced"] = length, produced
    else:
        s = int(rng.integers(0, S))
        valid = m.slots[s] is not None
        st_ = h.L.sprh_free(h.h, s)
        assert (st_ == 0) == valid, (op, s, st_)
        if valid:
            m.slots[s] = None


@settings(max_examples=150, deadline=None)
@given(st.integers(0, 2**32 - 1))
def test_random_call_sequences_match_the_model(seed):
    rng = np.random.default_rng(seed)
    h = Host(max_slots=S, max_ctx=MAX_CTX, kv_blocks=KV_BLOCKS)
    m = Model()
    for _ in range(60):
        step(h, m, rng)
        check(h, m)
    h.L.sprh_delete(h.h)
