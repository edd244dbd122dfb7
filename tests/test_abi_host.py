"""C ABI surface and host-side bookkeeping (no GPU needed).

The device library must load and export every entry point the header
declares.  The slot / KV-block bookkeeping that validates every call before
any work is enqueued is exercised through the host-only test library built
from the same source file (csrc/host_state.cpp).
"""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2403_12900_amd import binding
from paper_2403_12900_amd.configs import CONFIGS, LLAMA2_7B, TINY

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sprout.h")
# SPROUT_HOST_LIB selects another build of the same sources (the sanitizer build).
HOST_LIB = os.environ.get("SPROUT_HOST_LIB", os.path.join(ROOT, "paper_2403_12900_amd", "libsprout_host.so"))


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(spr_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = binding.load_library()
    names = declared_functions()
    assert "spr_decode_step" in names and "spr_prefill" in names and "spr_init" in names
    for n in names:
        assert hasattr(lib, n), n


def test_library_shares_torchs_hip_runtime():
    """One HIP runtime in the process: the library binds to the one torch brings, whose streams and
    device memory it is handed.  A second copy (the library loaded before torch) found no device."""
    binding.load_library()
    maps = open("/proc/self/maps").read().splitlines()
    hip = {line.split()[-1] for line in maps if "libamdhip64" in line and "/" in line}
    assert len(hip) == 1, hip


def test_workspace_bytes_and_invalid_configs():
    cfg = binding.make_config(LLAMA2_7B, 32, 2048, 32 * 128)
    n = binding.workspace_bytes(cfg)
    # Weights alone are 6.74e9 bf16 elements.
    assert n > 2 * LLAMA2_7B.weight_elements_per_step()
    bad = binding.make_config(LLAMA2_7B, 32, 2048, 32 * 128)
    bad.head_dim = 96
    assert binding.workspace_bytes(bad) == 0
    bad = binding.make_config(LLAMA2_7B, 65, 2048, 32 * 128)
    assert binding.workspace_bytes(bad) == 0
    bad = binding.make_config(TINY, 4, 64, 16)
    bad.kv_block = 32
    assert binding.workspace_bytes(bad) == 0


def test_init_rejects_bad_workspace_without_touching_the_device():
    lib = binding.load_library()
    cfg = binding.make_config(TINY, 4, 64, 16)
    h = ctypes.c_void_p()
    st = lib.spr_init(ctypes.byref(cfg), 1, None, 0, None, ctypes.byref(h))
    assert st == binding.SPR_ERR_WORKSPACE and not h.value
    st = lib.spr_init(ctypes.byref(cfg), 1, ctypes.c_void_p(4096 + 8), 1 << 30, None, ctypes.byref(h))
    assert st == binding.SPR_ERR_WORKSPACE  # misaligned
    st = lib.spr_init(ctypes.byref(cfg), 1, ctypes.c_void_p(4096), 16, None, ctypes.byref(h))
    assert st == binding.SPR_ERR_WORKSPACE  # too small
    assert b"needed" in lib.spr_last_error()


# ------------------------------------------------------------- bookkeeping

class Host:
    def __init__(self, max_slots=4, max_ctx=64, kv_blocks=8):
        L = ctypes.CDLL(HOST_LIB)
        I = ctypes.POINTER(ctypes.c_int32)
        L.sprh_new.restype = ctypes.c_void_p
        L.sprh_new.argtypes = [ctypes.POINTER(binding.SprConfig)]
        L.sprh_delete.argtypes = [ctypes.c_void_p]
        L.sprh_prefill.argtypes = [ctypes.c_void_p, ctypes.c_int, I, I, I, I]
        L.sprh_decode.argtypes = [ctypes.c_void_p, ctypes.c_int, I, I, I]
        L.sprh_rewind.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_int]
        L.sprh_free.argtypes = [ctypes.c_void_p, ctypes.c_int]
        L.sprh_free_blocks.argtypes = [ctypes.c_void_p]
        L.sprh_slot.argtypes = [ctypes.c_void_p, ctypes.c_int, I, I, I, I]
        L.sprh_block_row.argtypes = [ctypes.c_void_p, ctypes.c_int, I]
        L.sprh_last_error.restype = ctypes.c_char_p
        self.L = L
        self.cfg = binding.make_config(TINY, max_slots, max_ctx, kv_blocks)
        self.h = L.sprh_new(ctypes.byref(self.cfg))
        assert self.h

    @staticmethod
    def a(x):
        return np.ascontiguousarray(np.asarray(x, dtype=np.int32))

    def p(self, x):
        return x.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))

    def prefill(self, slots, seq, stop):
        s, q, t = self.a(slots), self.a(seq), self.a(stop)
        r = np.zeros(len(slots), dtype=np.int32)
        st = self.L.sprh_prefill(self.h, len(slots), self.p(s), self.p(q), self.p(t), self.p(r))
        return st, r

    def decode(self, slots, lens):
        s, l = self.a(slots), self.a(lens)
        r = np.zeros(len(slots), dtype=np.int32)
        st = self.L.sprh_decode(self.h, len(slots), self.p(s), self.p(l), self.p(r))
        return st, r

    def slot(self, s):
        v = [ctypes.c_int32() for _ in range(4)]
        self.L.sprh_slot(self.h, s, *[ctypes.byref(x) for x in v])
        return tuple(x.value for x in v)

    def row(self, s):
        mb = (self.cfg.max_ctx + 15) // 16
        out = np.zeros(mb, dtype=np.int32)
        self.L.sprh_block_row(self.h, s, self.p(out))
        return out

    def free_blocks(self):
        return self.L.sprh_free_blocks(self.h)


def test_prefill_reserves_blocks_for_prompt_and_generation():
    h = Host(max_slots=4, max_ctx=64, kv_blocks=8)
    st, r = h.prefill([2, 0], [20, 5], [13, 1])
    assert st == 0
    # slot 2: 20 + 13 - 1 = 32 positions -> 2 blocks; slot 0: 5 positions -> 1 block.
    assert h.free_blocks() == 5
    assert r.tolist() == [0, 1]                # stop_len 1: done at prefill
    assert h.slot(2) == (20, 1, 13, 1)          # len, produced, stop, state=active
    assert h.slot(0)[3] == 2                    # finished
    assert h.row(2)[:2].tolist() == [0, 1]      # blocks handed out from the bottom of the pool


def test_validation_changes_no_state():
    h = Host(max_slots=4, max_ctx=64, kv_blocks=4)
    assert h.prefill([0], [10], [7])[0] == 0
    before = (h.free_blocks(), h.slot(0))
    assert h.prefill([0], [4], [2])[0] == binding.SPR_ERR_STATE            # slot busy
    assert h.prefill([1, 1], [4, 4], [2, 2])[0] == binding.SPR_ERR_INVALID_ARG  # duplicate
    assert h.prefill([5], [4], [2])[0] == binding.SPR_ERR_INVALID_ARG       # out of range
    assert h.prefill([1], [60], [10])[0] == binding.SPR_ERR_INVALID_ARG     # exceeds max_ctx
    assert h.prefill([1], [0], [10])[0] == binding.SPR_ERR_INVALID_ARG      # empty prompt
    assert h.prefill([1], [4], [0])[0] == binding.SPR_ERR_INVALID_ARG       # stop_len < 1
    assert h.prefill([1, 2], [40, 40], [1, 1])[0] == binding.SPR_ERR_KV_FULL  # 3 + 3 blocks > 3 free
    assert h.decode([0], [11])[0] == binding.SPR_ERR_STATE                   # wrong length
    assert h.decode([1], [0])[0] == binding.SPR_ERR_STATE                    # free slot
    assert h.decode([0, 0], [10, 10])[0] == binding.SPR_ERR_INVALID_ARG
    assert (h.free_blocks(), h.slot(0)) == before


def test_decode_retires_at_stop_length_closed_form():
    """Request i emits g_0 at prefill and retires at decode step L_i - 1."""
    stops = [5, 1, 3, 8]
    seqs = [7, 3, 16, 1]
    h = Host(max_slots=4, max_ctx=64, kv_blocks=16)
    st, r = h.prefill([0, 1, 2, 3], seqs, stops)
    assert st == 0 and r.tolist() == [0, 1, 0, 0]
    lens = list(seqs)
    active = [i for i in range(4) if stops[i] > 1]
    step = 0
    while active:
        step += 1
        st, r = h.decode(active, [lens[i] for i in active])
        assert st == 0
        for k, i in enumerate(active):
            lens[i] += 1
            assert r[k] == (1 if step == stops[i] - 1 else 0)
        active = [i for k, i in enumerate(active) if not r[k]]
        assert active == [i for i in range(4) if stops[i] > step + 1]
    assert step == max(stops) - 1
    assert [h.slot(i)[0] for i in range(4)] == [seqs[i] + stops[i] - 1 for i in range(4)]
    assert h.decode([0], [lens[0]])[0] == binding.SPR_ERR_STATE              # finished


def test_rewind_and_free():
    h = Host(max_slots=2, max_ctx=64, kv_blocks=8)
    assert h.prefill([1], [10], [4])[0] == 0
    for L in (10, 11, 12):
        assert h.decode([1], [L])[0] == 0
    assert h.slot(1) == (13, 4, 4, 2)
    assert h.L.sprh_rewind(h.h, 1, 12, 2) == binding.SPR_ERR_INVALID_ARG     # inconsistent
    assert h.L.sprh_rewind(h.h, 1, 10, 1) == 0
    assert h.slot(1) == (10, 1, 4, 1)
    assert h.decode([1], [10])[0] == 0
    free = h.free_blocks()
    assert h.L.sprh_free(h.h, 1) == 0
    assert h.free_blocks() == free + 1
    assert h.L.sprh_free(h.h, 1) == binding.SPR_ERR_STATE
    assert h.prefill([1], [30], [3])[0] == 0                               # blocks reused


def test_all_configs_fit_one_gpu():
    """Every decode configuration's workspace fits in the 288 GB of one MI355X."""
    from paper_2403_12900_amd.workload import make_workload
    for k, c in CONFIGS.items():
        w = make_workload(c)
        max_ctx = int(np.max(w.seq_lens + w.stop_lens - 1))
        blocks = int(np.sum((w.seq_lens + w.stop_lens - 1 + 15) // 16))
        n = binding.workspace_bytes(binding.make_config(c.model, w.batch, max_ctx, blocks))
        assert 0 < n < 250e9, (k, n)
