"""Thin ctypes binding of the C ABI in include/sprout.h.

Argument marshalling only: every step of the decode runs in the HIP library.
PyTorch provides the device workspace and the stream.  Importing this module
raises if libsprout.so has not been built; there is no other code path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

from .configs import ModelConfig

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libsprout.so")

SPR_OK, SPR_ERR_INVALID_ARG, SPR_ERR_WORKSPACE, SPR_ERR_KV_FULL, SPR_ERR_STATE, SPR_ERR_HIP = 0, -1, -2, -3, -4, -5
SPR_ERR_DEVICE_CHECK = -6
SPR_F32, SPR_BF16 = 0, 1
KV_BLOCK = 16
TENSOR_IDS = {"embed": 0, "wq": 1, "wk": 2, "wv": 3, "wo": 4, "w1": 5, "w3": 6, "w2": 7, "lm_head": 8}


class SprConfig(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("d_ff", ctypes.c_int32),
                ("vocab", ctypes.c_int32), ("rope_base", ctypes.c_float), ("rms_eps", ctypes.c_float),
                ("dtype", ctypes.c_int32), ("kv_block", ctypes.c_int32), ("max_slots", ctypes.c_int32),
                ("max_ctx", ctypes.c_int32), ("kv_blocks", ctypes.c_int32), ("kv_dtype", ctypes.c_int32)]


class SproutError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"sprout status {status}: {msg}")
        self.status = status


_I32P = ctypes.POINTER(ctypes.c_int32)
_lib = None


MAX_LEVELS = 8  # SPR_MAX_LEVELS


class SprRequest(ctypes.Structure):
    _fields_ = [("tokens", _I32P), ("n_tokens", ctypes.c_int32), ("stop_len", ctypes.c_int32),
                ("arrival", ctypes.c_int32), ("level", ctypes.c_int32)]


class SprServeStats(ctypes.Structure):
    _fields_ = [("iterations", ctypes.c_int64), ("decode_steps", ctypes.c_int64), ("prefill_calls", ctypes.c_int64),
                ("decode_tokens", ctypes.c_int64), ("max_batch", ctypes.c_int32), ("mean_batch", ctypes.c_double),
                ("device_seconds", ctypes.c_double), ("level_requests", ctypes.c_int32 * MAX_LEVELS),
                ("level_tokens", ctypes.c_double * MAX_LEVELS), ("level_seconds", ctypes.c_double * MAX_LEVELS)]


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with `python -m paper_2403_12900_amd.build` "
                          "or __graft_entry__.build()")
    # torch carries its own HIP runtime.  The library must bind to that one (it is handed torch's
    # streams and device memory): loaded first, it would bring in the system runtime beside
    # torch's, and that second runtime finds no device once torch's holds it.
    import torch  # noqa: F401
    L = ctypes.CDLL(path)
    vp = ctypes.c_void_p
    L.spr_workspace_bytes.restype = ctypes.c_size_t
    L.spr_workspace_bytes.argtypes = [ctypes.POINTER(SprConfig)]
    L.spr_init.restype = ctypes.c_int
    L.spr_init.argtypes = [ctypes.POINTER(SprConfig), ctypes.c_uint64, vp, ctypes.c_size_t, vp, ctypes.POINTER(vp)]
    L.spr_prefill.restype = ctypes.c_int
    L.spr_prefill.argtypes = [vp, ctypes.c_int32, _I32P, _I32P, _I32P, _I32P, vp, vp, _I32P]
    L.spr_decode_step.restype = ctypes.c_int
    L.spr_decode_step.argtypes = [vp, ctypes.c_int32, _I32P, _I32P, vp, vp, _I32P]
    L.spr_decode_step_static_scratch.restype = ctypes.c_int
    L.spr_decode_step_static_scratch.argtypes = [vp, ctypes.c_int32, _I32P, _I32P, vp, vp, _I32P]
    L.spr_rewind_slot.restype = ctypes.c_int
    L.spr_rewind_slot.argtypes = [vp, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32]
    L.spr_free_slot.restype = ctypes.c_int
    L.spr_free_slot.argtypes = [vp, ctypes.c_int32]
    L.spr_slot_info.restype = ctypes.c_int
    L.spr_slot_info.argtypes = [vp, ctypes.c_int32, _I32P, _I32P, _I32P]
    L.spr_free_blocks.restype = ctypes.c_int32
    L.spr_free_blocks.argtypes = [vp]
    L.spr_export_weight_rows.restype = ctypes.c_int
    L.spr_export_weight_rows.argtypes = [vp, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, vp]
    L.spr_time_projection.restype = ctypes.c_int
    L.spr_time_projection.argtypes = [vp, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                      ctypes.POINTER(ctypes.c_float)]
    L.spr_test_write_lm_head_row.restype = ctypes.c_int
    L.spr_test_write_lm_head_row.argtypes = [vp, ctypes.c_int32, ctypes.c_int32, ctypes.c_float]
    L.spr_time_read_ceiling.restype = ctypes.c_int
    L.spr_time_read_ceiling.argtypes = [vp, ctypes.c_int32, ctypes.POINTER(ctypes.c_double),
                                        ctypes.POINTER(ctypes.c_uint64)]
    L.spr_serve.restype = ctypes.c_int
    L.spr_serve.argtypes = [vp, ctypes.c_int32, ctypes.POINTER(SprRequest), ctypes.c_int32, ctypes.c_int32, vp, vp,
                            _I32P, ctypes.POINTER(SprServeStats)]
    L.spr_release.restype = ctypes.c_int
    L.spr_release.argtypes = [vp]
    L.spr_last_error.restype = ctypes.c_char_p
    L.spr_last_error.argtypes = []
    _lib = L
    return L


def make_config(m: ModelConfig, max_slots: int, max_ctx: int, kv_blocks: int) -> SprConfig:
    return SprConfig(m.n_layers, m.d_model, m.n_heads, m.n_kv_heads, m.head_dim, m.d_ff, m.vocab,
                     m.rope_base, m.rms_eps, SPR_BF16 if m.bf16 else SPR_F32, KV_BLOCK, max_slots, max_ctx,
                     kv_blocks, SPR_BF16 if m.kv_is_bf16 else SPR_F32)


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(_I32P)


def _check(status: int):
    if status != SPR_OK:
        raise SproutError(status, load_library().spr_last_error().decode())


def workspace_bytes(cfg: SprConfig) -> int:
    return int(load_library().spr_workspace_bytes(ctypes.byref(cfg)))


class DecodeModel:
    """One model instance on one device, in a caller-owned torch workspace."""

    def __init__(self, model: ModelConfig, seed: int, max_slots: int, max_ctx: int,
                 kv_blocks: Optional[int] = None, device: int = 0):
        import torch
        self.torch = torch
        self.lib = load_library()
        self.model = model
        if kv_blocks is None:
            kv_blocks = max_slots * ((max_ctx + KV_BLOCK - 1) // KV_BLOCK)
        self.cfg = make_config(model, max_slots, max_ctx, kv_blocks)
        nbytes = workspace_bytes(self.cfg)
        if nbytes == 0:
            raise SproutError(SPR_ERR_INVALID_ARG, "invalid model configuration")
        self.device = torch.device("cuda", device)
        self.ws = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        self.stream = torch.cuda.current_stream(self.device)
        h = ctypes.c_void_p()
        _check(self.lib.spr_init(ctypes.byref(self.cfg), ctypes.c_uint64(seed), ctypes.c_void_p(self.ws.data_ptr()),
                                 nbytes, ctypes.c_void_p(self.stream.cuda_stream), ctypes.byref(h)))
        self.h = h
        self.max_slots = max_slots
        self.vocab = model.vocab

    def new_token_buffer(self):
        return self.torch.zeros(self.max_slots, dtype=self.torch.int32, device=self.device)

    def prefill(self, slots: Sequence[int], prompts: Sequence[Sequence[int]], stop_lens: Sequence[int], tok,
                want_logits: bool = False):
        n = len(slots)
        sl = _i32(slots)
        seq = _i32([len(p) for p in prompts])
        toks = _i32(np.concatenate([np.asarray(p, dtype=np.int32) for p in prompts]) if n else [])
        stops = _i32(stop_lens)
        retired = np.zeros(n, dtype=np.int32)
        logits = self.torch.empty((n, self.vocab), dtype=self.torch.float32, device=self.device) if want_logits else None
        _check(self.lib.spr_prefill(self.h, n, _ptr(sl), _ptr(toks), _ptr(seq), _ptr(stops),
                                    ctypes.c_void_p(tok.data_ptr()),
                                    ctypes.c_void_p(logits.data_ptr() if logits is not None else 0), _ptr(retired)))
        return logits, retired

    def decode_step(self, slots: Sequence[int], lens: Sequence[int], tok, want_logits: bool = False, logits=None):
        n = len(slots)
        sl = _i32(slots)
        ln = _i32(lens)
        retired = np.zeros(n, dtype=np.int32)
        if want_logits and logits is None:
            logits = self.torch.empty((n, self.vocab), dtype=self.torch.float32, device=self.device)
        _check(self.lib.spr_decode_step(self.h, n, _ptr(sl), _ptr(ln), ctypes.c_void_p(tok.data_ptr()),
                                        ctypes.c_void_p(logits.data_ptr() if want_logits else 0), _ptr(retired)))
        return (logits if want_logits else None), retired

    def decode_step_static_scratch(self, slots: Sequence[int], lens: Sequence[int], tok, want_logits: bool = False):
        """decode_step whose scratch is the library's static device array (spr_decode_step_static_scratch)."""
        n = len(slots)
        sl = _i32(slots)
        ln = _i32(lens)
        retired = np.zeros(n, dtype=np.int32)
        logits = self.torch.empty((n, self.vocab), dtype=self.torch.float32, device=self.device) if want_logits else None
        _check(self.lib.spr_decode_step_static_scratch(self.h, n, _ptr(sl), _ptr(ln), ctypes.c_void_p(tok.data_ptr()),
                                                       ctypes.c_void_p(logits.data_ptr() if want_logits else 0),
                                                       _ptr(retired)))
        return logits, retired

    def rewind(self, slot: int, length: int, produced: int):
        _check(self.lib.spr_rewind_slot(self.h, slot, length, produced))

    def free_slot(self, slot: int):
        _check(self.lib.spr_free_slot(self.h, slot))

    def slot_info(self, slot: int):
        a, b, c = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
        _check(self.lib.spr_slot_info(self.h, slot, ctypes.byref(a), ctypes.byref(b), ctypes.byref(c)))
        return a.value, b.value, c.value

    def free_blocks(self) -> int:
        return int(self.lib.spr_free_blocks(self.h))

    def export_weight_rows(self, tensor: str, layer: int, row0: int, nrows: int, cols: int):
        out = self.torch.empty((nrows, cols), dtype=self.torch.float32, device=self.device)
        _check(self.lib.spr_export_weight_rows(self.h, TENSOR_IDS[tensor], layer, row0, nrows,
                                               ctypes.c_void_p(out.data_ptr())))
        return out

    PROJECTIONS = {"o": 1, "gate_up": 2, "down": 3, "lm_head": 4}

    def time_projection(self, projection: str, n_rows: int, reps: int) -> float:
        """Mean launch duration (us) of one projection kernel, timed with HIP events on the model's stream."""
        out = ctypes.c_float()
        _check(self.lib.spr_time_projection(self.h, self.PROJECTIONS[projection], n_rows, reps, ctypes.byref(out)))
        return float(out.value)

    def test_write_lm_head_row(self, dst: int, src: int = -1, fill: float = 0.0):
        """Test aid: LM-head row dst := row src (src >= 0) or the constant fill (see spr_test_write_lm_head_row)."""
        _check(self.lib.spr_test_write_lm_head_row(self.h, dst, src, fill))

    def read_ceiling(self, reps: int = 5):
        """(GB/s, bytes per pass): plain streaming read of every weight matrix, timed on the model's stream."""
        gbps, nbytes = ctypes.c_double(), ctypes.c_uint64()
        _check(self.lib.spr_time_read_ceiling(self.h, reps, ctypes.byref(gbps), ctypes.byref(nbytes)))
        return float(gbps.value), int(nbytes.value)

    def serve(self, prompts: Sequence[Sequence[int]], stop_lens: Sequence[int], max_active: int,
              arrivals: Optional[Sequence[int]] = None, levels: Optional[Sequence[int]] = None, eos_id: int = -1):
        """Continuous batching of all requests (spr_serve).

        Returns (tokens per request, each cut to its length; stats dict with
        per-level lists for the level_* entries)."""
        n = len(prompts)
        arrivals = [0] * n if arrivals is None else list(arrivals)
        levels = [0] * n if levels is None else list(levels)
        keep = [_i32(p) for p in prompts]
        reqs = (SprRequest * max(n, 1))()
        for i in range(n):
            reqs[i] = SprRequest(_ptr(keep[i]), len(keep[i]), int(stop_lens[i]), int(arrivals[i]), int(levels[i]))
        total = int(sum(stop_lens))
        out = self.torch.full((max(total, 1),), -1, dtype=self.torch.int32, device=self.device)
        tok = self.new_token_buffer()
        lengths = np.zeros(max(n, 1), dtype=np.int32)
        st = SprServeStats()
        _check(self.lib.spr_serve(self.h, n, reqs, max_active, int(eos_id), ctypes.c_void_p(tok.data_ptr()),
                                  ctypes.c_void_p(out.data_ptr()), _ptr(lengths), ctypes.byref(st)))
        flat = out.cpu().numpy()
        off = np.concatenate([[0], np.cumsum(np.asarray(stop_lens, dtype=np.int64))]).astype(int)
        toks = [flat[off[i]:off[i] + lengths[i]].copy() for i in range(n)]
        stats = {}
        for f, _ in SprServeStats._fields_:
            v = getattr(st, f)
            stats[f] = list(v) if f.startswith("level_") else v
        return toks, stats

    def close(self):
        if getattr(self, "h", None) is not None and self.h.value:
            self.lib.spr_release(self.h)
            self.h = ctypes.c_void_p()
        self.ws = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
