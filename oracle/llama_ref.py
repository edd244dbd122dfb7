"""Plain fp64 CPU oracle of the Llama-2 greedy decode that Sprout serves.

TEST INFRASTRUCTURE ONLY.  Only tests/, __graft_entry__.smoke() and bench.py's
cpu_baseline leg may import or call this module.

What the method computes (cited by section of arXiv 2403.12900):
  * Section II-A ("Generative language model inference", Fig. 2): the model
    takes a prompt and predicts the next token again and again until an EOS
    token or a preset limit; keys and values of earlier tokens are kept in a
    KV cache and are reused, never recomputed.  Token generation, not the
    prompt prefill, dominates the cost.
  * Definition 1 and Section III-E ("Applying generation directive levels"): a
    directive level is a fixed text sequence that is placed as a system prompt
    *before* the user prompt (and before any system prompt it already has), so
    the directive tokens occupy the first positions and live in the KV cache
    like any other prompt token (Section II-B, Takeaway 2).
  * Section IV (Methodology): the served model is Llama 2; directive levels are
    L0 (none), L1 ("brief") and L2 ("very brief").

The paper gives no architecture detail beyond "Llama2".  The readings taken
here (pre-norm decoder, RMSNorm with eps 1e-5 and unit gains, RoPE on
interleaved adjacent pairs with base 10000, causal softmax attention with
grouped KV heads g(h) = floor(h / (H / Hkv)), SwiGLU MLP with W1 = gate,
W3 = up, W2 = down, no biases, untied embedding and LM head, greedy argmax with
the lowest index winning ties, retirement by per-request stop length) are the
published Llama-2 architecture, restated here in plain numpy.

Everything is fp64.  Weights are the exact fp32 / bf16 values drawn by the
counter-based generator in wgen.c, widened to fp64.  The KV cache is model
state kept in the model's KV-cache format: a key or value is rounded to bf16
or fp32, nearest-even, when it is cached, and attention reads the cached
values.  Nothing else is rounded.

Two forms of the same computation are provided:
  * ``forward_causal``  -- one causal pass over a whole token sequence, giving
    the logits at every position (the full-recompute definition);
  * ``KVCacheDecoder``  -- the paper's incremental loop: prefill fills the
    cache, every decode step feeds one token per active request and attends
    to the cached keys/values.
Their agreement (incremental == recompute) is one of the oracle's pins.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Sequence

import numpy as np

from . import _clib

# Tensor ids of the generator (oracle/wgen.c).  Layer-free tensors use layer 0.
TENSOR_IDS = {"embed": 0, "wq": 1, "wk": 2, "wv": 3, "wo": 4, "w1": 5, "w3": 6, "w2": 7, "lm_head": 8}


@dataclasses.dataclass(frozen=True)
class Shape:
    """Llama-2-architecture model shape (Section IV names Llama 2; sizes are the model's)."""
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    d_ff: int
    vocab: int
    rope_base: float = 10000.0
    rms_eps: float = 1e-5
    bf16: bool = True
    # Cached keys/values are stored in the KV-cache format (bf16 or fp32;
    # None: the weight format), rounded to nearest-even when written.
    # kv_round False keeps them exact (fp64), which only brute-force pins use.
    kv_round: bool = True
    kv_bf16: Optional[bool] = None

    def matrix_dims(self, name: str):
        d, hd = self.d_model, self.head_dim
        return {
            "embed": (self.vocab, d),
            "wq": (self.n_heads * hd, d),
            "wk": (self.n_kv_heads * hd, d),
            "wv": (self.n_kv_heads * hd, d),
            "wo": (d, self.n_heads * hd),
            "w1": (self.d_ff, d),
            "w3": (self.d_ff, d),
            "w2": (d, self.d_ff),
            "lm_head": (self.vocab, d),
        }[name]


class Weights:
    """The model's weights, drawn by the oracle's own generator.

    ``resident=True`` keeps every matrix once drawn; otherwise each layer's
    matrices are drawn when asked for and dropped afterwards (layer streaming,
    for shapes whose fp64 weights do not fit in host memory).
    """

    LAYER_MATS = ("wq", "wk", "wv", "wo", "w1", "w3", "w2")

    def __init__(self, shape: Shape, seed: int, resident: bool = True):
        self.shape = shape
        self.seed = int(seed)
        self.resident = resident
        self._cache: Dict[tuple, np.ndarray] = {}
        self._scratch: Dict[str, np.ndarray] = {}

    def matrix(self, name: str, layer: int = 0) -> np.ndarray:
        """The matrix (fp64).  Without residency, a matrix stays valid only until
        the same matrix of another layer is asked for (its buffer is reused)."""
        key = (name, layer)
        if key in self._cache:
            return self._cache[key]
        rows, cols = self.shape.matrix_dims(name)
        out = None if self.resident else self._scratch.get(name)
        m = _clib.wgen_rows(self.seed, TENSOR_IDS[name], layer, cols, 0, rows, self.shape.bf16, out=out)
        if self.resident:
            self._cache[key] = m
        else:
            self._scratch[name] = m
        return m

    def rows(self, name: str, layer: int, row0: int, nrows: int) -> np.ndarray:
        _, cols = self.shape.matrix_dims(name)
        return _clib.wgen_rows(self.seed, TENSOR_IDS[name], layer, cols, row0, nrows, self.shape.bf16)

    def layer(self, layer: int) -> Dict[str, np.ndarray]:
        return {n: self.matrix(n, layer) for n in self.LAYER_MATS}

    def gain(self) -> np.ndarray:
        # All RMSNorm gains are 1 for the random-init models.
        return np.ones(self.shape.d_model)


# --------------------------------------------------------------------------
# Building blocks (Llama-2 architecture; fp64)
# --------------------------------------------------------------------------

def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * g over the last axis."""
    x = np.asarray(x, dtype=np.float64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def rope_angles(positions: Sequence[int], head_dim: int, base: float) -> np.ndarray:
    """angle[t, i] = pos_t * base^(-2i/head_dim), i < head_dim/2 (fp64)."""
    i = np.arange(head_dim // 2, dtype=np.float64)
    theta = base ** (-2.0 * i / head_dim)
    return np.asarray(positions, dtype=np.float64)[:, None] * theta[None, :]


def apply_rope(x: np.ndarray, positions: Sequence[int], base: float) -> np.ndarray:
    """Rotates each adjacent pair (2i, 2i+1) of every head vector by pos * theta_i.

    x: [T, n_heads, head_dim]; positions: [T].
    """
    T, nh, hd = x.shape
    ang = rope_angles(positions, hd, base)            # [T, hd/2]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    even = x[..., 0::2]
    odd = x[..., 1::2]
    out = np.empty_like(x, dtype=np.float64)
    out[..., 0::2] = even * c - odd * s
    out[..., 1::2] = even * s + odd * c
    return out


def round_to_storage(x: np.ndarray, bf16: bool) -> np.ndarray:
    """Value of x once stored as fp32, or as bf16 (via fp32), round-to-nearest-even at each step."""
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    if bf16:
        u = f.view(np.uint32).astype(np.uint64)
        u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
        f = u.astype(np.uint32).view(np.float32)
    return f.astype(np.float64)


def cache_kv(shape: Shape, k: np.ndarray, v: np.ndarray):
    """Keys/values as the KV cache holds them (the model's storage format)."""
    if not shape.kv_round:
        return k, v
    kv_bf16 = shape.bf16 if shape.kv_bf16 is None else shape.kv_bf16
    return round_to_storage(k, kv_bf16), round_to_storage(v, kv_bf16)


def softmax(s: np.ndarray) -> np.ndarray:
    """Softmax over the last axis, with the row max subtracted first."""
    m = np.max(s, axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=-1, keepdims=True)


def kv_head_of(h: int, n_heads: int, n_kv_heads: int) -> int:
    """Grouped-query map: consecutive query heads share one KV head."""
    return h // (n_heads // n_kv_heads)


def attend(q: np.ndarray, K: np.ndarray, V: np.ndarray) -> np.ndarray:
    """One query position against cached keys/values.

    q: [H, hd]; K, V: [ctx, Hkv, hd] -> [H, hd].
    """
    H, hd = q.shape
    Hkv = K.shape[1]
    out = np.empty((H, hd))
    for h in range(H):
        g = kv_head_of(h, H, Hkv)
        scores = K[:, g, :] @ q[h] / math.sqrt(hd)   # [ctx]
        p = softmax(scores)
        out[h] = p @ V[:, g, :]
    return out


def causal_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray) -> np.ndarray:
    """Position t attends to positions 0..t: softmax(q k^T / sqrt(hd) + causal mask) v, per head.

    q: [T,H,hd], k,v: [T,Hkv,hd] -> [T,H,hd].  Query head h uses KV head
    h // (H / Hkv), i.e. each KV head is repeated for its group of query heads.
    """
    T, H, hd = q.shape
    group = H // k.shape[1]
    kh = np.repeat(k, group, axis=1).transpose(1, 2, 0)      # [H, hd, T]
    vh = np.repeat(v, group, axis=1).transpose(1, 0, 2)      # [H, T, hd]
    s = np.matmul(q.transpose(1, 0, 2), kh) / math.sqrt(hd)  # [H, T(query), T(key)]
    s[:, np.triu(np.ones((T, T), dtype=bool), k=1)] = -np.inf
    return np.matmul(softmax(s), vh).transpose(1, 0, 2)


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def swiglu(m: np.ndarray, w1: np.ndarray, w3: np.ndarray, w2: np.ndarray) -> np.ndarray:
    """(SiLU(m W1^T) * (m W3^T)) W2^T."""
    return (silu(m @ w1.T) * (m @ w3.T)) @ w2.T


def argmax_first(z: np.ndarray) -> np.ndarray:
    """Greedy token: index of the maximum logit; the lowest index wins ties."""
    return np.argmax(z, axis=-1)


# --------------------------------------------------------------------------
# Full causal recompute over one request's tokens
# --------------------------------------------------------------------------

def embed_rows(w: Weights, tokens: Sequence[int]) -> np.ndarray:
    """x_t = E[token_t] (fp64); draws only the rows asked for unless the weights are resident."""
    tokens = np.asarray(tokens, dtype=np.int64)
    if w.resident:
        return np.array(w.matrix("embed")[tokens], dtype=np.float64)
    uniq, inv = np.unique(tokens, return_inverse=True)
    rows = np.concatenate([w.rows("embed", 0, int(t), 1) for t in uniq]) if len(uniq) else np.zeros((0, w.shape.d_model))
    return rows[inv]


def forward_causal(w: Weights, tokens: Sequence[int], want_positions: Optional[Sequence[int]] = None,
                   n_layers: Optional[int] = None, progress=None) -> np.ndarray:
    """Logits [len(want_positions), V] of one request whose tokens sit at positions 0..T-1.

    Layers are processed one at a time so the weights can be streamed.
    ``n_layers`` truncates the model (used only by pins on toy shapes);
    ``progress(layer)`` is called after each layer if given.
    """
    return forward_causal_requests(w, [tokens], [want_positions], n_layers=n_layers, progress=progress)[0]


def forward_causal_requests(w: Weights, seqs: Sequence[Sequence[int]],
                            want_positions: Optional[Sequence[Optional[Sequence[int]]]] = None,
                            n_layers: Optional[int] = None, progress=None) -> List[np.ndarray]:
    """forward_causal for several independent requests: request i's tokens sit at positions
    0..len(seqs[i])-1 and it attends only to its own positions.  The row-wise steps (norms,
    projections, MLP) take all requests' rows in one product per matrix, so each layer's weights
    are drawn once for all of them; the result for a request is the same as forward_causal's.
    Returns one [len(want_positions[i]), V] array per request (all positions when None)."""
    sh = w.shape
    seqs = [np.asarray(t, dtype=np.int64) for t in seqs]
    if want_positions is None:
        want_positions = [None] * len(seqs)
    lens = [len(t) for t in seqs]
    off = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    g = w.gain()
    x = embed_rows(w, np.concatenate(seqs)) if seqs else np.zeros((0, sh.d_model))
    L = sh.n_layers if n_layers is None else n_layers
    for layer in range(L):
        W = w.layer(layer)
        a = rmsnorm(x, g, sh.rms_eps)
        q_all, k_all, v_all = a @ W["wq"].T, a @ W["wk"].T, a @ W["wv"].T
        o = np.empty((x.shape[0], sh.n_heads * sh.head_dim))
        for i, T in enumerate(lens):
            r = slice(off[i], off[i + 1])
            pos = np.arange(T)
            q = apply_rope(q_all[r].reshape(T, sh.n_heads, sh.head_dim), pos, sh.rope_base)
            k = apply_rope(k_all[r].reshape(T, sh.n_kv_heads, sh.head_dim), pos, sh.rope_base)
            k, v = cache_kv(sh, k, v_all[r].reshape(T, sh.n_kv_heads, sh.head_dim))
            o[r] = causal_attention(q, k, v).reshape(T, sh.n_heads * sh.head_dim)
        x = x + o @ W["wo"].T
        m = rmsnorm(x, g, sh.rms_eps)
        x = x + swiglu(m, W["w1"], W["w3"], W["w2"])
        del W
        if progress is not None:
            progress(layer)
    lm = w.matrix("lm_head")
    out = []
    for i, T in enumerate(lens):
        want = range(T) if want_positions[i] is None else want_positions[i]
        xs = rmsnorm(x[off[i] + np.asarray(want, dtype=np.int64)], g, sh.rms_eps)
        out.append(xs @ lm.T)
    return out


def teacher_forced_logits(w: Weights, prompt: Sequence[int], generated: Sequence[int],
                          steps: Optional[Sequence[int]] = None, progress=None) -> np.ndarray:
    """Logits that produced generated token g_s, for s in ``steps`` (default: all).

    g_0 comes from the last prompt position; g_s (s >= 1) from feeding g_{s-1}
    at position n + s - 1.  The sequence run is prompt ++ generated[:-1], so
    the oracle sees exactly the tokens the device saw.
    """
    return teacher_forced_logits_requests(w, [prompt], [generated], [steps], progress=progress)[0]


def teacher_forced_logits_requests(w: Weights, prompts: Sequence[Sequence[int]],
                                   generated: Sequence[Sequence[int]],
                                   steps: Optional[Sequence[Optional[Sequence[int]]]] = None,
                                   progress=None) -> List[np.ndarray]:
    """teacher_forced_logits for several requests in one pass over the layers."""
    if steps is None:
        steps = [None] * len(prompts)
    seqs, want = [], []
    for p, gen, st in zip(prompts, generated, steps):
        st = list(range(len(gen))) if st is None else list(st)
        n = len(p)
        seqs.append(list(p) + list(gen[:max(st)]))
        want.append([n - 1 + s for s in st])
    return forward_causal_requests(w, seqs, want, progress=progress)


# --------------------------------------------------------------------------
# The incremental loop with a KV cache (Section II-A), batched over requests
# --------------------------------------------------------------------------

class KVCacheDecoder:
    """Greedy decode of a closed batch with per-request stop lengths.

    A request with stop length L emits g_0 at prefill and g_1..g_{L-1} in
    L-1 decode steps, then retires; g_{L-1} is never fed back.  Requests are
    independent: each attends only to its own cache.
    """

    def __init__(self, w: Weights):
        self.w = w
        self.K: Dict[int, List[np.ndarray]] = {}
        self.V: Dict[int, List[np.ndarray]] = {}
        self.len: Dict[int, int] = {}

    def _alloc(self, rid: int, capacity: int):
        sh = self.w.shape
        self.K[rid] = [np.zeros((capacity, sh.n_kv_heads, sh.head_dim)) for _ in range(sh.n_layers)]
        self.V[rid] = [np.zeros((capacity, sh.n_kv_heads, sh.head_dim)) for _ in range(sh.n_layers)]
        self.len[rid] = 0

    def _layers(self, x: np.ndarray, rids: Sequence[int], positions: Sequence[int]) -> np.ndarray:
        """Runs all layers on the rows of x; row r belongs to request rids[r] at positions[r].

        Each row's keys/values are written to its request's cache before the
        attention reads the cache, so a row attends to itself and to every
        earlier position of the same request.
        """
        sh = self.w.shape
        g = self.w.gain()
        n = x.shape[0]
        for layer in range(sh.n_layers):
            W = self.w.layer(layer)
            a = rmsnorm(x, g, sh.rms_eps)
            q = (a @ W["wq"].T).reshape(n, sh.n_heads, sh.head_dim)
            k = (a @ W["wk"].T).reshape(n, sh.n_kv_heads, sh.head_dim)
            v = (a @ W["wv"].T).reshape(n, sh.n_kv_heads, sh.head_dim)
            q = apply_rope(q, positions, sh.rope_base)
            k = apply_rope(k, positions, sh.rope_base)
            k, v = cache_kv(sh, k, v)
            for r in range(n):
                self.K[rids[r]][layer][positions[r]] = k[r]
                self.V[rids[r]][layer][positions[r]] = v[r]
            o = np.empty((n, sh.n_heads, sh.head_dim))
            for r in range(n):
                ctx = positions[r] + 1
                o[r] = attend(q[r], self.K[rids[r]][layer][:ctx], self.V[rids[r]][layer][:ctx])
            x = x + o.reshape(n, -1) @ W["wo"].T
            m = rmsnorm(x, g, sh.rms_eps)
            x = x + swiglu(m, W["w1"], W["w3"], W["w2"])
        return x

    def _logits(self, x: np.ndarray) -> np.ndarray:
        sh = self.w.shape
        return rmsnorm(x, self.w.gain(), sh.rms_eps) @ self.w.matrix("lm_head").T

    def attach_cache(self, rid: int, capacity: int, length: int):
        """A request whose first `length` positions count as cached (zero-valued).

        Only for timing decode steps: the work of a step depends on the cache
        sizes, not on the cached values, so the prefill can be skipped.
        """
        self._alloc(rid, capacity)
        self.len[rid] = length

    def prefill(self, rid: int, tokens: Sequence[int], capacity: int) -> np.ndarray:
        """Fills the cache with the prompt (directive prefix first) and returns the logits of its last position."""
        self._alloc(rid, capacity)
        tokens = np.asarray(tokens, dtype=np.int64)
        T = len(tokens)
        x = embed_rows(self.w, tokens)
        x = self._layers(x, [rid] * T, list(range(T)))
        self.len[rid] = T
        return self._logits(x[-1:])[0]

    def step(self, rids: Sequence[int], tokens: Sequence[int]) -> np.ndarray:
        """One decode step: request rids[r] is fed tokens[r] at its next position.  Returns logits [n, V]."""
        tokens = np.asarray(tokens, dtype=np.int64)
        positions = [self.len[r] for r in rids]
        x = embed_rows(self.w, tokens)
        x = self._layers(x, list(rids), positions)
        for r in rids:
            self.len[r] += 1
        return self._logits(x)


def active_schedule(stop_lens: Sequence[int]) -> List[List[int]]:
    """Active request ids (ascending) at decode steps s = 1 .. max(L) - 1.

    Request i takes part in step s iff L_i > s: it emits g_s there and retires
    at the step where s == L_i - 1.
    """
    stop_lens = list(stop_lens)
    if not stop_lens:
        return []
    return [[i for i, L in enumerate(stop_lens) if L > s] for s in range(1, max(stop_lens))]


def greedy_decode(w: Weights, prompts: Sequence[Sequence[int]], stop_lens: Sequence[int],
                  forced: Optional[Sequence[Sequence[int]]] = None, record_logits: bool = True):
    """Runs the whole closed batch through the KV-cache loop.

    ``forced`` (teacher forcing) supplies the tokens to feed back instead of
    the oracle's own argmax: forced[i][s] replaces g_s of request i.
    Returns (tokens per request, logits per request [L_i, V] or None).
    """
    dec = KVCacheDecoder(w)
    n = len(prompts)
    toks: List[List[int]] = [[] for _ in range(n)]
    logits: List[List[np.ndarray]] = [[] for _ in range(n)]
    for i, p in enumerate(prompts):
        z = dec.prefill(i, p, len(p) + stop_lens[i])
        toks[i].append(int(argmax_first(z)))
        if record_logits:
            logits[i].append(z)
    for s, active in enumerate(active_schedule(stop_lens), start=1):
        feed = [(forced[i][s - 1] if forced is not None else toks[i][s - 1]) for i in active]
        Z = dec.step(active, feed)
        for r, i in enumerate(active):
            toks[i].append(int(argmax_first(Z[r])))
            if record_logits:
                logits[i].append(Z[r])
    return toks, ([np.stack(l) for l in logits] if record_logits else None)
