"""Oracle verifier forward pass (float64, NumPy) -- test infrastructure only.

Sec. III-A of the paper: an embedding layer maps tokens to x_0, every block
updates the residual stream x_{l+1} = x_l + f_l(x_l) with f_l = self-attention
then feed-forward, the LM head g maps the last hidden state to logits o_L, and
P(y_{t+1} | y_{1:t}) = softmax(o_L^t).  The paper does not fix the block; the
verifier here is the Llama-style instance: pre-RMSNorm, rotary position
embedding (rotate-half pairing, base rope_theta), multi-head causal attention
with scale 1/sqrt(head_dim), a SwiGLU feed-forward, no biases, untied LM head.
The paper's own cloud verifier is LLaMA-3.1-8B (Experiments, "Models"), whose
attention is grouped-query: with n_kv_heads < n_heads, query head h attends
with the K/V head floor(h / (n_heads / n_kv_heads)).

Readings the paper leaves open (each listed in the design notes):
* RMSNorm(x) = x / sqrt(mean(x^2) + eps) * g with eps = 1e-5;
* RoPE pairs feature i with i + head_dim/2 and rotates by pos * base^(-2i/hd);
* K and V are stored at the cache precision (bf16: round-to-nearest-even of
  the float32 value) after RoPE, and every attention read -- including the
  rows of the block being verified -- sees the stored values; queries are not
  rounded;
* a verify call appends gamma+1 rows, [pending, d_1 .. d_gamma], at
  positions L .. L+gamma of a cache holding L tokens (Algorithm 1: the d+1
  verifier distributions of one pass).

Everything runs in float64; bf16 weights are widened exactly.
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import Callable, Dict, List, Optional

import numpy as np


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns (uint16) to float64."""
    u32 = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u32.view(np.float32).astype(np.float64)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Value of x after storage as bf16: x is first rounded to float32, then
    to bf16 with round-to-nearest, ties-to-even on the 16 dropped bits."""
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    low = u & np.uint64(0xFFFF)
    high = u >> np.uint64(16)
    up = (low > 0x8000) | ((low == 0x8000) & ((high & np.uint64(1)) == 1))
    high = high + up.astype(np.uint64)
    r = (high << np.uint64(16)).astype(np.uint32).view(np.float32).astype(np.float64)
    return np.where(np.isfinite(f), r, f.astype(np.float64))


def rms_norm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * g over the last axis."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def rope_tables(positions: np.ndarray, head_dim: int, theta: float):
    """cos/sin of pos * theta^(-2i/head_dim), i < head_dim/2, in float64."""
    half = head_dim // 2
    inv = theta ** (-2.0 * np.arange(half, dtype=np.float64) / head_dim)
    ang = np.asarray(positions, dtype=np.float64)[:, None] * inv[None, :]
    return np.cos(ang), np.sin(ang)


def apply_rope(x: np.ndarray, cos: np.ndarray, sin: np.ndarray) -> np.ndarray:
    """x: [R, H, hd]; rotate pairs (i, i + hd/2) by the angle of each row."""
    half = x.shape[-1] // 2
    a, b = x[..., :half], x[..., half:]
    c, s = cos[:, None, :], sin[:, None, :]
    return np.concatenate([a * c - b * s, a * s + b * c], axis=-1)


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def softmax(z: np.ndarray, axis: int = -1) -> np.ndarray:
    m = np.max(z, axis=axis, keepdims=True)
    e = np.exp(z - m)
    return e / np.sum(e, axis=axis, keepdims=True)


@dataclass
class KVCache:
    """One request's cache: per layer K and V of shape [KV heads, capacity, hd]."""

    n_layers: int
    n_heads: int
    head_dim: int
    capacity: int
    length: int = 0
    k: List[np.ndarray] = field(default_factory=list)
    v: List[np.ndarray] = field(default_factory=list)

    def __post_init__(self):
        # Every stored value is already rounded to the cache precision (bf16
        # or float32), so float32 arrays hold it exactly; attention reads
        # widen it back to float64 without loss.
        if not self.k:
            shp = (self.n_heads, self.capacity, self.head_dim)
            self.k = [np.zeros(shp, dtype=np.float32) for _ in range(self.n_layers)]
            self.v = [np.zeros(shp, dtype=np.float32) for _ in range(self.n_layers)]

    def copy(self) -> "KVCache":
        return KVCache(self.n_layers, self.n_heads, self.head_dim, self.capacity, self.length,
                       [a.copy() for a in self.k], [a.copy() for a in self.v])


_LAYER_KINDS = ("g_attn", "wq", "wk", "wv", "wo", "g_ffn", "wg", "wu", "wd")


class Decoder:
    """The verifier M_p.  ``get(kind, layer)`` returns a weight tensor as
    stored: uint16 bf16 bits or float32 (row-major [out, in]), float32 gains."""

    def __init__(self, shape, get: Callable[[str, Optional[int]], np.ndarray],
                 keep_f64: bool = False):
        self.shape = shape
        self._get = get
        self._keep = keep_f64
        self._f64: Dict = {}

    def w(self, kind: str, layer: Optional[int] = None) -> np.ndarray:
        key = (kind, layer)
        if key in self._f64:
            return self._f64[key]
        t = self._get(kind, layer)
        t = bf16_bits_to_f64(t) if t.dtype == np.uint16 else np.asarray(t, dtype=np.float64)
        if self._keep:
            self._f64[key] = t
        return t

    def new_cache(self, capacity: int) -> KVCache:
        s = self.shape
        return KVCache(s.n_layers, s.kv_heads, s.head_dim, capacity)

    def _store(self, x: np.ndarray) -> np.ndarray:
        return bf16_round(x) if self.shape.kv_dtype == "bf16" else x.astype(np.float32).astype(np.float64)

    def block(self, l: int, W: Callable[[str], np.ndarray], cache: KVCache, x: np.ndarray) -> np.ndarray:
        """Residual block l (self-attention, then feed-forward) for the R rows
        x at positions cache.length .. +R-1; writes their K/V rows to the
        cache (the length is advanced by the caller).  ``W(kind)`` returns the
        block's weights."""
        s = self.shape
        R = x.shape[0]
        L = cache.length
        if L + R > cache.capacity:
            raise ValueError("cache capacity exceeded")
        H, hd = s.n_heads, s.head_dim
        KVH = s.kv_heads
        G = H // KVH  # query heads per K/V head
        pos = np.arange(L, L + R)
        cos, sin = rope_tables(pos, hd, s.rope_theta)
        scale = 1.0 / np.sqrt(hd)
        # attention sub-block
        h = rms_norm(x, W("g_attn"), s.rms_eps)
        q = (h @ W("wq").T).reshape(R, H, hd)
        k = (h @ W("wk").T).reshape(R, KVH, hd)
        v = (h @ W("wv").T).reshape(R, KVH, hd)
        q = apply_rope(q, cos, sin)
        k = apply_rope(k, cos, sin)
        cache.k[l][:, L:L + R, :] = self._store(k).transpose(1, 0, 2)
        cache.v[l][:, L:L + R, :] = self._store(v).transpose(1, 0, 2)
        # query head h reads K/V head h // G
        K = np.repeat(cache.k[l][:, :L + R, :], G, axis=0).astype(np.float64)  # [H, L+R, hd]
        Vv = np.repeat(cache.v[l][:, :L + R, :], G, axis=0).astype(np.float64)
        scores = np.matmul(q.transpose(1, 0, 2), K.transpose(0, 2, 1)) * scale  # [H, R, L+R]
        key_pos = np.arange(L + R)
        mask = key_pos[None, :] <= pos[:, None]  # row i sees keys <= L+i
        scores = np.where(mask[None, :, :], scores, -np.inf)
        p = softmax(scores, axis=-1)
        o = np.matmul(p, Vv).transpose(1, 0, 2).reshape(R, H * hd)
        x = x + o @ W("wo").T
        # feed-forward sub-block
        h = rms_norm(x, W("g_ffn"), s.rms_eps)
        a = silu(h @ W("wg").T) * (h @ W("wu").T)
        return x + a @ W("wd").T

    def head(self, x: np.ndarray) -> np.ndarray:
        """LM head: o_L = RMSNorm(x_L) W_lm^T for each row."""
        h = rms_norm(x, self.w("g_final"), self.shape.rms_eps)
        return h @ self.w("lm_head").T

    def forward(self, cache: KVCache, tokens: np.ndarray, want_logits: bool = True) -> Optional[np.ndarray]:
        """Append ``tokens`` (R ids) at positions cache.length .. +R-1 and
        return the R rows of next-token logits [R, V] (float64)."""
        tokens = np.asarray(tokens, dtype=np.int64)
        if cache.length + tokens.shape[0] > cache.capacity:
            raise ValueError("cache capacity exceeded")
        x = self.w("embed")[tokens]  # x_0
        for l in range(self.shape.n_layers):
            x = self.block(l, lambda kind: self.w(kind, l), cache, x)
        cache.length += tokens.shape[0]
        return self.head(x) if want_logits else None

    def forward_many(self, caches: List[KVCache], tokens: List[np.ndarray],
                     want_logits: bool = True) -> Optional[List[np.ndarray]]:
        """``forward`` for several independent requests, layer by layer: each
        layer's weights are fetched once and applied to every request in
        turn (the same arithmetic per request as ``forward``)."""
        toks = [np.asarray(t, dtype=np.int64) for t in tokens]
        for c, t in zip(caches, toks):
            if c.length + t.shape[0] > c.capacity:
                raise ValueError("cache capacity exceeded")
        E = self.w("embed")
        xs = [E[t] for t in toks]
        del E
        for l in range(self.shape.n_layers):
            Wl = {kind: self.w(kind, l) for kind in _LAYER_KINDS}
            for i, c in enumerate(caches):
                xs[i] = self.block(l, Wl.__getitem__, c, xs[i])
            del Wl
        for c, t in zip(caches, toks):
            c.length += t.shape[0]
        return [self.head(x) for x in xs] if want_logits else None

    def prefill(self, cache: KVCache, tokens: np.ndarray, chunk: int = 4096) -> None:
        """Run the cached prefix through the model (no logits needed)."""
        tokens = np.asarray(tokens)
        for i in range(0, len(tokens), chunk):
            self.forward(cache, tokens[i:i + chunk], want_logits=False)
