"""Seeded synthetic verifier weights.

Every tensor is generated in fixed-size chunks, each chunk from its own
counter-keyed PCG64 stream (``SeedSequence(seed, spawn_key=(layer, kind,
chunk))``), so the values do not depend on the number of threads used.

bf16 weights: each element is one of 65536 equiprobable values, the
quantiles of N(0, std) at (i + 0.5) / 65536 rounded to bf16 (round to nearest
even).  This is N(0, 0.02) as seen through bf16 storage, with the tails cut
at about 4.2 sigma.  fp32 weights: the N(0, std) quantile of a 32-bit uniform.
Norm gains are 1.0, or N(1, gain_std) for the scaled-down test shapes.

Layout of every matrix is row-major [out_features, in_features].
"""

from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, Iterator, Optional, Tuple

import numpy as np
from scipy.special import ndtri

from .configs import ModelShape

LAYER_KINDS = ("wq", "wk", "wv", "wo", "wg", "wu", "wd", "g_attn", "g_ffn")
GLOBAL_KINDS = ("embed", "g_final", "lm_head")
WEIGHT_KINDS = LAYER_KINDS + GLOBAL_KINDS
_KIND_ID = {k: i for i, k in enumerate(WEIGHT_KINDS)}
_GLOBAL_LAYER = 65535
CHUNK = 1 << 22


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bf16 (nearest, ties to even); returns uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounding = ((u >> 16) & 1) + np.uint32(0x7FFF)
    out = ((u + rounding) >> 16).astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        out[nan] = 0x7FC0
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


_TABLES: Dict[float, np.ndarray] = {}


def normal_table_bf16(std: float) -> np.ndarray:
    """65536 bf16 bit patterns: N(0, std) quantiles at (i + 0.5) / 65536."""
    t = _TABLES.get(std)
    if t is None:
        p = (np.arange(65536, dtype=np.float64) + 0.5) / 65536.0
        t = f32_to_bf16_bits((ndtri(p) * std).astype(np.float32))
        _TABLES[std] = t
    return t


def tensor_shape(shape: ModelShape, kind: str) -> Tuple[int, ...]:
    d, f, v = shape.d_model, shape.d_ffn, shape.vocab
    dkv = shape.kv_heads * shape.head_dim
    return {
        "wq": (d, d), "wk": (dkv, d), "wv": (dkv, d), "wo": (d, d),
        "wg": (f, d), "wu": (f, d), "wd": (d, f),
        "g_attn": (d,), "g_ffn": (d,), "g_final": (d,),
        "embed": (v, d), "lm_head": (v, d),
    }[kind]


def _rng(seed: int, layer: int, kind: str, chunk: int) -> np.random.Generator:
    ss = np.random.SeedSequence(seed, spawn_key=(layer, _KIND_ID[kind], chunk))
    return np.random.Generator(np.random.PCG64(ss))


def make_tensor(shape: ModelShape, kind: str, layer: Optional[int], seed: int,
                pool: Optional[ThreadPoolExecutor] = None) -> np.ndarray:
    """Generate one tensor.  bf16 matrices come back as uint16 bit patterns,
    fp32 matrices and all gains as float32."""
    dims = tensor_shape(shape, kind)
    lay = _GLOBAL_LAYER if layer is None else int(layer)
    n = int(np.prod(dims))
    if kind.startswith("g_"):
        if shape.gain_std == 0.0:
            return np.ones(dims, dtype=np.float32)
        r = _rng(seed, lay, kind, 0)
        return (1.0 + shape.gain_std * r.standard_normal(n)).astype(np.float32).reshape(dims)

    bf16 = shape.weight_dtype == "bf16"
    out = np.empty(n, dtype=np.uint16 if bf16 else np.float32)
    table = normal_table_bf16(shape.init_std) if bf16 else None
    nchunks = (n + CHUNK - 1) // CHUNK

    def fill(c: int) -> None:
        lo, hi = c * CHUNK, min(n, (c + 1) * CHUNK)
        r = _rng(seed, lay, kind, c)
        if bf16:
            idx = r.integers(0, 65536, size=hi - lo, dtype=np.uint16)
            np.take(table, idx, out=out[lo:hi])
        else:
            u = r.integers(0, 1 << 32, size=hi - lo, dtype=np.uint32)
            out[lo:hi] = (ndtri((u.astype(np.float64) + 0.5) * 2.0 ** -32)
                          * shape.init_std).astype(np.float32)

    if nchunks == 1:
        fill(0)
    elif pool is not None:
        list(pool.map(fill, range(nchunks)))
    else:
        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(fill, range(nchunks)))
    return out.reshape(dims)


def iter_weights(shape: ModelShape, seed: int) -> Iterator[Tuple[str, Optional[int], np.ndarray]]:
    """Yield (kind, layer, tensor) for every tensor, one at a time."""
    with ThreadPoolExecutor(_threads()) as pool:
        for kind in ("embed",):
            yield kind, None, make_tensor(shape, kind, None, seed, pool)
        for layer in range(shape.n_layers):
            for kind in LAYER_KINDS:
                yield kind, layer, make_tensor(shape, kind, layer, seed, pool)
        for kind in ("g_final", "lm_head"):
            yield kind, None, make_tensor(shape, kind, None, seed, pool)


def perturb_tensor(shape: ModelShape, kind: str, layer: Optional[int], t: np.ndarray, sigma: float,
                   noise_seed: int) -> np.ndarray:
    """A weight matrix plus sigma * init_std * N(0, 1) noise of its own seeded
    stream (normal quantiles, as for the weights), rounded back to the
    tensor's type; gains are returned unchanged.  A model built from these is
    a draft whose agreement with the unperturbed model falls as sigma grows."""
    if kind.startswith("g_") or sigma == 0.0:
        return t
    lay = _GLOBAL_LAYER if layer is None else int(layer)
    n = t.size
    table = normal_table_f32()
    out = np.empty(n, dtype=np.float32)
    base = bf16_bits_to_f32(t.ravel()) if t.dtype == np.uint16 else t.ravel().astype(np.float32)
    scale = np.float32(sigma * shape.init_std)
    for c in range((n + CHUNK - 1) // CHUNK):
        lo, hi = c * CHUNK, min(n, (c + 1) * CHUNK)
        r = _rng(noise_seed, lay, kind, c)
        out[lo:hi] = base[lo:hi] + scale * table[r.integers(0, 65536, size=hi - lo, dtype=np.uint16)]
    out = out.reshape(t.shape)
    return f32_to_bf16_bits(out) if t.dtype == np.uint16 else out


def normal_table_f32() -> np.ndarray:
    """65536 N(0, 1) quantiles at (i + 0.5) / 65536, float32."""
    t = _TABLES.get("f32")
    if t is None:
        p = (np.arange(65536, dtype=np.float64) + 0.5) / 65536.0
        t = ndtri(p).astype(np.float32)
        _TABLES["f32"] = t
    return t


def iter_weights_perturbed(shape: ModelShape, seed: int, sigma: float,
                           noise_seed: int) -> Iterator[Tuple[str, Optional[int], np.ndarray]]:
    """iter_weights with every matrix perturbed (perturb_tensor)."""
    for kind, layer, t in iter_weights(shape, seed):
        yield kind, layer, perturb_tensor(shape, kind, layer, t, sigma, noise_seed)


class ModelWeights:
    """All tensors of one model, generated on first use and kept."""

    def __init__(self, shape: ModelShape, seed: int):
        self.shape = shape
        self.seed = seed
        self._cache: Dict[Tuple[str, Optional[int]], np.ndarray] = {}
        self._pool: Optional[ThreadPoolExecutor] = None

    def get(self, kind: str, layer: Optional[int] = None) -> np.ndarray:
        key = (kind, layer)
        t = self._cache.get(key)
        if t is None:
            if self._pool is None:
                self._pool = ThreadPoolExecutor(_threads())
            t = make_tensor(self.shape, kind, layer, self.seed, self._pool)
            self._cache[key] = t
        return t

    def materialize(self) -> "ModelWeights":
        for layer in range(self.shape.n_layers):
            for kind in LAYER_KINDS:
                self.get(kind, layer)
        for kind in GLOBAL_KINDS:
            self.get(kind)
        return self

    def close(self) -> None:
        if self._pool is not None:
            self._pool.shutdown()
            self._pool = None
