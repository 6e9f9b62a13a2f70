"""Thin ctypes binding of ``libspade.so`` (include/spade.h).

Argument marshalling only: every step of the verify path runs in the HIP
library.  PyTorch provides the device buffers and the current stream.  If the
library is missing the import of a model fails loudly; there is no CPU path.
"""

from __future__ import annotations

import ctypes
import os
from typing import Iterable, Optional, Tuple

import numpy as np
import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libspade.so")

SPADE_OK = 0
GREEDY, SAMPLE = 0, 1
F32, BF16 = 0, 1
KINDS = {"wq": 0, "wk": 1, "wv": 2, "wo": 3, "wg": 4, "wu": 5, "wd": 6,
         "g_attn": 7, "g_ffn": 8, "embed": 9, "g_final": 10, "lm_head": 11}
GLOBAL_KINDS = ("embed", "g_final", "lm_head")
DERR_TOKEN, DERR_NAN, DERR_RESIDUAL, DERR_NOQ, DERR_CAPACITY, DERR_COMMIT = 1, 2, 4, 8, 16, 32

# include/spade.h: the calls of the method
EXPORTED = (
    "spade_weight_bytes", "spade_workspace_bytes", "spade_kv_bytes", "spade_model_create",
    "spade_model_load_tensor", "spade_kv_create", "spade_kv_set_state", "spade_kv_get_state",
    "spade_kv_snapshot", "spade_kv_restore", "spade_prefill", "spade_verify", "spade_kv_commit",
    "spade_accept_from_logits", "spade_get_device_error", "spade_last_error",
    "spade_model_destroy", "spade_kv_destroy", "spade_softmax", "spade_prefill_batch",
    "spade_accept_from_logits_noalloc",
)
# include/spade_tuning.h: schedule controls and measurement hooks
EXPORTED_TUNING = (
    "spade_model_set_wide_tiles", "spade_model_set_wide_k_splits", "spade_model_set_split_k",
    "spade_model_set_attn_merge", "spade_model_set_correction_slices", "spade_model_set_attn_grouped",
    "spade_model_set_prefill_rows", "spade_model_set_big_gemm", "spade_model_set_mid_gemm", "spade_profile_gemm",
    "spade_wide_tiling",
)


class SpadeError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"spade status {status}: {msg}")
        self.status = status


class SpadeConfig(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32),
                ("n_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("d_ffn", ctypes.c_int32), ("vocab", ctypes.c_int32),
                ("weight_dtype", ctypes.c_int32), ("kv_dtype", ctypes.c_int32),
                ("rms_eps", ctypes.c_float), ("rope_theta", ctypes.c_float),
                ("n_kv_heads", ctypes.c_int32)]


def config_from(shape) -> SpadeConfig:
    """spade_config from any object with the ModelShape attributes."""
    return SpadeConfig(shape.n_layers, shape.d_model, shape.n_heads, shape.head_dim, shape.d_ffn,
                       shape.vocab, BF16 if shape.weight_dtype == "bf16" else F32,
                       BF16 if shape.kv_dtype == "bf16" else F32, shape.rms_eps, shape.rope_theta,
                       getattr(shape, "n_kv_heads", 0))


_LIB = None
P, I, SZ, F = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t, ctypes.c_float


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built; run `python -m paper_2608_13076_amd.build` "
                           "(there is no CPU fallback)")
    lib = ctypes.CDLL(path)
    cfgp = ctypes.POINTER(SpadeConfig)
    sig = {
        "spade_weight_bytes": (SZ, [cfgp]),
        "spade_workspace_bytes": (SZ, [cfgp, I, I, I]),
        "spade_kv_bytes": (SZ, [cfgp, I, I]),
        "spade_model_create": (I, [cfgp, P, P, I, I, I, ctypes.POINTER(P)]),
        "spade_model_load_tensor": (I, [P, I, I, P, P]),
        "spade_kv_create": (I, [P, P, I, I, P, P, ctypes.POINTER(P)]),
        "spade_kv_set_state": (I, [P, I, P, P, P]),
        "spade_kv_get_state": (I, [P, I, P, P, P]),
        "spade_kv_snapshot": (I, [P, I, P, P, P]),
        "spade_kv_restore": (I, [P, I, P, P, P]),
        "spade_prefill": (I, [P, P, I, P, I, P]),
        "spade_verify": (I, [P, P, I, I, P, P, P, P, F, P, P, P, P]),
        "spade_kv_commit": (I, [P, I, P, P, P]),
        "spade_accept_from_logits": (I, [P, I, I, I, P, P, P, P, P, F, P, P, P]),
        "spade_accept_from_logits_noalloc": (I, [I, I, I, P, P, P, P, P, F, P, P, P, P]),
        "spade_profile_gemm": (I, [P, P, I, I, I, I, P]),
        "spade_get_device_error": (I, [P, P, P]),
        "spade_model_set_wide_tiles": (I, [P, I, I]),
        "spade_model_set_wide_k_splits": (I, [P, I]),
        "spade_model_set_attn_merge": (I, [P, I]),
        "spade_model_set_correction_slices": (I, [P, I]),
        "spade_model_set_attn_grouped": (I, [P, I]),
        "spade_model_set_prefill_rows": (I, [P, I]),
        "spade_model_set_big_gemm": (I, [P, I]),
        "spade_model_set_mid_gemm": (I, [P, I, I]),
        "spade_model_set_split_k": (I, [P, I]),
        "spade_softmax": (I, [P, I, I, F, P, P]),
        "spade_prefill_batch": (I, [P, P, I, P, I, P, P]),
        "spade_wide_tiling": (I, [I, I, I, I, I, P, P, P]),
        "spade_last_error": (ctypes.c_char_p, []),
        "spade_model_destroy": (None, [P]),
        "spade_kv_destroy": (None, [P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _LIB = lib
    return lib


def _check(status: int) -> None:
    if status != SPADE_OK:
        raise SpadeError(status, load_library().spade_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors passed to the library must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _to_device_u8(nbytes: int, device) -> torch.Tensor:
    # 256-byte alignment: torch's caching allocator returns 512-byte aligned blocks
    t = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)
    assert t.data_ptr() % 256 == 0
    return t


class Model:
    """Verifier weights + workspace on one GPU."""

    def __init__(self, shape, max_batch: int, max_gamma: int, max_len: int, device="cuda:0"):
        self.lib = load_library()
        self.shape = shape
        self.device = torch.device(device)
        self.cfg = config_from(shape)
        self.max_batch, self.max_gamma, self.max_len = max_batch, max_gamma, max_len
        wb = self.lib.spade_weight_bytes(ctypes.byref(self.cfg))
        if wb == 0:
            raise SpadeError(-4, "unsupported config: " + self.lib.spade_last_error().decode())
        ws = self.lib.spade_workspace_bytes(ctypes.byref(self.cfg), max_batch, max_gamma, max_len)
        if ws == 0:
            raise SpadeError(-2, "workspace size: " + self.lib.spade_last_error().decode())
        with torch.cuda.device(self.device):
            self.weights = _to_device_u8(wb, self.device)
            self.workspace = _to_device_u8(ws, self.device)
            h = ctypes.c_void_p()
            _check(self.lib.spade_model_create(ctypes.byref(self.cfg), _ptr(self.weights), _ptr(self.workspace),
                                               max_batch, max_gamma, max_len, ctypes.byref(h)))
        self.handle = h

    def weight_bytes(self) -> int:
        return self.weights.numel()

    def load_tensor(self, kind: str, layer: Optional[int], t: torch.Tensor) -> None:
        _check(self.lib.spade_model_load_tensor(self.handle, KINDS[kind], -1 if layer is None else layer,
                                                _ptr(t), _stream()))

    def load_numpy(self, kind: str, layer: Optional[int], arr: np.ndarray) -> None:
        a = np.ascontiguousarray(arr)
        if a.dtype == np.uint16:
            a = a.view(np.int16)
        t = torch.from_numpy(a).to(self.device)
        self.load_tensor(kind, layer, t)
        torch.cuda.current_stream(self.device).synchronize()

    def load_all(self, tensors: Iterable[Tuple[str, Optional[int], np.ndarray]]) -> None:
        for kind, layer, arr in tensors:
            self.load_numpy(kind, layer, arr)

    def set_wide_tiles(self, row_tiles: int, panels: int = 0) -> None:
        """Tiling of the batched projections: 16-row tiles per workgroup (0
        chosen per launch, 1..3 fixed, -1 skinny engine once per 32 rows) and
        weight panels per wave (0 chosen per launch, 1..2 fixed)."""
        _check(self.lib.spade_model_set_wide_tiles(self.handle, int(row_tiles), int(panels)))

    def set_attn_merge(self, mode: int) -> None:
        """Merge of one-chunk attention partials: 0 chosen per call, 1 by the
        last chunk workgroup, 2 in a second launch."""
        _check(self.lib.spade_model_set_attn_merge(self.handle, int(mode)))

    def set_attn_grouped(self, mode: int) -> None:
        """Grouped-query attention chunks (all query heads of a K/V head in one
        workgroup, with the second-launch merge): 0 where they apply, 1 off."""
        _check(self.lib.spade_model_set_attn_grouped(self.handle, int(mode)))

    def set_prefill_rows(self, rows: int) -> None:
        """Prompt rows per request of a prefill forward: 0 as many as the
        workspace holds (bf16 cache, head_dim 128), n > 0 at most n."""
        _check(self.lib.spade_model_set_prefill_rows(self.handle, int(rows)))

    def set_big_gemm(self, mode: int) -> None:
        """Projection GEMM of forwards with many rows: 0 where it fills the
        chip, 1 off, 2 for every launch of more than 16 rows (not the LM head)."""
        _check(self.lib.spade_model_set_big_gemm(self.handle, int(mode)))

    def set_mid_gemm(self, mode: int, k_splits: int = 0) -> None:
        """Projection GEMM of batched calls of up to 144 rows: mode 0 gate/up
        from 113 rows, O from 129, down from 137, 1 off, 2 every projection
        from 17 rows (not the LM head); k_splits 0 chosen per launch, 1..8
        fixed."""
        _check(self.lib.spade_model_set_mid_gemm(self.handle, int(mode), int(k_splits)))

    def set_correction_slices(self, mode: int) -> None:
        """Correction draw of sampling requests: 0 or 2 over vocabulary slices
        in a second launch, 1 in the accept workgroup."""
        _check(self.lib.spade_model_set_correction_slices(self.handle, int(mode)))

    def set_wide_k_splits(self, splits: int) -> None:
        """K splits of the batched O and down projections on the wide-row
        GEMM: 0 chosen per launch, 1 off, 2 or 4 fixed."""
        _check(self.lib.spade_model_set_wide_k_splits(self.handle, int(splits)))

    def set_split_k(self, splits: int) -> None:
        """K splits of the small-batch projections whose operand does not fit
        in LDS: 0 chosen per launch, 2 or 4 fixed, -1 off."""
        _check(self.lib.spade_model_set_split_k(self.handle, int(splits)))

    def device_error(self) -> int:
        v = ctypes.c_uint32()
        _check(self.lib.spade_get_device_error(self.handle, ctypes.byref(v), _stream()))
        return v.value

    def accept_from_logits(self, logits: torch.Tensor, drafts: torch.Tensor, draft_probs, uniforms,
                           modes: torch.Tensor, temperature: float = 1.0):
        B, R, V = logits.shape
        n = torch.empty(B, dtype=torch.int32, device=self.device)
        c = torch.empty(B, dtype=torch.int32, device=self.device)
        _check(self.lib.spade_accept_from_logits(self.handle, B, R - 1, V, _ptr(logits), _ptr(drafts),
                                                 _ptr(draft_probs), _ptr(uniforms), _ptr(modes),
                                                 float(temperature), _ptr(n), _ptr(c), _stream()))
        return n, c

    def close(self) -> None:
        if getattr(self, "handle", None):
            self.lib.spade_model_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class KVCache:
    """K/V storage plus per-request lens and pending tokens on the device."""

    def __init__(self, model: Model, max_batch: int, max_len: int):
        self.model = model
        self.lib = model.lib
        nbytes = self.lib.spade_kv_bytes(ctypes.byref(model.cfg), max_batch, max_len)
        with torch.cuda.device(model.device):
            self.buf = _to_device_u8(nbytes, model.device)
            self.lens = torch.zeros(max_batch, dtype=torch.int32, device=model.device)
            self.pending = torch.zeros(max_batch, dtype=torch.int32, device=model.device)
        h = ctypes.c_void_p()
        _check(self.lib.spade_kv_create(model.handle, _ptr(self.buf), max_batch, max_len, _ptr(self.lens),
                                        _ptr(self.pending), ctypes.byref(h)))
        self.handle = h
        self.max_batch, self.max_len = max_batch, max_len

    def set_state(self, lens, pending) -> None:
        l = np.ascontiguousarray(lens, dtype=np.int32)
        p = np.ascontiguousarray(pending, dtype=np.int32)
        _check(self.lib.spade_kv_set_state(self.handle, len(l), l.ctypes.data_as(P), p.ctypes.data_as(P),
                                           _stream()))

    def get_state(self, B: int):
        l = np.zeros(B, dtype=np.int32)
        p = np.zeros(B, dtype=np.int32)
        _check(self.lib.spade_kv_get_state(self.handle, B, l.ctypes.data_as(P), p.ctypes.data_as(P), _stream()))
        return l, p

    def snapshot(self, B: int):
        lens = torch.empty(B, dtype=torch.int32, device=self.model.device)
        pending = torch.empty(B, dtype=torch.int32, device=self.model.device)
        _check(self.lib.spade_kv_snapshot(self.handle, B, _ptr(lens), _ptr(pending), _stream()))
        return lens, pending

    def restore(self, lens: torch.Tensor, pending: torch.Tensor) -> None:
        _check(self.lib.spade_kv_restore(self.handle, lens.numel(), _ptr(lens), _ptr(pending), _stream()))

    def prefill(self, b: int, tokens) -> None:
        t = torch.as_tensor(np.asarray(tokens, dtype=np.int32)).to(self.model.device)
        _check(self.lib.spade_prefill(self.model.handle, self.handle, b, _ptr(t), t.numel(), _stream()))
        torch.cuda.current_stream(self.model.device).synchronize()

    def prefill_batch(self, prompts) -> None:
        """Prefill requests 0..len(prompts)-1 at once (spade_prefill_batch)."""
        B = len(prompts)
        ld = max(len(p) for p in prompts)
        arr = np.zeros((B, ld), dtype=np.int32)
        for b, p in enumerate(prompts):
            arr[b, :len(p)] = np.asarray(p, dtype=np.int32)
        counts = np.array([len(p) for p in prompts], dtype=np.int32)
        t = torch.from_numpy(arr).to(self.model.device)
        _check(self.lib.spade_prefill_batch(self.model.handle, self.handle, B, _ptr(t), ld,
                                            counts.ctypes.data_as(P), _stream()))
        torch.cuda.current_stream(self.model.device).synchronize()

    def commit(self, n: torch.Tensor, corr: torch.Tensor) -> None:
        _check(self.lib.spade_kv_commit(self.handle, n.numel(), _ptr(n), _ptr(corr), _stream()))

    def close(self) -> None:
        if getattr(self, "handle", None):
            self.lib.spade_kv_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class VerifyBuffers:
    """Device copies of one call's inputs and its outputs."""

    def __init__(self, model: Model, drafts, draft_probs, uniforms, modes, want_logits=True):
        dev = model.device
        drafts = np.ascontiguousarray(drafts, dtype=np.int32)
        self.B, self.gamma = drafts.shape
        self.drafts = torch.from_numpy(drafts).to(dev)
        self.q = None if draft_probs is None else torch.from_numpy(
            np.ascontiguousarray(draft_probs, dtype=np.float32)).to(dev)
        self.u = None if uniforms is None else torch.from_numpy(
            np.ascontiguousarray(uniforms, dtype=np.float32)).to(dev)
        self.mode = torch.from_numpy(np.ascontiguousarray(modes, dtype=np.uint8)).to(dev)
        self.n = torch.empty(self.B, dtype=torch.int32, device=dev)
        self.corr = torch.empty(self.B, dtype=torch.int32, device=dev)
        self.logits = (torch.empty((self.B, self.gamma + 1, model.shape.vocab), dtype=torch.float32, device=dev)
                       if want_logits else None)


def verify(model: Model, kv: KVCache, buf: VerifyBuffers, temperature: float = 1.0) -> None:
    """Launch spade_verify on the current stream (asynchronous)."""
    _check(model.lib.spade_verify(model.handle, kv.handle, buf.B, buf.gamma, _ptr(buf.drafts), _ptr(buf.q),
                                  _ptr(buf.u), _ptr(buf.mode), float(temperature), _ptr(buf.n),
                                  _ptr(buf.corr), _ptr(buf.logits), _stream()))


def accept_from_logits_noalloc(logits: torch.Tensor, drafts: torch.Tensor, draft_probs, uniforms,
                               modes: torch.Tensor, temperature: float, n: torch.Tensor, corr: torch.Tensor,
                               err: torch.Tensor) -> None:
    """spade_accept_from_logits_noalloc on the current stream: writes n and
    corr, ORs error bits into err (int32 [1]); allocates nothing."""
    B, R, V = logits.shape
    _check(load_library().spade_accept_from_logits_noalloc(B, R - 1, V, _ptr(logits), _ptr(drafts),
                                                           _ptr(draft_probs), _ptr(uniforms), _ptr(modes),
                                                           float(temperature), _ptr(n), _ptr(corr), _ptr(err),
                                                           _stream()))


def softmax_into(logits: torch.Tensor, out: torch.Tensor, temperature: float = 1.0) -> None:
    """out = softmax(logits / temperature) row by row (float32, last dim V),
    on the current stream."""
    V = logits.shape[-1]
    rows = logits.numel() // V
    _check(load_library().spade_softmax(_ptr(logits), rows, V, float(temperature), _ptr(out), _stream()))


GEMM_KINDS = {"qkv": 0, "o": 1, "gu": 2, "down": 3, "lm": 4}


def gemm_weight_bytes(shape, kind: str) -> int:
    """Weight bytes one launch of a projection GEMM streams."""
    elt = 2 if shape.weight_dtype == "bf16" else 4
    d, f, v = shape.d_model, shape.d_ffn, shape.vocab
    dkv = getattr(shape, "kv_heads", shape.n_heads) * shape.head_dim
    n_k = {"qkv": (d + 2 * dkv, d), "o": (d, d), "gu": (2 * f, d), "down": (d, f), "lm": (v, d)}[kind]
    return n_k[0] * n_k[1] * elt


def wide_tiling(kind: str, rows: int, n_units: int, k: int, n_cu: int = 256) -> tuple:
    """(row tiles, panels per wave, k-splits) the wide-row GEMM picks for a
    projection of `rows` rows, `n_units` weight panels and `k` inputs."""
    lib = load_library()
    rt, p, ks = ctypes.c_int(), ctypes.c_int(), ctypes.c_int()
    _check(lib.spade_wide_tiling(GEMM_KINDS[kind], rows, n_units, k, n_cu, ctypes.byref(rt), ctypes.byref(p),
                                 ctypes.byref(ks)))
    return rt.value, p.value, ks.value


def gemm_roofline(model: Model, kv: KVCache, kind: str, B: int, gamma: int, reps: int, peak_gbs: float) -> dict:
    """Average duration of one launch of a projection GEMM (HIP events on the
    current stream around `reps` x n_layers launches of that kernel alone)
    and its algorithmic bytes: the weight matrix once, the fp32 input rows
    once, the fp32 output rows once."""
    s = model.shape
    L = s.n_layers if kind != "lm" else 1
    n = reps * L
    M = B * (gamma + 1)
    d, f, v = s.d_model, s.d_ffn, s.vocab
    k_in = f if kind == "down" else d
    n_out = {"qkv": 3 * d, "o": d, "gu": f, "down": d, "lm": v}[kind]
    alg = gemm_weight_bytes(s, kind) + M * k_in * 4 + M * n_out * 4
    _check(model.lib.spade_profile_gemm(model.handle, kv.handle, GEMM_KINDS[kind], B, gamma, L, _stream()))
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    _check(model.lib.spade_profile_gemm(model.handle, kv.handle, GEMM_KINDS[kind], B, gamma, n, _stream()))
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / n
    achieved = alg / (us * 1e-6) / 1e9
    return {"kernel": f"gemm_kernel<{kind}>", "bound": "hbm", "achieved": round(achieved, 1),
            "peak": peak_gbs, "unit": "GB/s", "frac": round(achieved / peak_gbs, 4), "traffic": None,
            "avg_launch_us": round(us, 3), "algorithmic_bytes_per_launch": alg, "launches_timed": n}
