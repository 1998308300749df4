"""ctypes binding of libqevict.so (include/qevict.h), same names as the C ABI.

Argument marshalling only: every step of the decode path runs in the HIP
kernels of the library.  PyTorch supplies device memory (the workspace and the
tensors) and the HIP stream.  Importing this module does not need a GPU;
creating a cache does, and there is no CPU fallback: a missing library raises.
"""
from __future__ import annotations

import ctypes
import math
import dataclasses
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libqevict.so")

ABI_VERSION = 4
OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_WORKSPACE, ERR_BAD_STATE, ERR_NONFINITE, \
    ERR_CAPACITY, ERR_DEVICE = 0, -1, -2, -3, -4, -5, -6, -7
TIER_UNUSED, TIER_OPEN, TIER_FULL, TIER_QUANT, TIER_EVICTED = 0, 1, 2, 3, 4
LEDGER_NONE, LEDGER_ACTIVE, LEDGER_DORMANT = 0, 1, 2
BITS_MIXED_4_2 = 42
OUT_F32, OUT_BF16 = 0, 1
FLAG_NO_PROMOTION, FLAG_DEBUG_MASSES, FLAG_ASYNC_ROUTING = 0x1, 0x2, 0x4
FLAG_ROUTING_QUEUE_WAIT, FLAG_ROUTING_DEVICE_WAIT = 0x8, 0x10
KERNEL_ATTEND, KERNEL_MERGE, KERNEL_RETIER, KERNEL_MIGRATE = range(4)
SCORE_CUMULATIVE, SCORE_DECAY, SCORE_KEY_NORM, SCORE_PNORM = 0, 1, 2, 3

# exported symbols declared in include/qevict.h
SYMBOLS = (
    "qevict_workspace_size", "qevict_cache_init", "qevict_cache_destroy", "qevict_prefill_assign",
    "qevict_decode_attend", "qevict_retier", "qevict_quantize_window", "qevict_promote_window",
    "qevict_get_state", "qevict_export_window", "qevict_debug_shift_keys", "qevict_debug_masses",
    "qevict_debug_last_masses", "qevict_debug_routing_gate", "qevict_routing_order",
    "qevict_profile_enable", "qevict_profile_read", "qevict_last_attend_bytes", "qevict_join_routing",
    "qevict_status_string", "qevict_last_error", "qevict_prefill_scores_scratch_size",
    "qevict_prefill_scores", "qevict_capacities_for_budget", "qevict_memory_report",
    "qevict_prefill_scores_noalloc",
)


class QEvictError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"qevict status {status}: {message}")
        self.status = status


class _Config(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "abi_version", "batch", "num_layers", "num_q_heads", "num_kv_heads", "head_dim",
        "window_tokens", "group_size", "quant_bits", "sink_tokens", "recent_tokens", "max_context",
        "capacity_full", "capacity_quant", "retier_interval", "out_dtype")] + [
        ("flags", ctypes.c_uint32), ("softmax_scale", ctypes.c_float), ("num_splits", ctypes.c_int32),
        ("score_mode", ctypes.c_int32), ("score_decay", ctypes.c_float), ("score_p", ctypes.c_float),
        ("rope_base", ctypes.c_float)]


class MemoryReport(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in (
        "sink", "recent", "full", "quant_codes", "quant_meta", "position", "ledger", "total")]

    def as_dict(self):
        return {n: getattr(self, n) for n, _ in self._fields_}


class RetierStats(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "promotions", "admissions_full", "first_quantizations", "reactivations", "evictions",
        "n_full", "n_quant_int4", "n_quant_int2")]

    def as_dict(self):
        return {n: getattr(self, n) for n, _ in self._fields_}


@dataclasses.dataclass
class Config:
    batch: int
    num_q_heads: int
    num_kv_heads: int
    window_tokens: int
    quant_bits: int
    max_context: int
    capacity_full: int
    capacity_quant: int
    num_layers: int = 1
    head_dim: int = 128
    group_size: int = 0          # 0: window_tokens (32 for 8-token windows)
    sink_tokens: int = 0
    recent_tokens: int = 0
    retier_interval: int = 1
    out_dtype: int = OUT_F32
    flags: int = 0
    softmax_scale: float = 0.0
    num_splits: int = 0
    score_mode: int = SCORE_CUMULATIVE
    score_decay: float = 0.0
    score_p: float = 0.0
    rope_base: float = 0.0

    def to_c(self) -> _Config:
        c = _Config()
        c.abi_version = ABI_VERSION
        for f in dataclasses.fields(self):
            setattr(c, f.name, getattr(self, f.name))
        if not self.group_size:   # the value group: 32 channels for 8-token windows, else W
            c.group_size = 32 if self.window_tokens == 8 else self.window_tokens
        return c


_lib = None


def load_library(path: str | None = None):
    """Load libqevict.so (built in-tree); raises if it has not been built."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(f"{p} is missing: build it with `python -m paper_2608_05326_amd.build`")
    # torch carries its own HIP runtime: load it first so that the library binds
    # to the runtime torch's device memory and streams come from (loaded the
    # other way round, creating a cache fails with "no ROCm-capable device")
    import torch  # noqa: F401
    lib = ctypes.CDLL(p)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    P = ctypes.POINTER
    sig = {
        "qevict_workspace_size": [P(_Config), P(ctypes.c_size_t)],
        "qevict_cache_init": [P(_Config), vp, ctypes.c_size_t, vp, P(vp)],
        "qevict_cache_destroy": [vp],
        "qevict_prefill_assign": [vp, i32, vp, vp, i32, vp],
        "qevict_decode_attend": [vp, i32, vp, vp, vp, vp],
        "qevict_retier": [vp, i32, P(RetierStats)],
        "qevict_quantize_window": [vp, i32, i32, i32],
        "qevict_promote_window": [vp, i32, i32, i32],
        "qevict_get_state": [vp, i32, i32, vp, vp, vp, vp, i32, P(i32)],
        "qevict_export_window": [vp, i32, i32, i32, vp, vp, vp, vp, vp, vp],
        "qevict_debug_shift_keys": [vp, i32, i32, i32, vp],
        "qevict_debug_masses": [vp, i32, vp, i32],
        "qevict_debug_last_masses": [vp, i32, vp],
        "qevict_debug_routing_gate": [vp, i64, i32],
        "qevict_routing_order": [vp, P(i32)],
        "qevict_profile_enable": [vp, i32],
        "qevict_profile_read": [vp, i32, P(ctypes.c_double), P(i64)],
        "qevict_last_attend_bytes": [vp, i32, P(i64)],
        "qevict_join_routing": [vp],
        "qevict_prefill_scores_scratch_size": [P(_Config), i32, i32, P(ctypes.c_size_t)],
        "qevict_prefill_scores": [vp, vp, i32, vp, i32, vp, ctypes.c_size_t, vp],
        "qevict_capacities_for_budget": [P(_Config), i64, i32, P(i32), P(i32)],
        "qevict_memory_report": [vp, i32, i32, P(MemoryReport)],
        "qevict_prefill_scores_noalloc": [vp, vp, i32, vp, i32, vp],
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = i32
    lib.qevict_status_string.argtypes = [i32]
    lib.qevict_status_string.restype = ctypes.c_char_p
    lib.qevict_last_error.argtypes = []
    lib.qevict_last_error.restype = ctypes.c_char_p
    if path is None:
        _lib = lib
    return lib


def _check(lib, status: int):
    if status != OK:
        raise QEvictError(status, lib.qevict_last_error().decode())


def workspace_size(cfg: Config) -> int:
    lib = load_library()
    n = ctypes.c_size_t()
    _check(lib, lib.qevict_workspace_size(ctypes.byref(cfg.to_c()), ctypes.byref(n)))
    return n.value


def capacities_for_budget(cfg: Config, budget_bytes: int, q_permille: int) -> tuple[int, int]:
    """(K_f, K_q) from a per-layer, per-sequence byte budget and quantized share q (thousandths)."""
    lib = load_library()
    kf, kq = ctypes.c_int32(), ctypes.c_int32()
    _check(lib, lib.qevict_capacities_for_budget(ctypes.byref(cfg.to_c()), budget_bytes, q_permille,
                                                 ctypes.byref(kf), ctypes.byref(kq)))
    return kf.value, kq.value


def prefill_scores_scratch_size(cfg: Config, prompt_len: int, n_obs: int) -> int:
    lib = load_library()
    n = ctypes.c_size_t()
    _check(lib, lib.qevict_prefill_scores_scratch_size(ctypes.byref(cfg.to_c()), prompt_len, n_obs,
                                                       ctypes.byref(n)))
    return n.value


def _ptr(t, torch_dtype=None, name="tensor", shape=None):
    """Device address of a contiguous tensor; with `shape`, the tensor must hold
    exactly that many elements (the kernels read and write whole extents)."""
    if not t.is_cuda or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous device tensor")
    if torch_dtype is not None and t.dtype != torch_dtype:
        raise ValueError(f"{name} must be {torch_dtype}, got {t.dtype}")
    if shape is not None and t.numel() != math.prod(shape):
        raise ValueError(f"{name} must hold {' x '.join(map(str, shape))} values, "
                         f"got shape {tuple(t.shape)}")
    return ctypes.c_void_p(t.data_ptr())


class Cache:
    """One tiered KV cache (all layers and sequences) in a torch-owned workspace."""

    def __init__(self, cfg: Config, device="cuda", stream=None):
        import torch

        self.torch = torch
        self.lib = load_library()
        self.cfg = cfg
        self.device = torch.device(device)
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
        self.workspace = torch.empty(workspace_size(cfg), dtype=torch.uint8, device=self.device)
        h = ctypes.c_void_p()
        _check(self.lib, self.lib.qevict_cache_init(
            ctypes.byref(cfg.to_c()), ctypes.c_void_p(self.workspace.data_ptr()),
            self.workspace.numel(), ctypes.c_void_p(self.stream.cuda_stream), ctypes.byref(h)))
        self.handle = h
        gr = cfg.group_size or (32 if cfg.window_tokens == 8 else cfg.window_tokens)
        self.n_cap = -(-(cfg.max_context - cfg.sink_tokens) // cfg.window_tokens)
        self._gr = gr

    # -- lifecycle --
    def close(self):
        if getattr(self, "handle", None):
            self.lib.qevict_cache_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _c(self, status):
        _check(self.lib, status)

    # -- the decode path --
    def prefill_assign(self, layer: int, k, v, init_scores=None):
        """k, v: bf16 [B, H_kv, T, d]; init_scores: float32 [B, n_w] (None with
        the key-norm score)."""
        t = self.torch
        c = self.cfg
        if k.dim() != 4:
            raise ValueError(f"k must be [B, H_kv, T, d], got shape {tuple(k.shape)}")
        T = k.shape[2]
        kv = (c.batch, c.num_kv_heads, T, c.head_dim)
        n_w = max(0, -(-(T - c.sink_tokens) // c.window_tokens))
        sc = None if init_scores is None or init_scores.numel() == 0 else \
            _ptr(init_scores, t.float32, "init_scores", (c.batch, n_w))
        self._c(self.lib.qevict_prefill_assign(
            self.handle, layer, _ptr(k, t.bfloat16, "k", kv), _ptr(v, t.bfloat16, "v", kv), T, sc))

    def prefill_scores(self, q_obs, k, scores=None, scratch=None):
        """Initial window scores from the observation queries' attention.
        q_obs: bf16 [B, H_q, n_obs, d]; k: bf16 [B, H_kv, T, d]; returns float32
        [B, n_w] (written into `scores` when given)."""
        t = self.torch
        cfg = self.cfg
        B, n_obs, T = cfg.batch, q_obs.shape[2], k.shape[2]
        if tuple(q_obs.shape) != (B, cfg.num_q_heads, n_obs, cfg.head_dim):
            raise ValueError(f"q_obs shape {tuple(q_obs.shape)}")
        if tuple(k.shape) != (B, cfg.num_kv_heads, T, cfg.head_dim):
            raise ValueError(f"k shape {tuple(k.shape)}")
        n_w = max(0, -(-(T - cfg.sink_tokens) // cfg.window_tokens))
        if scores is None:
            scores = t.empty((B, n_w), dtype=t.float32, device=self.device)
        if scores.numel() != B * n_w:
            raise ValueError(f"scores must hold {B} x {n_w} values")
        need = prefill_scores_scratch_size(cfg, T, n_obs)
        if scratch is None:
            scratch = t.empty(need, dtype=t.uint8, device=self.device)
        self._c(self.lib.qevict_prefill_scores(
            self.handle, _ptr(q_obs, t.bfloat16, "q_obs"), n_obs, _ptr(k, t.bfloat16, "k"), T,
            _ptr(scratch, None, "scratch"), scratch.numel() * scratch.element_size(),
            _ptr(scores, t.float32, "scores") if n_w else None))
        return scores

    def prefill_scores_noalloc(self, q_obs, k, scores):
        """qevict_prefill_scores on the library's fixed per-device scratch (no
        scratch argument; the call allocates nothing).  q_obs: bf16
        [B, H_q, n_obs, d]; k: bf16 [B, H_kv, T, d]; scores: float32 [B, n_w]."""
        t = self.torch
        cfg = self.cfg
        B, n_obs, T = cfg.batch, q_obs.shape[2], k.shape[2]
        if tuple(q_obs.shape) != (B, cfg.num_q_heads, n_obs, cfg.head_dim):
            raise ValueError(f"q_obs shape {tuple(q_obs.shape)}")
        if tuple(k.shape) != (B, cfg.num_kv_heads, T, cfg.head_dim):
            raise ValueError(f"k shape {tuple(k.shape)}")
        n_w = max(0, -(-(T - cfg.sink_tokens) // cfg.window_tokens))
        self._c(self.lib.qevict_prefill_scores_noalloc(
            self.handle, _ptr(q_obs, t.bfloat16, "q_obs"), n_obs, _ptr(k, t.bfloat16, "k"), T,
            _ptr(scores, t.float32, "scores", (B, n_w)) if n_w else None))
        return scores

    def memory_report(self, layer: int, seq: int) -> dict:
        """Persistent cache bytes of one (layer, sequence), by component."""
        m = MemoryReport()
        self._c(self.lib.qevict_memory_report(self.handle, layer, seq, ctypes.byref(m)))
        return m.as_dict()

    def decode_attend(self, layer: int, q, k_new, v_new, out):
        t = self.torch
        c = self.cfg
        odt = t.bfloat16 if c.out_dtype == OUT_BF16 else t.float32
        qs, ks = (c.batch, c.num_q_heads, c.head_dim), (c.batch, c.num_kv_heads, c.head_dim)
        self._c(self.lib.qevict_decode_attend(
            self.handle, layer, _ptr(q, t.bfloat16, "q", qs), _ptr(k_new, t.bfloat16, "k_new", ks),
            _ptr(v_new, t.bfloat16, "v_new", ks), _ptr(out, odt, "out", qs)))

    def retier(self, layer: int, stats: bool = False):
        if stats:
            s = RetierStats()
            self._c(self.lib.qevict_retier(self.handle, layer, ctypes.byref(s)))
            return s.as_dict()
        self._c(self.lib.qevict_retier(self.handle, layer, None))
        return None

    def join_routing(self):
        """Order the cache stream after all routing enqueued so far (async routing)."""
        self._c(self.lib.qevict_join_routing(self.handle))

    def quantize_window(self, layer: int, seq: int, window: int):
        self._c(self.lib.qevict_quantize_window(self.handle, layer, seq, window))

    def promote_window(self, layer: int, seq: int, window: int):
        self._c(self.lib.qevict_promote_window(self.handle, layer, seq, window))

    # -- inspection --
    def get_state(self, layer: int, seq: int) -> dict:
        cap = self.n_cap
        tiers = np.zeros(cap, np.int8)
        scores = np.zeros(cap, np.float32)
        ledger = np.zeros(cap, np.int8)
        bits = np.zeros(cap, np.int8)
        n = ctypes.c_int32()
        self._c(self.lib.qevict_get_state(
            self.handle, layer, seq, tiers.ctypes.data_as(ctypes.c_void_p),
            scores.ctypes.data_as(ctypes.c_void_p), ledger.ctypes.data_as(ctypes.c_void_p),
            bits.ctypes.data_as(ctypes.c_void_p), cap, ctypes.byref(n)))
        m = n.value
        return dict(tiers=tiers[:m], scores=scores[:m], ledger=ledger[:m], bits=bits[:m], n=m)

    def export_window(self, layer: int, seq: int, window: int, quant=True, full=False) -> dict:
        h, w, d = self.cfg.num_kv_heads, self.cfg.window_tokens, self.cfg.head_dim
        gr = self._gr
        out = {}
        ptrs = [None] * 6
        if quant:
            out["codes_k"] = np.zeros((h, w, d), np.uint8)
            out["codes_v"] = np.zeros((h, w, d), np.uint8)
            out["meta_k"] = np.zeros((h, 2, 1, d), np.uint16)   # one key group per channel
            out["meta_v"] = np.zeros((h, 2, w, d // gr), np.uint16)
            for i, k in enumerate(("codes_k", "codes_v", "meta_k", "meta_v")):
                ptrs[i] = out[k].ctypes.data_as(ctypes.c_void_p)
        if full:
            out["full_k"] = np.zeros((h, w, d), np.uint16)
            out["full_v"] = np.zeros((h, w, d), np.uint16)
            ptrs[4] = out["full_k"].ctypes.data_as(ctypes.c_void_p)
            ptrs[5] = out["full_v"].ctypes.data_as(ctypes.c_void_p)
        self._c(self.lib.qevict_export_window(self.handle, layer, seq, window, *ptrs))
        return out

    def debug_shift_keys(self, layer: int, seq: int, window: int, delta):
        dlt = np.ascontiguousarray(delta, dtype=np.float32)
        if dlt.size != self.cfg.num_kv_heads * self.cfg.head_dim:
            raise ValueError(f"delta must hold H_kv x d values, got shape {dlt.shape}")
        self._c(self.lib.qevict_debug_shift_keys(self.handle, layer, seq, window,
                                                 dlt.ctypes.data_as(ctypes.c_void_p)))

    ROUTING_SYNC, ROUTING_GATE, ROUTING_QUEUE_WAIT = 0, 1, 2

    def routing_order(self) -> int:
        o = ctypes.c_int32()
        self._c(self.lib.qevict_routing_order(self.handle, ctypes.byref(o)))
        return o.value

    def debug_routing_gate(self, timeout_us: int, release: bool):
        self._c(self.lib.qevict_debug_routing_gate(self.handle, int(timeout_us), int(bool(release))))

    def debug_last_masses(self, layer: int) -> np.ndarray:
        c = self.cfg
        m = np.zeros((c.batch, c.num_q_heads, self.n_cap + 1), np.float32)
        self._c(self.lib.qevict_debug_last_masses(self.handle, layer, m.ctypes.data_as(ctypes.c_void_p)))
        return m

    def debug_masses(self, layer: int) -> np.ndarray:
        c = self.cfg
        m = np.zeros((c.batch, c.num_q_heads, self.n_cap + 1), np.float32)
        self._c(self.lib.qevict_debug_masses(self.handle, layer, m.ctypes.data_as(ctypes.c_void_p),
                                             self.n_cap))
        return m

    def profile_enable(self, on: bool = True):
        self._c(self.lib.qevict_profile_enable(self.handle, 1 if on else 0))

    def profile_read(self, kernel: int):
        ms, n = ctypes.c_double(), ctypes.c_int64()
        self._c(self.lib.qevict_profile_read(self.handle, kernel, ctypes.byref(ms), ctypes.byref(n)))
        return ms.value, n.value

    def last_attend_bytes(self, layer: int) -> int:
        n = ctypes.c_int64()
        self._c(self.lib.qevict_last_attend_bytes(self.handle, layer, ctypes.byref(n)))
        return n.value
