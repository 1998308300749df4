"""Seeded synthetic workloads for the QEvict tiered decode step.

This module only draws random numbers and shapes them; it holds none of the
method's arithmetic (no attention, no scoring, no quantization, no routing).
Both the oracle-side tests and the GPU path consume the arrays it produces.

Workload shapes follow the paper's evaluation models (Llama-3-8B head layout,
RULER-style 32K context, a 70B-style GQA-8 layout); the tensors themselves
stand in for real KV activations, which are not available here.  Every array
is a deterministic function of (config id, seed, sequence, layer, stream).

Value types: bf16 tensors are returned as ``uint16`` bit patterns (rounded to
nearest-even from float32 by ``f32_to_bf16_bits``); scores are float32.
"""
from __future__ import annotations

import dataclasses
import math
from fractions import Fraction

import numpy as np

__all__ = [
    "Workload", "WORKLOADS", "get_workload", "f32_to_bf16_bits", "bf16_bits_to_f32",
    "prompt_kv", "decode_inputs", "init_scores", "shift_delta", "pick_shift_window",
    "observation_queries",
]

# stream identifiers inside one (config, seed, seq, layer) seed sequence
_S_PROMPT_K, _S_PROMPT_V, _S_DRIFT, _S_INIT, _S_DEC_Q, _S_DEC_K, _S_DEC_V, _S_OUTLIER, _S_SHIFT, \
    _S_OBS_Q = range(10)


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic decode workload (all sequences share prompt length)."""
    name: str
    config_id: int
    batch: int
    layers: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    prompt_len: int
    window: int              # W: tokens per window
    group: int               # G: value quantization group (channels); keys group over the window
    bits: int                # 4, 2, or 42 (= int4 for the top half of the quantized tier, int2 below)
    frac_full: str           # fraction of prefill windows kept in bf16 (decimal string, exact)
    frac_quant: str          # fraction kept quantized
    steps: int               # decode steps
    retier_interval: int     # R: steps between routing events
    sink: int = 0
    recent: int = 0
    key_dist: str = "normal"         # "normal" | "student_t3"
    outlier_frac: float = 0.0        # fraction of (kv head, channel) key channels scaled up
    outlier_scale: float = 1.0
    drift: bool = False              # rotating query mean
    drift_amp: float = 0.0
    drift_omega: float = 0.0
    forced_shift: bool = False       # periodic key shift on low-ranked quantized windows
    shift_every: int = 4
    shift_scale: float = 3.0
    init_sigma: float = 1.0          # log-normal spread of the prefill window scores
    budget_frac: str = ""            # byte budget as a fraction of the full cache (capacities
    q_frac: str = ""                 # from the byte-budget equation), and the quantized share

    @property
    def gqa(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    @property
    def n_hist_windows(self) -> int:
        """Complete windows in the prompt outside the sink and recent regions."""
        n = self.prompt_len - self.sink - self.recent
        return max(n, 0) // self.window

    @property
    def n_prompt_windows(self) -> int:
        """Windows touched by the prompt (complete or partial), outside the sink."""
        n = self.prompt_len - self.sink
        return max(0, -(-n // self.window))

    @property
    def capacity_full(self) -> int:
        return math.floor(Fraction(self.frac_full) * self.n_hist_windows)

    @property
    def capacity_quant(self) -> int:
        return math.floor(Fraction(self.frac_quant) * self.n_hist_windows)

    @property
    def max_context(self) -> int:
        return self.prompt_len + self.steps

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


def _drift_defaults():
    # Rotating query mean: amplitude and angular speed (radians per decode step).
    # Chosen by running the oracle on the 8B/32K shape: with A = 24 and
    # omega = 0.1, quantized->bf16 promotions average 2.06 per step over decode
    # steps 16..64 (A = 2 / 8 / 16 gave 0.2 / 0.35 / 1.0 per step).
    return dict(drift=True, drift_amp=24.0, drift_omega=0.1)


WORKLOADS = {
    # 1 layer, batch 1, 8/8 heads, 2048-token context, 64 windows of 32;
    # 16 bf16 + 24 int4 windows; 16 steps; periodic forced promotions.
    "c1": Workload("c1", 1, batch=1, layers=1, num_q_heads=8, num_kv_heads=8, head_dim=128,
                   prompt_len=2048, window=32, group=32, bits=4, frac_full="0.25",
                   frac_quant="0.375", steps=16, retier_interval=1, forced_shift=True),
    # Llama-3-8B-shaped layer: 32/8 heads, 32K context, 20% bf16 / 30% int4 / 50% evicted.
    "c2": Workload("c2", 2, batch=1, layers=1, num_q_heads=32, num_kv_heads=8, head_dim=128,
                   prompt_len=32768, window=32, group=32, bits=4, frac_full="0.2",
                   frac_quant="0.3", steps=128, retier_interval=1, **_drift_defaults()),
    # all 32 layers, batch 8, independent seeds per (sequence, layer)
    "c3": Workload("c3", 3, batch=8, layers=32, num_q_heads=32, num_kv_heads=8, head_dim=128,
                   prompt_len=32768, window=32, group=32, bits=4, frac_full="0.2",
                   frac_quant="0.3", steps=256, retier_interval=1, **_drift_defaults()),
    # 128K context, windows of 64, int2 group 64; heavy-tailed keys with outlier channels.
    "c4": Workload("c4", 4, batch=1, layers=1, num_q_heads=32, num_kv_heads=8, head_dim=128,
                   prompt_len=131072, window=64, group=64, bits=2, frac_full="0.1",
                   frac_quant="0.3", steps=64, retier_interval=1, key_dist="student_t3",
                   outlier_frac=0.01, outlier_scale=8.0),
    # 70B-shaped layer: 64/8 heads, batch 4, 64K context; mixed int4/int2 tier; routing every 8 steps.
    "c5": Workload("c5", 5, batch=4, layers=1, num_q_heads=64, num_kv_heads=8, head_dim=128,
                   prompt_len=65536, window=32, group=32, bits=42, frac_full="0.2",
                   frac_quant="0.4", steps=128, retier_interval=8, **_drift_defaults()),
    # The paper's default operating point on the 8B shape: five sink tokens, 32 recent
    # tokens, routing every 8 steps, int2 tier, quantized fraction q = 0.70 of the
    # historical byte budget (20% of the full cache), windows of 32 (the library's
    # smallest window); capacities from the byte-budget equation.
    "c6": Workload("c6", 6, batch=1, layers=1, num_q_heads=32, num_kv_heads=8, head_dim=128,
                   prompt_len=32768, window=32, group=32, bits=2, frac_full="0", frac_quant="0",
                   steps=128, retier_interval=8, sink=5, recent=32, budget_frac="0.2", q_frac="0.7",
                   **_drift_defaults()),
    # The paper's default point with its 8-token windows (Omega = 8): values in groups
    # of 32 channels, keys per channel across the window; byte-budget capacities.
    "c6w8": Workload("c6w8", 8, batch=1, layers=1, num_q_heads=32, num_kv_heads=8, head_dim=128,
                     prompt_len=32768, window=8, group=32, bits=2, frac_full="0", frac_quant="0",
                     steps=128, retier_interval=8, sink=5, recent=32, budget_frac="0.2", q_frac="0.7",
                     **_drift_defaults()),
}

# Reduced-size variants with the same head layouts and tier policies: they span
# several windows per split and end with a ragged (partial) window, and the
# oracle finishes them in seconds.
WORKLOADS.update({
    "c1s": WORKLOADS["c1"].replace(name="c1s", prompt_len=2048 + 19),
    "c2s": WORKLOADS["c2"].replace(name="c2s", prompt_len=32 * 96 + 13, steps=40),
    "c3s": WORKLOADS["c3"].replace(name="c3s", batch=2, layers=2, prompt_len=32 * 64 + 5, steps=24),
    "c4s": WORKLOADS["c4"].replace(name="c4s", prompt_len=64 * 80 + 37, steps=24),
    "c5s": WORKLOADS["c5"].replace(name="c5s", batch=2, prompt_len=32 * 96 + 29, steps=40),
    "c6s": WORKLOADS["c6"].replace(name="c6s", prompt_len=32 * 96 + 23, steps=40),
    # a sink of two and a half windows, a recent region that is not a whole number
    # of windows, routing every 3 steps, mixed int4 / int2
    "c7s": WORKLOADS["c5"].replace(name="c7s", config_id=7, batch=2, prompt_len=32 * 90 + 3, steps=30,
                                   sink=80, recent=70, retier_interval=3, frac_full="0.2",
                                   frac_quant="0.3"),
    "c6w8s": WORKLOADS["c6w8"].replace(name="c6w8s", prompt_len=8 * 300 + 13, steps=40),
})


def get_workload(name: str) -> Workload:
    return WORKLOADS[name]


def _rng(wl: Workload, seed: int, seq: int, layer: int, stream: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(
        [wl.config_id, seed, seq, layer, stream])))


def f32_to_bf16_bits(x) -> np.ndarray:
    """float32 -> bf16 bit pattern, round to nearest even (finite inputs)."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (b >> 16) & 1          # finite inputs: the sum below stays below 2^32
    r += 0x7FFF
    r += b
    r >>= 16
    return r.astype(np.uint16)


def bf16_bits_to_f32(b) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _outlier_mask(wl: Workload, seed: int, seq: int, layer: int) -> np.ndarray:
    scale = np.ones((wl.num_kv_heads, wl.head_dim), dtype=np.float32)
    n = int(round(wl.outlier_frac * wl.num_kv_heads * wl.head_dim))
    if n:
        idx = _rng(wl, seed, seq, layer, _S_OUTLIER).choice(
            wl.num_kv_heads * wl.head_dim, size=n, replace=False)
        scale.reshape(-1)[idx] = wl.outlier_scale
    return scale


def _keys(wl: Workload, rng: np.random.Generator, shape, scale) -> np.ndarray:
    """Keys of the workload's distribution, drawn one leading-axis slice at a time."""
    out = np.empty(shape, dtype=np.float32)
    for i in range(shape[0]):
        x = rng.standard_normal(shape[1:], dtype=np.float32)
        if wl.key_dist == "student_t3":
            # Student-t with 3 degrees of freedom: Z / sqrt(chi^2_3 / 3)
            chi = np.zeros(shape[1:], dtype=np.float32)
            for _ in range(3):
                y = rng.standard_normal(shape[1:], dtype=np.float32)
                y *= y
                chi += y
            chi /= 3.0
            np.sqrt(chi, out=chi)
            x /= chi
        elif wl.key_dist != "normal":
            raise ValueError(wl.key_dist)
        x *= scale[i]
        out[i] = x
    return out


def _normal(rng: np.random.Generator, shape) -> np.ndarray:
    out = np.empty(shape, dtype=np.float32)
    for i in range(shape[0]):
        out[i] = rng.standard_normal(shape[1:], dtype=np.float32)
    return out


def prompt_kv(wl: Workload, seed: int, seq: int, layer: int):
    """Prompt keys and values, bf16 bits, shape [H_kv, prompt_len, d]."""
    shape = (wl.num_kv_heads, wl.prompt_len, wl.head_dim)
    scale = _outlier_mask(wl, seed, seq, layer)[:, None, :]
    k = f32_to_bf16_bits(_keys(wl, _rng(wl, seed, seq, layer, _S_PROMPT_K), shape, scale))
    v = f32_to_bf16_bits(_normal(_rng(wl, seed, seq, layer, _S_PROMPT_V), shape))
    return k, v


def _drift_basis(wl: Workload, seed: int, seq: int, layer: int):
    a = _rng(wl, seed, seq, layer, _S_DRIFT).standard_normal((2, wl.head_dim))
    u = a[0] / np.linalg.norm(a[0])
    v = a[1] - (a[1] @ u) * u
    v /= np.linalg.norm(v)
    return u, v


def decode_inputs(wl: Workload, seed: int, seq: int, layer: int, steps: int | None = None):
    """Per-step queries and new keys / values for decode steps 1..steps.

    Returns bf16 bits: q [steps, H_q, d], k [steps, H_kv, d], v [steps, H_kv, d].
    With drift, q_{t,h} = mu_t + eps, mu_t = A (cos(w t) u + sin(w t) v), where
    u, v are orthonormal directions shared by all heads of the layer.
    """
    n = wl.steps if steps is None else steps
    qs = _rng(wl, seed, seq, layer, _S_DEC_Q).standard_normal(
        (n, wl.num_q_heads, wl.head_dim), dtype=np.float32)
    if wl.drift:
        u, v = _drift_basis(wl, seed, seq, layer)
        t = np.arange(1, n + 1, dtype=np.float64)[:, None]
        mu = wl.drift_amp * (np.cos(wl.drift_omega * t) * u + np.sin(wl.drift_omega * t) * v)
        qs = qs + mu[:, None, :].astype(np.float32)
    scale = _outlier_mask(wl, seed, seq, layer)
    ks = _keys(wl, _rng(wl, seed, seq, layer, _S_DEC_K), (n, wl.num_kv_heads, wl.head_dim),
               np.broadcast_to(scale, (n,) + scale.shape))
    vs = _normal(_rng(wl, seed, seq, layer, _S_DEC_V), (n, wl.num_kv_heads, wl.head_dim))
    return f32_to_bf16_bits(qs), f32_to_bf16_bits(ks), f32_to_bf16_bits(vs)


def observation_queries(wl: Workload, seed: int, seq: int, layer: int, n_obs: int) -> np.ndarray:
    """Queries of the last n_obs prompt positions, bf16 bits [H_q, n_obs, d].

    The decode query recipe continued backwards: i.i.d. normal, plus (with
    drift) the rotating mean at steps 1 - n_obs .. 0.
    """
    qs = _rng(wl, seed, seq, layer, _S_OBS_Q).standard_normal(
        (wl.num_q_heads, n_obs, wl.head_dim), dtype=np.float32)
    if wl.drift:
        u, v = _drift_basis(wl, seed, seq, layer)
        t = np.arange(1 - n_obs, 1, dtype=np.float64)[:, None]
        mu = wl.drift_amp * (np.cos(wl.drift_omega * t) * u + np.sin(wl.drift_omega * t) * v)
        qs = qs + mu[None, :, :].astype(np.float32)
    return f32_to_bf16_bits(qs)


def init_scores(wl: Workload, seed: int, seq: int, layer: int) -> np.ndarray:
    """Prefill window scores, float32 [n_prompt_windows].

    A heavy-tailed (log-normal) positive score per window, normalised so the
    scores sum to W: the size of mass that W observation queries would hand
    out.  The prompt-scoring step itself sits outside the decode path; these
    values are inputs to it.
    """
    n = wl.n_prompt_windows
    z = _rng(wl, seed, seq, layer, _S_INIT).standard_normal(n)
    x = np.exp(wl.init_sigma * z)
    return (wl.window * x / x.sum()).astype(np.float32)


def pick_shift_window(wl: Workload, seed: int, seq: int, layer: int, event: int,
                      quant_windows_low_to_high) -> int:
    """Choose the window whose keys get shifted before a forced-promotion step.

    ``quant_windows_low_to_high`` lists the currently quantized windows from
    the lowest-ranked upward.  One of the lowest ceil(K_q / 4) is drawn
    uniformly (a seeded draw per event).
    """
    cands = list(quant_windows_low_to_high)[: max(1, -(-wl.capacity_quant // 4))]
    r = _rng(wl, seed, seq, layer, _S_SHIFT + 16 * (event + 1))
    return int(cands[int(r.integers(len(cands)))])


def shift_delta(wl: Workload, q_bits_step: np.ndarray) -> np.ndarray:
    """Key shift per KV head toward that step's query direction, float32 [H_kv, d].

    delta_g = shift_scale * sqrt(d) * qbar_g / |qbar_g|: the scale is counted in
    units of the norm of an N(0, I) key (sqrt(d)).  qbar_g is the mean query of
    the heads in KV group g (the single query head when GQA is 1).
    """
    q = bf16_bits_to_f32(q_bits_step).astype(np.float64).reshape(
        wl.num_kv_heads, wl.gqa, wl.head_dim).mean(axis=1)
    q /= np.linalg.norm(q, axis=1, keepdims=True)
    return (wl.shift_scale * np.sqrt(wl.head_dim) * q).astype(np.float32)
