"""QEvict per-decode-step method as a plain float64 CPU oracle.

TEST INFRASTRUCTURE.  This module exists to check the GPU path: only tests,
``__graft_entry__.smoke()`` and the benchmark's CPU-baseline leg may import or
run it.  It shares no code with the GPU library and imports nothing from it.

What it computes, and where the paper defines it (QEvict, arXiv 2608.05326):

* Decode attention of each query head over the accessible keys and values,
  softmax(q K^T / sqrt(d)) V, with grouped KV heads (Sec. 4.1, Preliminaries).
* The cache partition into sink, recent region and windows, with each
  historical window Full, Quantized or Evicted (Sec. 4.3, partition equation).
* The cumulative window score: each window's attention mass averaged over the
  H_q query heads, added at every decode step (Sec. 4.2, cumulative window
  score equation; the per-step reading is listed with the other readings).
  Optionally the exponentially decayed score S_t = lambda S_{t-R} + u_t of the
  appendix on alternative ranking functions (decayed score equation), u_t the
  attention a window received since the previous routing event, the
  attention p-norm (sum over routing periods r of u_r^p)^(1/p) (p-norm
  equation), or the attention-free key-norm score of the same appendix
  (key-norm equation).
* Routing: the candidate pool is the previous Full and Quantized windows plus
  the windows that left the recent region; the top K_f by score go to Full,
  the next K_q to Quantized, the rest are evicted (Sec. 4.3, candidate pool
  and TopK equations; Algorithm 1).
* Initial window scores from prompt attention: the mean over query heads of
  the causal attention mass that the last n_obs prompt queries put on each
  window (Sec. 4.2: prompt attention initialises the scores; the observation
  window is a reading).
* RoPE-aware Quantized tier (Sec. 4.3: keys are quantized in the pre-RoPE
  domain and re-rotated at their original positions after dequantization):
  the cache receives keys as attention consumes them (post-RoPE); a window's
  first quantization un-rotates them, and dequantized keys are rotated back
  for attention and for promotion.
* Migration-stable asymmetric quantization: keys per channel across tokens,
  values per token across channels; codes are produced once, at a window's
  first demotion, and reused on every later move; promotion reconstructs the
  low-bit values in bf16 and keeps the codes dormant (Sec. 4.3, paragraph on
  migration-stable quantization; Algorithm 1).

Everything is float64 except where the method stores a narrower format:
bf16 keys/values, fp16 quantization scale and zero point, integer codes.
Those roundings are exact (see ``numerics``).

Readings where the paper is silent (window size W and routing interval R are
separate parameters; scale/zero rounding; tie-breaks; mixed-precision rule;
one-way policy) are spelled out next to the code that takes them.
"""
from __future__ import annotations

import dataclasses
import math
from fractions import Fraction

import numpy as np

from .numerics import FP16_MAX, rd_fp16, rne_bf16, rne_fp16, ru_fp16

__all__ = [
    "OPEN", "AGED", "FULL", "QUANT", "EVICTED", "ACTIVE", "DORMANT",
    "OracleConfig", "QEvictUnit", "quantize_groups", "quantize_window",
    "dequantize_window", "route_order", "tier_split", "QuantRangeError", "CapacityError",
    "prefill_window_scores", "window_costs", "tier_capacities", "memory_report",
    "rope_cos_sin", "rope_rotate", "rope_unrotate_f32",
]

# window states; OPEN and AGED are both inside / just out of the recent region
OPEN, AGED, FULL, QUANT, EVICTED = 0, 1, 2, 3, 4
# ledger entry states (Algorithm 1: an entry is active, dormant, or absent)
ACTIVE, DORMANT = 1, 2


class QuantRangeError(ValueError):
    """A group's values fall outside the fp16 range of the scale/zero point."""


class CapacityError(ValueError):
    """A single-window move would put more than K_f / K_q windows in a tier."""


@dataclasses.dataclass
class OracleConfig:
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    window: int                   # W, tokens per window
    group: int                    # G, quantization group length
    bits: int                     # 4, 2, or 42 (mixed: int4 for the upper half of the quantized tier)
    capacity_full: int            # K_f
    capacity_quant: int           # K_q
    sink: int = 0
    recent: int = 0
    softmax_scale: float | None = None   # default 1/sqrt(head_dim)
    no_promotion: bool = False    # one-way Full -> Quantized -> Evicted policy
    score_decay: float = 1.0      # lambda of the decayed score; 1.0 = cumulative score
    key_norm: bool = False        # key-norm score instead of attention
    score_p: float = 0.0          # p of the attention p-norm score; 0 = not used
    rope_base: float = 0.0        # RoPE base of the Quantized tier's keys; 0 = no RoPE

    @property
    def scale(self) -> float:
        return self.softmax_scale if self.softmax_scale else 1.0 / math.sqrt(self.head_dim)

    @property
    def gqa(self) -> int:
        return self.num_q_heads // self.num_kv_heads


# ----------------------------------------------------------------------------
# Quantization (Sec. 4.3, migration-stable quantization)
# ----------------------------------------------------------------------------

def _fp16_step(v: np.ndarray, direction: int) -> np.ndarray:
    """Next fp16 value above (direction=+1) or below (-1) each non-negative v."""
    b = v.astype(np.float16).view(np.uint16).astype(np.int32)
    b = np.where(direction > 0, b + 1, np.maximum(b - 1, 0))
    return b.astype(np.uint16).view(np.float16).astype(np.float64)


def quantize_groups(x, bits: int):
    """Asymmetric b-bit quantization of every row of ``x`` (one row = one group).

    Reading of the paper's "asymmetric low-bit quantization" with fp16
    parameters:
      z = largest fp16 value <= min(x)            (zero point, rounded down)
      s = smallest fp16 value >= 0 with z + s (2^b - 1) >= max(x)
      c = round-half-even((x - z) / s), and c = 0 for every element when s = 0.
    Then 0 <= c <= 2^b - 1 and |x - (z + s c)| <= s / 2 for every element.

    Exactness: z and s are fp16 values (multiples of 2^-24 below 2^16 in
    magnitude), so z + k s / 2 for an integer k <= 31 is a multiple of 2^-25
    below 2^21 and is exact in float64.  The scale test and every rounding
    boundary of the codes are therefore compared exactly; the float64
    quotient only supplies a first guess that the comparisons correct.
    """
    x = np.asarray(x, dtype=np.float64)
    if x.ndim != 2:
        raise ValueError("expected [groups, group_len]")
    n = float(2 ** bits - 1)
    lo = x.min(axis=1)
    hi = x.max(axis=1)
    if np.any(lo < -FP16_MAX) or np.any(hi > FP16_MAX) or not np.all(np.isfinite(x)):
        raise QuantRangeError("group outside the fp16 range")
    z = rd_fp16(lo)
    s = ru_fp16((hi - z) / n)
    for _ in range(4):   # at most one fp16 step away; loop until stable
        small = z + s * n < hi
        s = np.where(small, _fp16_step(s, +1), s)
        prev = _fp16_step(s, -1)
        big = (s > 0) & (z + prev * n >= hi)
        s = np.where(big, prev, s)
        if not (small.any() or big.any()):
            break
    assert np.all(z + s * n >= hi) and np.all((s == 0) | (z + _fp16_step(s, -1) * n < hi))

    zc = z[:, None]
    sc = np.where(s > 0, s, 1.0)[:, None]
    c = np.rint((x - zc) / sc)
    for _ in range(4):
        lower = zc + (c - 0.5) * sc
        upper = zc + (c + 0.5) * sc
        moved = (x < lower) | (x > upper)
        c = np.where(x < lower, c - 1, np.where(x > upper, c + 1, c))
        if not moved.any():
            break
    lower = zc + (c - 0.5) * sc
    upper = zc + (c + 0.5) * sc
    assert np.all((x >= lower) & (x <= upper))
    odd = np.mod(c, 2) == 1
    c = np.where((x == upper) & odd, c + 1, c)      # tie at c + 1/2: go to the even neighbour
    c = np.where((x == lower) & odd, c - 1, c)      # tie at c - 1/2
    c = np.where(s[:, None] > 0, c, 0.0)
    assert np.all((c >= 0) & (c <= n))
    return z, s, c.astype(np.int64)


def quantize_window(k, v, bits: int, group: int) -> dict:
    """Quantize one window: k, v float64 [H_kv, W, d] (bf16 values).

    Keys: one group per (KV head, channel) across the window's W tokens ->
    per-channel scale/zero across the token dimension.  Values: one group per
    (KV head, token, G consecutive channels) -> per-token scale/zero across
    channels (Sec. 4.3, migration-stable quantization; the group sizes are
    readings: the window for keys, G for values).
    """
    h, w, d = k.shape
    if d % group:
        raise ValueError("the value group must divide the head dim")
    kg = k.transpose(0, 2, 1).reshape(-1, w)            # [H_kv * d, W]: one row per channel
    kz, ks, kc = quantize_groups(kg, bits)
    kc = kc.reshape(h, d, w).transpose(0, 2, 1)
    vg = v.reshape(-1, group)
    vz, vs, vc = quantize_groups(vg, bits)
    return dict(bits=bits, group=group,
                kz=kz.reshape(h, 1, d), ks=ks.reshape(h, 1, d), kc=kc,
                vz=vz.reshape(h, w, d // group), vs=vs.reshape(h, w, d // group),
                vc=vc.reshape(h, w, d), state=ACTIVE)


def dequantize_window(e: dict):
    """x_hat = z + s c for keys and values (exact in float64)."""
    g = e["group"]
    vz = np.repeat(e["vz"], g, axis=2)
    vs = np.repeat(e["vs"], g, axis=2)
    return e["kz"] + e["ks"] * e["kc"], vz + vs * e["vc"]


# ----------------------------------------------------------------------------
# Rotary position embedding of the Quantized tier (Sec. 4.3)
# ----------------------------------------------------------------------------
# Half-split RoPE over d channels: channel i < d/2 pairs with i + d/2 and turns
# by the angle p * base^(-2i/d) at position p.  cos and sin are taken in
# float64 from the C library (Python's math module) and stored as float32, the
# table both sides use.

def rope_cos_sin(base: float, head_dim: int, positions):
    """float32 cos, sin [len(positions), head_dim / 2]."""
    half = head_dim // 2
    inv = [math.pow(base, -2.0 * i / head_dim) for i in range(half)]
    cs = np.empty((len(positions), half), dtype=np.float32)
    sn = np.empty((len(positions), half), dtype=np.float32)
    for r, p in enumerate(positions):
        for i in range(half):
            ang = float(p) * inv[i]
            cs[r, i] = math.cos(ang)
            sn[r, i] = math.sin(ang)
    return cs, sn


def rope_rotate(x, cos, sin):
    """R(p) x in float64 (each product and sum rounded in float64).
    x [H, n, d]; cos, sin [n, d/2] (float32 values)."""
    h = x.shape[-1] // 2
    c = cos.astype(np.float64)[None]
    s = sin.astype(np.float64)[None]
    a, b = x[..., :h], x[..., h:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def rope_unrotate_f32(x, cos, sin):
    """R(-p) x with every product and sum rounded to float32 (x holds bf16 values)."""
    h = x.shape[-1] // 2
    a = x[..., :h].astype(np.float32)
    b = x[..., h:].astype(np.float32)
    c, s = cos[None], sin[None]
    return np.concatenate([a * c + b * s, b * c - a * s], axis=-1)


# ----------------------------------------------------------------------------
# Byte-constrained tier allocation (Sec. 4.3; memory accounting appendix)
# ----------------------------------------------------------------------------

def window_costs(num_kv_heads: int, head_dim: int, window: int, group: int, bits: int):
    """Bytes one window occupies in the Full tier (M_f) and in the Quantized tier
    (M_q), for one layer and sequence.

    Full: bf16 keys and values, plus a slot index and a position (4 bytes each).
    Quantized: packed b-bit codes of keys and values (b = 4 for the mixed
    int4/int2 tier, whose slots hold the larger record), fp16 scale and zero
    point per key group (one per channel) and per value group (token x d/G
    channel groups), slot index and position, and a 2-byte ledger entry
    (state, bit width) -- the codes, parameters, positions and persistent
    indexing state the paper lists.
    """
    b = 2 if bits == 2 else 4
    kv_elems = 2 * num_kv_heads * window * head_dim
    m_f = 2 * kv_elems + 4 + 4
    params = 2 * 2 * num_kv_heads * head_dim \
        + 2 * 2 * num_kv_heads * window * (head_dim // group)
    m_q = kv_elems * b // 8 + params + 4 + 4 + 2
    return m_f, m_q


def tier_capacities(budget_bytes: int, q_permille: int, num_kv_heads: int, head_dim: int,
                    window: int, group: int, bits: int, sink: int, recent: int):
    """K_f = floor((1 - q) B_hist / M_f), K_q = floor(q B_hist / M_q) (tier
    capacities equation), B_hist = the budget left after the protected sink and
    recent tokens (bf16 keys and values).  Exact rational arithmetic."""
    protected = 2 * 2 * num_kv_heads * head_dim * (sink + recent)
    if budget_bytes < protected:
        raise ValueError("budget below the protected regions")
    b_hist = budget_bytes - protected
    q = Fraction(q_permille, 1000)
    m_f, m_q = window_costs(num_kv_heads, head_dim, window, group, bits)
    return math.floor((1 - q) * b_hist / m_f), math.floor(q * b_hist / m_q)


def memory_report(unit: "QEvictUnit") -> dict:
    """Persistent bytes of a unit by the memory accounting appendix's terms:
    sink and recent tokens (bf16 K and V), Full windows, Quantized codes and
    their scale / zero points, 8 bytes of slot index and position per Full or
    Quantized window, and the ledger: dormant entries keep their codes and
    parameters, every entry costs 2 bytes.  "recent" counts the tokens after
    the windows that have been routed."""
    c = unit.cfg
    H, d, W, G = c.num_kv_heads, c.head_dim, c.window, c.group
    tok = 2 * 2 * H * d
    meta = 2 * 2 * H * d + 2 * 2 * H * W * (d // G)
    r = dict(sink=tok * min(c.sink, unit.T), recent=0, full=0, quant_codes=0, quant_meta=0,
             position=0, ledger=0)
    routed = int(np.sum((unit.state == FULL) | (unit.state == QUANT) | (unit.state == EVICTED)))
    r["recent"] = tok * max(0, unit.T - c.sink - W * routed)
    for w in np.nonzero(unit.state >= 0)[0]:
        st = unit.state[w]
        if st == FULL:
            r["full"] += tok * W
            r["position"] += 8
        elif st == QUANT:
            e = unit.ledger[w]
            r["quant_codes"] += 2 * H * W * d * e["bits"] // 8
            r["quant_meta"] += meta
            r["position"] += 8
    for w, e in unit.ledger.items():
        r["ledger"] += 2
        if e["state"] == DORMANT:
            r["ledger"] += 2 * H * W * d * e["bits"] // 8 + meta
    r["total"] = sum(r.values())
    return r


# ----------------------------------------------------------------------------
# Initial window scores from prompt attention (Sec. 4.2)
# ----------------------------------------------------------------------------

def prefill_window_scores(q_obs, k, sink: int, window: int, scale: float | None = None):
    """Score of every prompt window before the first routing event.

    q_obs: float64 [H_q, n_obs, d], the queries of prompt positions
    T - n_obs .. T - 1; k: float64 [H_kv, T, d] prompt keys (query head h reads
    KV head h // (H_q / H_kv)).  Each observation query attends causally to
    keys 0 .. its own position with softmax(q k^T * scale); the score of window
    w (tokens sink + w W .. sink + (w + 1) W - 1, the last one possibly
    partial) is the attention mass its tokens receive, summed over the
    observation queries and averaged over the H_q heads (the cumulative score of
    Sec. 4.2 with the observation queries in place of decode steps).  Sink
    tokens take part in the softmax and belong to no window.
    Returns float64 [n_w], n_w = ceil((T - sink) / W).
    """
    H_q, n_obs, d = q_obs.shape
    H_kv, T, _ = k.shape
    gqa = H_q // H_kv
    scale = scale if scale else 1.0 / math.sqrt(d)
    n_w = max(0, -(-(T - sink) // window))
    owner = np.full(T, -1)
    owner[sink:] = (np.arange(sink, T) - sink) // window
    scores = np.zeros(n_w)
    for h in range(H_q):
        kk = k[h // gqa]
        for j in range(n_obs):
            tau = T - n_obs + j
            logits = (kk[:tau + 1] @ q_obs[h, j]) * scale
            e = np.exp(logits - logits.max())
            p = e / e.sum()
            win = owner[:tau + 1] >= 0
            scores += np.bincount(owner[:tau + 1][win], weights=p[win], minlength=n_w)
    return scores / H_q


# ----------------------------------------------------------------------------
# Routing (Sec. 4.3 candidate pool and TopK equations; Algorithm 1)
# ----------------------------------------------------------------------------

def route_order(cands, scores) -> list:
    """Candidates by descending score; equal scores go to the lower window index."""
    return sorted(cands, key=lambda w: (-scores[w], w))


def tier_split(order, k_f: int, k_q: int, was_quantized=frozenset(), no_promotion=False):
    """F = top K_f, Q = next K_q of the rest, E = remainder.

    One-way policy reading: a window already in the quantized tier may not be
    chosen for Full, so Full takes the top K_f of the candidates that are not
    quantized; Quantized then takes the top K_q of everything else.
    """
    if no_promotion:
        full = [w for w in order if w not in was_quantized][:k_f]
    else:
        full = list(order[:k_f])
    fs = set(full)
    rest = [w for w in order if w not in fs]
    quant = rest[:k_q]
    evict = rest[k_q:]
    return full, quant, evict


# ----------------------------------------------------------------------------
# One (sequence, layer) cache
# ----------------------------------------------------------------------------

class QEvictUnit:
    """The tiered cache of one sequence in one layer, stepped in float64."""

    def __init__(self, cfg: OracleConfig, max_tokens: int):
        self.cfg = cfg
        c = cfg
        self.max_tokens = max_tokens
        self.n_win_cap = max(0, -(-(max_tokens - c.sink) // c.window))
        # original bf16 keys / values of every token ever appended
        self.k = np.zeros((c.num_kv_heads, max_tokens, c.head_dim))
        self.v = np.zeros((c.num_kv_heads, max_tokens, c.head_dim))
        # every token position as attention reads it now: the originals for sink,
        # open and aged tokens, the bf16 copy for Full windows, z + s c for
        # Quantized ones; att_live marks the positions attention sees (evicted
        # windows' rows are masked out).  Refreshed whenever a window changes tier
        # or its ledger changes (see _refresh); accessible() is the same set
        # assembled from the tier map.
        self.att_k = np.zeros((c.num_kv_heads, max_tokens, c.head_dim))
        self.att_v = np.zeros((c.num_kv_heads, max_tokens, c.head_dim))
        self.att_live = np.zeros(max_tokens, dtype=bool)
        self.owner = np.full(max_tokens, -1, dtype=np.int64)   # window of each position, -1 = sink
        if max_tokens > c.sink:
            self.owner[c.sink:] = (np.arange(c.sink, max_tokens) - c.sink) // c.window
        self.T = 0
        self.state = np.full(self.n_win_cap, -1, dtype=np.int64)   # -1: not started
        self.score = np.zeros(self.n_win_cap)
        self.full_k: dict[int, np.ndarray] = {}
        self.full_v: dict[int, np.ndarray] = {}
        self.ledger: dict[int, dict] = {}
        self.stats = dict(promotions=0, admissions_full=0, first_quantizations=0,
                          reactivations=0, evictions=0)
        self.quant_count = 0          # quantizations performed over the lifetime
        # decayed score: the first step after a routing event (or prefill) starts a new
        # period, S = lambda S_previous_event + (attention received during the period)
        self.new_period = False
        # p-norm score: u of every completed routing period, per window, and the
        # attention received in the period in progress
        self.u_hist: list[list[float]] = [[] for _ in range(self.n_win_cap)]
        self.u_cur = np.zeros(self.n_win_cap)

    # -- geometry ---------------------------------------------------------
    def win_range(self, w: int):
        a = self.cfg.sink + w * self.cfg.window
        return a, a + self.cfg.window

    def _rope(self, w: int):
        a, b = self.win_range(w)
        return rope_cos_sin(self.cfg.rope_base, self.cfg.head_dim, range(a, b))

    def _quantize(self, w: int, k, v, bits: int):
        """First quantization of window w from its bf16 keys (as attention uses
        them) and values; with RoPE the keys are first un-rotated (float32) and
        rounded to bf16: the pre-RoPE keys the codes describe."""
        if self.cfg.rope_base:
            k = rne_bf16(rope_unrotate_f32(k, *self._rope(w)).astype(np.float64))
        return quantize_window(k, v, bits, self.cfg.group)

    def _dequantize(self, w: int):
        """Keys and values of a ledger entry in the attention domain (float64):
        with RoPE the keys are rotated back to their positions."""
        kh, vh = dequantize_window(self.ledger[w])
        if self.cfg.rope_base:
            kh = rope_rotate(kh, *self._rope(w))
        return kh, vh

    def _refresh(self, w: int):
        """Rewrite window w's rows of the attention-domain copy from its tier:
        bf16 copy (Full), z + s c (Quantized), originals (open / aged), or
        masked out (Evicted)."""
        a, b = self.win_range(w)
        b = min(b, self.T)
        st = self.state[w]
        if st == EVICTED:
            self.att_live[a:b] = False
            return
        if st == FULL:
            kk, vv = self.full_k[w], self.full_v[w]
        elif st == QUANT:
            kk, vv = self._dequantize(w)
        else:
            kk, vv = self.k[:, a:b], self.v[:, a:b]
        self.att_k[:, a:b] = kk[:, :b - a]
        self.att_v[:, a:b] = vv[:, :b - a]
        self.att_live[a:b] = True

    def _age(self):
        """OPEN -> AGED once a window is complete and older than the recent region."""
        c = self.cfg
        for w in np.nonzero(self.state == OPEN)[0]:
            if self.win_range(w)[1] <= self.T - c.recent:
                self.state[w] = AGED

    def _start_windows(self):
        c = self.cfg
        n = max(0, -(-(self.T - c.sink) // c.window))
        for w in range(n):
            if self.state[w] == -1:
                self.state[w] = OPEN

    # -- prefill (Sec. 4.2: prompt attention initialises the scores and the first assignment)
    def prefill(self, k, v, init_scores, route=True):
        """k, v: float64 [H_kv, T, d] bf16 values; init_scores: per window
        (unused with the key-norm score, which the keys determine).  With
        route=False the first assignment waits for finish_prefill(), so that a
        lockstep comparison can look at the scores first."""
        c = self.cfg
        T = k.shape[1]
        self.k[:, :T] = k
        self.v[:, :T] = v
        self.att_k[:, :T] = k
        self.att_v[:, :T] = v
        self.att_live[:T] = True
        self.T = T
        self._start_windows()
        n = int(np.sum(self.state >= 0))
        if c.key_norm:
            for w in range(n):
                a, b = self.win_range(w)
                self.score[w] = -self._key_norms(a, min(b, T)).sum() / c.window
        else:
            init = np.asarray(init_scores, dtype=np.float64)
            self.score[:n] = init[:n]
            if c.score_p:                 # prompt attention is the first period's u
                if np.any(init[:n] < 0):
                    raise ValueError("p-norm score: negative initial score")
                for w in range(n):
                    self.u_hist[w] = [float(init[w])]
                self._pnorm_scores(np.arange(n))
        if route:
            self.finish_prefill()

    def finish_prefill(self):
        """The first assignment after the prompt (Sec. 4.2)."""
        self._age()
        self.route()

    def _pnorm_scores(self, windows):
        """score = S^p = sum over completed periods of u_r^p plus u^p of the period
        in progress (appendix, p-norm equation; S^p orders windows as S does)."""
        p = self.cfg.score_p
        for w in windows:
            self.score[w] = sum(u ** p for u in self.u_hist[w]) + self.u_cur[w] ** p

    def _key_norms(self, a, b):
        """L2 norm of each token's key in [a, b) over all KV heads and channels
        (appendix on alternative ranking functions, key-norm equation)."""
        return np.sqrt(np.sum(self.k[:, a:b, :] ** 2, axis=(0, 2)))

    # -- one decode step ----------------------------------------------------
    def append(self, k_new, v_new):
        c = self.cfg
        self.k[:, self.T] = k_new
        self.v[:, self.T] = v_new
        self.att_k[:, self.T] = k_new       # sink or open-window token: attended as given
        self.att_v[:, self.T] = v_new
        self.att_live[self.T] = True
        self.T += 1
        self._start_windows()
        if c.key_norm and self.T - 1 >= c.sink:   # the token's share of its window's key-norm score
            w = (self.T - 1 - c.sink) // c.window
            self.score[w] -= self._key_norms(self.T - 1, self.T)[0] / c.window
        self._age()

    def accessible(self):
        """Keys, values [H_kv, n, d] and owning window [n] (-1 = sink) of every token attended to.

        Windows appear in index order (chronological); Quantized windows enter as
        their dequantized values z + s c.
        """
        c = self.cfg
        ks, vs, owner = [], [], []
        ns = min(c.sink, self.T)
        if ns:
            ks.append(self.k[:, :ns])
            vs.append(self.v[:, :ns])
            owner.append(np.full(ns, -1))
        for w in np.nonzero(self.state >= 0)[0]:
            st = self.state[w]
            a, b = self.win_range(w)
            b = min(b, self.T)
            if st == FULL:
                kk, vv = self.full_k[w], self.full_v[w]
            elif st == QUANT:
                kk, vv = self._dequantize(w)
            elif st in (OPEN, AGED):
                kk, vv = self.k[:, a:b], self.v[:, a:b]
            else:
                continue
            ks.append(kk)
            vs.append(vv)
            owner.append(np.full(kk.shape[1], w))
        return np.concatenate(ks, axis=1), np.concatenate(vs, axis=1), np.concatenate(owner)

    def attend(self, q):
        """Attention of all query heads; accumulate window scores.

        q: float64 [H_q, d].  Returns (out [H_q, d], mass [H_q, n_win_cap],
        sink_mass [H_q]).  Each query head attends with softmax(q k^T * scale)
        over the accessible tokens (the live rows of the attention-domain copy,
        i.e. the set accessible() lists); the score update adds, for every
        accessible window, the attention mass its tokens received averaged over
        the H_q heads.
        """
        c = self.cfg
        T = self.T
        out = np.zeros((c.num_q_heads, c.head_dim))
        mass = np.zeros((c.num_q_heads, self.n_win_cap))
        sink_mass = np.zeros(c.num_q_heads)
        live = self.att_live[:T]
        owner = self.owner[:T][live]
        win = owner >= 0
        for g in range(c.num_kv_heads):
            hs = slice(g * c.gqa, (g + 1) * c.gqa)       # the query heads reading KV head g
            logits = (self.att_k[g, :T] @ q[hs].T) * c.scale    # [T, heads of the group]
            logits[~live] = -np.inf
            e = np.exp(logits - logits.max(axis=0))
            p = e / e.sum(axis=0)
            out[hs] = p.T @ self.att_v[g, :T]
            for j in range(c.gqa):
                h = g * c.gqa + j
                pl = p[live, j]
                mass[h] = np.bincount(owner[win], weights=pl[win], minlength=self.n_win_cap)
                sink_mass[h] = pl[~win].sum()
        live_w = (self.state >= 0) & (self.state != EVICTED)
        if self.new_period and c.score_decay != 1.0:
            self.score[live_w] *= c.score_decay
        self.new_period = False
        if c.score_p:
            self.u_cur[live_w] += mass[:, live_w].sum(axis=0) / c.num_q_heads
            self._pnorm_scores(np.nonzero(live_w)[0])
        elif not c.key_norm:
            self.score[live_w] += mass[:, live_w].sum(axis=0) / c.num_q_heads
        return out, mass, sink_mass

    def step(self, q, k_new, v_new):
        self.append(k_new, v_new)
        return self.attend(q)

    # -- routing event (Sec. 4.3 candidate pool, TopK and state transitions; Algorithm 1)
    def candidates(self):
        return [int(w) for w in np.nonzero((self.state == FULL) | (self.state == QUANT)
                                           | (self.state == AGED))[0]]

    def adopt_scores(self, scores):
        """Take another implementation's scores (lockstep comparison)."""
        n = min(len(scores), self.n_win_cap)
        live = (self.state[:n] >= 0) & (self.state[:n] != EVICTED)
        self.score[:n][live] = np.asarray(scores, dtype=np.float64)[:n][live]

    # What a routing event does to one candidate, by (its state before the event,
    # the tier the ranking gives it, its ledger entry before the event; None = no
    # entry).  The moves are those of the state diagram Full <-> Quantized ->
    # Evicted under the write-once ledger (Sec. 4.3, migration-stable
    # quantization and the state-transition equation; Algorithm 1 applies the
    # same moves): codes are made once, at a window's first entry into the
    # quantized tier, a promotion leaves them dormant and a later demotion
    # reactivates them.  A candidate ranked below K_f + K_q is evicted whatever
    # its state: its copies are released and its entry deleted.
    MOVES = {
        (FULL, FULL, None): "keep",
        (FULL, FULL, DORMANT): "keep",
        (QUANT, QUANT, ACTIVE): "keep",
        (QUANT, FULL, ACTIVE): "promote",      # bf16 copy of z + s c; the entry goes dormant
        (AGED, FULL, None): "admit",           # bf16 copy of the original tokens
        (FULL, QUANT, None): "quantize",       # first demotion: codes from the bf16 copy
        (AGED, QUANT, None): "quantize",       # codes from the original tokens
        (FULL, QUANT, DORMANT): "reactivate",  # the earlier codes, no requantization
    }

    def route(self):
        c = self.cfg
        cand = self.candidates()
        order = route_order(cand, self.score)
        was_q = frozenset(w for w in cand if self.state[w] == QUANT)
        full, quant, evict = tier_split(order, c.capacity_full, c.capacity_quant,
                                        was_q, c.no_promotion)
        new_tier = dict.fromkeys(full, FULL)
        new_tier.update(dict.fromkeys(quant, QUANT))
        new_tier.update(dict.fromkeys(evict, EVICTED))
        # mixed widths: an entry created now takes 4 bits in the upper half of the
        # new quantized tier (by rank), 2 below, and keeps them for its lifetime
        q_rank = {w: r for r, w in enumerate(quant)}
        half = -(-c.capacity_quant // 2)
        for w in order:
            nt = new_tier[w]
            e = self.ledger.get(w)
            move = "evict" if nt == EVICTED else \
                self.MOVES[(int(self.state[w]), nt, None if e is None else e["state"])]
            if move == "promote":
                kh, vh = self._dequantize(w)
                self.full_k[w] = rne_bf16(kh)
                self.full_v[w] = rne_bf16(vh)
                e["state"] = DORMANT
                self.stats["promotions"] += 1
            elif move == "admit":
                a, b = self.win_range(w)
                self.full_k[w] = self.k[:, a:b].copy()
                self.full_v[w] = self.v[:, a:b].copy()
                self.stats["admissions_full"] += 1
            elif move == "quantize":
                if self.state[w] == FULL:
                    src_k, src_v = self.full_k[w], self.full_v[w]
                else:
                    a, b = self.win_range(w)
                    src_k, src_v = self.k[:, a:b], self.v[:, a:b]
                bits = c.bits if c.bits in (2, 4) else (4 if q_rank[w] < half else 2)
                self.ledger[w] = self._quantize(w, src_k, src_v, bits)
                self.stats["first_quantizations"] += 1
                self.quant_count += 1
            elif move == "reactivate":
                e["state"] = ACTIVE
                self.stats["reactivations"] += 1
            elif move == "evict":
                self.ledger.pop(w, None)
                self.stats["evictions"] += 1
            if nt != FULL:
                self.full_k.pop(w, None)
                self.full_v.pop(w, None)
            self.state[w] = nt
            if move != "keep":
                self._refresh(w)
        self.new_period = True
        if c.score_p:                     # the routing event closes the period
            for w in np.nonzero(self.state >= 0)[0]:
                self.u_hist[w].append(float(self.u_cur[w]))
                self.u_cur[w] = 0.0
        return full, quant, evict

    # -- single-window moves outside a routing event --------------------------
    # The same transitions Algorithm 1 applies to a window entering Q or F,
    # for one window chosen by the caller, within the tier capacities.
    def quantize_one(self, w: int):
        """Full -> Quantized: reactivate a dormant ledger entry as it is, or
        quantize the window's bf16 values once (mixed-width caches give such a
        new entry the upper width, 4 bits)."""
        c = self.cfg
        if self.state[w] != FULL:
            raise ValueError(f"window {w} is not in the Full tier")
        if int(np.sum(self.state == QUANT)) >= c.capacity_quant:
            raise CapacityError("the Quantized tier already holds K_q windows")
        e = self.ledger.get(w)
        if e is None:
            bits = c.bits if c.bits in (2, 4) else 4
            self.ledger[w] = self._quantize(w, self.full_k[w], self.full_v[w], bits)
            self.quant_count += 1
        else:
            e["state"] = ACTIVE
        del self.full_k[w], self.full_v[w]
        self.state[w] = QUANT
        self._refresh(w)

    def promote_one(self, w: int):
        """Quantized -> Full: bf16 values from the ledger (RNE of z + s c), the
        entry stays as a dormant record."""
        c = self.cfg
        if self.state[w] != QUANT:
            raise ValueError(f"window {w} is not in the Quantized tier")
        if c.no_promotion:
            raise ValueError("promotion is disabled (one-way policy)")
        if int(np.sum(self.state == FULL)) >= c.capacity_full:
            raise CapacityError("the Full tier already holds K_f windows")
        kh, vh = self._dequantize(w)
        self.full_k[w] = rne_bf16(kh)
        self.full_v[w] = rne_bf16(vh)
        self.ledger[w]["state"] = DORMANT
        self.state[w] = FULL
        self._refresh(w)

    # -- perturbation used by the forced-promotion workload -------------------
    def shift_key_zero_points(self, w: int, delta):
        """z_c <- RNE_fp16(z_c + delta_c) for every key group of window w.

        delta: [H_kv, d] (float32 values); the sum is formed in float64 first.
        Shifting every key zero point by delta_c moves each dequantized key of
        the window by (about) delta_c along channel c.
        """
        e = self.ledger[w]
        d = np.asarray(delta, dtype=np.float32).astype(np.float64)
        e["kz"] = rne_fp16(e["kz"] + d[:, None, :])
        if self.state[w] == QUANT:
            self._refresh(w)

    # -- views used by tests -------------------------------------------------
    def tiers(self):
        return self.state.copy()

    def ledger_states(self):
        out = np.zeros(self.n_win_cap, dtype=np.int64)
        for w, e in self.ledger.items():
            out[w] = e["state"]
        return out
