"""Pins for the oracle's quantizer (Sec. 4.3, migration-stable quantization).

* the hand-derived examples in tests/golden/quant_worked_examples.json;
* a brute-force reference in exact rational arithmetic (fractions.Fraction)
  that searches the whole fp16 table for the zero point and the scale;
* the invariants the definition guarantees: |x - x_hat| <= s/2,
  z <= min, z + s (2^b - 1) >= max, s minimal, 0 <= c <= 2^b - 1.
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle.qevict_oracle import dequantize_window, quantize_groups, quantize_window

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "quant_worked_examples.json")


def _fp16_table():
    v = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16).view(np.float16).astype(np.float64)
    return sorted(set(float(a) for a in v[np.isfinite(v)]))


_TABLE = _fp16_table()
_NONNEG = [t for t in _TABLE if t >= 0]
_TABLE_F = [Fraction(t) for t in _TABLE]
_NONNEG_F = [Fraction(t) for t in _NONNEG]


def _first_true(table, pred):
    """Smallest index i with pred(table[i]) for a monotone predicate (binary search)."""
    a, b = 0, len(table)
    while a < b:
        m = (a + b) // 2
        if pred(table[m]):
            b = m
        else:
            a = m + 1
    return a


def brute_force_group(x, bits):
    """Exact rational reference over the full fp16 table: z, s, then codes by RNE."""
    n = 2 ** bits - 1
    fx = [Fraction(float(a)) for a in x]
    lo, hi = min(fx), max(fx)
    z = _TABLE_F[_first_true(_TABLE_F, lambda t: t > lo) - 1]
    s = _NONNEG_F[_first_true(_NONNEG_F, lambda t: z + t * n >= hi)]
    codes = [0 if s == 0 else round((a - z) / s) for a in fx]   # Fraction rounds half to even
    return float(z), float(s), codes


def test_golden_examples():
    with open(GOLDEN) as f:
        g = json.load(f)
    for case in g["quant"]:
        x = np.array([[float.fromhex(a) for a in case["x"]]])
        z, s, c = quantize_groups(x, case["bits"])
        assert z[0] == float.fromhex(case["z"]), case["name"]
        assert s[0] == float.fromhex(case["s"]), case["name"]
        assert list(c[0]) == case["codes"], case["name"]
        bz, bs, bc = brute_force_group(x[0], case["bits"])
        assert (bz, bs, bc) == (z[0], s[0], list(c[0])), case["name"]


def _bf16_round(x):
    b = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    b = ((b + 0x7FFF + ((b >> 16) & 1)) >> 16) << 16
    return b.astype(np.uint32).view(np.float32).astype(np.float64)


@pytest.mark.parametrize("bits", [2, 4])
def test_matches_exact_brute_force(bits):
    rng = np.random.default_rng(10 + bits)
    groups = []
    for i in range(120):
        kind = i % 6
        if kind == 0:
            g = rng.normal(size=8)
        elif kind == 1:
            g = rng.standard_t(3, size=8) * 8
        elif kind == 2:
            g = rng.normal(size=8) * 1e-5          # near / below the fp16 normal range
        elif kind == 3:
            g = np.full(8, rng.normal())           # constant group
        elif kind == 4:
            g = rng.integers(-4, 5, size=8) / 4.0  # lands exactly on rounding boundaries
        else:
            g = rng.normal(size=8) * 300
        groups.append(_bf16_round(g))
    x = np.array(groups)
    z, s, c = quantize_groups(x, bits)
    for i in range(len(x)):
        bz, bs, bc = brute_force_group(x[i], bits)
        assert (z[i], s[i]) == (bz, bs), i
        assert list(c[i]) == bc, i


@pytest.mark.parametrize("bits", [2, 4])
def test_error_bound_and_minimality(bits):
    rng = np.random.default_rng(20 + bits)
    x = _bf16_round(rng.standard_t(3, size=(4000, 32)) * rng.choice([1e-3, 1, 30], size=(4000, 1)))
    z, s, c = quantize_groups(x, bits)
    n = 2 ** bits - 1
    xhat = z[:, None] + s[:, None] * c
    assert np.all(np.abs(x - xhat) <= s[:, None] / 2)
    assert np.all(z <= x.min(1)) and np.all(z + s * n >= x.max(1))
    assert np.all((c >= 0) & (c <= n))
    prev = np.where(s > 0, np.nextafter(s.astype(np.float16), np.float16(0)).astype(np.float64), 0)
    assert np.all((s == 0) | (z + prev * n < x.max(1)))


@pytest.mark.parametrize("w,g", [(32, 32), (64, 64), (8, 32)])
def test_window_layout_groups(w, g):
    """Keys: one (s, z) per channel across the window's tokens; values: per token per G
    channels (8-token windows keep 32-channel value groups)."""
    rng = np.random.default_rng(7)
    h, d = 2, 128
    k = _bf16_round(rng.normal(size=(h, w, d)))
    v = _bf16_round(rng.normal(size=(h, w, d)))
    e = quantize_window(k, v, 4, g)
    assert e["kz"].shape == (h, 1, d) and e["vz"].shape == (h, w, d // g)
    # channel 5 of head 1 is one key group
    z, s, c = quantize_groups(k[1, :, 5][None, :], 4)
    assert e["kz"][1, 0, 5] == z[0] and e["ks"][1, 0, 5] == s[0]
    assert np.array_equal(e["kc"][1, :, 5], c[0])
    # token 7, channels g .. 2g - 1 of head 0 is one value group
    z, s, c = quantize_groups(v[0, 7, g:2 * g][None, :], 4)
    assert e["vz"][0, 7, 1] == z[0] and np.array_equal(e["vc"][0, 7, g:2 * g], c[0])
    kh, vh = dequantize_window(e)
    assert np.all(np.abs(kh - k) <= e["ks"] / 2)
    assert np.all(np.abs(vh - v) <= np.repeat(e["vs"], g, axis=2) / 2)
