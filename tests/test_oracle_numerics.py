"""Pins for the oracle's exact rounding helpers.

Each helper is checked against something other than itself: numpy's
float64->float16 conversion (correctly rounded), torch's float32->bfloat16
conversion, and a brute-force search over every finite value of the target
format.
"""
import numpy as np
import pytest
import torch

from oracle.numerics import rd_fp16, rne_bf16, rne_fp16, ru_fp16


def _all_fp16():
    v = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16).view(np.float16).astype(np.float64)
    return np.unique(v[np.isfinite(v)])


def _all_bf16():
    b = np.arange(1 << 16, dtype=np.uint32) << 16
    v = b.view(np.float32)
    return np.unique(v[np.isfinite(v)].astype(np.float64))


def _samples(rng, n=20000):
    mags = np.exp2(rng.uniform(-30, 17, size=n))
    x = mags * rng.choice([-1.0, 1.0], size=n)
    return np.concatenate([x, rng.normal(size=n), [0.0, -0.0, 1.0, -1.0, 65504.0, -65504.0]])


def _midpoints(table):
    t = table[(table > -60000) & (table < 60000)]
    return (t[:-1] + t[1:]) / 2


def test_rne_fp16_matches_numpy():
    rng = np.random.default_rng(1)
    x = _samples(rng)
    x = x[np.abs(x) < 65504]
    mid = _midpoints(_all_fp16())   # exact halfway points: ties to even
    for v in (x, mid):
        assert np.array_equal(rne_fp16(v), v.astype(np.float16).astype(np.float64))


def test_rd_ru_fp16_brute_force():
    table = _all_fp16()
    rng = np.random.default_rng(2)
    x = _samples(rng)
    x = x[np.abs(x) <= 65504]
    x = np.concatenate([x, table[::97], _midpoints(table)[::31]])
    lo = table[np.searchsorted(table, x, side="right") - 1]
    hi = table[np.searchsorted(table, x, side="left")]
    assert np.array_equal(rd_fp16(x), lo)
    assert np.array_equal(ru_fp16(x), hi)


def test_rne_bf16_matches_torch_on_float32_inputs():
    rng = np.random.default_rng(3)
    x = _samples(rng).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(rne_bf16(x.astype(np.float64)), ref)


def test_rne_bf16_brute_force_nearest_even():
    table = _all_bf16()
    rng = np.random.default_rng(4)
    x = _samples(rng, 5000)
    x = np.concatenate([x, _midpoints(table[(table > -1e4) & (table < 1e4)])[::53]])
    idx = np.searchsorted(table, x)
    lo, hi = table[idx - 1], table[idx]
    exact = table[np.minimum(idx, len(table) - 1)] == x
    dlo, dhi = x - lo, hi - x
    lo_bits = lo.astype(np.float32).view(np.uint32) >> 16
    pick_lo = (dlo < dhi) | ((dlo == dhi) & ((lo_bits & 1) == 0))
    ref = np.where(exact, x, np.where(pick_lo, lo, hi))
    assert np.array_equal(rne_bf16(x), ref)


@pytest.mark.parametrize("f", [rne_fp16, rd_fp16, ru_fp16, rne_bf16])
def test_results_are_fixed_points(f):
    rng = np.random.default_rng(5)
    y = f(_samples(rng, 2000))
    y = y[np.isfinite(y)]
    assert np.array_equal(f(y), y)
