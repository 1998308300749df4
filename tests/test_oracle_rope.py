"""Pins for the oracle's RoPE-aware Quantized tier (Sec. 4.3: keys quantized in
the pre-RoPE domain, rotated back at their original positions after
dequantization).

* the rotation equals a complex multiplication of the channel pairs
  (i, i + d/2) by exp(i p theta_i), theta_i = base^(-2i/d), written here with
  numpy complex numbers; the float32 inverse rotation undoes it;
* rotations compose by adding positions and preserve the dot product's
  dependence on relative position only: (R(p) q).(R(p') k) = q.(R(p' - p) k);
* a cache whose windows all stay Full is unaffected by the RoPE setting;
* a RoPE cache's codes are those of the pre-RoPE keys (un-rotated here with
  complex numbers, then rounded to bf16), promoted keys lie within the
  quantization error of the keys the cache received, and the attention output
  equals plain softmax attention over the rotated dequantized keys.
"""
import math

import numpy as np
import pytest

from oracle.numerics import rne_bf16
from oracle.qevict_oracle import (FULL, QUANT, OracleConfig, QEvictUnit, dequantize_window,
                                  quantize_window, rope_cos_sin, rope_rotate, rope_unrotate_f32)

D = 16


def _complex_rotate(x, positions, base, sign=1.0):
    h = x.shape[-1] // 2
    theta = base ** (-2.0 * np.arange(h) / x.shape[-1])
    z = x[..., :h] + 1j * x[..., h:]
    z = z * np.exp(1j * sign * np.asarray(positions, dtype=np.float64)[:, None] * theta)
    return np.concatenate([z.real, z.imag], axis=-1)


def test_rotation_is_a_complex_multiplication():
    rng = np.random.default_rng(0)
    pos = [0, 1, 7, 1000, 32767]
    x = rng.normal(size=(2, len(pos), D))
    cs, sn = rope_cos_sin(10000.0, D, pos)
    assert np.allclose(rope_rotate(x, cs, sn), _complex_rotate(x, pos, 10000.0), rtol=1e-6, atol=1e-6)
    assert np.array_equal(cs[0], np.ones(D // 2, np.float32)) and not np.any(sn[0])
    # float32 inverse rotation of bf16 values undoes the rotation up to float32 rounding
    xb = rne_bf16(x)
    back = rope_unrotate_f32(rope_rotate(xb, cs, sn), cs, sn).astype(np.float64)
    assert np.allclose(back, xb, rtol=0, atol=1e-5)
    assert np.allclose(rope_unrotate_f32(xb, cs, sn), _complex_rotate(xb, pos, 10000.0, -1.0),
                       rtol=1e-5, atol=1e-5)


def test_relative_position_property():
    rng = np.random.default_rng(1)
    q, k = rng.normal(size=(1, 1, D)), rng.normal(size=(1, 1, D))
    for p, pk in [(5, 9), (100, 3), (4000, 4000)]:
        cq, sq = rope_cos_sin(500000.0, D, [p])
        ck, sk = rope_cos_sin(500000.0, D, [pk])
        cd, sd = rope_cos_sin(500000.0, D, [pk - p]) if pk >= p else (None, None)
        lhs = float((rope_rotate(q, cq, sq) * rope_rotate(k, ck, sk)).sum())
        rel = _complex_rotate(k[0], [pk - p], 500000.0)[None]
        assert lhs == pytest.approx(float((q * rel).sum()), rel=1e-5, abs=1e-6)
        if cd is not None:
            assert lhs == pytest.approx(float((q * rope_rotate(k, cd, sd)).sum()), rel=1e-5, abs=1e-6)


def _unit(rope, kf, kq, n_win=8, W=4, sink=2):
    cfg = OracleConfig(4, 2, D, W, W, 4, kf, kq, sink=sink, rope_base=rope)
    u = QEvictUnit(cfg, sink + W * n_win + 8)
    rng = np.random.default_rng(3)
    T = sink + W * n_win
    k = rne_bf16(rng.normal(size=(2, T, D)))
    v = rne_bf16(rng.normal(size=(2, T, D)))
    u.prefill(k, v, rng.permutation(n_win) / n_win)
    return u, k, v, rng


def test_all_full_cache_ignores_rope():
    a, _, _, rng = _unit(0.0, 8, 0)
    b, _, _, _ = _unit(10000.0, 8, 0)
    for _ in range(5):
        q = rne_bf16(rng.normal(size=(4, D)))
        kn, vn = rne_bf16(rng.normal(size=(2, D))), rne_bf16(rng.normal(size=(2, D)))
        oa, _, _ = a.step(q, kn, vn)
        ob, _, _ = b.step(q, kn, vn)
        a.route()
        b.route()
        assert np.array_equal(oa, ob)


def test_codes_describe_the_pre_rope_keys_and_promotion_rotates_back():
    base, W, sink = 10000.0, 4, 2
    u, k, v, rng = _unit(base, 2, 4)
    quant = [w for w in range(8) if u.state[w] == QUANT]
    assert quant
    for w in quant:
        a = sink + w * W
        pos = list(range(a, a + W))
        # the pre-RoPE keys the codes describe (the float32 un-rotation rounded to
        # bf16) agree with the exact float64 un-rotation to within one bf16 step
        exact = _complex_rotate(k[:, a:a + W], pos, base, -1.0)
        recipe = rne_bf16(rope_unrotate_f32(k[:, a:a + W], *rope_cos_sin(base, D, pos)).astype(np.float64))
        assert np.all(np.abs(recipe - exact) <= 2.0 ** -7 * np.abs(exact) + 2.0 ** -133)
        # and the ledger holds exactly the quantization of those keys
        e = quantize_window(recipe, v[:, a:a + W], 4, W)
        led = u.ledger[w]
        assert np.array_equal(led["kc"], e["kc"]) and np.array_equal(led["ks"], e["ks"])
        assert np.array_equal(led["kz"], e["kz"]) and np.array_equal(led["vc"], e["vc"])
        # dequantized keys rotated back lie within the quantization error of the received keys
        kh, _ = dequantize_window(led)
        back = _complex_rotate(kh, pos, base)
        bound = (led["ks"][..., :D // 2] + led["ks"][..., D // 2:]) / 2   # pairs mix two channels
        err = np.abs(back - k[:, a:a + W])
        bound = np.concatenate([bound, bound], axis=-1) + 2.0 ** -7 * np.abs(k[:, a:a + W])
        assert np.all(err <= bound + 1e-12)
    # promotion stores the rotated dequantized keys, rounded to bf16 (a cache with room:
    # 4 Full and 4 of 6 Quantized; demote a Full window, then promote a Quantized one)
    u, k, v, rng = _unit(base, 4, 6)
    w = [x for x in range(8) if u.state[x] == QUANT][0]
    u.quantize_one([x for x in range(8) if u.state[x] == FULL][0])
    u.promote_one(w)
    a = sink + w * W
    kh, _ = dequantize_window(u.ledger[w])
    assert np.array_equal(u.full_k[w], rne_bf16(rope_rotate(kh, *rope_cos_sin(base, D, range(a, a + W)))))


def test_attention_uses_rotated_dequantized_keys():
    base, W, sink = 10000.0, 4, 2
    u, k, v, rng = _unit(base, 2, 4)
    q = rne_bf16(rng.normal(size=(4, D)))
    kn, vn = rne_bf16(rng.normal(size=(2, D))), rne_bf16(rng.normal(size=(2, D)))
    out, _, _ = u.step(q, kn, vn)
    # independent assembly: sink and bf16 tiers as received, quantized windows rotated back
    T = u.T
    keys, vals = [k[:, :sink]], [v[:, :sink]]
    allk = np.concatenate([k, kn[:, None]], axis=1)
    allv = np.concatenate([v, vn[:, None]], axis=1)
    for w in range(-(-(T - sink) // W)):
        a, b = sink + w * W, min(sink + (w + 1) * W, T)
        if u.state[w] == QUANT:
            kh, vh = dequantize_window(u.ledger[w])
            keys.append(_complex_rotate(kh, list(range(a, b)), base))
            vals.append(vh)
        elif u.state[w] == FULL or u.state[w] in (0, 1):
            keys.append(allk[:, a:b])
            vals.append(allv[:, a:b])
    K, V = np.concatenate(keys, axis=1), np.concatenate(vals, axis=1)
    for h in range(4):
        lg = K[h // 2] @ q[h] / math.sqrt(D)
        p = np.exp(lg - lg.max())
        p /= p.sum()
        assert np.allclose(out[h], p @ V[h // 2], rtol=1e-5, atol=1e-6)   # float32 cos, sin table
