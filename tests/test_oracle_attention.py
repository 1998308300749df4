"""Pins for the oracle's attention and window scores (Sec. 4.1, Sec. 4.2).

* With every window in the bf16 tier the output equals ordinary softmax
  attention over all tokens (torch's scaled_dot_product_attention, float64).
* With a quantized tier it equals ordinary attention over the token set whose
  quantized windows are replaced by z + s c.
* Per head and step the window masses plus the sink mass sum to 1, so the sum
  of all window scores grows by exactly 1 - (mean sink mass) per step.
* Evicted tokens receive no attention.
"""
import numpy as np
import torch

from oracle.qevict_oracle import (AGED, EVICTED, FULL, QUANT, OracleConfig, QEvictUnit,
                                  dequantize_window)
from synthetic import bf16_bits_to_f32, f32_to_bf16_bits


def _bf16(rng, shape, scale=1.0):
    return bf16_bits_to_f32(f32_to_bf16_bits(rng.normal(size=shape) * scale)).astype(np.float64)


def _sdpa(q, k, v, scale):
    """torch reference: q [H_q, d], k/v [H_kv, n, d]; GQA by repeating KV heads."""
    hq, hkv = q.shape[0], k.shape[0]
    kk = torch.from_numpy(k).repeat_interleave(hq // hkv, dim=0)
    vv = torch.from_numpy(v).repeat_interleave(hq // hkv, dim=0)
    qq = torch.from_numpy(q)[:, None, :]
    o = torch.nn.functional.scaled_dot_product_attention(qq, kk, vv, scale=scale)
    return o[:, 0, :].numpy()


def _unit(hq=8, hkv=2, d=64, w=16, T=16 * 10 + 5, kf=100, kq=0, sink=0, recent=0, steps=4, seed=0,
          bits=4):
    rng = np.random.default_rng(seed)
    cfg = OracleConfig(hq, hkv, d, w, w, bits, kf, kq, sink=sink, recent=recent)
    u = QEvictUnit(cfg, T + steps)
    k, v = _bf16(rng, (hkv, T, d)), _bf16(rng, (hkv, T, d))
    n = -(-(T - sink) // w)
    u.prefill(k, v, rng.uniform(0, 1, size=n))
    return u, rng


def test_all_full_equals_plain_attention():
    u, rng = _unit(kf=1000, sink=3, recent=7)
    for _ in range(3):
        q = _bf16(rng, (8, 64))
        kn, vn = _bf16(rng, (2, 64)), _bf16(rng, (2, 64))
        out, mass, sink_mass = u.step(q, kn, vn)
        T = u.T
        ref = _sdpa(q, u.k[:, :T], u.v[:, :T], u.cfg.scale)
        np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-12)
        assert np.all(u.state[u.state >= 0] != EVICTED)


def test_quantized_tier_equals_attention_over_dequantized_tokens():
    u, rng = _unit(kf=3, kq=4, T=16 * 9, steps=2, seed=3)
    q = _bf16(rng, (8, 64))
    kn, vn = _bf16(rng, (2, 64)), _bf16(rng, (2, 64))
    u.append(kn, vn)
    # assemble the accessible set by hand from the tier map
    ks, vs = [], []
    for w in range(u.n_win_cap):
        a, b = u.win_range(w)
        b = min(b, u.T)
        if a >= u.T:
            break
        st = u.state[w]
        if st == FULL:
            ks.append(u.full_k[w]), vs.append(u.full_v[w])
        elif st == QUANT:
            e = u.ledger[w]
            kh = e["kz"].repeat(e["group"], 1) + e["ks"].repeat(e["group"], 1) * e["kc"]
            vh = e["vz"].repeat(e["group"], 2) + e["vs"].repeat(e["group"], 2) * e["vc"]
            ks.append(kh), vs.append(vh)
        elif st != EVICTED:
            ks.append(u.k[:, a:b]), vs.append(u.v[:, a:b])
    assert np.sum(u.state == QUANT) == 4 and np.sum(u.state == FULL) == 3
    ref = _sdpa(q, np.concatenate(ks, 1), np.concatenate(vs, 1), u.cfg.scale)
    out, _, _ = u.attend(q)
    np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-12)


def test_masses_sum_to_one_and_scores_grow_by_non_sink_mass():
    u, rng = _unit(kf=4, kq=3, sink=5, recent=9, steps=20, seed=5)
    for _ in range(20):
        before = u.score.sum()
        q = _bf16(rng, (8, 64), 2.0)
        out, mass, sink_mass = u.step(q, _bf16(rng, (2, 64)), _bf16(rng, (2, 64)))
        np.testing.assert_allclose(mass.sum(1) + sink_mass, 1.0, rtol=0, atol=1e-12)
        after = u.score.sum()
        np.testing.assert_allclose(after - before, 1.0 - sink_mass.mean(), rtol=0, atol=1e-12)
        ev = u.state == EVICTED
        assert np.all(mass[:, ev] == 0)
        u.route()


def test_gqa_heads_share_kv():
    """Two query heads of one KV group with equal queries give equal outputs and masses."""
    u, rng = _unit(hq=8, hkv=2, kf=5, kq=2, seed=9)
    q = _bf16(rng, (8, 64))
    q[1] = q[0]
    out, mass, _ = u.step(q, _bf16(rng, (2, 64)), _bf16(rng, (2, 64)))
    np.testing.assert_array_equal(out[1], out[0])
    np.testing.assert_array_equal(mass[1], mass[0])


def test_promoted_window_holds_bf16_of_dequantized_values():
    u, rng = _unit(kf=2, kq=3, T=16 * 8, seed=11)
    qw = [w for w in range(u.n_win_cap) if u.state[w] == QUANT]
    w = qw[-1]
    u.score[w] = 1e6
    u.route()
    assert u.state[w] == FULL and u.ledger[w]["state"] == 2
    kh, vh = dequantize_window(u.ledger[w])
    ref_k = torch.from_numpy(kh).to(torch.float32)
    # kh is a multiple of 2^-24 below 2^21, exact in float32 only when it has <= 24 bits;
    # compare through float32 only where that holds, and bit-for-bit on the oracle's own grid
    exact32 = ref_k.to(torch.float64).numpy() == kh
    bf = ref_k.to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(u.full_k[w][exact32], bf[exact32])
    assert np.all(np.abs(u.full_k[w] - kh) <= np.abs(kh) * 2.0 ** -8)


def test_attention_copy_follows_every_tier_change():
    """attend() reads the live rows of the oracle's attention-domain copy; along a
    trajectory with promotions, first quantizations, reactivations, evictions,
    admissions, manual moves and a key shift, it equals textbook attention over
    the set accessible() assembles from the tier map, and the masses equal the
    per-window sums of those probabilities."""
    u, rng = _unit(hq=8, hkv=2, kf=3, kq=4, T=16 * 12 + 5, sink=5, recent=9, steps=40, seed=21)
    kinds = set()
    for t in range(40):
        q = _bf16(rng, (8, 64), 1.5)
        kn, vn = _bf16(rng, (2, 64)), _bf16(rng, (2, 64))
        u.append(kn, vn)
        kk, vv, owner = u.accessible()
        ref = _sdpa(q, kk, vv, u.cfg.scale)
        logits = np.einsum("hnd,hd->hn", np.repeat(kk, 4, axis=0), q) * u.cfg.scale
        p = np.exp(logits - logits.max(axis=1, keepdims=True))
        p /= p.sum(axis=1, keepdims=True)
        out, mass, sink_mass = u.attend(q)
        np.testing.assert_allclose(out, ref, rtol=1e-11, atol=1e-12)
        for w in range(u.n_win_cap):
            np.testing.assert_allclose(mass[:, w], p[:, owner == w].sum(axis=1), rtol=0, atol=1e-12)
        np.testing.assert_allclose(sink_mass, p[:, owner < 0].sum(axis=1), rtol=0, atol=1e-12)
        # stir the scores so that windows move both ways, then route
        live = (u.state >= 0) & (u.state != EVICTED)
        u.score[live] += rng.uniform(0, 0.3, size=live.sum())
        if t % 3 == 0:
            u.score[u.state == AGED] += 5.0      # some aged windows enter Full directly
        before = dict(u.stats)
        u.route()
        kinds |= {k for k in before if u.stats[k] > before[k]}
        if t == 10:
            qw = np.nonzero(u.state == QUANT)[0]
            u.shift_key_zero_points(int(qw[0]), rng.normal(size=(2, 64)).astype(np.float32))
        if t == 20:
            fw = np.nonzero(u.state == FULL)[0]
            if np.sum(u.state == QUANT) < 4:
                u.quantize_one(int(fw[0]))
            qw = np.nonzero(u.state == QUANT)[0]
            if np.sum(u.state == FULL) < 3:
                u.promote_one(int(qw[0]))
    assert {"promotions", "first_quantizations", "reactivations", "evictions",
            "admissions_full"} <= kinds, kinds
