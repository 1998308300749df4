"""Pins for the oracle's single-window moves (the transitions of Algorithm 1
for one window chosen by the caller, within the tier capacities).

* a manual demotion creates the same ledger entry as a routing demotion of
  the same window (twin caches), and the same entry as quantizing the
  window's bf16 values directly;
* a manual promotion gives the same bf16 values and ledger state as a
  routing promotion of the same window (twin caches);
* demote -> promote -> demote reactivates the dormant entry: codes are
  identical and no second quantization happens;
* capacity and state rules: a full tier refuses the move, only Full windows
  can be demoted, only Quantized windows promoted, the one-way policy
  refuses promotion, evicted windows never move.
"""
import copy

import numpy as np
import pytest

from oracle.qevict_oracle import (ACTIVE, DORMANT, EVICTED, FULL, QUANT, CapacityError,
                                  OracleConfig, QEvictUnit, quantize_window)


def _bf16(rng, shape, scale=1.0):
    x = (rng.normal(size=shape) * scale).astype(np.float32)
    b = x.view(np.uint32).astype(np.uint64)
    b = ((b + 0x7FFF + ((b >> 16) & 1)) >> 16) << 16
    return b.astype(np.uint32).view(np.float32).astype(np.float64)


def _unit(seed, kf, kq, bits=4, no_promotion=False, W=4, n_win=10):
    rng = np.random.default_rng(seed)
    T0 = W * n_win
    cfg = OracleConfig(4, 2, 16, W, W, bits, kf, kq, no_promotion=no_promotion)
    u = QEvictUnit(cfg, T0 + 8)
    u.prefill(_bf16(rng, (2, T0, 16)), _bf16(rng, (2, T0, 16)), rng.permutation(n_win).astype(float))
    return u


def _same_ledger(a, b):
    return all(np.array_equal(a[k], b[k]) for k in ("kc", "vc", "ks", "kz", "vs", "vz")) \
        and a["bits"] == b["bits"]


def test_manual_demotion_matches_direct_quantization():
    u = _unit(0, kf=4, kq=7)                 # 10 windows: 4 Full, 6 Quantized, room for one more
    w = int(np.nonzero(u.state == FULL)[0][0])
    ref = quantize_window(u.full_k[w], u.full_v[w], 4, u.cfg.group)
    n_before = u.quant_count
    u.quantize_one(w)
    assert u.state[w] == QUANT and w not in u.full_k
    assert u.ledger[w]["state"] == ACTIVE and _same_ledger(u.ledger[w], ref)
    assert u.quant_count == n_before + 1


def test_manual_demotion_matches_routing_demotion():
    u = _unit(1, kf=4, kq=7)
    w = int(np.nonzero(u.state == FULL)[0][0])
    twin = copy.deepcopy(u)
    u.quantize_one(w)
    # routing: w falls below the Full cut, the best Quantized window takes its place
    q_best = int(np.nonzero(twin.state == QUANT)[0][0])
    live = np.nonzero((twin.state == FULL) | (twin.state == QUANT))[0]
    twin.score[live] = 10.0
    twin.score[w] = 1.0
    twin.score[q_best] = 20.0
    twin.route()
    assert twin.state[w] == QUANT
    assert _same_ledger(u.ledger[w], twin.ledger[w])


def test_manual_promotion_matches_routing_promotion():
    u = _unit(2, kf=4, kq=7)
    f0 = int(np.nonzero(u.state == FULL)[0][0])
    u.quantize_one(f0)                       # frees one Full slot
    w = int(np.nonzero(u.state == QUANT)[0][-1])
    twin = copy.deepcopy(u)
    u.promote_one(w)
    # routing with w ranked right after the current Full windows fills the free slot with w
    fulls = np.nonzero(twin.state == FULL)[0]
    live = np.nonzero((twin.state == FULL) | (twin.state == QUANT))[0]
    twin.score[live] = 1.0
    twin.score[fulls] = 10.0
    twin.score[w] = 5.0
    twin.route()
    assert np.array_equal(u.state, twin.state)
    assert np.array_equal(u.full_k[w], twin.full_k[w]) and np.array_equal(u.full_v[w], twin.full_v[w])
    assert u.ledger[w]["state"] == twin.ledger[w]["state"] == DORMANT


def test_demote_promote_demote_reactivates():
    u = _unit(3, kf=4, kq=7)
    w = int(np.nonzero(u.state == FULL)[0][1])
    u.quantize_one(w)
    first = copy.deepcopy(u.ledger[w])
    n = u.quant_count
    u.promote_one(w)
    assert u.ledger[w]["state"] == DORMANT
    u.quantize_one(w)
    assert u.quant_count == n and u.ledger[w]["state"] == ACTIVE
    assert _same_ledger(u.ledger[w], first)


def test_capacity_and_state_rules():
    u = _unit(4, kf=4, kq=6)                 # both tiers full
    f = int(np.nonzero(u.state == FULL)[0][0])
    q = int(np.nonzero(u.state == QUANT)[0][0])
    with pytest.raises(CapacityError):
        u.quantize_one(f)
    with pytest.raises(CapacityError):
        u.promote_one(q)
    with pytest.raises(ValueError):
        u.quantize_one(q)
    with pytest.raises(ValueError):
        u.promote_one(f)
    u2 = _unit(5, kf=3, kq=3)                # 4 of 10 windows evicted
    e = int(np.nonzero(u2.state == EVICTED)[0][0])
    with pytest.raises(ValueError):
        u2.quantize_one(e)
    with pytest.raises(ValueError):
        u2.promote_one(e)
    u3 = _unit(6, kf=4, kq=7, no_promotion=True)
    u3.quantize_one(int(np.nonzero(u3.state == FULL)[0][0]))
    with pytest.raises(ValueError):
        u3.promote_one(int(np.nonzero(u3.state == QUANT)[0][0]))


def test_mixed_width_manual_ledger_is_upper_width():
    u = _unit(7, kf=4, kq=7, bits=42)
    w = int(np.nonzero(u.state == FULL)[0][0])
    u.quantize_one(w)
    assert u.ledger[w]["bits"] == 4
