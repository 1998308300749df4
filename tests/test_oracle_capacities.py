"""Pins for the byte-constrained tier capacities (Sec. 4.3 tier capacities
equation; memory accounting appendix) and the library's copy of them.

* a worked example at the paper's default point on the 8B shape (32K prompt,
  20% of the full cache, q = 0.70, int2, W = 32, five sink and 32 recent
  tokens), with the byte counts written out by hand below;
* floor properties: the chosen capacities fit their shares and one more
  window would not; q = 0 and q = 1 leave one tier empty;
* the host function of the library returns the same capacities over a sweep
  of configurations (no GPU needed).
"""
from fractions import Fraction

import pytest

from oracle.qevict_oracle import tier_capacities, window_costs


def test_worked_example_paper_default_8b():
    # full cache of one layer: 2 (K, V) x 8 heads x 128 channels x 32768 tokens x 2 B
    full = 134_217_728
    budget = 26_843_545                      # floor(0.2 x full)
    # protected: 37 tokens x 4 KiB (bf16 K and V over 8 heads) = 151,552 B
    b_hist = 26_691_993
    # M_f = 131,072 (bf16 window) + 8;  M_q = 16,384 (int2 codes) + 4,096 (key params)
    #       + 4,096 (value params) + 10
    assert window_costs(8, 128, 32, 32, 2) == (131_080, 24_586)
    assert budget == int(Fraction(2, 10) * full)
    # K_f = floor(0.3 x 26,691,993 / 131,080) = floor(61.09), K_q = floor(0.7 x ... / 24,586) = floor(759.96)
    assert tier_capacities(budget, 700, 8, 128, 32, 32, 2, 5, 32) == (61, 759)
    assert budget - b_hist == 151_552


def test_paper_default_point_eight_token_windows():
    """The same budget with the paper's 8-token windows (values in 32-channel groups)."""
    # M_f = 2 x 8 x 8 x 128 x 2 B + 8 = 32,776;  M_q = 4,096 (int2 codes) + 4,096 (key
    # scale / zero per channel) + 1,024 (value scale / zero per token and 32 channels) + 10
    assert window_costs(8, 128, 8, 32, 2) == (32_776, 9_226)
    # K_f = floor(0.3 x 26,691,993 / 32,776) = floor(244.31), K_q = floor(0.7 x ... / 9,226) = floor(2025.18)
    assert tier_capacities(26_843_545, 700, 8, 128, 8, 32, 2, 5, 32) == (244, 2025)


@pytest.mark.parametrize("q", [0, 150, 500, 700, 999, 1000])
@pytest.mark.parametrize("bits,W", [(2, 32), (4, 32), (42, 32), (2, 64)])
def test_floor_properties(q, bits, W):
    budget, sink, recent = 9_876_543, 5, 32
    kf, kq = tier_capacities(budget, q, 8, 128, W, W, bits, sink, recent)
    m_f, m_q = window_costs(8, 128, W, W, bits)
    b_hist = budget - 4 * 8 * 128 * (sink + recent)
    qf = Fraction(q, 1000)
    assert kf * m_f <= (1 - qf) * b_hist < (kf + 1) * m_f
    assert kq * m_q <= qf * b_hist < (kq + 1) * m_q
    assert kf * m_f + kq * m_q <= b_hist
    if q == 0:
        assert kq == 0
    if q == 1000:
        assert kf == 0


def test_budget_below_protected_regions():
    with pytest.raises(ValueError):
        tier_capacities(4 * 8 * 128 * 37 - 1, 700, 8, 128, 32, 32, 2, 5, 32)


def test_library_matches_oracle():
    import paper_2608_05326_amd as qv
    for H_kv, W, bits, sink, recent, budget, q in [
        (8, 32, 2, 5, 32, 26_843_545, 700), (8, 32, 4, 0, 0, 13_421_772, 300),
        (8, 64, 2, 64, 128, 50_000_000, 900), (8, 32, 42, 40, 70, 7_000_000, 550),
        (1, 32, 4, 0, 100, 3_000_000, 0), (4, 64, 2, 3, 0, 1_000_000, 1000),
        (8, 8, 2, 5, 32, 26_843_545, 700), (8, 8, 42, 0, 16, 5_000_000, 400),
    ]:
        G = 32 if W == 8 else W
        cfg = qv.Config(batch=1, num_q_heads=4 * H_kv, num_kv_heads=H_kv, window_tokens=W,
                        quant_bits=bits, max_context=65536, capacity_full=0, capacity_quant=0,
                        sink_tokens=sink, recent_tokens=recent)
        assert qv.qevict.capacities_for_budget(cfg, budget, q) == \
            tier_capacities(budget, q, H_kv, 128, W, G, bits, sink, recent)
    with pytest.raises(qv.QEvictError):
        qv.qevict.capacities_for_budget(cfg, 10, 500)
    with pytest.raises(qv.QEvictError):
        qv.qevict.capacities_for_budget(cfg, budget, 1001)


def test_memory_report_of_a_routed_cache():
    """A prompt of 11.25 windows of 4 tokens after 3 sink tokens, 5 recent
    tokens, 2 Full and 3 int4 windows: the bytes counted by hand, and the total
    agrees with the per-window costs of the capacity equation; then a smaller
    cache where a promotion leaves a dormant ledger entry."""
    import numpy as np
    from oracle.qevict_oracle import FULL, QUANT, OracleConfig, QEvictUnit, memory_report
    H, d, W = 2, 8, 4
    cfg = OracleConfig(4, H, d, W, W, 4, 2, 3, sink=3, recent=5)
    u = QEvictUnit(cfg, 3 + 4 * 12)
    T = 3 + 4 * 10 + 5
    rng = np.random.default_rng(0)
    u.prefill(rng.normal(size=(H, T, d)), rng.normal(size=(H, T, d)), rng.permutation(12) / 12.0)
    r = memory_report(u)
    tok = 2 * 2 * H * d                       # 64 bytes per token
    assert r["sink"] == 3 * 64 and tok == 64
    # windows tile [3, 48): 11 complete and one of a single token; routed are the complete
    # windows ending at or before T - 5 = 43, windows 0..9 (tokens 3..42), so
    # 48 - 3 - 40 = 5 tokens count as recent
    assert r["recent"] == 5 * 64
    assert r["full"] == 2 * 4 * 64
    codes = 2 * H * W * d * 4 // 8            # 64 bytes of int4 codes per window
    # fp16 scale and zero point: keys per (head, channel) = 2 x 8 x 4 B, values per
    # (head, token, group of 4 channels) = 2 x 4 x 2 x 4 B
    meta = 64 + 64
    assert r["quant_codes"] == 3 * codes and r["quant_meta"] == 3 * meta
    assert r["position"] == 5 * 8
    assert r["ledger"] == 3 * 2
    m_f, m_q = window_costs(H, d, W, W, 4)
    assert r["total"] == r["sink"] + r["recent"] + 2 * m_f + 3 * m_q
    # four routed windows (2 Full, 2 Quantized, one Quantized slot free): demote a Full
    # window, then promote a Quantized one, whose ledger turns dormant
    v = QEvictUnit(cfg, 3 + 4 * 6)
    T = 3 + 4 * 4 + 5
    v.prefill(rng.normal(size=(H, T, d)), rng.normal(size=(H, T, d)), rng.permutation(6) / 6.0)
    r = memory_report(v)
    assert (r["full"], r["quant_codes"], r["ledger"]) == (2 * 4 * 64, 2 * codes, 2 * 2)
    q = [w for w in range(6) if v.state[w] == QUANT][0]
    f = [w for w in range(6) if v.state[w] == FULL][0]
    v.quantize_one(f)
    v.promote_one(q)
    r2 = memory_report(v)
    assert (r2["full"], r2["quant_codes"]) == (r["full"], r["quant_codes"])
    assert r2["ledger"] == 3 * 2 + codes + meta    # three entries, one of them dormant
