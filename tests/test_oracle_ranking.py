"""Pins for the oracle's window ranking functions (Sec. 4.2 cumulative window
score equation; the decayed score S_t = lambda S_{t-R} + u_t of the appendix on
alternative ranking functions, u_t the attention a window received since the
previous routing event).

* with all keys zero every query attends uniformly, so a window's mass at a
  step is (its tokens) / (tokens held); the scores then follow a recurrence
  written out here independently of the oracle: plain sums for the
  cumulative score, and for the decayed score one multiplication by lambda at
  the first step of every routing period (R = 1 and R = 3);
* lambda just below 1 stays on the cumulative trajectory, on random inputs
  with routing;
* a small lambda changes which windows survive: recent attention outweighs
  old attention that the cumulative score still remembers;
* key-norm score: a closed form for keys whose norm is the token index + 1
  (prefill and decode), independence from the queries, routing keeps the
  lowest-norm windows (a zero-key window first; doubling a window's keys
  doubles its score), and windows completed during decode score as a prefill
  of the same tokens does;
* attention p-norm: the uniform-attention periods (R = 1 to 4, several p),
  p = 1 equals the cumulative score, and with all windows in Full the score
  equals the p-th powers of the cumulative increments between routing
  events, within the power-mean bounds of the largest period.
"""
import numpy as np
import pytest

from oracle.qevict_oracle import EVICTED, FULL, QUANT, OracleConfig, QEvictUnit

W = 4


def _uniform_unit(decay, n_win=3, kf=16):
    cfg = OracleConfig(2, 1, 8, W, W, 4, kf, 0, score_decay=decay)
    u = QEvictUnit(cfg, W * n_win + 40)
    T0 = W * n_win
    u.prefill(np.zeros((1, T0, 8)), np.ones((1, T0, 8)), np.arange(1, n_win + 1) / 8.0)
    return u


def _expected_scores(init, steps, R, decay, T0):
    """Scores of the uniform-attention cache after `steps` decode steps."""
    s = {w: float(v) for w, v in enumerate(init)}
    new_period = True                    # prefill is a routing event
    for t in range(1, steps + 1):
        T = T0 + t
        n_started = -(-T // W)
        for w in range(n_started):
            s.setdefault(w, 0.0)
        if new_period:
            for w in s:
                s[w] *= decay
            new_period = False
        for w in range(n_started):
            s[w] += min(W, T - W * w) / T
        if t % R == 0:
            new_period = True
    return s


@pytest.mark.parametrize("decay,R", [(1.0, 1), (0.9, 1), (0.5, 3), (0.75, 3)])
def test_uniform_attention_recurrence(decay, R):
    u = _uniform_unit(decay)
    T0 = u.T
    init = u.score[:3].copy()
    steps = 13
    for t in range(1, steps + 1):
        u.step(np.ones((2, 8)), np.zeros((1, 8)), np.ones((1, 8)))
        if t % R == 0:
            u.route()
    exp = _expected_scores(init, steps, R, decay, T0)
    assert sorted(exp) == list(np.nonzero(u.state >= 0)[0])
    for w, v in exp.items():
        assert u.score[w] == pytest.approx(v, rel=1e-13, abs=1e-15), (w, v, u.score[w])
    assert all(u.state[w] == FULL for w in range(3))


def _bf16(rng, shape):
    x = rng.normal(size=shape).astype(np.float32)
    b = x.view(np.uint32).astype(np.uint64)
    b = ((b + 0x7FFF + ((b >> 16) & 1)) >> 16) << 16
    return b.astype(np.uint32).view(np.float32).astype(np.float64)


def _random_run(decay, seed=3, steps=12):
    rng = np.random.default_rng(seed)
    n_win = 10
    cfg = OracleConfig(4, 2, 16, W, W, 4, 3, 3, score_decay=decay)
    u = QEvictUnit(cfg, W * n_win + steps + 1)
    u.prefill(_bf16(rng, (2, W * n_win, 16)), _bf16(rng, (2, W * n_win, 16)),
              rng.permutation(n_win) / 10.0)
    traj = []
    for _ in range(steps):
        out, _, _ = u.step(_bf16(rng, (4, 16)) * 3.0, _bf16(rng, (2, 16)), _bf16(rng, (2, 16)))
        u.route()
        traj.append((out.copy(), u.score.copy(), u.state.copy()))
    return traj


def test_decay_near_one_follows_the_cumulative_score():
    """lambda = 1 - 1e-12 runs the decay arithmetic and stays on the cumulative
    trajectory: same outputs and tiers, scores within 1e-9 relative."""
    a = _random_run(1.0)
    b = _random_run(1.0 - 1e-12)
    for (oa, sa, ta), (ob, sb, tb) in zip(a, b):
        assert np.array_equal(ta, tb)
        assert np.allclose(oa, ob, rtol=1e-9, atol=1e-12)
        assert np.allclose(sa, sb, rtol=1e-9, atol=1e-12)
    assert OracleConfig(4, 2, 16, W, W, 4, 3, 3).score_decay == 1.0


def test_strong_decay_prefers_recent_attention():
    """Window 0 starts with a large score, window 1 (Quantized) then receives
    almost all attention.  After three steps the cumulative score still keeps
    window 0 in Full; with lambda = 0.5 window 1 has overtaken it (promoted,
    window 0 demoted)."""
    def run(decay):
        cfg = OracleConfig(1, 1, 8, W, W, 4, 1, 1, score_decay=decay)
        u = QEvictUnit(cfg, 3 * W + 20)
        k = np.zeros((1, 3 * W, 8))
        k[0, W:2 * W, 0] = 4.0          # window 1's keys respond to queries along channel 0
        u.prefill(k, np.ones((1, 3 * W, 8)), np.array([5.0, 0.0, 0.0]))
        assert u.state[0] == FULL and u.state[1] == QUANT and u.state[2] == EVICTED
        q = np.zeros((1, 8))
        q[0, 0] = 4.0
        for _ in range(3):
            u.step(q, np.zeros((1, 8)), np.ones((1, 8)))
            u.route()
        return u
    cum, dec = run(1.0), run(0.5)
    assert cum.state[0] == FULL and cum.state[1] == QUANT
    assert dec.state[1] == FULL and dec.state[0] == QUANT
    assert cum.score[0] > cum.score[1] and dec.score[1] > dec.score[0]


# ---- key-norm score (appendix, key-norm equation) ----

def _kn_unit(n_win, kf, kq, max_extra=40, heads=2):
    cfg = OracleConfig(4, heads, 8, W, W, 4, kf, kq, key_norm=True)
    return QEvictUnit(cfg, W * n_win + max_extra)


def _ramp_keys(T, heads=2):
    """Token i's key: head 0, channel 0 holds i + 1, everything else 0 (|k_i| = i + 1)."""
    k = np.zeros((heads, T, 8))
    k[0, :, 0] = np.arange(1, T + 1)
    return k


def test_key_norm_closed_form_prefill_and_decode():
    n_win, steps = 4, 9
    u = _kn_unit(n_win, 16, 0)
    T0 = W * n_win
    u.prefill(_ramp_keys(T0), np.ones((2, T0, 8)), None)
    rng = np.random.default_rng(0)
    for t in range(steps):
        kn = np.zeros((2, 8))
        kn[0, 0] = T0 + t + 1
        u.step(rng.normal(size=(4, 8)), kn, np.ones((2, 8)))
        u.route()
    T = T0 + steps
    for w in range(-(-T // W)):
        n_tok = min(W, T - w * W)
        expect = -sum(range(w * W + 1, w * W + n_tok + 1)) / W
        assert u.score[w] == pytest.approx(expect, rel=1e-14), w


def test_key_norm_ignores_attention():
    def run(seed):
        rng = np.random.default_rng(seed)
        u = _kn_unit(8, 2, 2)
        T0 = 8 * W
        kk = np.random.default_rng(7).normal(size=(2, T0 + 12, 8))
        u.prefill(kk[:, :T0], np.ones((2, T0, 8)), None)
        for t in range(12):
            u.step(rng.normal(size=(4, 8)) * 5, kk[:, T0 + t], np.ones((2, 8)))
            u.route()
        return u
    a, b = run(1), run(2)
    assert np.array_equal(a.score, b.score) and np.array_equal(a.state, b.state)


def test_key_norm_keeps_the_lowest_norm_windows():
    """Windows' keys scaled by distinct factors: Full gets the smallest norm,
    Quantized the next, the rest are evicted; a zero-key window (score 0, the
    largest possible) goes first."""
    n_win = 6
    factors = [3.0, 0.0, 5.0, 1.0, 2.0, 4.0]
    u = _kn_unit(n_win, 2, 2)
    rng = np.random.default_rng(3)
    base = rng.normal(size=(2, W, 8))
    k = np.concatenate([base * f for f in factors], axis=1)
    u.prefill(k, np.ones((2, n_win * W, 8)), None)
    order = sorted(range(n_win), key=lambda w: (factors[w], w))
    assert [u.state[w] for w in order] == [FULL, FULL, QUANT, QUANT, EVICTED, EVICTED]
    assert u.score[1] == 0.0
    # scaling a window's keys by 2 doubles its score exactly
    assert u.score[4] == pytest.approx(2.0 * u.score[3], rel=1e-15)


def test_key_norm_decode_accumulation_matches_prefill():
    """Scores of windows completed during decode equal the scores a prefill of
    the same tokens gives."""
    n0, steps = 5 * W, 3 * W + 2
    kk = np.random.default_rng(11).normal(size=(2, n0 + steps, 8))
    a = _kn_unit(8, 16, 0)
    a.prefill(kk[:, :n0], np.ones((2, n0, 8)), None)
    for t in range(steps):
        a.step(np.zeros((4, 8)), kk[:, n0 + t], np.ones((2, 8)))
    b = _kn_unit(8, 16, 0)
    b.prefill(kk, np.ones((2, n0 + steps, 8)), None)
    n = -(-(n0 + steps) // W)
    assert np.allclose(a.score[:n], b.score[:n], rtol=1e-13, atol=0)


# ---- attention p-norm (appendix, p-norm equation) ----

def _pnorm_uniform_unit(p, n_win=3):
    cfg = OracleConfig(2, 1, 8, W, W, 4, 16, 0, score_p=p)
    u = QEvictUnit(cfg, W * n_win + 40)
    T0 = W * n_win
    u.prefill(np.zeros((1, T0, 8)), np.ones((1, T0, 8)), np.arange(1, n_win + 1) / 8.0)
    return u


@pytest.mark.parametrize("p,R", [(3.0, 1), (3.0, 3), (2.0, 4), (1.5, 2)])
def test_pnorm_uniform_attention(p, R):
    """Uniform attention: the attention of a period is a sum of (tokens of the
    window) / (tokens held) over its steps; the score is the sum of the
    periods' p-th powers, the prompt score being the first period."""
    u = _pnorm_uniform_unit(p)
    T0 = u.T
    init = [1 / 8, 2 / 8, 3 / 8]
    periods = {w: [init[w]] for w in range(3)}
    cur: dict[int, float] = {}
    steps = 13
    for t in range(1, steps + 1):
        u.step(np.ones((2, 8)), np.zeros((1, 8)), np.ones((1, 8)))
        T = T0 + t
        for w in range(-(-T // W)):
            cur[w] = cur.get(w, 0.0) + min(W, T - W * w) / T
        expect = {w: sum(x ** p for x in periods.get(w, [])) + cur[w] ** p for w in cur}
        for w, v in expect.items():
            assert u.score[w] == pytest.approx(v, rel=1e-13), (t, w)
        if t % R == 0:
            u.route()
            for w, x in cur.items():
                periods.setdefault(w, []).append(x)
            cur = {w: 0.0 for w in cur}


def _run_scores(seed=5, steps=12, R=1, **kw):
    rng = np.random.default_rng(seed)
    n_win = 10
    cfg = OracleConfig(4, 2, 16, W, W, 4, 3, 3, **kw)
    u = QEvictUnit(cfg, W * n_win + steps + 1)
    u.prefill(_bf16(rng, (2, W * n_win, 16)), _bf16(rng, (2, W * n_win, 16)),
              rng.permutation(n_win) / 10.0)
    traj = []
    for t in range(steps):
        out, _, _ = u.step(_bf16(rng, (4, 16)) * 3.0, _bf16(rng, (2, 16)), _bf16(rng, (2, 16)))
        if (t + 1) % R == 0:
            u.route()
        traj.append((out.copy(), u.score.copy(), u.state.copy()))
    return traj, u


@pytest.mark.parametrize("R", [1, 3])
def test_pnorm_with_p_one_is_the_cumulative_score(R):
    a, _ = _run_scores(R=R)
    b, _ = _run_scores(R=R, score_p=1.0)
    for (oa, sa, ta), (ob, sb, tb) in zip(a, b):
        assert np.array_equal(ta, tb)
        assert np.allclose(oa, ob, rtol=1e-12, atol=1e-14)
        assert np.allclose(sa, sb, rtol=1e-12, atol=1e-14)


def test_pnorm_from_the_cumulative_increments():
    """With every window in Full (no routing decision depends on the score) the
    attention is the same under any ranking, so the periods' u_r are the
    increments of the cumulative score between routing events.  The p-norm run
    must give S^p = sum_r u_r^p of those, and S must lie between max_r u_r and
    n^(1/p) max_r u_r (p = 16 comes close to the maximum)."""
    R, steps, n_win = 2, 12, 10

    def run(**kw):
        rng = np.random.default_rng(9)
        cfg = OracleConfig(4, 2, 16, W, W, 4, 16, 0, **kw)
        u = QEvictUnit(cfg, W * n_win + steps + 1)
        u.prefill(_bf16(rng, (2, W * n_win, 16)), _bf16(rng, (2, W * n_win, 16)),
                  rng.permutation(n_win) / 10.0)
        at_events = [u.score.copy()]
        for t in range(steps):
            u.step(_bf16(rng, (4, 16)) * 3.0, _bf16(rng, (2, 16)), _bf16(rng, (2, 16)))
            if (t + 1) % R == 0:
                at_events.append(u.score.copy())
                u.route()
        return u, at_events

    cum, ev = run()
    for p in (3.0, 16.0):
        pn, _ = run(score_p=p)
        assert np.array_equal(cum.state, pn.state)
        n = -(-cum.T // W)
        for w in range(n):
            u_r = [ev[0][w]] + [ev[i][w] - ev[i - 1][w] for i in range(1, len(ev))]
            expect = sum(x ** p for x in u_r)
            assert pn.score[w] == pytest.approx(expect, rel=1e-9), (p, w)
            S, m = pn.score[w] ** (1 / p), max(u_r)
            assert m * (1 - 1e-9) <= S <= len(u_r) ** (1 / p) * m * (1 + 1e-9)
