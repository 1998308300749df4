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
  old attention that the cumulative score still remembers.
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
