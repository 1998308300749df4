"""Pins for the oracle's initial window scores from prompt attention (Sec. 4.2:
prompt attention initialises the window scores; the observation queries are
the last n_obs prompt positions).

* zero queries attend uniformly: query at position tau gives window w the
  share |w within [0, tau]| / (tau + 1), written out here;
* torch's scaled_dot_product_attention (float64, CPU) with a causal mask and
  the window-indicator matrix as values returns each query's per-window
  masses directly; the KV heads are repeated for the query heads, which pins
  the head-to-group mapping;
* every query's probabilities sum to one: window scores plus the sink's mass
  equal n_obs;
* scores add over observation queries, and a query sees only keys up to its
  own position (splitting the observation window and truncating the prompt
  gives the same sum);
* a query aligned with one window's keys puts nearly all its mass there.
"""
import math

import numpy as np
import pytest
import torch

from oracle.qevict_oracle import prefill_window_scores


def _owner(T, sink, W):
    o = np.full(T, -1)
    o[sink:] = (np.arange(sink, T) - sink) // W
    return o


@pytest.mark.parametrize("T,n_obs,sink,W", [(37, 5, 0, 8), (40, 16, 3, 8), (9, 9, 1, 4)])
def test_uniform_attention_closed_form(T, n_obs, sink, W):
    H_q, H_kv, d = 4, 2, 8
    s = prefill_window_scores(np.zeros((H_q, n_obs, d)), np.random.default_rng(0).normal(size=(H_kv, T, d)),
                              sink, W)
    n_w = -(-(T - sink) // W)
    expect = np.zeros(n_w)
    for j in range(n_obs):
        tau = T - n_obs + j
        for w in range(n_w):
            a, b = sink + w * W, min(sink + (w + 1) * W, tau + 1)
            expect[w] += max(0, b - a) / (tau + 1)
    assert np.allclose(s, expect, rtol=1e-13, atol=1e-15)


@pytest.mark.parametrize("gqa", [1, 4])
def test_matches_torch_sdpa_with_window_indicator_values(gqa):
    rng = np.random.default_rng(gqa)
    H_kv, T, d, n_obs, sink, W = 2, 45, 16, 7, 5, 8
    H_q = H_kv * gqa
    q = rng.normal(size=(H_q, n_obs, d)) * 2
    k = rng.normal(size=(H_kv, T, d))
    scale = 0.3
    s = prefill_window_scores(q, k, sink, W, scale)
    owner = _owner(T, sink, W)
    n_w = owner.max() + 1
    ind = np.zeros((T, n_w))
    ind[np.arange(T)[owner >= 0], owner[owner >= 0]] = 1.0
    pos_q = np.arange(T - n_obs, T)
    mask = torch.from_numpy(np.arange(T)[None, :] <= pos_q[:, None])   # True = attend
    kt = torch.from_numpy(np.repeat(k, gqa, axis=0))
    vt = torch.from_numpy(np.broadcast_to(ind, (H_q, T, n_w)).copy())
    m = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q), kt, vt, attn_mask=mask, scale=scale)        # [H_q, n_obs, n_w]
    ref = m.sum(dim=(0, 1)).numpy() / H_q
    assert np.allclose(s, ref, rtol=1e-12, atol=1e-14)


def test_mass_conservation():
    rng = np.random.default_rng(3)
    H_q, H_kv, T, d, n_obs, sink, W = 8, 2, 50, 8, 12, 0, 16
    s = prefill_window_scores(rng.normal(size=(H_q, n_obs, d)), rng.normal(size=(H_kv, T, d)), sink, W)
    assert s.sum() == pytest.approx(n_obs, rel=1e-13)
    # with a sink the windows get what the sink does not
    k = rng.normal(size=(H_kv, T, d))
    k[:, :4] = 0.0
    q = np.zeros((H_q, n_obs, d))
    s4 = prefill_window_scores(q, k, 4, W)
    sink_mass = sum(4 / (T - n_obs + j + 1) for j in range(n_obs))
    assert s4.sum() + sink_mass == pytest.approx(n_obs, rel=1e-13)


def test_additive_over_queries_and_causal():
    """The last query's share plus the rest's on the prompt without its last
    token (which they cannot see) gives the whole."""
    rng = np.random.default_rng(4)
    H_q, H_kv, T, d, n_obs, sink, W = 4, 1, 33, 8, 6, 2, 8
    q = rng.normal(size=(H_q, n_obs, d))
    k = rng.normal(size=(H_kv, T, d))
    whole = prefill_window_scores(q, k, sink, W)
    last = prefill_window_scores(q[:, -1:], k, sink, W)
    rest = prefill_window_scores(q[:, :-1], k[:, :-1], sink, W)
    rest = np.pad(rest, (0, len(whole) - len(rest)))
    assert np.allclose(whole, last + rest, rtol=1e-13, atol=1e-15)


def test_aligned_query_concentrates_on_one_window():
    H_q, H_kv, T, d, n_obs, W = 2, 1, 64, 8, 4, 16
    k = np.zeros((H_kv, T, d))
    k[0, 2 * W:3 * W, 0] = 20.0
    q = np.zeros((H_q, n_obs, d))
    q[:, :, 0] = 20.0 * math.sqrt(d)
    s = prefill_window_scores(q, k, 0, W)
    assert s[2] > n_obs * (1 - 1e-9)
    assert np.argmax(s) == 2
