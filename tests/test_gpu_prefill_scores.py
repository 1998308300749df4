"""GPU parity of the initial-window-score kernels (qevict_prefill_scores)
against the float64 oracle: scores within 1e-4 relative (floor 1e-7 of the
total), on seeded synthetic prompts: several key blocks with a ragged tail,
more query rows than one LDS chunk, n_obs = 1, n_obs = T, sinks with partial
windows, every window size, GQA 1 to 8, and the full 32K / 64K prompt
shapes of the 8B and 70B layouts.  Also: bitwise repeatability and the
prefill that consumes the scores.
"""
import numpy as np
import pytest

import synthetic as syn

pytestmark = pytest.mark.gpu

TOL = 1e-4


def _rel_err(got, ref):
    floor = 1e-7 * np.abs(ref).sum()
    return np.abs(got - ref) / np.maximum(np.abs(ref), floor)


def _cache(B, H_q, H_kv, W, T, sink, max_extra=64, **kw):
    import paper_2608_05326_amd as qv
    cfg = qv.Config(batch=B, num_q_heads=H_q, num_kv_heads=H_kv, window_tokens=W, quant_bits=4,
                    max_context=T + max_extra, capacity_full=4, capacity_quant=4, sink_tokens=sink,
                    **kw)
    return qv.Cache(cfg)


def _bf16(rng, shape, scale=1.0):
    return syn.f32_to_bf16_bits((rng.standard_normal(shape) * scale).astype(np.float32))


CASES = [
    # B, H_q, H_kv, W, T, n_obs, sink
    (2, 32, 8, 32, 1037, 32, 0),     # 8B heads, five key blocks, ragged tail
    (1, 8, 1, 64, 300, 17, 5),       # one KV head, rows not a multiple of 16, sink
    (1, 64, 8, 32, 777, 32, 4),      # GQA 8: 256 rows (two LDS chunks)
    (1, 4, 4, 32, 256, 1, 0),        # GQA 1, one query, exactly one block
    (1, 16, 2, 64, 40, 40, 3),       # every prompt query observes, one partial block
    (1, 8, 2, 32, 20, 4, 20),        # the whole prompt is sink: no window
    (1, 32, 8, 8, 1037, 32, 5),      # 8-token windows: eight per 64-key block, sink, ragged tail
    (2, 8, 2, 8, 300, 9, 0),         # 8-token windows, GQA 4, batch 2
]


@pytest.mark.parametrize("case", CASES, ids=[f"B{c[0]}-Hq{c[1]}-Hkv{c[2]}-W{c[3]}-T{c[4]}-obs{c[5]}-s{c[6]}"
                                              for c in CASES])
def test_prefill_scores_match_oracle(case):
    import torch
    from oracle.qevict_oracle import prefill_window_scores
    from tests.gpu_harness import to_dev_bf16
    B, H_q, H_kv, W, T, n_obs, sink = case
    print(f"[prefill_scores] case {case}", flush=True)
    rng = np.random.default_rng(sum(case))
    q = _bf16(rng, (B, H_q, n_obs, 128), 2.0)
    k = _bf16(rng, (B, H_kv, T, 128))
    cache = _cache(B, H_q, H_kv, W, T, sink)
    try:
        got = cache.prefill_scores(to_dev_bf16(q), to_dev_bf16(k)).cpu().numpy()
        torch.cuda.synchronize()
    finally:
        cache.close()
    n_w = max(0, -(-(T - sink) // W))
    assert got.shape == (B, n_w)
    for b in range(B):
        ref = prefill_window_scores(syn.bf16_bits_to_f32(q[b]).astype(np.float64),
                                    syn.bf16_bits_to_f32(k[b]).astype(np.float64), sink, W)
        err = _rel_err(got[b].astype(np.float64), ref)
        print(f"[prefill_scores] seq {b}: max rel err {err.max(initial=0):.2e}", flush=True)
        assert np.all(err <= TOL)


@pytest.mark.parametrize("name,seqs", [("c2", [0]), ("c5", [0, 3])])
def test_prefill_scores_full_prompt(name, seqs):
    """The 8B / 32K and 70B / 64K (batch 4) prompt shapes, W observation
    queries from the synthetic query recipe; the oracle checks the listed
    sequences."""
    import torch
    from oracle.qevict_oracle import prefill_window_scores
    from tests.gpu_harness import to_dev_bf16
    wl = syn.get_workload(name)
    n_obs = wl.window
    print(f"[prefill_scores] {name} prompt={wl.prompt_len} B={wl.batch} n_obs={n_obs}", flush=True)
    ks, qs = [], []
    for b in range(wl.batch):
        k, _ = syn.prompt_kv(wl, 0, b, 0)
        ks.append(k)
        qs.append(syn.observation_queries(wl, 0, b, 0, n_obs))
    K, Q = to_dev_bf16(np.stack(ks)), to_dev_bf16(np.stack(qs))
    cache = _cache(wl.batch, wl.num_q_heads, wl.num_kv_heads, wl.window, wl.prompt_len, wl.sink)
    try:
        got = cache.prefill_scores(Q, K)
        again = cache.prefill_scores(Q, K)
        torch.cuda.synchronize()
        assert torch.equal(got, again), "not bitwise repeatable"
        got = got.cpu().numpy()
    finally:
        cache.close()
    del K, Q
    for b in seqs:
        ref = prefill_window_scores(syn.bf16_bits_to_f32(qs[b]).astype(np.float64),
                                    syn.bf16_bits_to_f32(ks[b]).astype(np.float64), wl.sink, wl.window)
        err = _rel_err(got[b].astype(np.float64), ref)
        print(f"[prefill_scores] {name} seq {b}: max rel err {err.max():.2e}, "
              f"sum {got[b].sum():.4f} (oracle {ref.sum():.4f})", flush=True)
        assert np.all(err <= TOL)


def test_prefill_scores_feed_prefill():
    """Lockstep on the reduced 8B workload with the GPU's observation scores
    as the prompt scores of both sides (checked against the oracle's first)."""
    from tests.gpu_harness import Lockstep
    wl = syn.get_workload("c2s")
    ls = Lockstep(wl, steps=8, observed_init=True)
    print(f"[lockstep] c2s observed init, steps={ls.steps}", flush=True)
    try:
        ls.run()
    finally:
        ls.close()
    print(f"[lockstep] c2s observed init: max out err {ls.max_out_err:.2e}, "
          f"max score err {ls.max_score_err:.2e}", flush=True)
