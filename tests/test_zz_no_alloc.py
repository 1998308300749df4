"""The allocation-free initial-score call (qevict_prefill_scores_noalloc, on
the library's fixed per-device scratch) against qevict_prefill_scores with a
caller scratch buffer: bitwise the same scores on two calls in a row, the
second with a smaller prompt (the fixed scratch still holds the first call's
contents), and a prompt that needs more scratch than the fixed array is
refused without touching the output."""
import numpy as np
import pytest

import synthetic as syn

pytestmark = pytest.mark.gpu

FIXED_BYTES = 16 << 20   # QEVICT_STATIC_SCRATCH_BYTES


def _dev(bits):
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def test_noalloc_matches_caller_scratch():
    import torch
    import paper_2608_05326_amd as qv
    base = syn.get_workload("c2")
    cfg = qv.Config(batch=1, num_q_heads=base.num_q_heads, num_kv_heads=base.num_kv_heads,
                    window_tokens=base.window, group_size=base.group, quant_bits=base.bits,
                    max_context=base.prompt_len + 64, capacity_full=base.capacity_full,
                    capacity_quant=base.capacity_quant)
    cache = qv.Cache(cfg)
    try:
        # the 8B / 32K prompt with 32 observation queries, then a smaller ragged one
        for T, n_obs in ((base.prompt_len, 32), (32 * 128 + 17, 8)):
            need = qv.qevict.prefill_scores_scratch_size(cfg, T, n_obs)
            assert need <= FIXED_BYTES, need
            wl = base.replace(prompt_len=T)
            K = _dev(syn.prompt_kv(wl, 3, 0, 0)[0][None])
            Q = _dev(syn.observation_queries(wl, 3, 0, 0, n_obs)[None])
            n_w = -(-T // cfg.window_tokens)
            print(f"[no-alloc] prompt {T}, {n_obs} observation queries, scratch {need} bytes",
                  flush=True)
            ref = cache.prefill_scores(Q, K)
            got = torch.full((1, n_w), float("nan"), dtype=torch.float32, device="cuda")
            cache.prefill_scores_noalloc(Q, K, got)
            torch.cuda.synchronize()
            assert torch.equal(got, ref), \
                f"prompt {T}: max diff {(got - ref).abs().max().item():.3e}"
        # more scratch than the fixed array: refused, nothing enqueued
        T, n_obs = base.prompt_len, 128
        assert qv.qevict.prefill_scores_scratch_size(cfg, T, n_obs) > FIXED_BYTES
        K = torch.zeros((1, cfg.num_kv_heads, T, 128), dtype=torch.bfloat16, device="cuda")
        Q = torch.zeros((1, cfg.num_q_heads, n_obs, 128), dtype=torch.bfloat16, device="cuda")
        out = torch.full((1, T // 32), -7.0, dtype=torch.float32, device="cuda")
        with pytest.raises(qv.QEvictError) as ei:
            cache.prefill_scores_noalloc(Q, K, out)
        assert ei.value.status == qv.ERR_WORKSPACE
        torch.cuda.synchronize()
        assert bool((out == -7.0).all())
    finally:
        cache.close()
