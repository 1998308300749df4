"""GPU parity at the full workload sizes, in the launch configuration the
benchmark times (default split count), against the float64 oracle.

Each case runs its workload's whole decode length in lockstep (outputs, per-head
window masses, scores, tiers, ledgers, codes, promoted values; see gpu_harness
for the bars).  Where a workload has several sequences or layers, every
sequence runs on the GPU and a sample of them is mirrored by the oracle.  One
mirrored sequence per case also runs an independent oracle trajectory on its
own float64 scores; its first divergence from the GPU, if any, must be a
near-tie.
"""
import pytest

import synthetic as syn

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def _lockstep(name, independent=(0,), **kw):
    from tests.gpu_harness import Lockstep
    wl = syn.get_workload(name)
    ls = Lockstep(wl, independent_seqs=independent, progress_every=32, **kw)
    print(f"[fullsize] {name} prompt={wl.prompt_len} B={wl.batch} steps={ls.steps} "
          f"layers={ls.layer_ids} checked seqs={ls.check_seqs}", flush=True)
    try:
        ls.run()
    finally:
        ls.close()
    print(f"[fullsize] {name}: max out err {ls.max_out_err:.2e}, max score err {ls.max_score_err:.2e}, "
          f"promotions {ls.promotions} over {ls.events} events", flush=True)
    for line in ls.report_independent():
        print(f"[fullsize] {name} independent {line}", flush=True)
    return ls


def test_8b_32k_bench_config():
    # 128 decode steps, routing every step (about two promotions per step)
    ls = _lockstep("c2")
    assert ls.events == 128


def test_8b_128k_int2_w64():
    # 64 decode steps at 128K context, int2 windows of 64 tokens
    ls = _lockstep("c4")
    assert ls.events == 64


def test_70b_64k_mixed_bits_batch4():
    # 128 steps, routing every 8: 16 routing events; sequences 0 and 3 mirrored
    ls = _lockstep("c5", check_seqs=[0, 3])
    assert ls.events == 16


def test_8b_32k_batch8_two_layers():
    # layers 0 and 31 of the 32, all 8 sequences of each on the GPU, 256 steps
    # routing every step; sequences 0 and 7 mirrored
    ls = _lockstep("c3", layer_ids=(0, 31), check_seqs=[0, 7])
    assert ls.events == 2 * 256


def test_8b_32k_paper_default_point():
    # 5 sink + 32 recent tokens, int2, capacities from a 20% byte budget with q = 0.70
    # (61 bf16 + 759 int2 windows), 128 steps, routing every 8 steps
    ls = _lockstep("c6")
    assert ls.events == 16


def test_max_candidates_4000_windows():
    # 4000 routed prompt windows of 32 tokens (the re-rank kernel sorts up to 4096
    # candidates in one workgroup): K_f = 1000, K_q = 3000, two routing events
    wl = syn.get_workload("c2").replace(name="cmax", prompt_len=32 * 4000 + 5, steps=2,
                                        frac_full="0.25", frac_quant="0.75")
    from tests.gpu_harness import Lockstep
    ls = Lockstep(wl, steps=2, independent_seqs=[0])
    print(f"[fullsize] cmax prompt={wl.prompt_len} K_f={ls.cfg.capacity_full} "
          f"K_q={ls.cfg.capacity_quant}", flush=True)
    try:
        ls.run()
    finally:
        ls.close()
    print(f"[fullsize] cmax: max out err {ls.max_out_err:.2e}, max score err {ls.max_score_err:.2e}",
          flush=True)


def test_8b_32k_rope():
    # the benchmark shape with the RoPE-aware Quantized tier (Llama-3 base 500000)
    _lockstep("c2", steps=16, rope_base=500000.0)


def test_8b_32k_paper_default_eight_token_windows():
    # the paper's default point with its 8-token windows: sink 5, recent 32, int2,
    # byte budget 20% with q = 0.70 (244 bf16 + 2025 int2 windows of 4091), routing
    # every 8 steps, 128 steps
    ls = _lockstep("c6w8")
    assert ls.events == 16
