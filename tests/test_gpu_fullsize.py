"""GPU parity at the full workload sizes, in the launch configuration the
benchmark times (default split count), against the float64 oracle.

Each case runs a few lockstep steps (outputs, scores, tiers, ledgers, codes,
promoted values; see gpu_harness for the bars).  Where a workload has
several sequences or layers, every sequence runs on the GPU and a sample of
them is mirrored by the oracle.
"""
import pytest

import synthetic as syn

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def _lockstep(name, **kw):
    from tests.gpu_harness import Lockstep
    wl = syn.get_workload(name)
    ls = Lockstep(wl, **kw)
    print(f"[fullsize] {name} prompt={wl.prompt_len} B={wl.batch} steps={ls.steps} "
          f"layers={ls.layer_ids} checked seqs={ls.check_seqs}", flush=True)
    try:
        ls.run()
    finally:
        ls.close()
    print(f"[fullsize] {name}: max out err {ls.max_out_err:.2e}, max score err {ls.max_score_err:.2e}, "
          f"promotions {ls.promotions} over {ls.events} events", flush=True)
    return ls


def test_8b_32k_bench_config():
    _lockstep("c2", steps=6)


def test_8b_128k_int2_w64():
    _lockstep("c4", steps=3)


def test_70b_64k_mixed_bits_batch4():
    # routing every 8 steps: step 8 is the first routing event
    _lockstep("c5", steps=9, check_seqs=[0, 3])


def test_8b_32k_batch8_layer_sample():
    # one of the 32 layers, all 8 sequences on the GPU, two mirrored
    _lockstep("c3", steps=3, layer_ids=(31,), check_seqs=[0, 7])


def test_8b_32k_paper_default_point():
    # 5 sink + 32 recent tokens, int2, capacities from a 20% byte budget with q = 0.70
    # (61 bf16 + 759 int2 windows), routing every 8 steps: step 8 is the first event
    _lockstep("c6", steps=9)


def test_max_candidates_4000_windows():
    # 4000 routed prompt windows of 32 tokens (the re-rank kernel sorts up to 4096
    # candidates in one workgroup): K_f = 1000, K_q = 3000, two routing events
    wl = syn.get_workload("c2").replace(name="cmax", prompt_len=32 * 4000 + 5, steps=2,
                                        frac_full="0.25", frac_quant="0.75")
    from tests.gpu_harness import Lockstep
    ls = Lockstep(wl, steps=2)
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
    _lockstep("c2", steps=4, rope_base=500000.0)
