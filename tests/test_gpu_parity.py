"""GPU parity of the HIP decode path against the float64 oracle (lockstep).

Every case drives the C ABI through the ctypes binding on the GPU and the
oracle on the CPU with the same seeded inputs; see gpu_harness for the bars.
"""
import numpy as np
import pytest

import synthetic as syn

pytestmark = pytest.mark.gpu


def _lockstep(name, **kw):
    from tests.gpu_harness import Lockstep
    wl = syn.get_workload(name)
    ls = Lockstep(wl, **kw)
    print(f"[lockstep] {name} seed={ls.seed} steps={ls.steps}", flush=True)
    try:
        ls.run()
    finally:
        ls.close()
    print(f"[lockstep] {name}: max out err {ls.max_out_err:.2e}, max score err {ls.max_score_err:.2e}, "
          f"promotions {ls.promotions} over {ls.events} events", flush=True)
    return ls


def test_c1_forced_promotions():
    ls = _lockstep("c1", independent_seqs=[0])
    assert ls.promotions >= ls.wl.steps // ls.wl.shift_every
    print("[lockstep] c1 independent " + "; ".join(ls.report_independent()), flush=True)


@pytest.mark.parametrize("name", ["c1s", "c2s", "c4s", "c5s", "c3s"])
def test_small_workloads_lockstep(name):
    ls = _lockstep(name, independent_seqs=[0])
    print(f"[lockstep] {name} independent " + "; ".join(ls.report_independent()), flush=True)


@pytest.mark.parametrize("name,decay", [("c2s", 0.99), ("c5s", 0.9)])
def test_decayed_score_lockstep(name, decay):
    """Exponentially decayed ranking (lambda per routing period; c5s routes every
    8 steps): scores and routing against the oracle."""
    _lockstep(name, score_decay=decay)


@pytest.mark.parametrize("name", ["c2s", "c4s"])
def test_key_norm_lockstep(name):
    """Key-norm ranking (scores from the keys alone, computed by the prefill
    kernel and the merge's per-token update): scores and routing against the
    oracle."""
    _lockstep(name, key_norm=True)


@pytest.mark.parametrize("name", ["c2s", "c5s"])
def test_pnorm_lockstep(name):
    """Attention p-norm ranking, p = 3 (per step on c2s; periods of 8 steps on
    c5s): scores (held as S^p) and routing against the oracle."""
    _lockstep(name, score_p=3.0)


@pytest.mark.parametrize("name", ["c6s", "c7s"])
def test_sink_and_recent_lockstep(name):
    """Protected sink and recent regions: c6s is the paper's default point (5
    sink and 32 recent tokens, routing every 8 steps, int2, capacities from a
    20% byte budget with q = 0.70); c7s has a sink of two and a half windows,
    a recent region of 70 tokens, routing every 3 steps and mixed bits."""
    ls = _lockstep(name)
    assert ls.events > 0


@pytest.mark.parametrize("name,splits", [("c2s", 1), ("c2s", 7), ("c5s", 64)])
def test_split_counts(name, splits):
    """One split, an odd count, and 64 splits of 4 waves for about 50 items
    (most waves get no window): outputs and masses against the oracle."""
    _lockstep(name, num_splits=splits, steps=12)


@pytest.mark.parametrize("kf,kq", [(0, 28), (19, 0), (40, 60)])
def test_tier_extremes(kf, kq):
    """Quantized tier only (K_f = 0), eviction only (K_q = 0, the two-tier
    policy) and more capacity than windows (nothing is evicted)."""
    ls = _lockstep("c2s", capacity_full=kf, capacity_quant=kq, steps=16)
    assert ls.events == 16


@pytest.mark.parametrize("name,base", [("c2s", 10000.0), ("c4s", 500000.0), ("c5s", 500000.0),
                                       ("c7s", 10000.0)])
def test_rope_lockstep(name, base):
    """RoPE-aware Quantized tier: codes of the un-rotated keys (bit-exact),
    attention over dequantized keys rotated back to their positions, promotions
    rotated in float64 (bit-exact), on int4 W 32, int2 W 64, mixed bits with
    8-step periods, and sink / recent regions."""
    ls = _lockstep(name, rope_base=base)
    assert ls.events > 0


@pytest.mark.parametrize("prompt,sink,steps", [(5, 0, 100), (16, 16, 70)])
def test_short_prompts(prompt, sink, steps):
    """A prompt shorter than one window (nothing routed at prefill) and a prompt
    that is only sink tokens (no prompt window, no initial scores): windows are
    started, aged and routed during decode (K_f = 1, K_q = 1)."""
    from tests.gpu_harness import Lockstep
    wl = syn.get_workload("c2s").replace(name=f"short{prompt}", prompt_len=prompt, sink=sink, steps=steps)
    ls = Lockstep(wl, capacity_full=1, capacity_quant=1)
    print(f"[lockstep] short prompt {prompt} sink {sink} steps {steps}", flush=True)
    try:
        ls.run()
    finally:
        ls.close()
    print(f"[lockstep] short: max out err {ls.max_out_err:.2e}, promotions {ls.promotions}", flush=True)
    assert ls.events == steps


@pytest.mark.parametrize("hq,hkv", [(24, 2), (12, 4), (32, 2), (1, 1), (2, 1), (2, 2)])
def test_head_layouts(hq, hkv):
    """Query-head counts that are not powers of two (the merge sums heads through
    LDS instead of a butterfly) and GQA ratios 12 and 16 (four 4-head groups per
    wave in the attention kernel), plus GQA 3; one and two query heads (the
    per-head split statistics are folded by 64 threads of one wave, and the
    window masses must still sum to one per head)."""
    from tests.gpu_harness import Lockstep
    wl = syn.get_workload("c2s").replace(name=f"h{hq}x{hkv}", num_q_heads=hq, num_kv_heads=hkv, steps=16)
    ls = Lockstep(wl)
    print(f"[lockstep] heads {hq}/{hkv}", flush=True)
    try:
        ls.run()
    finally:
        ls.close()
    print(f"[lockstep] heads {hq}/{hkv}: max out err {ls.max_out_err:.2e}, "
          f"max score err {ls.max_score_err:.2e}, promotions {ls.promotions}", flush=True)


@pytest.mark.parametrize("bits", [4, 42])
def test_window64_bit_widths(bits):
    """64-token windows with int4 and with the mixed int4 / int2 tier (c4s is int2)."""
    wl_name = "c4s"
    from tests.gpu_harness import Lockstep
    wl = syn.get_workload(wl_name).replace(name=f"w64b{bits}", bits=bits, steps=16)
    ls = Lockstep(wl)
    try:
        ls.run()
    finally:
        ls.close()
    print(f"[lockstep] W 64 bits {bits}: max out err {ls.max_out_err:.2e}, promotions {ls.promotions}",
          flush=True)


@pytest.mark.parametrize("bits", [2, 4, 42])
def test_window8_paper_default(bits):
    """The paper's 8-token windows at its default point (sink 5, recent 32,
    routing every 8 steps, byte-budget capacities with q = 0.70) at reduced
    size: int2 as in the paper, int4, and the mixed tier."""
    from tests.gpu_harness import Lockstep
    wl = syn.get_workload("c6w8s").replace(name=f"c6w8s-b{bits}", bits=bits)
    ls = Lockstep(wl, independent_seqs=[0])
    print(f"[lockstep] {wl.name} steps={ls.steps}", flush=True)
    try:
        ls.run()
    finally:
        ls.close()
    print(f"[lockstep] W 8 bits {bits}: max out err {ls.max_out_err:.2e}, max score err "
          f"{ls.max_score_err:.2e}, promotions {ls.promotions} over {ls.events} events; "
          + "; ".join(ls.report_independent()), flush=True)


def test_window8_routing_every_step():
    """8-token windows on the 8B head layout with a routing event after every
    step (windows age, are admitted, quantized and promoted each step), int4."""
    from tests.gpu_harness import Lockstep
    wl = syn.get_workload("c2s").replace(name="w8r1", window=8, group=32, prompt_len=8 * 200 + 3,
                                         steps=40)
    ls = Lockstep(wl, independent_seqs=[0])
    try:
        ls.run()
    finally:
        ls.close()
    print(f"[lockstep] W 8 R 1: max out err {ls.max_out_err:.2e}, promotions {ls.promotions}; "
          + "; ".join(ls.report_independent()), flush=True)
    assert ls.promotions > 0


@pytest.mark.parametrize("name,window,R,steps", [("c6w8s", 8, 10, 40), ("c6s", 32, 40, 90)])
def test_split_plans_over_routing_periods(name, window, R, steps):
    """The re-rank kernel writes split plans for the steps up to the next routing
    event, one slot per count of recent-region windows (two slots); with a
    routing interval longer than W + 1 some steps of a period need a third count
    and split the list in the attention kernel.  Outputs and masses against the
    oracle across those boundaries, 8- and 32-token windows."""
    from tests.gpu_harness import Lockstep
    wl = syn.get_workload(name).replace(name=f"{name}-r{R}", retier_interval=R, steps=steps)
    assert wl.window == window and R - 1 > window
    ls = Lockstep(wl)
    print(f"[lockstep] {wl.name}", flush=True)
    try:
        ls.run()
    finally:
        ls.close()
    print(f"[lockstep] plans W {window} R {R}: max out err {ls.max_out_err:.2e}, "
          f"max score err {ls.max_score_err:.2e}, events {ls.events}", flush=True)
    assert ls.events >= 2


@pytest.mark.parametrize("hq,hkv,splits", [(8, 8, 0), (6, 2, 0), (4, 2, 1), (32, 8, 64), (16, 2, 0)])
def test_window8_head_layouts_and_splits(hq, hkv, splits):
    """8-token windows with at most four query heads per KV head are computed in
    pairs, one window per column block of the QK^T tile: GQA 1 and 3 (blocks
    partly empty), GQA 2 on one split (every wave a long run of pairs), and 64
    splits (short runs: waves with one window, an unpaired last window, or none),
    with the paper's sink / recent regions and int2 codes; GQA 8 takes the
    one-window-at-a-time path."""
    from tests.gpu_harness import Lockstep
    wl = syn.get_workload("c6w8s").replace(name=f"w8h{hq}x{hkv}s{splits}", num_q_heads=hq,
                                           num_kv_heads=hkv, steps=24)
    ls = Lockstep(wl, num_splits=splits)
    print(f"[lockstep] {wl.name}", flush=True)
    try:
        ls.run()
    finally:
        ls.close()
    print(f"[lockstep] W 8 heads {hq}/{hkv} splits {splits}: max out err {ls.max_out_err:.2e}, "
          f"max score err {ls.max_score_err:.2e}, promotions {ls.promotions}", flush=True)
    assert ls.events > 0


@pytest.mark.parametrize("pattern", ["all_equal", "three_values", "coarse_grid", "outlier"])
@pytest.mark.parametrize("wl_name", ["c2s", "c5s"])
def test_tier_selection_with_tied_scores(wl_name, pattern):
    """The re-rank kernel selects tier positions by counting keys per bucket of
    the score range.  Planted prompt scores make buckets hold many equal keys
    (all equal, three values: the general refinement), a few equal keys
    (coarse grid: ranked pairwise within the bucket) or squeeze the bulk into
    one bucket beside a far outlier; tiers must still follow the total order
    (score descending, then window) at the prefill routing and every later
    event, on the 8B head layout (int4) and the 70B one (mixed int4 / int2)."""
    from tests.gpu_harness import Lockstep

    def transform(x):
        if pattern == "all_equal":
            return np.ones_like(x)
        if pattern == "three_values":
            return np.choose(np.arange(x.size) % 3, [0.5, 1.0, 2.0]).astype(np.float32)
        if pattern == "coarse_grid":
            return np.round(x * 8.0) / 8.0
        y = x.copy()
        y[y.size // 2] = 1e30
        return y

    wl = syn.get_workload(wl_name).replace(steps=9)   # the 70B layout routes every 8 steps
    ls = Lockstep(wl, init_transform=transform)
    try:
        ls.run()
    finally:
        ls.close()
    print(f"[lockstep] {wl_name} {pattern}: max out err {ls.max_out_err:.2e}, events {ls.events}",
          flush=True)
