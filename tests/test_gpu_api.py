"""GPU tests of the C ABI beyond lockstep parity: single-window moves against
the oracle, protocol and argument errors, latched device errors, the one-way
policy, bf16 output, run-to-run determinism, the all-Full special case
against plain attention, and the smoke entry point.
"""
import ctypes

import numpy as np
import pytest

import synthetic as syn

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    return torch


# ---------------------------------------------------------------------------
# single-window moves (qevict_quantize_window / qevict_promote_window)
# ---------------------------------------------------------------------------

def test_manual_moves_match_oracle():
    from tests.gpu_harness import Lockstep
    from oracle.qevict_oracle import FULL, QUANT
    wl = syn.get_workload("c1s")
    # 64 prompt windows: 8 Full, 56 Quantized, room for 4 more Quantized
    ls = Lockstep(wl, capacity_full=8, capacity_quant=60, steps=4)
    try:
        ls.prefill()
        u, c = ls.units[(0, 0)], ls.cache
        f = [int(w) for w in np.nonzero(u.state == FULL)[0]]
        w = f[2]
        c.quantize_window(0, 0, w)          # first quantization
        u.quantize_one(w)
        ls.compare_state(0, 0)
        ls.compare_ledgers(0, 0, [w])
        first = c.export_window(0, 0, w, quant=True)
        c.promote_window(0, 0, w)           # dequantize-promote, ledger dormant
        u.promote_one(w)
        ls.compare_state(0, 0)
        ls.compare_full(0, 0, [w])
        c.quantize_window(0, 0, w)          # reactivation: same codes, no requantization
        u.quantize_one(w)
        ls.compare_state(0, 0)
        again = c.export_window(0, 0, w, quant=True)
        for k in first:
            assert np.array_equal(first[k], again[k]), k
        q = [int(x) for x in np.nonzero(u.state == QUANT)[0]]
        c.promote_window(0, 0, q[-1])       # a Quantized window with a fresh ledger
        u.promote_one(q[-1])
        ls.compare_state(0, 0)
        ls.compare_full(0, 0, [q[-1]])
        # attention and routing keep agreeing after the moves
        for _ in range(ls.steps):
            ls.step()
    finally:
        ls.close()


def test_manual_move_errors():
    import paper_2608_05326_amd as qv
    from tests.gpu_harness import Lockstep
    from oracle.qevict_oracle import EVICTED, FULL, QUANT
    wl = syn.get_workload("c1s")         # 16 Full, 24 Quantized, 24 evicted: both tiers full
    ls = Lockstep(wl, steps=0)
    try:
        ls.prefill()
        u, c = ls.units[(0, 0)], ls.cache
        f = int(np.nonzero(u.state == FULL)[0][0])
        q = int(np.nonzero(u.state == QUANT)[0][0])
        e = int(np.nonzero(u.state == EVICTED)[0][0])
        cases = [(c.quantize_window, f, qv.ERR_CAPACITY), (c.promote_window, q, qv.ERR_CAPACITY),
                 (c.quantize_window, q, qv.ERR_BAD_STATE), (c.promote_window, f, qv.ERR_BAD_STATE),
                 (c.quantize_window, e, qv.ERR_BAD_STATE), (c.promote_window, e, qv.ERR_BAD_STATE),
                 (c.quantize_window, 10 ** 6, qv.ERR_INVALID_ARG)]
        for fn, w, code in cases:
            with pytest.raises(qv.QEvictError) as ex:
                fn(0, 0, w)
            assert ex.value.status == code, (fn.__name__, w, ex.value)
        ls.compare_state(0, 0)               # nothing changed
    finally:
        ls.close()


# ---------------------------------------------------------------------------
# protocol, arguments and latched device errors
# ---------------------------------------------------------------------------

def _small_cache(flags=0, out_dtype=None, max_context=None, layers=1):
    import paper_2608_05326_amd as qv
    from tests.gpu_harness import gpu_config
    wl = syn.get_workload("c2s")
    if max_context is not None:
        wl = wl.replace(steps=max_context - wl.prompt_len)
    cfg = gpu_config(wl, layers, flags, out_dtype=qv.OUT_F32 if out_dtype is None else out_dtype)
    return wl, qv.Cache(cfg)


def _prompt(wl, seq=0, layer=0):
    from tests.gpu_harness import to_dev_bf16
    torch = _torch()
    k, v = syn.prompt_kv(wl, 0, seq, layer)
    s = syn.init_scores(wl, 0, seq, layer)
    return to_dev_bf16(k[None]), to_dev_bf16(v[None]), torch.from_numpy(s[None].copy()).cuda()


def _step_inputs(wl, t, seq=0, layer=0):
    from tests.gpu_harness import to_dev_bf16
    qs, ks, vs = syn.decode_inputs(wl, 0, seq, layer, t + 1)
    return to_dev_bf16(qs[t][None]), to_dev_bf16(ks[t][None]), to_dev_bf16(vs[t][None])


def test_protocol_and_argument_errors():
    import paper_2608_05326_amd as qv
    torch = _torch()
    wl, c = _small_cache(max_context=32 * 96 + 13 + 2)
    try:
        out = torch.empty((1, wl.num_q_heads, 128), dtype=torch.float32, device="cuda")
        q, kn, vn = _step_inputs(wl, 0)
        with pytest.raises(qv.QEvictError) as ex:          # decode before prefill
            c.decode_attend(0, q, kn, vn, out)
        assert ex.value.status == qv.ERR_BAD_STATE
        with pytest.raises(qv.QEvictError) as ex:          # routing before prefill
            c.retier(0)
        assert ex.value.status == qv.ERR_BAD_STATE
        with pytest.raises(qv.QEvictError) as ex:          # layer out of range
            c.retier(1)
        assert ex.value.status == qv.ERR_INVALID_ARG
        K, V, S = _prompt(wl)
        # extents that differ from the configuration are rejected on the host
        with pytest.raises(ValueError):                    # two sequences for a batch of one
            c.prefill_assign(0, torch.cat([K, K]), torch.cat([V, V]), S)
        with pytest.raises(ValueError):                    # scores for one window too many
            c.prefill_assign(0, K, V, torch.cat([S, S[:, :1]], dim=1))
        with pytest.raises(ValueError):
            c.decode_attend(0, torch.cat([q, q]), kn, vn, out)
        with pytest.raises(ValueError):
            c.decode_attend(0, q, kn[:, :1].contiguous(), vn, out)
        c.prefill_assign(0, K, V, S)
        with pytest.raises(qv.QEvictError) as ex:          # second prefill of a layer
            c.prefill_assign(0, K, V, S)
        assert ex.value.status == qv.ERR_BAD_STATE
        lib, h = c.lib, c.handle
        null = ctypes.c_void_p(None)
        p = lambda t: ctypes.c_void_p(t.data_ptr())
        st = lib.qevict_decode_attend(h, 0, null, p(kn), p(vn), p(out))
        assert st == qv.ERR_INVALID_ARG
        st = lib.qevict_decode_attend(h, 0, ctypes.c_void_p(q.data_ptr() + 2), p(kn), p(vn), p(out))
        assert st == qv.ERR_INVALID_ARG                     # misaligned query
        # the cache is still usable after rejected calls
        for t in range(2):
            q, kn, vn = _step_inputs(wl, t)
            c.decode_attend(0, q, kn, vn, out)
            c.retier(0)
        q, kn, vn = _step_inputs(wl, 2)
        with pytest.raises(qv.QEvictError) as ex:          # max_context reached
            c.decode_attend(0, q, kn, vn, out)
        assert ex.value.status == qv.ERR_BAD_STATE
        assert torch.isfinite(out).all()
    finally:
        c.close()


def test_nonfinite_initial_score_latches_error():
    import paper_2608_05326_amd as qv
    wl, c = _small_cache()
    try:
        K, V, S = _prompt(wl)
        S[0, 3] = float("nan")
        c.prefill_assign(0, K, V, S)                        # enqueued; checked on the device
        with pytest.raises(qv.QEvictError) as ex:
            c.get_state(0, 0)
        assert ex.value.status == qv.ERR_NONFINITE
        with pytest.raises(qv.QEvictError) as ex:          # the cache now only accepts destroy
            c.retier(0)
        assert ex.value.status == qv.ERR_BAD_STATE
    finally:
        c.close()


# ---------------------------------------------------------------------------
# policies, output type, determinism
# ---------------------------------------------------------------------------

def test_one_way_policy_lockstep():
    import paper_2608_05326_amd as qv
    from tests.gpu_harness import Lockstep
    ls = Lockstep(syn.get_workload("c2s"), flags=qv.FLAG_NO_PROMOTION, steps=16)
    try:
        ls.run()
    finally:
        ls.close()
    assert ls.promotions == 0 and ls.events == 16


def _run_gpu_only(wl, steps, out_dtype, flags=0):
    torch = _torch()
    wl_, c = _small_cache(flags=flags, out_dtype=out_dtype)
    outs, states = [], []
    try:
        K, V, S = _prompt(wl)
        c.prefill_assign(0, K, V, S)
        dt = torch.bfloat16 if out_dtype == 1 else torch.float32
        for t in range(steps):
            q, kn, vn = _step_inputs(wl, t)
            out = torch.empty((1, wl.num_q_heads, 128), dtype=dt, device="cuda")
            c.decode_attend(0, q, kn, vn, out)
            c.retier(0)
            outs.append(out.cpu())
            st = c.get_state(0, 0)
            states.append(st)
    finally:
        c.close()
    return outs, states


def test_repeat_runs_are_bitwise_identical():
    wl = syn.get_workload("c2s")
    o1, s1 = _run_gpu_only(wl, 8, 0)
    o2, s2 = _run_gpu_only(wl, 8, 0)
    for a, b in zip(o1, o2):
        assert _torch().equal(a, b)
    for a, b in zip(s1, s2):
        for k in ("tiers", "scores", "ledger", "bits"):
            assert np.array_equal(a[k], b[k]), k


def test_bf16_output_is_rounded_fp32_output():
    torch = _torch()
    wl = syn.get_workload("c2s")
    o32, s32 = _run_gpu_only(wl, 6, 0)
    o16, s16 = _run_gpu_only(wl, 6, 1)
    for a, b in zip(o32, o16):
        assert torch.equal(a.to(torch.bfloat16), b)
    for a, b in zip(s32, s16):
        assert np.array_equal(a["scores"], b["scores"])


# ---------------------------------------------------------------------------
# all-Full special case: plain attention over every token
# ---------------------------------------------------------------------------

def test_all_full_equals_plain_attention():
    import paper_2608_05326_amd as qv
    from tests.gpu_harness import gpu_config, to_dev_bf16
    from oracle.numerics import from_bf16_bits
    torch = _torch()
    wl = syn.get_workload("c2s")
    n_hist = wl.n_hist_windows
    cfg = gpu_config(wl, 1, capacity_full=n_hist, capacity_quant=0)
    c = qv.Cache(cfg)
    try:
        k, v = syn.prompt_kv(wl, 0, 0, 0)
        c.prefill_assign(0, to_dev_bf16(k[None]), to_dev_bf16(v[None]),
                         torch.from_numpy(syn.init_scores(wl, 0, 0, 0)[None].copy()).cuda())
        qs, ks, vs = syn.decode_inputs(wl, 0, 0, 0, 5)
        K = torch.from_numpy(from_bf16_bits(k))          # float64 [H_kv, T, d]
        V = torch.from_numpy(from_bf16_bits(v))
        G = wl.num_q_heads // wl.num_kv_heads
        for t in range(5):
            out = torch.empty((1, wl.num_q_heads, 128), dtype=torch.float32, device="cuda")
            c.decode_attend(0, to_dev_bf16(qs[t][None]), to_dev_bf16(ks[t][None]),
                            to_dev_bf16(vs[t][None]), out)
            c.retier(0)
            K = torch.cat([K, torch.from_numpy(from_bf16_bits(ks[t]))[:, None]], dim=1)
            V = torch.cat([V, torch.from_numpy(from_bf16_bits(vs[t]))[:, None]], dim=1)
            q = torch.from_numpy(from_bf16_bits(qs[t])).view(wl.num_kv_heads, G, 128)
            ref = torch.softmax(q @ K.transpose(1, 2) / np.sqrt(128.0), dim=-1) @ V   # [H_kv, G, d]
            ref = ref.reshape(wl.num_q_heads, 128).numpy()
            got = out[0].cpu().numpy().astype(np.float64)
            err = np.abs(got - ref).max(axis=1) / np.linalg.norm(ref, axis=1)
            assert np.all(err <= 2e-3), err.max()
        st = c.get_state(0, 0)
        assert not np.any(st["tiers"] == qv.TIER_QUANT) and not np.any(st["tiers"] == qv.TIER_EVICTED)
    finally:
        c.close()


def test_smoke_entry_point():
    import __graft_entry__
    __graft_entry__.smoke()


# ---------------------------------------------------------------------------
# asynchronous routing (routing stream + per-layer ordering)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("name,kw,order", [("c2s", {}, None), ("c3s", {}, None),
                                           ("c5s", {"rope_base": 500000.0}, None),
                                           ("c5s", {"score_p": 3.0}, None), ("c2s", {"score_decay": 0.9}, None),
                                           ("c4s", {}, None), ("c6w8s", {}, "device"), ("c2s", {}, "queue")])
def test_async_routing_lockstep(name, kw, order):
    """Routing on its own stream, also with RoPE, the p-norm over 8-step periods
    and the decayed score (the period bookkeeping happens at enqueue time), with
    the ordering the cache chooses (queue-level wait for c4s and c5s, the
    device-side gate for the others) or a forced one (`order`)."""
    import paper_2608_05326_amd as qv
    from tests.gpu_harness import Lockstep
    extra = {None: 0, "device": qv.FLAG_ROUTING_DEVICE_WAIT, "queue": qv.FLAG_ROUTING_QUEUE_WAIT}[order]
    ls = Lockstep(syn.get_workload(name), flags=qv.FLAG_ASYNC_ROUTING | extra, steps=12, **kw)
    try:
        ls.run()
    finally:
        ls.close()


@pytest.mark.parametrize("n_layers,twice,queue_wait", [(4, False, False), (9, False, False),
                                                       (16, False, False), (5, True, False),
                                                       (4, False, True), (9, False, True)])
def test_async_routing_interleaved_layers_match_sync(n_layers, twice, queue_wait):
    """Several layers stepped back to back with no host synchronisation: the
    routing of each layer overlaps the attention of the others and every
    output and final state equals the single-stream run bit for bit.  Routing
    requests are launched in batches, one re-rank and one migration launch per
    batch (2 layers with 4 layers, 4 with 9, 8 with 16), so with 9 layers the
    last layer's request is still queued when its state is read; with `twice`
    every layer is routed twice per step, and a layer already queued starts a
    new batch.  Batches follow the cache stream through the device-side wait,
    or with `queue_wait` a queue-level wait (QEVICT_FLAG_ROUTING_QUEUE_WAIT)."""
    import paper_2608_05326_amd as qv
    from tests.gpu_harness import gpu_config, to_dev_bf16
    torch = _torch()
    wl = syn.get_workload("c2s")
    steps = 10

    def run(flags):
        c = qv.Cache(gpu_config(wl, n_layers, flags))
        outs = []
        try:
            for l in range(n_layers):
                k, v = syn.prompt_kv(wl, 0, 0, l)
                s = syn.init_scores(wl, 0, 0, l)
                c.prefill_assign(l, to_dev_bf16(k[None]), to_dev_bf16(v[None]),
                                 torch.from_numpy(s[None].copy()).cuda())
            dec = [syn.decode_inputs(wl, 0, 0, l, steps) for l in range(n_layers)]
            ins = [[tuple(to_dev_bf16(x[t][None]) for x in dec[l]) for t in range(steps)]
                   for l in range(n_layers)]
            for t in range(steps):
                for l in range(n_layers):
                    out = torch.empty((1, wl.num_q_heads, 128), dtype=torch.float32, device="cuda")
                    c.decode_attend(l, *ins[l][t], out)
                    c.retier(l)
                    if twice:
                        c.retier(l)
                    outs.append(out)
            last = c.get_state(n_layers - 1, 0)
            c.join_routing()
            torch.cuda.synchronize()
            states = [c.get_state(l, 0) for l in range(n_layers)]
            return [o.cpu() for o in outs], states + [last]
        finally:
            c.close()

    o_sync, s_sync = run(0)
    o_async, s_async = run(qv.FLAG_ASYNC_ROUTING | (qv.FLAG_ROUTING_QUEUE_WAIT if queue_wait else 0))
    for a, b in zip(o_sync, o_async):
        assert torch.equal(a, b)
    for a, b in zip(s_sync, s_async):
        for k in ("tiers", "scores", "ledger", "bits"):
            assert np.array_equal(a[k], b[k]), k


@pytest.mark.parametrize("name,kw,flags,order", [
    ("c2s", {}, "async", "gate"),                     # 32-token windows, GQA 4: 204 + 204 + 79 registers
    ("c6s", {}, "async", "gate"),
    ("c2s", {"rope_base": 500000.0}, "async", "queue"),   # RoPE-aware attention: 256 registers
    ("c4s", {}, "async", "queue"),                    # 64-token windows: 256 registers
    ("c5s", {}, "async", "queue"),                    # GQA 8: 217 + 217 + 79
    ("c6w8s", {}, "async", "queue"),                  # 8-token windows: 222 + 222 + 96
    ("c2s", {}, "async+queue", "queue"),
    ("c6w8s", {}, "async+device", "gate"),
    ("c2s", {}, "sync", "sync"),
])
def test_routing_order_follows_kernel_footprints(name, kw, flags, order):
    """Routing batches follow the cache stream through the device-side wait
    where a migration workgroup fits on a compute unit beside two attention
    workgroups, else through the queue-level wait; either flag forces one."""
    import paper_2608_05326_amd as qv
    from tests.gpu_harness import gpu_config
    f = {"async": qv.FLAG_ASYNC_ROUTING, "async+queue": qv.FLAG_ASYNC_ROUTING | qv.FLAG_ROUTING_QUEUE_WAIT,
         "async+device": qv.FLAG_ASYNC_ROUTING | qv.FLAG_ROUTING_DEVICE_WAIT, "sync": 0}[flags]
    c = qv.Cache(gpu_config(syn.get_workload(name), 1, f, **kw))
    try:
        want = {"gate": c.ROUTING_GATE, "queue": c.ROUTING_QUEUE_WAIT, "sync": c.ROUTING_SYNC}[order]
        assert c.routing_order() == want
    finally:
        c.close()


def test_routing_gate_time_out_skips_routing_and_reports():
    """The routing stream waits on the device for the cache stream's published
    sequence number.  Forced from the host to time out (the cache stream stops
    publishing, 2 ms limit): the waiting batch's re-rank and migrations leave
    the layer as it was, the layer's next synchronous call reports
    QEVICT_ERR_BAD_STATE naming the skipped routing, later calls report the
    poisoned cache, and destroying the cache returns (every wait ended)."""
    import paper_2608_05326_amd as qv
    from paper_2608_05326_amd.qevict import QEvictError
    from tests.gpu_harness import gpu_config, to_dev_bf16
    torch = _torch()
    wl = syn.get_workload("c2s")
    for flags in (0, qv.FLAG_ASYNC_ROUTING | qv.FLAG_ROUTING_QUEUE_WAIT):
        c = qv.Cache(gpu_config(wl, 2, flags))
        try:
            with pytest.raises(QEvictError) as ei:
                c.debug_routing_gate(2000, False)      # no device-side wait to test
            assert ei.value.status == -1
        finally:
            c.close()
    c = qv.Cache(gpu_config(wl, 2, qv.FLAG_ASYNC_ROUTING))
    try:
        for l in range(2):
            k, v = syn.prompt_kv(wl, 0, 0, l)
            s = syn.init_scores(wl, 0, 0, l)
            c.prefill_assign(l, to_dev_bf16(k[None]), to_dev_bf16(v[None]),
                             torch.from_numpy(s[None].copy()).cuda())
        with pytest.raises(QEvictError):
            c.debug_routing_gate(0, False)
        dec = [syn.decode_inputs(wl, 0, 0, l, 1) for l in range(2)]
        out = torch.empty((1, wl.num_q_heads, 128), dtype=torch.float32, device="cuda")
        # a routed step first: the gate releases it
        c.decode_attend(0, *(to_dev_bf16(x[0][None]) for x in dec[0]), out)
        c.retier(0)
        c.join_routing()
        torch.cuda.synchronize()
        c.get_state(0, 0)
        c.debug_routing_gate(2000, False)
        c.decode_attend(1, *(to_dev_bf16(x[0][None]) for x in dec[1]), out)
        c.retier(1)
        c.join_routing()
        torch.cuda.synchronize()
        with pytest.raises(QEvictError) as ei:
            c.get_state(1, 0)
        assert ei.value.status == -4 and "routing skipped" in str(ei.value), str(ei.value)
        with pytest.raises(QEvictError) as ei:
            c.get_state(0, 0)
        assert ei.value.status == -4
    finally:
        c.close()


def test_debug_last_masses_matches_debug_masses():
    """The debug call for the cache's full window capacity returns the per-head
    window masses of the last step (each head's masses, sink included, sum to 1)."""
    import paper_2608_05326_amd as qv
    from tests.gpu_harness import gpu_config, to_dev_bf16
    torch = _torch()
    wl = syn.get_workload("c2s")
    c = qv.Cache(gpu_config(wl, 1, qv.FLAG_DEBUG_MASSES))
    try:
        k, v = syn.prompt_kv(wl, 0, 0, 0)
        s = syn.init_scores(wl, 0, 0, 0)
        c.prefill_assign(0, to_dev_bf16(k[None]), to_dev_bf16(v[None]), torch.from_numpy(s[None].copy()).cuda())
        q, kn, vn = (to_dev_bf16(x[0][None]) for x in syn.decode_inputs(wl, 0, 0, 0, 1))
        out = torch.empty((1, wl.num_q_heads, 128), dtype=torch.float32, device="cuda")
        c.decode_attend(0, q, kn, vn, out)
        a, b = c.debug_masses(0), c.debug_last_masses(0)
        assert np.array_equal(a, b)
        assert np.allclose(b.sum(axis=-1, dtype=np.float64), 1.0, atol=1e-5)
    finally:
        c.close()
