"""Lockstep comparison of the HIP decode path with the float64 oracle.

Both sides receive the same seeded synthetic inputs.  At every routing event
the oracle first adopts the GPU's fp32 window scores (exactly, as float64), so
both rank identical numbers; tier decisions, ledger states, bit widths,
quantization codes and parameters, and promoted bf16 values must then agree
bit for bit.  Attention outputs must agree to max-abs <= 2e-3 * ||o||_2 per
(sequence, head) row, cumulative scores to 1e-4 relative with the floor
1e-7 * sum of scores.

Independent trajectory: beside each lockstep unit, a sample of sequences also
has an oracle unit that never adopts the GPU's scores; it routes on its own
float64 scores.  Until its tier map first differs from the GPU's, its outputs
and scores are held to the same bars; the first difference is recorded with
the relative score gap between the windows that changed places (per tier
boundary), and it must be a near-tie (gap <= 1e-4), the only way fp32 and
float64 scores may legitimately rank windows differently.
"""
from __future__ import annotations

import numpy as np
import torch

import paper_2608_05326_amd as qv
import synthetic as syn
from oracle.numerics import from_bf16_bits, from_fp16_bits
from oracle.qevict_oracle import DORMANT, OracleConfig, QEvictUnit, QUANT

OUT_TOL = 2e-3
SCORE_TOL = 1e-4
ORACLE_TO_ABI = np.array([0, 1, 1, 2, 3, 4])   # index = oracle state + 1


def abi_tiers(unit: QEvictUnit, n: int) -> np.ndarray:
    return ORACLE_TO_ABI[unit.state[:n] + 1].astype(np.int8)


def to_dev_bf16(bits: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def budget_capacities(wl: syn.Workload):
    """(K_f, K_q) of a workload given as a byte budget: a fraction of the full
    bf16 cache of the prompt (2 x H_kv x d x T x 2 bytes per layer and
    sequence) with quantized share q, through the library's capacity function."""
    from fractions import Fraction
    full = 2 * wl.num_kv_heads * wl.head_dim * wl.prompt_len * 2
    budget = int(Fraction(wl.budget_frac) * full)
    cfg = qv.Config(batch=wl.batch, num_q_heads=wl.num_q_heads, num_kv_heads=wl.num_kv_heads,
                    window_tokens=wl.window, group_size=wl.group, quant_bits=wl.bits,
                    max_context=wl.max_context, capacity_full=0, capacity_quant=0,
                    sink_tokens=wl.sink, recent_tokens=wl.recent, retier_interval=wl.retier_interval)
    return qv.qevict.capacities_for_budget(cfg, budget, int(Fraction(wl.q_frac) * 1000))


def gpu_config(wl: syn.Workload, layers: int, flags: int = 0, out_dtype: int = qv.OUT_F32,
               num_splits: int = 0, capacity_full=None, capacity_quant=None,
               score_decay: float | None = None, key_norm: bool = False,
               score_p: float | None = None, rope_base: float = 0.0) -> qv.Config:
    mode = qv.SCORE_KEY_NORM if key_norm else qv.SCORE_PNORM if score_p is not None else \
        qv.SCORE_DECAY if score_decay is not None else qv.SCORE_CUMULATIVE
    if wl.budget_frac:
        kf, kq = budget_capacities(wl)
        capacity_full = kf if capacity_full is None else capacity_full
        capacity_quant = kq if capacity_quant is None else capacity_quant
    return qv.Config(
        batch=wl.batch, num_layers=layers, num_q_heads=wl.num_q_heads, num_kv_heads=wl.num_kv_heads,
        window_tokens=wl.window, group_size=wl.group, quant_bits=wl.bits, max_context=wl.max_context,
        capacity_full=wl.capacity_full if capacity_full is None else capacity_full,
        capacity_quant=wl.capacity_quant if capacity_quant is None else capacity_quant,
        sink_tokens=wl.sink, recent_tokens=wl.recent, retier_interval=wl.retier_interval,
        out_dtype=out_dtype, flags=flags, num_splits=num_splits,
        score_mode=mode, score_decay=score_decay or 0.0, score_p=score_p or 0.0, rope_base=rope_base)


def oracle_config(cfg: qv.Config) -> OracleConfig:
    return OracleConfig(cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim, cfg.window_tokens,
                        cfg.group_size or cfg.window_tokens, cfg.quant_bits, cfg.capacity_full,
                        cfg.capacity_quant, sink=cfg.sink_tokens, recent=cfg.recent_tokens,
                        no_promotion=bool(cfg.flags & qv.FLAG_NO_PROMOTION),
                        score_decay=float(np.float32(cfg.score_decay))
                        if cfg.score_mode == qv.SCORE_DECAY else 1.0,
                        key_norm=cfg.score_mode == qv.SCORE_KEY_NORM,
                        score_p=float(np.float32(cfg.score_p))
                        if cfg.score_mode == qv.SCORE_PNORM else 0.0,
                        rope_base=float(np.float32(cfg.rope_base)))


class Lockstep:
    """Drive a GPU cache and oracle units with the same workload.

    layer_ids: which layers of the workload (seeds) the cache holds.
    check_seqs: sequences mirrored by the oracle (others run on the GPU only).
    """

    def __init__(self, wl: syn.Workload, seed: int = 0, layer_ids=(0,), check_seqs=None,
                 flags: int = 0, num_splits: int = 0, steps: int | None = None, log=print,
                 capacity_full=None, capacity_quant=None, score_decay: float | None = None,
                 key_norm: bool = False, score_p: float | None = None, observed_init: bool = False,
                 rope_base: float = 0.0, independent_seqs=None, progress_every: int = 0,
                 init_transform=None):
        self.wl, self.seed = wl, seed
        # optional map applied to the synthetic prompt scores (e.g. to plant ties)
        self.init_transform = init_transform
        self.layer_ids = list(layer_ids)
        self.check_seqs = list(range(wl.batch)) if check_seqs is None else list(check_seqs)
        self.steps = wl.steps if steps is None else steps
        self.cfg = gpu_config(wl, len(self.layer_ids), flags | qv.FLAG_DEBUG_MASSES,
                              num_splits=num_splits, capacity_full=capacity_full,
                              capacity_quant=capacity_quant, score_decay=score_decay,
                              key_norm=key_norm, score_p=score_p, rope_base=rope_base)
        self.key_norm = key_norm
        # modes whose prompt scores the GPU computes itself (key norms, u_0^p)
        self.gpu_prompt_scores = key_norm or score_p is not None
        # prompt scores from the observation queries' attention (GPU kernel,
        # checked against the oracle's, then given to both sides)
        self.observed_init = observed_init
        self.cache = qv.Cache(self.cfg)
        self.ocfg = oracle_config(self.cfg)
        self.units = {(li, b): QEvictUnit(self.ocfg, wl.max_context)
                      for li in range(len(self.layer_ids)) for b in self.check_seqs}
        # independent-trajectory units (own scores, never adopted)
        ind = [] if independent_seqs is None else list(independent_seqs)
        assert set(ind) <= set(self.check_seqs), "independent sequences must be mirrored"
        self.indep = {(li, b): QEvictUnit(self.ocfg, wl.max_context)
                      for li in range(len(self.layer_ids)) for b in ind}
        self.divergence = {}          # (li, b) -> first divergence record
        self.progress_every = progress_every
        self.log = log
        self.inputs = {}
        self.t = 0
        self.max_out_err = 0.0
        self.max_score_err = 0.0
        self.promotions = 0
        self.events = 0

    # ---- helpers ---------------------------------------------------------
    def _dec(self, li, b):
        key = (li, b)
        if key not in self.inputs:
            self.inputs[key] = syn.decode_inputs(self.wl, self.seed, b, self.layer_ids[li], self.steps)
        return self.inputs[key]

    def compare_ledgers(self, li, b, windows):
        u = self.units[(li, b)]
        for w in windows:
            e = u.ledger[w]
            ex = self.cache.export_window(li, b, int(w), quant=True)
            assert np.array_equal(ex["codes_k"], e["kc"].astype(np.uint8)), f"key codes, window {w}"
            assert np.array_equal(ex["codes_v"], e["vc"].astype(np.uint8)), f"value codes, window {w}"
            mk = from_fp16_bits(ex["meta_k"])
            mv = from_fp16_bits(ex["meta_v"])
            assert np.array_equal(mk[:, 0], e["ks"]) and np.array_equal(mk[:, 1], e["kz"]), \
                f"key scale / zero, window {w}"
            assert np.array_equal(mv[:, 0], e["vs"]) and np.array_equal(mv[:, 1], e["vz"]), \
                f"value scale / zero, window {w}"

    def compare_memory(self, li, b):
        from oracle.qevict_oracle import memory_report
        got = self.cache.memory_report(li, b)
        exp = memory_report(self.units[(li, b)])
        assert got == exp, f"memory report {got} != {exp}"

    def compare_full(self, li, b, windows):
        u = self.units[(li, b)]
        for w in windows:
            ex = self.cache.export_window(li, b, int(w), quant=False, full=True)
            assert np.array_equal(from_bf16_bits(ex["full_k"]), u.full_k[w]), f"bf16 keys, window {w}"
            assert np.array_equal(from_bf16_bits(ex["full_v"]), u.full_v[w]), f"bf16 values, window {w}"

    def compare_state(self, li, b, check_scores=True):
        u = self.units[(li, b)]
        st = self.cache.get_state(li, b)
        n = st["n"]
        assert np.array_equal(st["tiers"], abi_tiers(u, n)), \
            f"tiers differ at {np.nonzero(st['tiers'] != abi_tiers(u, n))[0][:10]}"
        assert np.array_equal(st["ledger"], u.ledger_states()[:n]), "ledger states"
        for w, e in u.ledger.items():
            assert st["bits"][w] == e["bits"], f"bit width, window {w}"
        if check_scores:
            live = (u.state[:n] >= 0) & (u.state[:n] != 4)
            so = u.score[:n][live]
            sg = st["scores"][live].astype(np.float64)
            floor = 1e-7 * np.abs(so).sum()
            err = np.abs(sg - so) / np.maximum(np.abs(so), floor)
            self.max_score_err = max(self.max_score_err, float(err.max(initial=0)))
            assert np.all(err <= SCORE_TOL), f"score rel err {err.max():.3e} at window {np.argmax(err)}"
        return st

    def check_scores(self, u, st, what):
        n = st["n"]
        live = (u.state[:n] >= 0) & (u.state[:n] != 4)
        so = u.score[:n][live]
        sg = st["scores"][live].astype(np.float64)
        floor = 1e-7 * np.abs(so).sum()
        err = np.abs(sg - so) / np.maximum(np.abs(so), floor)
        assert np.all(err <= SCORE_TOL), f"{what}: score rel err {err.max():.3e}"

    def compare_masses(self, got, mass, sink, u, t, b):
        """Per-head window masses of the step (the score increments before the
        head average): 1e-4 relative, floor 1e-7 (a head's masses sum to 1)."""
        n = min(u.n_win_cap, got.shape[1] - 1)
        ref = mass[:, :n]
        err = np.abs(got[:, :n].astype(np.float64) - ref) / np.maximum(np.abs(ref), 1e-7)
        assert np.all(err <= SCORE_TOL), \
            f"step {t} seq {b}: window mass rel err {err.max():.3e} (head, window " \
            f"{np.unravel_index(np.argmax(err), err.shape)})"
        tot = got[:, :n].astype(np.float64).sum(axis=1) + got[:, -1]
        assert np.all(np.abs(tot - 1.0) <= 1e-5), f"step {t} seq {b}: head masses sum to {tot}"

    def check_independent(self, li, b, pre_scores, where, st=None):
        """Tier maps (and bit widths) of the GPU and the independent unit after a
        routing event; the first difference is recorded and must be a near-tie."""
        ui = self.indep[(li, b)]
        if st is None:
            st = self.cache.get_state(li, b)
        n = st["n"]
        tg, ti = st["tiers"], abi_tiers(ui, n)
        bg = st["bits"][:n].astype(np.int64)
        bi = np.zeros(n, np.int64)
        for w, e in ui.ledger.items():
            if w < n:
                bi[w] = e["bits"]
        quant = tg == qv.TIER_QUANT
        diff = np.nonzero((tg != ti) | (quant & (ti == qv.TIER_QUANT) & (bg != bi)))[0]
        if len(diff) == 0:
            assert np.array_equal(st["ledger"], ui.ledger_states()[:n]), \
                f"independent ledger states at {where} (tiers agree)"
            return
        sc = ui.score if pre_scores is None else pre_scores
        groups = {}
        for w in diff:
            pair = tuple(sorted((int(tg[w]), int(ti[w]))))
            key = "bits" if pair[0] == pair[1] else {(2, 3): "full/quant", (3, 4): "quant/evict",
                                                     (2, 4): "full/evict"}.get(pair, str(pair))
            groups.setdefault(key, []).append(float(sc[w]))
        gaps = {k: (max(v) - min(v)) / max(abs(x) for x in v) if len(v) > 1 else float("inf")
                for k, v in groups.items()}
        self.divergence[(li, b)] = dict(where=where, n_windows=int(len(diff)),
                                        gaps={k: f"{g:.2e}" for k, g in gaps.items()})
        self.log(f"[lockstep] independent layer {li} seq {b}: first divergence at {where}, "
                 f"windows {diff[:8].tolist()}, relative score gaps {gaps}")
        assert all(g <= SCORE_TOL for g in gaps.values()), \
            f"independent run diverged at {where} without a near-tie: gaps {gaps}"

    # ---- phases ------------------------------------------------------------
    def prefill(self):
        wl = self.wl
        from concurrent.futures import ThreadPoolExecutor

        def gen(b, layer):
            k, v = syn.prompt_kv(wl, self.seed, b, layer)
            init = syn.init_scores(wl, self.seed, b, layer)
            if self.init_transform is not None:
                init = np.ascontiguousarray(self.init_transform(init), dtype=np.float32)
            return k, v, init

        for li, layer in enumerate(self.layer_ids):
            with ThreadPoolExecutor(max_workers=min(8, wl.batch)) as ex:
                prompts = list(ex.map(lambda b: gen(b, layer), range(wl.batch)))
            ks = [p[0] for p in prompts]
            vs = [p[1] for p in prompts]
            inits = [p[2] for p in prompts]
            del prompts
            K = to_dev_bf16(np.stack(ks))
            V = to_dev_bf16(np.stack(vs))
            S = None if self.key_norm else torch.from_numpy(np.stack(inits)).cuda()
            if self.observed_init:
                from oracle.qevict_oracle import prefill_window_scores
                qo = [syn.observation_queries(wl, self.seed, b, layer, wl.window) for b in range(wl.batch)]
                S = self.cache.prefill_scores(to_dev_bf16(np.stack(qo)), K)
                got = S.cpu().numpy()
                for b in self.check_seqs:
                    ref = prefill_window_scores(from_bf16_bits(qo[b]), from_bf16_bits(ks[b]),
                                                wl.sink, wl.window)
                    err = np.abs(got[b] - ref) / np.maximum(np.abs(ref), 1e-7 * np.abs(ref).sum())
                    assert np.all(err <= SCORE_TOL), f"observed prompt score rel err {err.max():.3e}"
                    inits[b] = got[b]
            for b in range(wl.batch):
                if (li, b) in self.units:
                    # key-norm and p-norm prompt scores: the GPU computes its own
                    self.units[(li, b)].prefill(from_bf16_bits(ks[b]), from_bf16_bits(vs[b]), inits[b],
                                                route=not self.gpu_prompt_scores)
                if (li, b) in self.indep:
                    self.indep[(li, b)].prefill(from_bf16_bits(ks[b]), from_bf16_bits(vs[b]), inits[b])
            self.cache.prefill_assign(li, K, V, S)
            torch.cuda.synchronize()
            del K, V
            for b in self.check_seqs:
                u = self.units[(li, b)]
                if self.gpu_prompt_scores:
                    # fp32 against fp64 arithmetic: check the scores, then route both
                    # with the GPU's so that near-ties rank alike
                    st = self.cache.get_state(li, b)
                    n = st["n"]
                    so, sg = u.score[:n], st["scores"].astype(np.float64)
                    err = np.abs(sg - so) / np.maximum(np.abs(so), 1e-7 * np.abs(so).sum())
                    assert np.all(err <= SCORE_TOL), f"prefill score rel err {err.max():.3e}"
                    u.adopt_scores(sg)
                    u.finish_prefill()
                self.compare_state(li, b)
                self.compare_memory(li, b)
                self.compare_ledgers(li, b, sorted(u.ledger))
                if (li, b) in self.indep:
                    self.check_independent(li, b, None, "prefill")
                full = [w for w in range(u.n_win_cap) if u.state[w] == 2]
                self.compare_full(li, b, full[:: max(1, len(full) // 16)])

    def forced_shift(self, li, b_all):
        """Shift the keys of a low-ranked quantized window toward this step's query."""
        wl = self.wl
        ev = self.t // wl.shift_every
        for b in b_all:
            st = self.cache.get_state(li, b)
            q = np.nonzero(st["tiers"] == qv.TIER_QUANT)[0]
            low = sorted(q, key=lambda w: (st["scores"][w], -w))
            w = syn.pick_shift_window(wl, self.seed, b, self.layer_ids[li], ev, low)
            qbits = self._dec(li, b)[0][self.t]
            delta = syn.shift_delta(wl, qbits)
            self.cache.debug_shift_keys(li, b, w, delta)
            if (li, b) in self.units:
                self.units[(li, b)].shift_key_zero_points(w, delta)
            if (li, b) in self.indep and (li, b) not in self.divergence:
                self.indep[(li, b)].shift_key_zero_points(w, delta)

    def step(self):
        wl, t = self.wl, self.t
        B, Hq, d = wl.batch, wl.num_q_heads, wl.head_dim
        routing = (t + 1) % wl.retier_interval == 0
        for li in range(len(self.layer_ids)):
            if wl.forced_shift and t % wl.shift_every == 0:
                self.forced_shift(li, range(B))
            qs = np.stack([self._dec(li, b)[0][t] for b in range(B)])
            kn = np.stack([self._dec(li, b)[1][t] for b in range(B)])
            vn = np.stack([self._dec(li, b)[2][t] for b in range(B)])
            out = torch.empty((B, Hq, d), dtype=torch.float32, device="cuda")
            self.cache.decode_attend(li, to_dev_bf16(qs), to_dev_bf16(kn), to_dev_bf16(vn), out)
            out = out.cpu().numpy()
            gm = self.cache.debug_masses(li)
            pre_scores = {}
            for b in self.check_seqs:
                u = self.units[(li, b)]
                o, mass, sink = u.step(from_bf16_bits(qs[b]), from_bf16_bits(kn[b]),
                                       from_bf16_bits(vn[b]))
                err = np.abs(out[b] - o).max(axis=1) / np.linalg.norm(o, axis=1)
                self.max_out_err = max(self.max_out_err, float(err.max()))
                assert np.all(err <= OUT_TOL), f"step {t} seq {b}: out rel err {err.max():.3e}"
                if not self.key_norm:
                    self.compare_masses(gm[b], mass, sink, u, t, b)
                st = self.compare_state(li, b)
                pre_scores[b] = st["scores"].astype(np.float64)
                if routing:
                    u.adopt_scores(pre_scores[b])
                if (li, b) in self.indep and (li, b) not in self.divergence:
                    ui = self.indep[(li, b)]
                    oi, _, _ = ui.step(from_bf16_bits(qs[b]), from_bf16_bits(kn[b]), from_bf16_bits(vn[b]))
                    erri = np.abs(out[b] - oi).max(axis=1) / np.linalg.norm(oi, axis=1)
                    assert np.all(erri <= OUT_TOL), f"independent step {t} seq {b}: out rel err {erri.max():.3e}"
                    self.check_scores(ui, st, f"independent step {t} seq {b}")
            if routing:
                stats = self.cache.retier(li, stats=True)
                self.events += 1
                self.promotions += stats["promotions"]
                for b in self.check_seqs:
                    u = self.units[(li, b)]
                    before_ledger = set(u.ledger)
                    before_state = u.state.copy()
                    u.route()
                    st = self.compare_state(li, b, check_scores=False)
                    self.compare_memory(li, b)
                    new_led = [w for w in u.ledger if w not in before_ledger]
                    self.compare_ledgers(li, b, new_led)
                    promoted = [w for w in range(u.n_win_cap)
                                if before_state[w] == QUANT and u.state[w] == 2]
                    admitted = [w for w in range(u.n_win_cap)
                                if before_state[w] in (0, 1) and u.state[w] == 2]
                    self.compare_full(li, b, promoted + admitted)
                    for w in promoted:
                        assert u.ledger[w]["state"] == DORMANT
                    if (li, b) in self.indep and (li, b) not in self.divergence:
                        ui = self.indep[(li, b)]
                        pre = ui.score.copy()
                        ui.route()
                        self.check_independent(li, b, pre, f"step {t}", st)
        self.t += 1
        if self.progress_every and self.t % self.progress_every == 0:
            self.log(f"[lockstep] {self.wl.name}: step {self.t}/{self.steps}, max out err "
                     f"{self.max_out_err:.2e}, max score err {self.max_score_err:.2e}, "
                     f"promotions {self.promotions}, diverged {sorted(self.divergence)}")

    def run(self):
        self.prefill()
        for _ in range(self.steps):
            self.step()
        return self

    def report_independent(self):
        """One line per independent unit: no divergence, or its first divergence."""
        lines = []
        for key in sorted(self.indep):
            d = self.divergence.get(key)
            lines.append(f"layer {key[0]} seq {key[1]}: " +
                         ("no divergence" if d is None else
                          f"first divergence at {d['where']}: {d['n_windows']} windows, "
                          f"boundaries {d['gaps']}"))
        return lines

    def close(self):
        self.cache.close()
