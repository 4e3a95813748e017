"""Drive the GPU library and the CPU oracle over the same seeded inputs.

Inputs come only from ``synth`` (host generator); expected values only from
``oracle``.  The GPU side goes through the C ABI (ctypes binding).
"""
from __future__ import annotations

import numpy as np

import oracle
from synth import gen

# acceptance bounds for attention outputs computed from bf16/fp32 K/V
ATOL = 2e-2
RTOL_NORM = 1e-2
ENTROPY_TOL = 1e-3
MARGIN = 1e-3


# --------------------------------------------------------------------------
# inputs
# --------------------------------------------------------------------------

class Inputs:
    """Host copies of a workload's inputs, generated on demand and cached."""

    def __init__(self, w, attempts=None):
        self.w = w
        self.attempts = attempts or {}
        self._kv = {}

    def kv(self, layer, seq):
        key = (layer, seq)
        if key not in self._kv:
            n = self.w.prefill[seq] + self.w.steps
            self._kv[key] = gen.kv_rows(self.w, layer, seq, 0, n, self.attempts.get(key))
        return self._kv[key]

    def prompt(self, layer, seq):
        K, V = self.kv(layer, seq)
        P = self.w.prefill[seq]
        return K[:P], V[:P]

    def new_token(self, layer, seq, t):
        K, V = self.kv(layer, seq)
        p = self.w.prefill[seq] + t - 1
        return K[p], V[p]

    def q(self, layer, seq, t):
        return gen.q_row(self.w, layer, seq, t)

    def logits(self, seq, t):
        return gen.logits_row(self.w, seq, t)


def fix_margin(w, max_rounds=20):
    """Re-draw keys until every relevance score keeps |s - tau| >= MARGIN at
    every step (tiny workloads; scores from the oracle over all positions)."""
    attempts = {}
    for _ in range(max_rounds):
        inp = Inputs(w, attempts)
        bad_any = False
        for l in range(w.n_layers):
            for b in range(w.batch):
                K, _ = inp.kv(l, b)
                P = w.prefill[b]
                bad = np.zeros(len(K), bool)
                for t in range(1, w.steps + 1):
                    n = P + t
                    s = oracle.relevance(inp.q(l, b, t), K[:n])
                    bad[:n] |= np.abs(s - w.tau) < MARGIN
                if bad.any():
                    bad_any = True
                    a = attempts.setdefault((l, b), np.zeros(len(K), np.int64))
                    a[bad] += 1
        if not bad_any:
            return attempts
    raise RuntimeError("margin not reached")


def score_quantile(w, qtl, layer=0, seq=0):
    inp = Inputs(w)
    K, _ = inp.kv(layer, seq)
    P = w.prefill[seq]
    s = np.concatenate([oracle.relevance(inp.q(layer, seq, t), K[: P + t])
                        for t in range(1, w.steps + 1)])
    return float(np.quantile(s, qtl))


# --------------------------------------------------------------------------
# oracle side
# --------------------------------------------------------------------------

def oracle_levels(w, inp, seq, modes=None, with_logits=True):
    """Recovery level applied after each step of one sequence."""
    if modes is None and with_logits:
        ent = [oracle.entropy(inp.logits(seq, t)) for t in range(1, w.steps + 1)]
        levels, rr = oracle.recovery_schedule(ent, w.entropy_spike, w.conf_drop)
        return levels, ent
    levels = []
    for t in range(1, w.steps + 1):
        m = 0 if modes is None else modes.get(t, 0)
        levels.append(m if m in (1, 2, 3) else 0)
    ent = ([oracle.entropy(inp.logits(seq, t)) for t in range(1, w.steps + 1)]
           if with_logits else None)
    return levels, ent


def _oracle_instance(w, inp, l, b, steps):
    K, V = inp.prompt(l, b)
    return oracle.Instance(K, V, w.window_K, w.tau, w.k_soft, capacity=w.prefill[b] + steps + 1,
                           history_W=w.history_W, relevance_kind=w.relevance,
                           candidates=w.candidates)


def _oracle_global(w, inp, b, steps):
    KV = [inp.prompt(l, b) for l in range(w.n_layers)]
    return oracle.GlobalInstance([k for k, _ in KV], [v for _, v in KV], w.window_K, w.tau,
                                 w.k_soft, capacity=w.prefill[b] + steps + 1,
                                 history_W=w.history_W, relevance_kind=w.relevance,
                                 candidates=w.candidates)


def _record(inst, t, out, rec):
    timer, count, frozen = inst.state()
    act = np.concatenate([np.nonzero(~frozen)[0], [inst.n]])
    return dict(t=t, out=out, frozen=frozen, timer=timer, count=count, active_next=act,
                scores=rec.scores, attended=rec.active)


def run_oracle(w, inp, instances, modes=None, with_logits=True, steps=None, record=None,
               on_scores=None):
    """Per instance: list over steps of dict(out, frozen, timer, count, active_next).
    on_scores(l_or_None, b, t, n, attended, scores) sees every step's relevance."""
    steps = w.steps if steps is None else steps
    res = {}
    if w.scope == "token":
        for b in sorted({b for _, b in instances}):
            levels, _ = oracle_levels(w, inp, b, modes, with_logits)
            inst = _oracle_global(w, inp, b, steps)
            layers = [l for l, bb in instances if bb == b]
            recs = {l: [] for l in layers}
            for t in range(1, steps + 1):
                kv = [inp.new_token(l, b, t) for l in range(w.n_layers)]
                rec = inst.step([inp.q(l, b, t) for l in range(w.n_layers)],
                                [k for k, _ in kv], [v for _, v in kv])
                if on_scores is not None:
                    on_scores(None, b, t, inst.n, rec.active, rec.scores)
                if levels[t - 1]:
                    inst.recover(levels[t - 1], w.wr_last_N)
                if record is None or record(t):
                    for l in layers:
                        recs[l].append(_record(inst, t, rec.out[l], rec))
            for l in layers:
                res[(l, b)] = recs[l]
        return res
    for (l, b) in instances:
        levels, _ = oracle_levels(w, inp, b, modes, with_logits)
        inst = _oracle_instance(w, inp, l, b, steps)
        recs = []
        for t in range(1, steps + 1):
            kn, vn = inp.new_token(l, b, t)
            rec = inst.step(inp.q(l, b, t), kn, vn)
            if on_scores is not None:
                on_scores(l, b, t, inst.n, rec.active, rec.scores)
            if levels[t - 1]:
                inst.recover(levels[t - 1], w.wr_last_N)
            if record is None or record(t):
                recs.append(_record(inst, t, rec.out, rec))
        res[(l, b)] = recs
    return res


def candidate_mask(w, A, n):
    """Which of the attended positions A the freeze loop may take, with n
    positions after the append: outside the window of the window_K most recent
    positions, or inside it when the workload takes candidates inside."""
    outside = A < n - w.window_K
    return outside if w.candidates == "outside" else ~outside


def fix_margin_run(w, margin, relative=False, modes=None, with_logits=True, max_rounds=40):
    """Re-draw keys until every score the oracle actually compares with tau
    (scored freeze candidates, in the run's own active sets) keeps
    |s - tau| >= margin (times tau when relative).  With token scope a
    token's keys are re-drawn in every layer.  Returns the attempts map."""
    attempts = {}
    instances = [(l, b) for l in range(w.n_layers) for b in range(w.batch)]
    lim = margin * abs(w.tau) if relative else margin
    for _ in range(max_rounds):
        bad = set()

        def on_scores(l, b, t, n, A, s):
            near = (np.abs(s - w.tau) < lim) & candidate_mask(w, A, n)
            for j in A[near]:
                for ll in (range(w.n_layers) if l is None else [l]):
                    bad.add((ll, b, int(j)))

        run_oracle(w, Inputs(w, attempts), instances, modes, with_logits, on_scores=on_scores)
        if not bad:
            return attempts
        for (l, b, j) in bad:
            a = attempts.setdefault((l, b), np.zeros(w.prefill[b] + w.steps, dtype=np.int64))
            a[j] += 1
    raise RuntimeError("could not keep the scores away from tau")


# --------------------------------------------------------------------------
# GPU side
# --------------------------------------------------------------------------

def _dev(x, dtype):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    if dtype == "bf16":
        t = t.to(torch.bfloat16)           # exact: values are bf16-representable
    return t.cuda()


def run_gpu(w, inp, instances, modes=None, with_logits=True, steps=None, record=None,
            timing=False, side_delay_us=0, streams=None, ctx=None):
    """Run the library; per instance a list of dict(out, unfreeze, count, frozen,
    active_next) for the recorded steps; per sequence the entropy monitor.
    streams(call, t, layer), when given, names the torch stream of each call
    ("prefill", "decode", "restore"; None = the current stream); such a stream
    first waits for the current stream, where the inputs were copied.  ctx, when
    given, is a context of the workload's configuration that has run no step
    (the caller keeps it); otherwise the run opens and closes its own."""
    import torch
    import paper_2512_11221_amd as A

    def on(call, t, layer):
        s = streams(call, t, layer) if streams else None
        if s is not None:
            s.wait_stream(torch.cuda.current_stream())
        return s

    steps = w.steps if steps is None else steps
    cfg = A.make_config(w.n_layers, w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim,
                        w.max_ctx, w.window_K, w.tau, w.k_soft, w.vocab,
                        entropy_spike=w.entropy_spike, conf_drop=w.conf_drop,
                        wr_last_N=w.wr_last_N, dtype=w.dtype, spill_min_D=w.spill_min_D,
                        device_rows=w.device_rows, history_W=w.history_W,
                        relevance=w.relevance, scope=w.scope, candidates=w.candidates)
    own = ctx is None
    if own:
        ctx = A.asrkf_init(cfg)
    if side_delay_us:
        A.asrkf_debug_delay_side(ctx, side_delay_us)
    res = {key: [] for key in instances}
    seqmon = {b: [] for b in range(w.batch)}
    stats = []
    try:
        for l in range(w.n_layers):
            for b in range(w.batch):
                K, V = inp.prompt(l, b)
                if len(K):
                    dk, dv = _dev(K, w.dtype), _dev(V, w.dtype)
                    A.asrkf_prefill(ctx, l, b, dk, dv, len(K), stream=on("prefill", 0, l))
                    torch.cuda.synchronize()
        torch.cuda.synchronize()
        for t in range(1, steps + 1):
            outs = []
            keep = []
            for l in range(w.n_layers):
                q = np.stack([inp.q(l, b, t) for b in range(w.batch)])
                kn = np.stack([inp.new_token(l, b, t)[0] for b in range(w.batch)])
                vn = np.stack([inp.new_token(l, b, t)[1] for b in range(w.batch)])
                dq, dk, dv = _dev(q, w.dtype), _dev(kn, w.dtype), _dev(vn, w.dtype)
                out = torch.empty((w.batch, w.n_q_heads, w.head_dim), dtype=torch.float32,
                                  device="cuda")
                A.asrkf_decode_step(ctx, l, dq, dk, dv, out, stream=on("decode", t, l))
                keep += [dq, dk, dv]
                outs.append(out)
            mode = A.AUTO if modes is None else modes.get(t, A.NONE)
            if with_logits:
                lg = _dev(np.stack([inp.logits(b, t) for b in range(w.batch)]), "f32")
                keep.append(lg)
                A.asrkf_restore(ctx, lg, mode, stream=on("restore", t, None))
            else:
                A.asrkf_restore(ctx, None, mode, stream=on("restore", t, None))
            torch.cuda.synchronize()
            if record is None or record(t):
                for (l, b) in instances:
                    st = A.asrkf_get_state(ctx, l, b, w.max_ctx)
                    st["out"] = outs[l][b].cpu().numpy()
                    st["t"] = t
                    if w.spill_min_D:
                        st.update(A.asrkf_get_residency(ctx, l, b, w.max_ctx))
                    res[(l, b)].append(st)
                for b in range(w.batch):
                    seqmon[b].append(A.asrkf_get_seq(ctx, b))
                stats.append(A.asrkf_stats(ctx))
            del keep
    finally:
        if own:
            A.asrkf_destroy(ctx)
    return res, seqmon, stats


# --------------------------------------------------------------------------
# comparison
# --------------------------------------------------------------------------

def compare_instance(gpu_recs, ora_recs, check_out=True):
    """Bit-exact states; attention outputs within the acceptance bound.
    Returns the largest absolute output error seen."""
    worst = 0.0
    assert len(gpu_recs) == len(ora_recs)
    for g, o in zip(gpu_recs, ora_recs):
        t = o["t"]
        assert g["t"] == t
        n = len(o["frozen"])
        assert g["n"] == n, (t, g["n"], n)
        np.testing.assert_array_equal(g["frozen"], o["frozen"], err_msg=f"frozen mask, step {t}")
        np.testing.assert_array_equal(g["count"], o["count"], err_msg=f"counts, step {t}")
        fz = o["frozen"]
        np.testing.assert_array_equal(g["unfreeze"][fz] - (t + 1), o["timer"][fz],
                                      err_msg=f"remaining timers, step {t}")
        np.testing.assert_array_equal(g["active"], o["active_next"], err_msg=f"active list, step {t}")
        if check_out:
            ref = o["out"]
            err = np.abs(g["out"].astype(np.float64) - ref)
            worst = max(worst, float(err.max()))
            assert err.max() <= ATOL, (t, float(err.max()))
            rel = np.linalg.norm(g["out"] - ref) / max(np.linalg.norm(ref), 1e-30)
            assert rel <= RTOL_NORM, (t, rel)
    return worst


def compare_residency(w, gpu_recs, ora_recs):
    """Spill mode, every step recorded: a position is held only on the host
    exactly while it is frozen by a freeze of d >= spill_min_D steps (d from
    its kept count, Eq. 3); resident positions hold distinct device rows; the
    host store holds every position that was ever released.  Returns the
    number of (position, step) restores seen."""
    seen = None
    restores = 0
    prev_host_only = None
    for g, o in zip(gpu_recs, ora_recs):
        t = o["t"]
        n = len(o["frozen"])
        d = np.array([oracle.freeze_duration(int(c), w.k_soft) for c in o["count"]])
        host_only = o["frozen"] & (d >= w.spill_min_D)
        row = g["device_row"]
        np.testing.assert_array_equal(row < 0, host_only, err_msg=f"host-only positions, step {t}")
        live = row[row >= 0]
        assert len(np.unique(live)) == len(live), f"device row held twice, step {t}"
        pool = w.device_rows or (w.max_ctx + 1 + 63) // 64 * 64
        assert live.size == 0 or (live.min() >= 0 and live.max() < pool), t
        seen = host_only.copy() if seen is None else np.concatenate([seen, [False] * (n - len(seen))]) | host_only
        np.testing.assert_array_equal(g["on_host"], seen, err_msg=f"host store contents, step {t}")
        if prev_host_only is not None:
            restores += int(np.count_nonzero(prev_host_only & ~host_only[:len(prev_host_only)]))
        prev_host_only = host_only
    return restores


def run_gpu_device(w, instances, record_steps, seqs_for_entropy=None, check_state=None):
    """Run a large workload exactly as the bench does (device-generated inputs,
    the library's own launch configuration).  Returns per instance the attention
    output of every step and the token states at ``record_steps``; per sequence
    the entropy monitor of every step.  check_state(layer, seq, t, state), when
    given, sees the token states of every (layer, sequence) at ``record_steps``."""
    import torch
    import paper_2512_11221_amd as A
    from synth.device import DeviceGen

    L, B, Hq, Hkv, D = w.n_layers, w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim
    tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    cfg = A.make_config(L, B, Hq, Hkv, D, w.max_ctx, w.window_K, w.tau, w.k_soft, w.vocab,
                        entropy_spike=w.entropy_spike, conf_drop=w.conf_drop,
                        wr_last_N=w.wr_last_N, dtype=w.dtype, spill_min_D=w.spill_min_D,
                        device_rows=w.device_rows)
    ctx = A.asrkf_init(cfg)
    outs = {key: [] for key in instances}
    states = {key: {} for key in instances}
    ent = {b: [] for b in (seqs_for_entropy or range(B))}
    try:
        dg = DeviceGen(w)
        Pmax = max(w.prefill)
        sk = torch.empty(Pmax * Hkv * D, dtype=tdt, device="cuda")
        sv = torch.empty_like(sk)
        for l in range(L):
            for b in range(B):
                dg.kv_rows(l, b, 0, w.prefill[b], sk, sv)
                A.asrkf_prefill(ctx, l, b, sk, sv, w.prefill[b])
        torch.cuda.synchronize()
        del sk, sv
        S = w.steps
        Q = torch.empty((S, L, B, Hq, D), dtype=tdt, device="cuda")
        Kn = torch.empty((S, L, B, Hkv, D), dtype=tdt, device="cuda")
        Vn = torch.empty_like(Kn)
        LG = torch.empty((S, B, w.vocab), dtype=torch.float32, device="cuda")
        dg.q(1, S, Q)
        dg.new_kv(1, S, Kn, Vn)
        dg.logits(1, S, LG)
        out = torch.empty((L, B, Hq, D), dtype=torch.float32, device="cuda")
        for t in range(1, S + 1):
            for l in range(L):
                A.asrkf_decode_step(ctx, l, Q[t - 1, l], Kn[t - 1, l], Vn[t - 1, l], out[l])
            A.asrkf_restore(ctx, LG[t - 1], A.AUTO)
            torch.cuda.synchronize()
            for (l, b) in instances:
                outs[(l, b)].append(out[l, b].cpu().numpy())
                if t in record_steps:
                    st = A.asrkf_get_state(ctx, l, b, w.max_ctx)
                    st["t"] = t
                    states[(l, b)][t] = st
            if check_state is not None and t in record_steps:
                for l in range(L):
                    for b in range(B):
                        st = A.asrkf_get_state(ctx, l, b, w.max_ctx)
                        check_state(l, b, t, st)
            for b in ent:
                ent[b].append(A.asrkf_get_seq(ctx, b))
    finally:
        A.asrkf_destroy(ctx)
    return outs, states, ent


def compare_sampled(w, inp, instances, outs, states, record_steps):
    """Oracle on the sampled instances over every step: outputs each step within
    the acceptance bound, states at record_steps bit-exact."""
    worst = 0.0
    for (l, b) in instances:
        ora = run_oracle(w, inp, [(l, b)], record=lambda t: True)[(l, b)]
        for o in ora:
            t = o["t"]
            g = outs[(l, b)][t - 1]
            err = np.abs(g.astype(np.float64) - o["out"])
            worst = max(worst, float(err.max()))
            assert err.max() <= ATOL, (l, b, t, float(err.max()))
            rel = np.linalg.norm(g - o["out"]) / max(np.linalg.norm(o["out"]), 1e-30)
            assert rel <= RTOL_NORM, (l, b, t, rel)
            if t in record_steps:
                gs = states[(l, b)][t]
                gs["out"] = g
                compare_instance([gs], [o], check_out=False)
    return worst


def score_quantile_run(w, qtl, steps=8):
    """The qtl quantile of the scores of the freeze candidates over the first
    steps of the workload with nothing frozen (tau below every score)."""
    vals = []
    wq = w.replace(tau=-1.0, steps=steps, flat_logit_steps=())

    def on_scores(l, b, t, n, A, s):
        vals.append(s[candidate_mask(w, A, n)])

    instances = [(l, b) for l in range(w.n_layers) for b in range(w.batch)]
    run_oracle(wq, Inputs(wq), instances, with_logits=False, on_scores=on_scores)
    return float(np.quantile(np.concatenate(vals), qtl))
