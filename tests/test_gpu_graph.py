"""A decode step captured in a HIP graph (torch.cuda.CUDAGraph over the C ABI)
and replayed: the step index comes from the device, so one captured step
(every layer's decode_step and the restore, reading static input buffers)
replays step after step.  Each replay follows eager copies of that step's
inputs and is followed by a synchronization and eager state reads; outputs,
token states and the entropy monitor must equal an eager run's bit for bit,
and the eager run matches the oracle."""
import numpy as np
import pytest

from synth import gen
from tests import _harness as H

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2512_11221_amd as A
    A.load()
    return torch


def _workload(**kw):
    args = dict(name="graph-hh", seed=gen.SEED + 95, n_layers=2, batch=2, n_q_heads=32,
                n_kv_heads=8, head_dim=128, dtype="bf16", prefill=[300, 170], steps=24,
                window_K=16, tau=0.5, k_soft=2.0, vocab=1024, logit_sigma=2.0, recipe="hh",
                f_hh=[0.35, 0.25], entropy_spike=6.5, flat_logit_steps=(12, 13))
    args.update(kw)
    return gen.Workload(**args)


class _Static:
    """Static device buffers of one step's inputs and outputs."""

    def __init__(self, w):
        import torch
        L, B = w.n_layers, w.batch
        self.q = torch.empty((L, B, w.n_q_heads, w.head_dim), dtype=torch.bfloat16, device="cuda")
        self.k = torch.empty((L, B, w.n_kv_heads, w.head_dim), dtype=torch.bfloat16, device="cuda")
        self.v = torch.empty_like(self.k)
        self.lg = torch.empty((B, w.vocab), dtype=torch.float32, device="cuda")
        self.out = torch.empty((L, B, w.n_q_heads, w.head_dim), dtype=torch.float32, device="cuda")

    def load(self, w, inp, t):
        """Eager copies of step t's inputs into the static buffers."""
        L, B = w.n_layers, w.batch
        self.q.copy_(H._dev(np.stack([[inp.q(l, b, t) for b in range(B)] for l in range(L)]), "bf16"))
        self.k.copy_(H._dev(np.stack([[inp.new_token(l, b, t)[0] for b in range(B)] for l in range(L)]), "bf16"))
        self.v.copy_(H._dev(np.stack([[inp.new_token(l, b, t)[1] for b in range(B)] for l in range(L)]), "bf16"))
        self.lg.copy_(H._dev(np.stack([inp.logits(b, t) for b in range(B)]), "f32"))

    def step(self, A, ctx, w):
        for l in range(w.n_layers):
            A.asrkf_decode_step(ctx, l, self.q[l], self.k[l], self.v[l], self.out[l])
        A.asrkf_restore(ctx, self.lg, A.AUTO)


def _open(A, w):
    cfg = A.make_config(w.n_layers, w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.max_ctx,
                        w.window_K, w.tau, w.k_soft, w.vocab, entropy_spike=w.entropy_spike,
                        wr_last_N=w.wr_last_N, dtype=w.dtype, spill_min_D=w.spill_min_D)
    ctx = A.asrkf_init(cfg)
    inp = H.Inputs(w)
    for l in range(w.n_layers):
        for b in range(w.batch):
            K, V = inp.prompt(l, b)
            A.asrkf_prefill(ctx, l, b, H._dev(K, w.dtype), H._dev(V, w.dtype), len(K))
    return ctx, inp


def _capture(torch, A, ctx, w, buf):
    g = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        buf.step(A, ctx, w)
    torch.cuda.synchronize()
    return g


# two layers; four layers with some 10k tokens per layer, where the
# first-tile records are built inside the captured restore and used by the
# captured attention launches
_REPLAYED = [dict(), dict(name="graph-hh-records", n_layers=4, batch=4, prefill=[2600, 2400, 2800, 2300],
                          f_hh=[0.35, 0.25, 0.3, 0.2], steps=20)]


@pytest.mark.parametrize("case", range(len(_REPLAYED)))
def test_captured_step_replays_like_eager_steps(case):
    import torch
    import paper_2512_11221_amd as A
    w = _workload(**_REPLAYED[case])
    s_cold, s_hot = gen.hh_relevance_bounds(w)
    assert s_cold < w.tau - H.MARGIN and s_hot > w.tau + H.MARGIN
    inst = [(l, b) for l in range(w.n_layers) for b in range(w.batch)]
    eager, mon_e, st_e = H.run_gpu(w, H.Inputs(w), inst)
    o = H.run_oracle(w, H.Inputs(w), inst)
    for key in inst:
        H.compare_instance(eager[key], o[key])
    warm = 4
    ctx, inp = _open(A, w)
    buf = _Static(w)
    try:
        torch.cuda.synchronize()
        for t in range(1, warm + 1):                   # eager steps before the capture
            buf.load(w, inp, t)
            buf.step(A, ctx, w)
        g = _capture(torch, A, ctx, w, buf)
        assert A.asrkf_stats(ctx)["step"] == warm       # capturing ran nothing
        for t in range(warm + 1, w.steps + 1):
            buf.load(w, inp, t)
            g.replay()
            torch.cuda.synchronize()
            out = buf.out.cpu().numpy()
            for (l, b) in inst:
                st = A.asrkf_get_state(ctx, l, b, w.max_ctx)
                ref = eager[(l, b)][t - 1]
                assert ref["t"] == t
                np.testing.assert_array_equal(out[l, b], ref["out"], err_msg=f"out {l} {b} step {t}")
                for f in ("unfreeze", "count", "frozen", "active"):
                    np.testing.assert_array_equal(st[f], ref[f], err_msg=f"{f} {l} {b} step {t}")
            for b in range(w.batch):
                assert A.asrkf_get_seq(ctx, b) == mon_e[b][t - 1], (b, t)
            stats = A.asrkf_stats(ctx)
            assert stats["step"] == t
            for key in ("attended_total", "active_positions", "total_positions", "recoveries",
                        "rr_requests"):
                assert stats[key] == st_e[t - 1][key], (key, t)
    finally:
        A.asrkf_destroy(ctx)


def test_forced_recovery_in_a_graph_is_counted():
    """A restore without logits and a forced level, captured and replayed:
    every replay applies it (states equal an eager run) and the recovery
    counter counts it on the device."""
    import torch
    import paper_2512_11221_amd as A
    w = _workload(steps=10, entropy_spike=float("inf"), flat_logit_steps=())
    inst = [(l, b) for l in range(w.n_layers) for b in range(w.batch)]
    modes = {t: (A.SR if t > 3 else A.NONE) for t in range(1, w.steps + 1)}
    eager, _, st_e = H.run_gpu(w, H.Inputs(w), inst, modes=modes, with_logits=False)
    ctx, inp = _open(A, w)
    buf = _Static(w)
    try:
        torch.cuda.synchronize()
        for t in range(1, 4):
            buf.load(w, inp, t)
            for l in range(w.n_layers):
                A.asrkf_decode_step(ctx, l, buf.q[l], buf.k[l], buf.v[l], buf.out[l])
            A.asrkf_restore(ctx, None, A.NONE)
        g = torch.cuda.CUDAGraph()
        torch.cuda.synchronize()
        with torch.cuda.graph(g):
            for l in range(w.n_layers):
                A.asrkf_decode_step(ctx, l, buf.q[l], buf.k[l], buf.v[l], buf.out[l])
            A.asrkf_restore(ctx, None, A.SR)
        for t in range(4, w.steps + 1):
            buf.load(w, inp, t)
            g.replay()
            torch.cuda.synchronize()
            for (l, b) in inst:
                st = A.asrkf_get_state(ctx, l, b, w.max_ctx)
                for f in ("unfreeze", "count", "active"):
                    np.testing.assert_array_equal(st[f], eager[(l, b)][t - 1][f], err_msg=f"{f} step {t}")
        stats = A.asrkf_stats(ctx)
        assert stats["recoveries"] == st_e[-1]["recoveries"]
        assert stats["recoveries"][1] == w.batch * (w.steps - 3)
    finally:
        A.asrkf_destroy(ctx)


def test_capture_refused_before_the_first_step_and_in_spill_mode():
    import torch
    import paper_2512_11221_amd as A
    from paper_2512_11221_amd import _lib as L
    for spill in (False, True):
        w = _workload(steps=6, spill_min_D=2 if spill else 0)
        ctx, inp = _open(A, w)
        buf = _Static(w)
        try:
            torch.cuda.synchronize()
            if spill:                                  # spill mode: refused even after a step
                buf.load(w, inp, 1)
                buf.step(A, ctx, w)
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            s = torch.cuda.Stream()
            with torch.cuda.stream(s):
                g.capture_begin()
                try:
                    with pytest.raises(A.AsrkfError) as e:
                        A.asrkf_decode_step(ctx, 0, buf.q[0], buf.k[0], buf.v[0], buf.out[0])
                finally:
                    g.capture_end()                    # an empty graph: nothing was queued
            assert e.value.code == L.ESTATE
            torch.cuda.synchronize()
        finally:
            A.asrkf_destroy(ctx)


def test_replays_past_max_ctx_are_refused_on_the_device():
    """Replays do not pass the host's capacity check: the rebuild refuses a
    step that would pass max_ctx (nothing out of bounds), and the next waiting
    call reports ECAPACITY."""
    import torch
    import paper_2512_11221_amd as A
    from paper_2512_11221_amd import _lib as L
    w = _workload(steps=12)
    w = w.replace(max_ctx=max(w.prefill) + 6)
    ctx, inp = _open(A, w)
    buf = _Static(w)
    try:
        torch.cuda.synchronize()
        for t in range(1, 3):
            buf.load(w, inp, t)
            buf.step(A, ctx, w)
        g = _capture(torch, A, ctx, w, buf)
        for t in range(3, 9):                          # steps 7 and 8 pass max_ctx (306)
            buf.load(w, inp, t)
            g.replay()
        torch.cuda.synchronize()
        with pytest.raises(A.AsrkfError) as e:
            A.asrkf_stats(ctx)
        assert e.value.code == L.ECAPACITY and "max_ctx" in str(e.value)
    finally:
        A.asrkf_destroy(ctx)
