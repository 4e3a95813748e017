"""GPU parity for the parts of the recovery ladder (Sec. 3.6) beyond the
entropy trigger: the confidence-drop trigger (p_max below theta_p), Rewalk
Regeneration requests after four or more consecutive spikes, Window Reset over
a span other than the default, logits with -inf entries, and the ordering of
calls that switch streams.  Every level, escalation count and recovery counter
is compared with the oracle exactly, entropy and p_max within tolerance."""
import math

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


def _tiny_freezing(**kw):
    w0 = gen.tiny()
    w = gen.tiny(tau=H.score_quantile(w0, 0.6), **kw)
    return w, H.Inputs(w, H.fix_margin(w))


def _run(w, inp, modes=None):
    g, mon, stats = H.run_gpu(w, inp, [(0, 0)], modes)
    o = H.run_oracle(w, inp, [(0, 0)], modes)
    worst = H.compare_instance(g[(0, 0)], o[(0, 0)])
    print(f"{w.name}: worst |out - oracle| = {worst:.3e}")
    return mon[0], stats


def _check_monitor(w, inp, mon, stats):
    """Entropy, p_max, escalation count and level of every step against the
    oracle; recovery and Rewalk Regeneration counters against its flags."""
    ent = [H.oracle.entropy(inp.logits(0, t)) for t in range(1, w.steps + 1)]
    levels, rr = H.oracle.recovery_schedule(ent, w.entropy_spike, w.conf_drop)
    count = 0
    for t, (m, (e, pm), lv) in enumerate(zip(mon, ent, levels), 1):
        spike = (e > w.entropy_spike) or (w.conf_drop > 0 and pm < w.conf_drop)
        count = count + 1 if spike else 0
        assert m["level"] == lv, (t, m["level"], lv)
        assert m["escalation"] == count, (t, m["escalation"], count)
        assert abs(m["entropy"] - e) <= H.ENTROPY_TOL, (t, m["entropy"], e)
        assert abs(m["pmax"] - pm) <= 1e-5 * pm, (t, m["pmax"], pm)
    last = stats[-1]
    assert last["recoveries"][1:] == [levels.count(1), levels.count(2), levels.count(3)]
    assert last["rr_requests"] == sum(rr)
    return levels, rr


def test_confidence_drop_trigger():
    """theta_H is +inf, so only the p_max trigger can fire: planted flat steps
    (p_max ~ 1.3e-3) fall below theta_p = 5e-3; every other step stays above
    2.2e-2.  Steps 45-47 drop three times in a row: SR, WR, FR."""
    flat = (20, 30, 31, 45, 46, 47)
    w, inp = _tiny_freezing(entropy_spike=math.inf, conf_drop=5e-3, flat_logit_steps=flat)
    pm = [H.oracle.entropy(inp.logits(0, t))[1] for t in range(1, w.steps + 1)]
    assert [t for t, p in enumerate(pm, 1) if p < w.conf_drop] == list(flat)
    assert min(abs(p - w.conf_drop) / w.conf_drop for p in pm) >= 0.5
    mon, stats = _run(w, inp)
    levels, rr = _check_monitor(w, inp, mon, stats)
    assert [t for t, lv in enumerate(levels, 1) if lv] == list(flat)
    assert max(levels) == 3 and not any(rr)


def test_rewalk_regeneration_requests():
    """Six consecutive spike steps: SR, WR, FR, then FR again with a Rewalk
    Regeneration request at each of the last three (count 4, 5, 6)."""
    flat = (30, 31, 32, 33, 34, 35)
    w, inp = _tiny_freezing(entropy_spike=6.5, flat_logit_steps=flat)
    ent = [H.oracle.entropy(inp.logits(0, t))[0] for t in range(1, w.steps + 1)]
    assert min(abs(e - w.entropy_spike) for e in ent) >= 1e-2
    assert [t for t, e in enumerate(ent, 1) if e > w.entropy_spike] == list(flat)
    mon, stats = _run(w, inp)
    levels, rr = _check_monitor(w, inp, mon, stats)
    assert levels[29:35] == [1, 2, 3, 3, 3, 3]
    assert [t for t, r in enumerate(rr, 1) if r] == [33, 34, 35]
    assert stats[-1]["rr_requests"] == 3


@pytest.mark.parametrize("span", [1, 40, 200])
def test_window_reset_span(span):
    """Window Reset over the last 1, 40 or 200 positions (default 4K = 128):
    forced at three steps in one run, reached by the entropy ladder (two
    consecutive spikes) in another."""
    import paper_2512_11221_amd as A
    flat = (50, 51)
    w, inp = _tiny_freezing(entropy_spike=6.5, flat_logit_steps=flat, wr_last_N=span)
    assert w.wr_last_N == span
    _run(w, inp, modes={24: A.WR, 37: A.WR, 58: A.WR})
    mon, stats = _run(w, inp)
    levels, _ = _check_monitor(w, inp, mon, stats)
    assert [t for t, lv in enumerate(levels, 1) if lv] == [50, 51] and levels[50] == 2


class _NegInfLogits(H.Inputs):
    """Logits with -inf at every seventh entry (masked vocabulary entries);
    at step 5 only the first entry is finite (a one-point distribution)."""

    def logits(self, seq, t):
        x = super().logits(seq, t).copy()
        x[::7] = -np.inf
        if t == 5:
            x[1:] = -np.inf
            x[0] = 1.5
        return x


def test_entropy_with_negative_infinite_logits():
    flat = (20, 40, 41)
    w0, _ = _tiny_freezing(entropy_spike=6.5, flat_logit_steps=flat)
    inp = _NegInfLogits(w0, H.fix_margin(w0))
    ent = [H.oracle.entropy(inp.logits(0, t)) for t in range(1, w0.steps + 1)]
    assert all(math.isfinite(e) for e, _ in ent)
    assert ent[4] == (0.0, 1.0)
    assert min(abs(e - w0.entropy_spike) for e, _ in ent) >= 1e-2
    assert [t for t, (e, _) in enumerate(ent, 1) if e > w0.entropy_spike] == list(flat)
    mon, stats = _run(w0, inp)
    _check_monitor(w0, inp, mon, stats)
    assert mon[4]["entropy"] == 0.0 and mon[4]["pmax"] == 1.0


def _three_layer_hh(spill=False):
    return gen.Workload(name="streams-hh", seed=gen.SEED + 93, n_layers=3, batch=2, n_q_heads=32,
                        n_kv_heads=8, head_dim=128, dtype="bf16", prefill=[300, 170], steps=24,
                        window_K=16, tau=0.5, k_soft=2.0, vocab=1024, logit_sigma=2.0,
                        recipe="hh", f_hh=[0.35, 0.25], entropy_spike=6.5,
                        flat_logit_steps=(12, 13), spill_min_D=2 if spill else 0)


@pytest.mark.parametrize("spill", [False, True], ids=["resident", "spill"])
def test_calls_on_alternating_streams(spill):
    """Prefill, each layer's decode_step and restore on different streams of
    the caller's (layer l on stream l % 2, restore on a third), with no host
    synchronization inside a step: the outputs and states are bitwise those of
    a run on one stream, because a call on a new stream waits for the
    context's previous work (layer l + 1 reuses the split partials of layer l)."""
    import torch
    w = _three_layer_hh(spill)
    s_cold, s_hot = gen.hh_relevance_bounds(w)
    assert s_cold < w.tau - H.MARGIN and s_hot > w.tau + H.MARGIN
    inp = H.Inputs(w)
    for b in range(w.batch):
        ent = [H.oracle.entropy(inp.logits(b, t))[0] for t in range(1, w.steps + 1)]
        assert min(abs(e - w.entropy_spike) for e in ent) >= 1e-2
        assert [t for t, e in enumerate(ent, 1) if e > w.entropy_spike] == [12, 13]
    inst = [(l, b) for l in range(w.n_layers) for b in range(w.batch)]
    rec = lambda t: t % 4 == 0 or t == w.steps
    one, mon1, _ = H.run_gpu(w, inp, inst, record=rec)
    pool = [torch.cuda.Stream() for _ in range(3)]

    def streams(call, t, layer):
        if call == "restore":
            return pool[2]
        return pool[layer % 2]

    many, mon2, _ = H.run_gpu(w, inp, inst, record=rec, streams=streams)
    torch.cuda.synchronize()
    for key in inst:
        for a, b in zip(one[key], many[key]):
            for f in ("out", "unfreeze", "count", "frozen", "active"):
                np.testing.assert_array_equal(a[f], b[f], err_msg=f"{key} step {a['t']} {f}")
    assert [m["level"] for m in mon1[0]] == [m["level"] for m in mon2[0]]
    o = H.run_oracle(w, inp, inst, record=rec)
    for key in inst:
        H.compare_instance(one[key], o[key])
