"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Freeze masks, counts, remaining timers and active lists are compared bit for
bit; attention outputs within 2e-2 max-abs and 1e-2 relative (norm); entropy
within 1e-3 nats.  Inputs come from the seeded generator; every relevance
score stays at least 1e-3 away from tau (by construction for the heavy-hitter
recipe, by re-drawing keys for the Gaussian recipe).
"""
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
    A.load()          # raises when the library is not built: no fallback
    return torch


def _all_instances(w):
    return [(l, b) for l in range(w.n_layers) for b in range(w.batch)]


def _parity(w, inp, modes=None, with_logits=True, instances=None, record=None, check_out=True):
    instances = instances or _all_instances(w)
    g, mon, stats = H.run_gpu(w, inp, instances, modes, with_logits, record=record)
    o = H.run_oracle(w, inp, instances, modes, with_logits, record=record)
    worst = 0.0
    for key in instances:
        worst = max(worst, H.compare_instance(g[key], o[key], check_out))
    print(f"{w.name}: worst |out - oracle| = {worst:.3e}")
    return g, o, mon, stats


def _tiny_freezing(**kw):
    w0 = gen.tiny()
    tau = H.score_quantile(w0, 0.6)
    w = gen.tiny(tau=tau, **kw)
    return w, H.Inputs(w, H.fix_margin(w))


def test_tiny_freezing_nothing_is_dense():
    w = gen.tiny()                          # scores ~6.4 >> tau = 0.5
    inp = H.Inputs(w)
    g, o, _, _ = _parity(w, inp)
    for r in o[(0, 0)]:
        assert not r["frozen"].any()
    for r in g[(0, 0)]:
        assert len(r["active"]) == r["n"] + 1


def test_tiny_with_freezing():
    w, inp = _tiny_freezing()
    g, o, _, _ = _parity(w, inp)
    frac = np.mean([r["frozen"].mean() for r in o[(0, 0)]])
    assert 0.05 < frac < 0.9, frac           # the run does freeze and restore


def test_tiny_entropy_driven_recovery():
    flat = (40, 50, 51, 60, 61, 62)
    w, inp = _tiny_freezing(entropy_spike=6.5, flat_logit_steps=flat)
    # every step's entropy stays 1e-2 away from theta_H; spikes only where planted
    ent = [H.oracle.entropy(inp.logits(0, t))[0] for t in range(1, w.steps + 1)]
    assert min(abs(e - 6.5) for e in ent) >= 1e-2
    assert [t for t, e in enumerate(ent, 1) if e > 6.5] == list(flat)
    g, o, mon, stats = _parity(w, inp)
    levels, _ = H.oracle_levels(w, inp, 0)
    assert [m["level"] for m in mon[0]] == levels
    assert max(levels) == 3
    for m, e in zip(mon[0], ent):
        assert abs(m["entropy"] - e) <= H.ENTROPY_TOL
    assert stats[-1]["recoveries"][1:] == [3, 2, 1]


@pytest.mark.parametrize("with_logits", [False, True])
def test_forced_recovery_modes(with_logits):
    import paper_2512_11221_amd as A
    w, inp = _tiny_freezing()
    modes = {20: A.SR, 33: A.WR, 47: A.FR, 55: A.SR}
    _parity(w, inp, modes=modes, with_logits=with_logits)


def test_llama8b_one_layer_full_run():
    w = gen.llama8b_1layer()
    inp = H.Inputs(w)
    g, o, mon, stats = _parity(w, inp)
    ent = [H.oracle.entropy(inp.logits(0, t))[0] for t in range(1, w.steps + 1)]
    for m, e in zip(mon[0], ent):
        assert abs(m["entropy"] - e) <= H.ENTROPY_TOL
    # heavy-hitter recipe: active fraction between the hitter share and 1
    last = o[(0, 0)][-1]
    assert 0.3 < 1 - last["frozen"].mean() <= 1.0


@pytest.mark.parametrize("tau", [-1.0, math.inf])
def test_bf16_gaussian_multilayer_ragged(tau):
    """Strong logits (q, k ~ N(0,1) at D = 128), two layers, three sequences of
    very different prompt lengths; tau below every score (dense) or above
    every score (every out-of-window token flagged each step)."""
    w = gen.Workload(name="bf16-gauss", seed=gen.SEED + 21, n_layers=2, batch=3, n_q_heads=32,
                     n_kv_heads=8, head_dim=128, dtype="bf16", prefill=[700, 1, 300], steps=40,
                     window_K=16, tau=tau, k_soft=2.0, vocab=1000, logit_sigma=2.0,
                     recipe="gauss")
    _parity(w, H.Inputs(w))


@pytest.mark.parametrize("shape", [
    dict(n_q_heads=8, n_kv_heads=8, head_dim=128, dtype="bf16"),    # G = 1
    dict(n_q_heads=16, n_kv_heads=2, head_dim=128, dtype="bf16"),   # G = 8
    dict(n_q_heads=64, n_kv_heads=8, head_dim=128, dtype="bf16"),   # G = 8, two waves per token
    dict(n_q_heads=32, n_kv_heads=32, head_dim=128, dtype="bf16"),  # multi-head, four waves per token
    dict(n_q_heads=32, n_kv_heads=16, head_dim=64, dtype="bf16"),   # G = 2, two waves per token
    dict(n_q_heads=16, n_kv_heads=16, head_dim=256, dtype="bf16"),  # rows of 256, multi-head
    dict(n_q_heads=16, n_kv_heads=8, head_dim=256, dtype="bf16"),   # rows of 256, G = 2
    dict(n_q_heads=32, n_kv_heads=8, head_dim=256, dtype="bf16"),   # rows of 256, G = 4 split
    dict(n_q_heads=8, n_kv_heads=4, head_dim=64, dtype="bf16"),     # G = 2, D = 64
    dict(n_q_heads=8, n_kv_heads=2, head_dim=128, dtype="f32"),     # fp32, D = 128
])
def test_shapes_flag_all(shape):
    w = gen.Workload(name="shape", seed=gen.SEED + 31, n_layers=1, batch=2, prefill=[190, 77],
                     steps=70, window_K=0, tau=math.inf, k_soft=0.75, vocab=64,
                     logit_sigma=1.0, recipe="gauss", **shape)
    _parity(w, H.Inputs(w))


def test_ragged_heavy_hitters_multilayer():
    w = gen.Workload(name="hh-ragged", seed=gen.SEED + 41, n_layers=2, batch=6, n_q_heads=32,
                     n_kv_heads=8, head_dim=128, dtype="bf16",
                     prefill=[1, 17, 64, 333, 1000, 2049], steps=48, window_K=32, tau=0.5,
                     k_soft=2.0, vocab=128256, logit_sigma=3.0, recipe="hh",
                     f_hh=[0.2, 0.3, 0.5, 0.35, 0.25, 0.45])
    s_cold, s_hot = gen.hh_relevance_bounds(w)
    assert s_cold < w.tau - H.MARGIN and s_hot > w.tau + H.MARGIN
    _parity(w, H.Inputs(w))


def test_short_and_empty_lists_among_long_ones():
    """Twelve sequences whose lists range from the new token alone to a few
    thousand entries.  With so few tokens the launch cuts ranges of ~32
    entries, so ranges end inside a sequence's virtual cost tokens, straddle
    sequence boundaries, or hold only virtual tokens: every such plan must
    still cover each real entry exactly once."""
    w = gen.Workload(name="short-lists", seed=gen.SEED + 43, n_layers=2, batch=12, n_q_heads=32,
                     n_kv_heads=8, head_dim=128, dtype="bf16",
                     prefill=[0, 1, 2, 30, 47, 48, 49, 95, 500, 1500, 3, 64], steps=30,
                     window_K=8, tau=math.inf, k_soft=1.0, vocab=64, logit_sigma=1.0,
                     recipe="gauss")
    _parity(w, H.Inputs(w))


def test_bitwise_determinism():
    w, inp = _tiny_freezing()
    a, _, _ = H.run_gpu(w, inp, [(0, 0)])
    b, _, _ = H.run_gpu(w, inp, [(0, 0)])
    for x, y in zip(a[(0, 0)], b[(0, 0)]):
        np.testing.assert_array_equal(x["out"], y["out"])
        np.testing.assert_array_equal(x["unfreeze"], y["unfreeze"])
        np.testing.assert_array_equal(x["active"], y["active"])


_LAYOUTS = [  # (q heads, KV heads, head_dim, dtype), every layout family the kernel has
    (8, 2, 64, "f32"), (8, 8, 128, "bf16"), (32, 8, 128, "bf16"), (16, 2, 128, "bf16"),
    (64, 8, 128, "bf16"), (32, 32, 128, "bf16"), (32, 16, 64, "bf16"), (16, 8, 256, "bf16"),
    (4, 4, 64, "f32"), (2, 1, 128, "bf16"), (64, 32, 64, "bf16"), (16, 16, 256, "bf16"),
]


@pytest.mark.parametrize("case", range(len(_LAYOUTS)))
def test_seeded_random_runs(case):
    """For each head layout, a run whose sizes are drawn from a seeded generator:
    2-4 sequences with prompts of 0..700 tokens, 1-2 layers, a window of 0..40
    and k in [0.5, 3], every out-of-window token flagged each step (tau = +inf)
    or none (tau = -inf), so that freezing, restores and the planner's ranges
    all vary while no score sits near tau."""
    rng = np.random.default_rng([0x2512, case])
    hq, hkv, d, dtype = _LAYOUTS[case]
    batch = int(rng.integers(2, 5))
    w = gen.Workload(name=f"random-{case}", seed=gen.SEED + 200 + case,
                     n_layers=int(rng.integers(1, 3)), batch=batch, n_q_heads=hq, n_kv_heads=hkv,
                     head_dim=d, dtype=dtype,
                     prefill=[int(x) for x in rng.integers(0, 700, size=batch)],
                     steps=int(rng.integers(12, 30)), window_K=int(rng.integers(0, 41)),
                     tau=math.inf if case % 3 else -math.inf,
                     k_soft=float(np.round(rng.uniform(0.5, 3.0), 2)), vocab=64, logit_sigma=1.0,
                     recipe="gauss")
    _parity(w, H.Inputs(w))


def _max_batch(**kw):
    rng = np.random.default_rng(0x1024)
    args = dict(name="max-batch", seed=gen.SEED + 81, n_layers=1, batch=1024, n_q_heads=32,
                n_kv_heads=8, head_dim=128, dtype="bf16",
                prefill=[int(x) for x in rng.integers(0, 61, size=1024)], steps=10,
                window_K=8, tau=math.inf, k_soft=1.0, vocab=64, logit_sigma=1.0, recipe="gauss")
    args.update(kw)
    return gen.Workload(**args)


@pytest.mark.parametrize("spill_min_D", [0, 2])
def test_maximum_batch(spill_min_D):
    """The largest batch the library takes (1024 sequences) with prompts of 0 to
    60 tokens: each workgroup's range covers several sequences, most lists are
    shorter than the per-sequence cost the planner charges, and every
    out-of-window token is flagged each step."""
    w = _max_batch(spill_min_D=spill_min_D)
    _parity(w, H.Inputs(w))


@pytest.mark.parametrize("k_soft,window_K,forced", [
    (2.0 ** -8, 4, True),      # d = floor(256 sqrt(c)): a token flagged once is gone for the run
    (2.0 ** 16, 4, False),     # d = 0 for every count: nothing ever freezes
    (1.7, 3, False),           # k not a power of two: the schedule is the exact floor for fp32 1.7
    (0.3, 1000, False),        # the window covers every position: no candidate at all
])
def test_schedule_and_window_extremes(k_soft, window_K, forced):
    """The ends of the k range the library accepts, a k that is not dyadic, and
    a window wider than every sequence; every candidate is flagged at every
    step (tau = +inf).  With k = 2^-8 the forced SR, WR and FR bring the
    long-frozen tokens back."""
    import paper_2512_11221_amd as A
    w = gen.Workload(name="extremes", seed=gen.SEED + 91, n_layers=2, batch=3, n_q_heads=8,
                     n_kv_heads=2, head_dim=64, dtype="f32", prefill=[50, 7, 0], steps=24,
                     window_K=window_K, tau=math.inf, k_soft=k_soft, vocab=64, logit_sigma=1.0,
                     recipe="gauss")
    modes = {6: A.SR, 11: A.WR, 17: A.FR} if forced else None
    g, o, _, stats = _parity(w, H.Inputs(w), modes=modes, with_logits=False)
    frozen = [bool(r["frozen"].any()) for key in o for r in o[key]]
    if k_soft >= 2.0 ** 16 or window_K >= 1000:
        assert not any(frozen)
    else:
        assert any(frozen)


@pytest.mark.parametrize("batch", [20, 40, 200])
def test_entropy_and_combine_across_batch_sizes(batch):
    """Batch sizes at which the launches take other shapes: the entropy pass
    splits a sequence's 128256 logits over 16, 8 or 4 workgroups (32 below
    batch 17), and the split combine folds a sequence's partial slots with 4 or
    1 slot groups.  Entropy and the confidence of every sequence at every step
    against the oracle; states bit-exact and outputs in tolerance."""
    rng = np.random.default_rng(0x5EED + batch)
    w = gen.Workload(name=f"batch-{batch}", seed=gen.SEED + 101 + batch, n_layers=1, batch=batch,
                     n_q_heads=8, n_kv_heads=2, head_dim=64, dtype="f32",
                     prefill=[int(x) for x in rng.integers(1, 90, size=batch)], steps=3,
                     window_K=8, tau=math.inf, k_soft=1.0, vocab=128256, logit_sigma=3.0,
                     recipe="gauss")
    inp = H.Inputs(w)
    _, _, mon, _ = _parity(w, inp)
    for b in range(batch):
        for t in range(1, w.steps + 1):
            e, pmax = H.oracle.entropy(inp.logits(b, t))
            m = mon[b][t - 1]
            assert abs(m["entropy"] - e) <= H.ENTROPY_TOL, (b, t, m["entropy"], e)
            assert abs(m["pmax"] - pmax) <= 1e-6 + 1e-4 * pmax, (b, t, m["pmax"], pmax)


@pytest.mark.parametrize("batch,vocab", [(3, 1), (3, 7), (40, 7), (3, 1001), (40, 1001)])
def test_entropy_small_and_unaligned_vocab(batch, vocab):
    """Vocabularies that take the entropy pass's element-wise path (not a
    multiple of four logits), fewer logits than the workgroups a sequence is
    split over (so some of them fold nothing), and the one-logit distribution
    (entropy 0, confidence 1)."""
    rng = np.random.default_rng(0xE17 + vocab + batch)
    w = gen.Workload(name=f"vocab-{vocab}", seed=gen.SEED + 131 + vocab + batch, n_layers=1,
                     batch=batch, n_q_heads=8, n_kv_heads=2, head_dim=64, dtype="f32",
                     prefill=[int(x) for x in rng.integers(1, 40, size=batch)], steps=2,
                     window_K=8, tau=math.inf, k_soft=1.0, vocab=vocab, logit_sigma=3.0,
                     recipe="gauss")
    inp = H.Inputs(w)
    _, _, mon, _ = _parity(w, inp)
    for b in range(batch):
        for t in range(1, w.steps + 1):
            e, pmax = H.oracle.entropy(inp.logits(b, t))
            m = mon[b][t - 1]
            assert abs(m["entropy"] - e) <= H.ENTROPY_TOL, (b, t, m["entropy"], e)
            assert abs(m["pmax"] - pmax) <= 1e-6 + 1e-4 * pmax, (b, t, m["pmax"], pmax)
            if vocab == 1:
                assert m["entropy"] == 0.0 and m["pmax"] == 1.0
