"""GPU parity for the optional readings: a finite history window W for the
detection count, relevance by attention weight, and token-global scope (one
token state per sequence shared by every layer).  Same bar as the default
path: states bit for bit, outputs within 2e-2 max-abs and 1e-2 relative.
Inputs keep every score the oracle compares with tau away from it (1e-3
absolute for |q.k| scores, 1e-5 relative for attention weights, five times
the fp32 error of the weight computation)."""
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


def _parity(w, attempts, modes=None, with_logits=True):
    inp = H.Inputs(w, attempts)
    instances = [(l, b) for l in range(w.n_layers) for b in range(w.batch)]
    g, mon, stats = H.run_gpu(w, inp, instances, modes, with_logits)
    o = H.run_oracle(w, inp, instances, modes, with_logits)
    for key in instances:
        H.compare_instance(g[key], o[key])
    frozen = np.mean([r["frozen"].mean() for key in instances for r in o[key]])
    print(f"{w.name}: mean frozen fraction {frozen:.3f}")
    assert frozen > 0.02                      # the run does freeze
    return g, o, mon, stats


def _tuned(w, qtl, relative=False, **fix):
    w = w.replace(tau=H.score_quantile_run(w, qtl))
    margin = 1e-5 if relative else H.MARGIN
    return w, H.fix_margin_run(w, margin, relative=relative, **fix)


def _multi(**kw):
    args = dict(name="multi", seed=gen.SEED + 61, n_layers=3, batch=2, n_q_heads=8, n_kv_heads=2,
                head_dim=64, dtype="f32", prefill=[300, 170], steps=48, window_K=16, tau=0.0,
                k_soft=1.0, vocab=512, logit_sigma=2.0, recipe="gauss")
    args.update(kw)
    return gen.Workload(**args)


@pytest.mark.parametrize("W", [4, 9, 64])
def test_history_window(W):
    w, att = _tuned(gen.tiny(k_soft=1.0, history_W=W), 0.6)
    _parity(w, att)


def test_history_window_heavy_hitters():
    w = gen.llama8b_1layer(steps=96, history_W=16)
    _parity(w, {})


def test_softmax_relevance_layer_scope():
    w, att = _tuned(gen.tiny(relevance="softmax"), 0.5, relative=True)
    _parity(w, att)


def test_token_scope_abs():
    w, att = _tuned(_multi(scope="token"), 0.55)
    g, o, _, _ = _parity(w, att)
    for b in range(w.batch):                   # one state per sequence, seen from every layer
        for l in range(1, w.n_layers):
            for x, y in zip(g[(0, b)], g[(l, b)]):
                np.testing.assert_array_equal(x["active"], y["active"])


def test_token_scope_softmax_with_window():
    w, att = _tuned(_multi(scope="token", relevance="softmax", history_W=6), 0.5, relative=True)
    _parity(w, att)


def test_token_scope_recovery():
    flat = (20, 30, 31, 40, 41, 42)
    w0 = _multi(scope="token", entropy_spike=6.0, flat_logit_steps=flat, logit_sigma=2.0)
    w, att = _tuned(w0, 0.55)
    g, o, mon, stats = _parity(w, att)
    levels, _ = H.oracle_levels(w, H.Inputs(w, att), 0)
    assert max(levels) == 3
    assert [m["level"] for m in mon[0]] == levels


def test_token_scope_forced_modes():
    import paper_2512_11221_amd as A
    w, att = _tuned(_multi(scope="token"), 0.55, with_logits=False)
    _parity(w, att, modes={12: A.SR, 25: A.WR, 37: A.FR}, with_logits=False)


def test_token_scope_heavy_hitters_two_layers():
    """Two layers: a token that is a heavy hitter in either layer scores at
    least 1.39 / 2 on average, a cold one at most 0.253 (the recipe's bounds)."""
    w = gen.Workload(name="hh-token", seed=gen.SEED + 63, n_layers=2, batch=3, n_q_heads=32,
                     n_kv_heads=8, head_dim=128, dtype="bf16", prefill=[1000, 17, 2049],
                     steps=40, window_K=32, tau=0.5, k_soft=2.0, vocab=128256, logit_sigma=3.0,
                     recipe="hh", f_hh=[0.35, 0.3, 0.2], scope="token")
    s_cold, s_hot = gen.hh_relevance_bounds(w)
    assert s_cold < w.tau - H.MARGIN and s_hot / 2 > w.tau + H.MARGIN
    _parity(w, {})


@pytest.mark.parametrize("relevance,scope", [("abs", "layer"), ("abs", "token"),
                                             ("softmax", "layer"), ("softmax", "token")])
def test_wide_query_groups(relevance, scope):
    """64 query heads over 8 KV heads (G = 8): a lane keeps half of a KV head's
    query heads, two waves share every token, and the two parts of each
    token's score are summed after the tiles, for both readings of the score
    and both state scopes."""
    w0 = _multi(name="wide", n_layers=2, n_q_heads=64, n_kv_heads=8, head_dim=128, dtype="bf16",
                prefill=[260, 130], steps=40, relevance=relevance, scope=scope)
    softmax = relevance == "softmax"
    w, att = _tuned(w0, 0.5 if softmax else 0.55, relative=softmax)
    _parity(w, att)


@pytest.mark.parametrize("relevance,scope", [("abs", "layer"), ("softmax", "token")])
def test_multi_head_attention(relevance, scope):
    """32 query heads over 32 KV heads (plain multi-head attention): four waves
    share every token, each with 8 of its KV heads."""
    w0 = _multi(name="mha", n_layers=2, n_q_heads=32, n_kv_heads=32, head_dim=128, dtype="bf16",
                prefill=[260, 130], steps=40, relevance=relevance, scope=scope)
    softmax = relevance == "softmax"
    w, att = _tuned(w0, 0.5 if softmax else 0.55, relative=softmax)
    _parity(w, att)


def _inside(**kw):
    """Freeze candidates inside a window of 96 positions; k = 0.5 freezes a
    token for 2 steps at its first detection, so the window's tokens come and go."""
    args = dict(name="inside", candidates="inside", window_K=96, k_soft=0.5)
    args.update(kw)
    return _multi(**args)


@pytest.mark.parametrize("relevance,scope", [("abs", "layer"), ("abs", "token"),
                                             ("softmax", "layer"), ("softmax", "token")])
def test_candidates_inside_window(relevance, scope):
    """Freeze candidates taken inside the window of the K most recent positions
    (the wording of Sec. 3.2) for both scores and both state scopes."""
    softmax = relevance == "softmax"
    w, att = _tuned(_inside(relevance=relevance, scope=scope), 0.5 if softmax else 0.55,
                    relative=softmax)
    _parity(w, att)


@pytest.mark.parametrize("shape", [
    dict(n_q_heads=32, n_kv_heads=8, head_dim=128, dtype="bf16"),    # one wave per token
    dict(n_q_heads=64, n_kv_heads=8, head_dim=128, dtype="bf16"),    # two waves share a token
    dict(n_q_heads=32, n_kv_heads=32, head_dim=128, dtype="bf16"),   # four waves share a token
])
def test_candidates_inside_window_layouts(shape):
    w, att = _tuned(_inside(name="inside-layout", n_layers=2, prefill=[400, 97], steps=40,
                            **shape), 0.55)
    _parity(w, att)


def test_candidates_inside_window_flag_all_hand_count():
    """Every candidate flagged (tau = +inf), K = 32, k = 2, a 14-token prompt
    and 255 steps: by the hand derivation each (layer, sequence) ends with the
    tokens of relative steps 16, 18, ..., 32 frozen, 260 of 269 active."""
    w = gen.Workload(name="inside-flag-all", seed=gen.SEED + 71, n_layers=2, batch=3,
                     n_q_heads=32, n_kv_heads=8, head_dim=128, dtype="bf16",
                     prefill=[14, 14, 14], steps=255, window_K=32, tau=float("inf"), k_soft=2.0,
                     vocab=64, logit_sigma=1.0, recipe="gauss", candidates="inside")
    inp = H.Inputs(w)
    instances = [(l, b) for l in range(w.n_layers) for b in range(w.batch)]
    g, _, stats = H.run_gpu(w, inp, instances, with_logits=False,
                            record=lambda t: t in (1, 100, w.steps))
    for key in instances:
        last = g[key][-1]
        assert len(last["frozen"]) == 269
        assert int((~last["frozen"]).sum()) == 260
        assert list(np.nonzero(last["frozen"])[0]) == sorted(269 - r for r in range(16, 33, 2))
    assert stats[-1]["active_positions"] == 260 * len(instances)
