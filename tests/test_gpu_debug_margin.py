"""The debug margin check: with debug_margin > 0 the library counts the freeze
decisions taken on a relevance within the margin of tau (decisions that
rounding could flip).  A heavy-hitter run whose scores are proven to keep a
distance from tau counts none; a run with tau placed among the scores counts
what the oracle's fp64 scores say, up to the rounding of the scores
themselves.  The count is exact in every mode (layer and token scope, Eq. 2
and softmax relevance, spill mode)."""
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


def _margin_hits(w, inp, margin):
    """Run the library with the margin check on; returns its margin_hits."""
    import paper_2512_11221_amd as A
    cfg = A.make_config(w.n_layers, w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.max_ctx,
                        w.window_K, w.tau, w.k_soft, w.vocab, entropy_spike=w.entropy_spike,
                        conf_drop=w.conf_drop, wr_last_N=w.wr_last_N, dtype=w.dtype,
                        spill_min_D=w.spill_min_D, history_W=w.history_W,
                        relevance=w.relevance, scope=w.scope, candidates=w.candidates,
                        debug_margin=margin)
    ctx = A.asrkf_init(cfg)
    try:
        inst = [(l, b) for l in range(w.n_layers) for b in range(w.batch)]
        H.run_gpu(w, inp, inst, record=lambda t: False, ctx=ctx)
        return A.asrkf_stats(ctx)["margin_hits"]
    finally:
        A.asrkf_destroy(ctx)


def _oracle_bounds(w, inp, margin, eps):
    """Freeze decisions whose fp64 score is within margin - eps of tau (the
    library must count them) and within margin + eps (it may count them)."""
    lo = hi = 0

    def see(l, b, t, n, attended, scores):
        nonlocal lo, hi
        cand = H.candidate_mask(w, np.asarray(attended), n)
        d = np.abs(np.asarray(scores, np.float64) - w.tau)[cand]
        lo += int((d < margin - eps).sum())
        hi += int((d < margin + eps).sum())

    inst = [(l, b) for l in range(w.n_layers) for b in range(w.batch)]
    H.run_oracle(w, inp, inst, record=lambda t: False, on_scores=see)
    return lo, hi


def test_no_hits_when_scores_keep_their_distance():
    w = gen.Workload(name="margin-hh", seed=gen.SEED + 101, n_layers=2, batch=2, n_q_heads=32,
                     n_kv_heads=8, head_dim=128, dtype="bf16", prefill=[300, 170], steps=24,
                     window_K=16, tau=0.5, k_soft=2.0, vocab=1024, logit_sigma=2.0, recipe="hh",
                     f_hh=[0.35, 0.25])
    s_cold, s_hot = gen.hh_relevance_bounds(w)
    gap = min(w.tau - s_cold, s_hot - w.tau)
    assert gap > H.MARGIN
    inp = H.Inputs(w)
    assert _margin_hits(w, inp, 0.5 * gap) == 0
    assert _margin_hits(w, inp, 0.0) == 0                 # off


@pytest.mark.parametrize("case", ["abs-layer", "abs-token", "softmax-layer", "spill"])
def test_hits_match_the_oracle(case):
    """tau at the median candidate score, so many decisions fall near it; the
    inputs keep every decision 1e-3 (softmax: 1e-5 relative) from tau, so the
    run follows the oracle's, and the margin is wide against the rounding of a
    score (eps)."""
    kw = {"abs-layer": {}, "abs-token": dict(scope="token", n_layers=2),
          "softmax-layer": dict(relevance="softmax"), "spill": dict(spill_min_D=2)}[case]
    relative = case == "softmax-layer"
    w = gen.tiny(**kw)
    w = w.replace(tau=H.score_quantile_run(w, 0.5))
    attempts = H.fix_margin_run(w, 1e-5 if relative else H.MARGIN, relative=relative)
    inp = H.Inputs(w, attempts)
    margin = 0.1 * abs(w.tau)
    eps = 1e-5 * abs(w.tau) if relative else 1e-4
    lo, hi = _oracle_bounds(w, inp, margin, eps)
    assert lo > 20, lo                                    # the check has something to count
    got = _margin_hits(w, inp, margin)
    print(f"{case}: tau {w.tau:.6g} margin {margin:.4g}: library {got}, oracle [{lo}, {hi}]")
    assert lo <= got <= hi
