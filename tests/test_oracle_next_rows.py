"""Pins of the oracle's extensions: the history window W of Eq. 3, relevance
by attention weight, and the token-global freeze scope (one token state per
sequence, relevance averaged over layers).  Each pin compares the oracle with
a hand derivation, a closed form, an invariant or a reduction to the pinned
per-layer oracle; planted mistakes at the end fail them."""
import json
import math
import os

import numpy as np
import pytest

from oracle import asrkf_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _flag_all(P, steps, K, k_soft, W=0, cls=O.Instance):
    inst = cls(np.zeros((P, 1, 1)), np.zeros((P, 1, 1)), K, math.inf, k_soft,
               capacity=P + steps + 1, history_W=W)
    z = np.zeros((1, 1))
    recs = [inst.step(z, z, z) for _ in range(steps)]
    return inst, recs


# --------------------------------------------------------------------------
# history window W (Eq. 3)
# --------------------------------------------------------------------------

def _window_trajectory(cls=O.Instance):
    g = _golden("history_window_trajectory.json")
    inst = cls(np.zeros((33, 1, 1)), np.zeros((33, 1, 1)), 32, math.inf, g["k"],
               capacity=200, history_W=g["W"])
    z = np.zeros((1, 1))
    attends, counts = set(), {}
    for t in range(1, 101):
        rec = inst.step(z, z, z)
        if 0 in rec.active:
            attends.add(t)
            counts[t] = int(inst.count[0])
    return g, attends, counts


def test_history_window_hand_trajectory():
    g, attends, counts = _window_trajectory()
    for t in g["excluded_at_steps"]:
        assert t not in attends, t
    for t in g["attends_at_steps"]:
        assert t in attends, t
    for t, c in g["count_after_step"]:
        assert counts[t] == c, (t, counts[t], c)


def test_long_window_is_the_cumulative_count():
    """W at least the run length counts every detection: Table 1's 170 of 514."""
    paper = _golden("paper_numbers.json")
    hp, tb = paper["hyperparameters"], paper["table1"]
    inst, _ = _flag_all(14, tb["total_tokens"] - 14, hp["window_K"], hp["k"], W=10 ** 6)
    assert int((~inst.frozen[: inst.n]).sum()) == tb["active_kv"]


@pytest.mark.parametrize("W,k", [(3, 2.0), (1, 1.0001), (15, 4.0)])
def test_window_shorter_than_k_squared_never_freezes(W, k):
    """c <= W < k^2 gives d = floor(sqrt(c)/k) = 0: nothing is ever frozen."""
    inst, recs = _flag_all(40, 120, 8, k, W=W)
    assert not inst.frozen.any()
    assert all(len(r.active) == 40 + t for t, r in enumerate(recs, 1))


# --------------------------------------------------------------------------
# relevance by attention weight
# --------------------------------------------------------------------------

def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


def test_softmax_relevance_sums_to_one():
    q, K = _rand((8, 16), 1), _rand((300, 2, 16), 2)
    s = O.relevance_softmax(q, K)
    assert abs(s.sum() - 1.0) < 1e-12 and (s > 0).all()


def test_softmax_relevance_equal_keys_is_uniform():
    q = _rand((4, 8), 3)
    K = np.repeat(_rand((1, 1, 8), 4), 37, axis=0)
    np.testing.assert_allclose(O.relevance_softmax(q, K), 1.0 / 37, rtol=1e-13)


def test_softmax_relevance_two_tokens_is_logistic():
    """Two keys whose logits differ by delta under every head: s_1 = 1/(1+e^-delta/sqrt(d))."""
    D = 16
    q = np.zeros((2, D))
    q[:, 0] = 1.0
    K = np.zeros((2, 1, D))
    K[0, 0, 0], K[1, 0, 0] = 3.0, -1.0                 # q.k difference 4
    s = O.relevance_softmax(q, K)
    expect = 1.0 / (1.0 + math.exp(-4.0 / math.sqrt(D)))
    assert abs(s[0] - expect) < 1e-15 and abs(s[1] - (1 - expect)) < 1e-15


def test_attend_rows_softmax_kind_matches_definition():
    q, K, V = _rand((8, 16), 5), _rand((50, 2, 16), 6), _rand((50, 2, 16), 7)
    Kh, Vh = K.transpose(1, 0, 2), V.transpose(1, 0, 2)
    out, s = O.attend_rows(q, Kh, Vh, "softmax")
    np.testing.assert_allclose(s, O.relevance_softmax(q, K), rtol=1e-12)
    np.testing.assert_allclose(out, O.attention(q, K, V), rtol=1e-12)


# --------------------------------------------------------------------------
# token-global scope
# --------------------------------------------------------------------------

def _inputs(L, P, steps, Hq=4, Hkv=2, D=8, seed=10):
    K = [_rand((P + steps, Hkv, D), seed + l) for l in range(L)]
    V = [_rand((P + steps, Hkv, D), seed + 100 + l) for l in range(L)]
    Q = [[_rand((Hq, D), seed + 1000 * (l + 1) + t) for t in range(steps)] for l in range(L)]
    return K, V, Q


def test_global_scope_one_layer_is_the_layer_scope():
    P, S = 60, 40
    K, V, Q = _inputs(1, P, S)
    a = O.Instance(K[0][:P], V[0][:P], 8, 2.5, 2.0, capacity=P + S + 1)
    b = O.GlobalInstance([K[0][:P]], [V[0][:P]], 8, 2.5, 2.0, capacity=P + S + 1)
    for t in range(S):
        ra = a.step(Q[0][t], K[0][P + t], V[0][P + t])
        rb = b.step([Q[0][t]], [K[0][P + t]], [V[0][P + t]])
        np.testing.assert_array_equal(ra.active, rb.active)
        np.testing.assert_allclose(rb.out[0], ra.out, rtol=1e-13)
        for x, y in zip(a.state(), b.state()):
            np.testing.assert_array_equal(x, y)
    assert a.frozen.any()                      # the run does freeze


def test_global_scope_identical_layers_match_one_layer():
    P, S, L = 60, 40, 3
    K, V, Q = _inputs(1, P, S)
    a = O.Instance(K[0][:P], V[0][:P], 8, 2.5, 2.0, capacity=P + S + 1)
    b = O.GlobalInstance([K[0][:P]] * L, [V[0][:P]] * L, 8, 2.5, 2.0, capacity=P + S + 1)
    for t in range(S):
        ra = a.step(Q[0][t], K[0][P + t], V[0][P + t])
        rb = b.step([Q[0][t]] * L, [K[0][P + t]] * L, [V[0][P + t]] * L)
        np.testing.assert_array_equal(ra.active, rb.active)
    for x, y in zip(a.state(), b.state()):
        np.testing.assert_array_equal(x, y)


def _two_layer_scores(s0, s1):
    """Three prompt tokens, two layers; |q.k| of token j in layer l is s_l[j]
    (one head, one dimension), window 0, tau 0.5.  Returns the tokens flagged
    at step 1 (count 1)."""
    K0 = np.array(s0, dtype=np.float64).reshape(3, 1, 1)
    K1 = np.array(s1, dtype=np.float64).reshape(3, 1, 1)
    inst = O.GlobalInstance([K0, K1], [K0, K1], 0, 0.5, 0.5, capacity=8)
    q = np.ones((1, 1))
    inst.step([q, q], [np.full((1, 1), 9.0)] * 2, [np.zeros((1, 1))] * 2)
    return [j for j in range(3) if inst.count[j] == 1]


def test_global_scope_averages_over_layers():
    # means: 0.4 (flag), 0.6 (keep), 0.475 (flag); a sum, a min or a max flags other tokens
    assert _two_layer_scores([0.4, 0.2, 0.4], [0.4, 1.0, 0.55]) == [0, 2]


def test_global_scope_flag_all_reproduces_table1():
    paper = _golden("paper_numbers.json")
    hp, tb = paper["hyperparameters"], paper["table1"]
    steps = tb["total_tokens"] - 14
    z = np.zeros((14, 1, 1))
    inst = O.GlobalInstance([z, z], [z, z], hp["window_K"], math.inf, hp["k"], capacity=600)
    q = np.zeros((1, 1))
    for _ in range(steps):
        inst.step([q, q], [q, q], [q, q])
    assert int((~inst.frozen[: inst.n]).sum()) == tb["active_kv"]


# --------------------------------------------------------------------------
# planted mistakes
# --------------------------------------------------------------------------

class _WindowOneLonger(O.Instance):
    def detect(self, j):
        hist = self.detections[j]
        hist.append(self.t)
        self.count[j] = sum(1 for s in hist if s >= self.t - self.history_W)
        return self.count[j]


def test_planted_window_off_by_one_breaks_trajectory():
    g, attends, counts = _window_trajectory(_WindowOneLonger)
    assert any(t in attends for t in g["excluded_at_steps"]) or \
        any(counts.get(t) != c for t, c in g["count_after_step"])


def test_planted_unscaled_softmax_breaks_logistic(monkeypatch):
    def unscaled(q, K):
        q = np.asarray(q, dtype=np.float64)
        s = np.zeros(K.shape[0])
        for h in range(q.shape[0]):
            x = K[:, 0, :] @ q[h]
            w = np.exp(x - x.max())
            s += w / w.sum()
        return s / q.shape[0]
    monkeypatch.setattr(O, "relevance_softmax", unscaled)
    with pytest.raises(AssertionError):
        test_softmax_relevance_two_tokens_is_logistic()


# --------------------------------------------------------------------------
# freeze candidates inside the window (the wording of Sec. 3.2)
# --------------------------------------------------------------------------

def _flag_all_inside(P, steps, K, k_soft, cls=O.Instance, hook=None):
    inst = cls(np.zeros((P, 1, 1)), np.zeros((P, 1, 1)), K, math.inf, k_soft,
               capacity=P + steps + 1, candidates="inside")
    z = np.zeros((1, 1))
    for t in range(1, steps + 1):
        rec = inst.step(z, z, z)
        if hook:
            hook(t, rec, inst)
    return inst


@pytest.mark.parametrize("P", [0, 1, 14, 40, 100])
def test_inside_window_frozen_at_end(P):
    g = _golden("inside_window_trajectory.json")
    for K, frozen in g["frozen_at_end_by_K"]:
        for steps in (K + 2, K + 37, 150):
            inst = _flag_all_inside(P, steps, K, g["k"])
            assert int(inst.frozen[: inst.n].sum()) == frozen, (P, K, steps)


def test_inside_window_token_trajectory():
    g = _golden("inside_window_trajectory.json")
    tr = g["token_appended_at_step_1"]
    P = 14
    attends = set()
    _flag_all_inside(P, 220, tr["K"], g["k"],
                     hook=lambda t, rec, inst: attends.add(t) if P in rec.active else None)
    for t in tr["excluded_at_steps"]:
        assert t not in attends, t
    for t in tr["attends_at_steps"]:
        assert t in attends, t
    excluded = set(range(1, 221)) - attends
    assert excluded == set(tr["excluded_at_steps"])


def test_inside_window_table_runs():
    g = _golden("inside_window_trajectory.json")
    for n, active in g["table_runs"]:
        inst = _flag_all_inside(14, n - 14, 32, g["k"])
        assert inst.n == n and int((~inst.frozen[:n]).sum()) == active


def test_inside_window_only_window_tokens_are_counted():
    """Tokens outside the window are never detected: their counts stop when
    they leave it, and the protected region of the default reading is exactly
    where detections happen now."""
    inst = _flag_all_inside(20, 120, 8, 2.0)
    n = inst.n
    assert (inst.count[: n - 8] <= 8).all()
    assert (inst.count[20: n - 8] == 8).all()        # decode tokens: 8 steps inside, never frozen


def test_inside_window_token_scope_matches_layer_scope_when_all_flagged():
    P, steps, K = 14, 90, 32
    a = _flag_all_inside(P, steps, K, 2.0)
    L = 3
    z = np.zeros((P, 1, 1))
    gi = O.GlobalInstance([z] * L, [z] * L, K, math.inf, 2.0, capacity=P + steps + 1,
                          candidates="inside")
    q = np.zeros((1, 1))
    for _ in range(steps):
        gi.step([q] * L, [q] * L, [q] * L)
    assert (gi.frozen[: gi.n] == a.frozen[: a.n]).all()
    assert (gi.count[: gi.n] == a.count[: a.n]).all()


def test_unknown_candidates_value_is_refused():
    with pytest.raises(ValueError):
        O.Instance(np.zeros((1, 1, 1)), np.zeros((1, 1, 1)), 4, 0.0, 2.0, candidates="all")


class _InsideWindowOneWider(O.Instance):
    """Planted: a window of K + 1 positions."""
    def outside_window(self, j):
        return j < self.n - 1 - self.window_K


class _InsideWindowOneNarrower(O.Instance):
    """Planted: the window leaves out the token appended this step."""
    def outside_window(self, j):
        return j < self.n - self.window_K or j == self.n - 1


@pytest.mark.parametrize("cls", [_InsideWindowOneWider, _InsideWindowOneNarrower])
def test_planted_inside_window_edges_break_the_hand_counts(cls):
    g = _golden("inside_window_trajectory.json")
    got = [int(_flag_all_inside(14, 120, K, g["k"], cls=cls).frozen.sum())
           for K, _ in g["frozen_at_end_by_K"]]
    assert got != [f for _, f in g["frozen_at_end_by_K"]]
