"""Pins of the CPU oracle against what the paper prints and what mathematics fixes.

Every check here compares the oracle with something other than itself: values
printed in the paper (tests/golden/), hand derivations, closed forms, library
routines (math.isqrt, torch SDPA, scipy entropy) and invariants.  The planted
mistakes at the end show that plausible errors in the oracle fail these pins.
"""
import json
import math
import os

import numpy as np
import pytest

import oracle
from oracle import asrkf_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


PAPER = _golden("paper_numbers.json")


# --------------------------------------------------------------------------
# Eq. 3
# --------------------------------------------------------------------------

def test_eq3_printed_examples():
    g = PAPER["eq3_examples"]
    for c, d in g["count_to_duration"]:
        assert oracle.freeze_duration(c, g["k"]) == d, (c, d)


@pytest.mark.parametrize("num,den", [(2, 1), (3, 2), (3, 4), (5, 2), (1, 1), (7, 8)])
def test_eq3_integer_sqrt_closed_form(num, den):
    # k = num/den: floor(sqrt(c)/k) = floor(sqrt(den^2 c) / num) = isqrt(den^2 c) // num
    k = num / den
    for c in range(0, 5000):
        assert oracle.freeze_duration(c, k) == math.isqrt(den * den * c) // num, (c, k)


def test_eq3_first_detection_never_freezes_at_default_k():
    # "First detection yields d = 0 (no freeze)" (Sec. 3.4) for the default k = 2
    assert oracle.freeze_duration(1, PAPER["hyperparameters"]["k"]) == 0


# --------------------------------------------------------------------------
# Algorithm 1: schedule-only replays
# --------------------------------------------------------------------------

def _flag_all(P, steps, K, k_soft=2.0, hook=None, inst_cls=O.Instance):
    """Every out-of-window active token is flagged (tau = +inf); values unused."""
    inst = inst_cls(np.zeros((P, 1, 1)), np.zeros((P, 1, 1)), K, float("inf"), k_soft,
                    capacity=P + steps + 1)
    z = np.zeros((1, 1))
    for t in range(1, steps + 1):
        rec = inst.step(z, z, z)
        if hook:
            hook(t, rec, inst)
    return inst


def _active_after(inst):
    return int((~inst.frozen[: inst.n]).sum())


def test_single_token_hand_trajectory():
    g = _golden("single_token_trajectory.json")
    reached, attends = {}, set()

    def hook(t, rec, inst):
        if 0 in rec.active:
            attends.add(t)
        reached.setdefault(int(inst.count[0]), t)

    # 33-token prompt, window 32: position 0 is outside the window from step 1
    _flag_all(33, 2100, 32, g["k"], hook)
    for c, t in g["count_reached_at_step"]:
        assert reached[c] == t, (c, reached.get(c), t)
    for t in g["attends_at_steps"]:
        assert t in attends, t
    for t in g["excluded_at_steps"]:
        assert t not in attends, t


@pytest.mark.parametrize("table", ["table1", "table3"])
@pytest.mark.parametrize("P", [1, 14, 33])
def test_paper_active_kv_counts(table, P):
    """Tables 1 and 3 follow from the schedule alone with the paper's K and k,
    for any prompt of at most K + 1 tokens (prompt length is not printed)."""
    hp, tb = PAPER["hyperparameters"], PAPER[table]
    inst = _flag_all(P, tb["total_tokens"] - P, hp["window_K"], hp["k"])
    assert inst.n == tb["total_tokens"]
    active = _active_after(inst)
    assert active == tb["active_kv"]
    assert round(100.0 * (1 - active / inst.n), 2) == tb["compression_pct"]


def test_figure1_trajectory_settles():
    hp, fig = PAPER["hyperparameters"], PAPER["figure1_prose"]
    traj = []
    _flag_all(14, 500, hp["window_K"], hp["k"],
              lambda t, r, inst: traj.append(_active_after(inst)))
    late = traj[199:]
    assert fig["low"] - 5 <= min(late) and max(late) <= fig["high"]
    assert traj[-1] < 514 / 2          # sublinear: well under the full cache


def test_window_tokens_never_freeze():
    inst = _flag_all(40, 300, 32)
    n = inst.n
    assert not inst.frozen[n - 32:n].any()


# --------------------------------------------------------------------------
# Eq. 1 (attention)
# --------------------------------------------------------------------------

def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


def test_attention_matches_torch_sdpa():
    torch = pytest.importorskip("torch")
    Hq, Hkv, D, n = 8, 2, 16, 37
    q, K, V = _rand((Hq, D), 1), _rand((n, Hkv, D), 2), _rand((n, Hkv, D), 3)
    got = oracle.attention(q, K, V)
    G = Hq // Hkv
    tq = torch.tensor(q)[:, None, :]                             # [Hq][1][D]
    tk = torch.tensor(K).permute(1, 0, 2).repeat_interleave(G, 0)  # [Hq][n][D]
    tv = torch.tensor(V).permute(1, 0, 2).repeat_interleave(G, 0)
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk.contiguous(), tv.contiguous())
    np.testing.assert_allclose(got, ref[:, 0, :].numpy(), rtol=1e-12, atol=1e-12)


def test_attention_special_cases():
    Hq, Hkv, D = 4, 2, 8
    q = _rand((Hq, D), 4)
    V = _rand((5, Hkv, D), 5)
    # a single active token: output is its value row
    np.testing.assert_allclose(oracle.attention(q, _rand((1, Hkv, D), 6), V[:1]),
                               V[0, [0, 0, 1, 1], :], atol=1e-15)
    # equal keys: output is the mean value row
    K = np.repeat(_rand((1, Hkv, D), 7), 5, axis=0)
    np.testing.assert_allclose(oracle.attention(q, K, V), V.mean(0)[[0, 0, 1, 1]], atol=1e-12)
    # one dominant logit: output is that value row
    K = np.zeros((5, Hkv, D))
    K[3] = 200.0
    np.testing.assert_allclose(oracle.attention(np.abs(q) + 0.5, K, V), V[3, [0, 0, 1, 1], :],
                               atol=1e-9)
    # permutation invariance over the attended set
    K, perm = _rand((5, Hkv, D), 8), np.array([4, 2, 0, 1, 3])
    np.testing.assert_allclose(oracle.attention(q, K[perm], V[perm]), oracle.attention(q, K, V),
                               atol=1e-13)


def test_fused_pass_equals_the_definitions():
    Hq, Hkv, D, n = 8, 2, 16, 41
    q, K, V = _rand((Hq, D), 21), _rand((n, Hkv, D), 22), _rand((n, Hkv, D), 23)
    out, s = oracle.attend_rows(q, [K[:, g] for g in range(Hkv)], [V[:, g] for g in range(Hkv)])
    np.testing.assert_allclose(out, oracle.attention(q, K, V), rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(s, oracle.relevance(q, K), rtol=1e-13, atol=1e-14)


def test_freezing_nothing_is_dense_attention():
    """tau below every score: nothing is flagged, every step attends all tokens."""
    Hq, Hkv, D, P, steps = 4, 2, 8, 20, 6
    K, V = _rand((P + steps, Hkv, D), 9), _rand((P + steps, Hkv, D), 10)
    Q = _rand((steps, Hq, D), 11)
    inst = O.Instance(K[:P], V[:P], 4, -1.0, 2.0, capacity=P + steps)
    for t in range(steps):
        rec = inst.step(Q[t], K[P + t], V[P + t])
        assert list(rec.active) == list(range(P + t + 1))
        np.testing.assert_allclose(rec.out, oracle.attention(Q[t], K[: P + t + 1], V[: P + t + 1]))


# --------------------------------------------------------------------------
# Eq. 2 (relevance)
# --------------------------------------------------------------------------

def test_relevance_closed_forms():
    Hq, Hkv, D = 8, 2, 4
    e0 = np.eye(D)[0]
    # all heads the unit query e0, key c*e0 in both KV heads: s = |c|
    q = np.tile(e0, (Hq, 1))
    K = np.zeros((1, Hkv, D))
    K[0, :, 0] = -3.0
    assert oracle.relevance(q, K)[0] == pytest.approx(3.0, abs=1e-15)
    # signs alternate across heads: the absolute value keeps them from cancelling
    q = np.array([(-1) ** h * e0 for h in range(Hq)])
    assert oracle.relevance(q, K)[0] == pytest.approx(3.0, abs=1e-15)
    # head h = (h+1) e0, KV head g key = (g+1) e0, grouping h -> h // 4:
    # (1+2+3+4)*1 + (5+6+7+8)*2 = 62, over 8 heads = 7.75
    q = np.array([(h + 1) * e0 for h in range(Hq)])
    K = np.zeros((1, Hkv, D))
    K[0, 0, 0], K[0, 1, 0] = 1.0, 2.0
    assert oracle.relevance(q, K)[0] == pytest.approx(7.75, abs=1e-14)
    # orthogonal query and key: zero relevance
    K = np.zeros((1, Hkv, D))
    K[0, :, 1] = 5.0
    assert oracle.relevance(np.tile(e0, (Hq, 1)), K)[0] == 0.0


# --------------------------------------------------------------------------
# Entropy (Sec. 3.6 reading: nats of softmax at T = 1)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("V,expected", [(1024, 6.931471805599453), (128256, 11.761783545564427)])
def test_entropy_uniform(V, expected):
    H, pmax = oracle.entropy(np.full(V, 0.37))
    assert H == pytest.approx(expected, abs=1e-12)
    assert pmax == pytest.approx(1.0 / V, rel=1e-12)


@pytest.mark.parametrize("a,x", [(1, 5.0), (3, -2.0), (100, 1.5), (1000, 0.25)])
def test_entropy_two_level_closed_form(a, x):
    V = 1024
    logits = np.zeros(V)
    logits[:a] = x
    Z = a * math.exp(x) + V - a
    expected = math.log(Z) - a * x * math.exp(x) / Z
    assert oracle.entropy(logits)[0] == pytest.approx(expected, abs=1e-12)


def test_entropy_matches_scipy_and_shift_invariance():
    scipy_stats = pytest.importorskip("scipy.stats")
    x = 2.0 * _rand(1024, 12)
    p = np.exp(x - x.max())
    p /= p.sum()
    H, pmax = oracle.entropy(x)
    assert H == pytest.approx(scipy_stats.entropy(p), abs=1e-12)
    assert pmax == pytest.approx(p.max(), abs=1e-15)
    assert oracle.entropy(x + 123.0)[0] == pytest.approx(H, abs=1e-11)


def test_entropy_single_dominant_logit_is_zero():
    x = np.zeros(1024)
    x[7] = 1000.0
    H, pmax = oracle.entropy(x)
    assert H == pytest.approx(0.0, abs=1e-12) and pmax == pytest.approx(1.0)


# --------------------------------------------------------------------------
# Recovery ladder (Sec. 3.6).  The paper prints no numbers for it; the pins are
# hand-derived expected states (tests/golden/recovery_levels.json) under the
# readings of SR, WR, FR and the trigger stated there.
# --------------------------------------------------------------------------

RECOVERY = _golden("recovery_levels.json")
_LEVEL = {"none": 0, "SR": O.SR, "WR": O.WR, "FR": O.FR}


def test_escalation_ladder_sequence():
    spikes = {3, 5, 6, 9, 10, 11, 12, 13}
    ent = [(10.0 if t in spikes else 1.0, 0.5) for t in range(15)]
    levels, rr = oracle.recovery_schedule(ent, theta_H=5.0, theta_p=0.0)
    assert levels == [0, 0, 0, 1, 0, 1, 2, 0, 0, 1, 2, 3, 3, 3, 0]
    assert [t for t, r in enumerate(rr) if r] == [12, 13]


@pytest.mark.parametrize("case", RECOVERY["escalation"]["cases"],
                         ids=lambda c: f"thH{c['theta_H']}-thp{c['theta_p']}")
def test_escalation_with_confidence_drop(case):
    steps = [tuple(x) for x in RECOVERY["escalation"]["steps"]]
    levels, rr = oracle.recovery_schedule(steps, float(case["theta_H"]), case["theta_p"])
    assert levels == case["levels"]
    assert [t for t, r in enumerate(rr) if r] == case["rr_steps"]


def _static_state(cls=O.TokenStates):
    g = RECOVERY["static_state"]
    n = g["n"]
    inst = cls(n + 1, 0, 0.0, 2.0)
    inst.n = n
    for j, rem in g["frozen_remaining"]:
        inst.frozen[j] = True
        inst.timer[j] = rem
    inst.count[:n] = g["counts"]
    return inst


@pytest.mark.parametrize("level", ["SR", "WR", "FR"])
def test_recovery_levels_static_state(level):
    g = RECOVERY["static_state"]
    inst = _static_state()
    inst.recover(_LEVEL[level], g["wr_last_N"])
    assert np.nonzero(inst.frozen[: g["n"]])[0].tolist() == g["frozen_after"][level]
    assert inst.count[: g["n"]].tolist() == g["counts"]        # detection counts are kept


def _recovery_case(case, inst_cls=O.Instance):
    g = RECOVERY["single_token"]
    lo, hi = g["window"]
    attends = []

    def hook(t, rec, inst):
        if lo <= t <= hi and 0 in rec.active:
            attends.append(t)
        if t == case["after_step"] and case["level"] != "none":
            inst.recover(_LEVEL[case["level"]], case["wr_last_N"])

    _flag_all(g["prompt"], hi, g["window_K"], g["k"], hook, inst_cls=inst_cls)
    return attends


@pytest.mark.parametrize("case", RECOVERY["single_token"]["cases"],
                         ids=lambda c: f"{c['level']}-after{c['after_step']}-N{c['wr_last_N']}")
def test_recovery_on_the_single_token_trajectory(case):
    assert _recovery_case(case) == case["attends"]


def _copy_instance(inst):
    import copy
    return copy.deepcopy(inst)


# --------------------------------------------------------------------------
# Planted mistakes: each must break at least one pin above
# --------------------------------------------------------------------------

class _WindowWithoutCurrent(O.Instance):
    def outside_window(self, j):
        return j < self.n - 1 - self.window_K


class _TimerSkipsNewlyFrozen(O.Instance):
    def freeze_loop(self, A, s):
        before = self.frozen.copy()
        super().freeze_loop(A, s)
        self._new = self.frozen & ~before

    def timer_loop(self):
        for j in np.nonzero(self.frozen[: self.n] & ~self._new[: self.n])[0]:
            self.timer[j] -= 1
            if self.timer[j] <= 0:
                self.frozen[j] = False


class _InsideWindowCandidates(O.Instance):
    def outside_window(self, j):
        return j >= self.n - self.window_K


@pytest.mark.parametrize("cls,expect_not", [(_WindowWithoutCurrent, 170),
                                            (_TimerSkipsNewlyFrozen, 170),
                                            (_InsideWindowCandidates, 170)])
def test_planted_schedule_mistakes_break_table1(cls, expect_not):
    inst = _flag_all(14, 500, 32, 2.0, inst_cls=cls)
    assert _active_after(inst) != expect_not


def test_planted_eq3_mistake_breaks_printed_examples(monkeypatch):
    def ceil_variant(c, k_soft):
        return math.ceil(math.sqrt(c) / k_soft)
    monkeypatch.setattr(O, "freeze_duration", ceil_variant)
    g = PAPER["eq3_examples"]
    assert any(O.freeze_duration(c, g["k"]) != d for c, d in g["count_to_duration"])


def test_planted_relevance_mistake_breaks_closed_form(monkeypatch):
    real = O.relevance

    def over_kv_heads(q, K):
        return real(q, K) * q.shape[0] / K.shape[1]
    monkeypatch.setattr(oracle, "relevance", over_kv_heads)
    with pytest.raises(AssertionError):
        test_relevance_closed_forms()


def test_planted_attention_scale_mistake_breaks_sdpa(monkeypatch):
    real = O.attention

    def unscaled(q, K, V):
        return real(np.asarray(q) * np.sqrt(np.asarray(q).shape[1]), K, V)
    monkeypatch.setattr(oracle, "attention", unscaled)
    with pytest.raises(AssertionError):
        test_attention_matches_torch_sdpa()


# Planted mistakes in the recovery ladder: each must break a hand-derived pin.

class _SoftResetAtOne(O.Instance):
    """SR also restores tokens with one step to go."""
    def recover(self, level, last_N):
        if level == O.SR:
            F = np.nonzero(self.frozen[: self.n])[0]
            sel = F[self.timer[F] >= 1]
            self.frozen[sel] = False
            self.timer[sel] = 0
        else:
            super().recover(level, last_N)


class _WindowResetOneWider(O.Instance):
    """WR reaches one position further back (positions >= n - N - 1)."""
    def recover(self, level, last_N):
        super().recover(level, last_N + 1 if level == O.WR else last_N)


class _WindowResetOneNarrower(O.Instance):
    """WR stops one position short (positions >= n - N + 1)."""
    def recover(self, level, last_N):
        super().recover(level, last_N - 1 if level == O.WR else last_N)


class _FullResetClearsCounts(O.Instance):
    """FR also clears the detection counts."""
    def recover(self, level, last_N):
        super().recover(level, last_N)
        if level == O.FR:
            self.count[: self.n] = 0


@pytest.mark.parametrize("cls", [_SoftResetAtOne, _WindowResetOneWider, _WindowResetOneNarrower,
                                 _FullResetClearsCounts])
def test_planted_recovery_mistakes_break_the_trajectories(cls):
    cases = RECOVERY["single_token"]["cases"]
    assert any(_recovery_case(c, cls) != c["attends"] for c in cases)


def _trigger_ignores_theta_p(count, H, pmax, theta_H, theta_p):
    spike = H > theta_H
    count = count + 1 if spike else 0
    return count, min(count, O.FR), count > O.FR


def _trigger_non_strict_drop(count, H, pmax, theta_H, theta_p):
    spike = (H > theta_H) or (theta_p > 0 and pmax <= theta_p)
    count = count + 1 if spike else 0
    return count, min(count, O.FR), count > O.FR


def _trigger_rr_at_level_three(count, H, pmax, theta_H, theta_p):
    spike = (H > theta_H) or (theta_p > 0 and pmax < theta_p)
    count = count + 1 if spike else 0
    return count, min(count, O.FR), count >= O.FR


@pytest.mark.parametrize("variant", [_trigger_ignores_theta_p, _trigger_non_strict_drop,
                                     _trigger_rr_at_level_three])
def test_planted_trigger_mistakes_break_the_escalation_pin(monkeypatch, variant):
    monkeypatch.setattr(O, "escalate", variant)
    broken = False
    for case in RECOVERY["escalation"]["cases"]:
        try:
            test_escalation_with_confidence_drop(case)
        except AssertionError:
            broken = True
    assert broken
