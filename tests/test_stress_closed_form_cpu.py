"""The closed form behind the recovery-stress test, checked against the oracle
stepped in full on a small heavy-hitter instance (CPU only)."""
import numpy as np

import oracle
from synth import gen
from tests import _harness as H
from tests._closed_form import ClosedForm, base_trajectory


def test_closed_form_matches_stepped_oracle():
    w = gen.recovery_stress(prefill=[700], steps=140, window_K=32, name="stress-small")
    s_cold, s_hot = gen.hh_relevance_bounds(w)
    assert s_cold < w.tau - H.MARGIN and s_hot > w.tau + H.MARGIN
    P, S = w.prefill[0], w.steps
    K, V = gen.kv_rows(w, 0, 0, 0, P + S)
    cf = ClosedForm(w, gen.hh_mask(w, 0, 0, 0, P + S), base_trajectory(w.k_soft, S + 1))
    inst = oracle.Instance(K[:P], V[:P], w.window_K, w.tau, w.k_soft, capacity=P + S + 1)
    for t in range(1, S + 1):
        rec = inst.step(gen.q_row(w, 0, 0, t), K[P + t - 1], V[P + t - 1])
        np.testing.assert_array_equal(rec.active, cf.active(t), err_msg=f"attended, step {t}")
        timer, count, frozen = inst.state()
        c, f, r = cf.state(t)
        np.testing.assert_array_equal(count, c, err_msg=f"counts, step {t}")
        np.testing.assert_array_equal(frozen, f, err_msg=f"frozen, step {t}")
        np.testing.assert_array_equal(timer[frozen], r[frozen], err_msg=f"timers, step {t}")


def test_closed_form_matches_stepped_oracle_on_a_32layer_instance():
    """The same closed form on one (layer, sequence) of the 32-layer, batch-8,
    32k-context workload (the one whose 256 instances the GPU test checks with
    it), over its first 20 steps, which include the dense steps and the first
    freezes."""
    w = gen.llama8b_32layer(steps=20)
    l, b = 5, 3
    P, S = w.prefill[b], w.steps
    K, V = gen.kv_rows(w, l, b, 0, P + S)
    cf = ClosedForm(w, gen.hh_mask(w, l, b, 0, P + S), base_trajectory(w.k_soft, S + 1), seq=b)
    inst = oracle.Instance(K[:P], V[:P], w.window_K, w.tau, w.k_soft, capacity=P + S + 1)
    for t in range(1, S + 1):
        rec = inst.step(gen.q_row(w, l, b, t), K[P + t - 1], V[P + t - 1])
        np.testing.assert_array_equal(rec.active, cf.active(t), err_msg=f"attended, step {t}")
        timer, count, frozen = inst.state()
        c, f, r = cf.state(t)
        np.testing.assert_array_equal(count, c, err_msg=f"counts, step {t}")
        np.testing.assert_array_equal(frozen, f, err_msg=f"frozen, step {t}")
        np.testing.assert_array_equal(timer[frozen], r[frozen], err_msg=f"timers, step {t}")
    assert frozen.any()
