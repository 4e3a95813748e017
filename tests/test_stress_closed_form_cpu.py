"""The closed form behind the recovery-stress test, checked against the oracle
stepped in full on a small heavy-hitter instance (CPU only)."""
import numpy as np

import oracle
from synth import gen
from tests import _harness as H
from tests.test_gpu_recovery_stress import ClosedForm, _base_trajectory


def test_closed_form_matches_stepped_oracle():
    w = gen.recovery_stress(prefill=[700], steps=140, window_K=32, name="stress-small")
    s_cold, s_hot = gen.hh_relevance_bounds(w)
    assert s_cold < w.tau - H.MARGIN and s_hot > w.tau + H.MARGIN
    P, S = w.prefill[0], w.steps
    K, V = gen.kv_rows(w, 0, 0, 0, P + S)
    cf = ClosedForm(w, gen.hh_mask(w, 0, 0, 0, P + S), _base_trajectory(w.k_soft, S + 1))
    inst = oracle.Instance(K[:P], V[:P], w.window_K, w.tau, w.k_soft, capacity=P + S + 1)
    for t in range(1, S + 1):
        rec = inst.step(gen.q_row(w, 0, 0, t), K[P + t - 1], V[P + t - 1])
        np.testing.assert_array_equal(rec.active, cf.active(t), err_msg=f"attended, step {t}")
        timer, count, frozen = inst.state()
        c, f, r = cf.state(t)
        np.testing.assert_array_equal(count, c, err_msg=f"counts, step {t}")
        np.testing.assert_array_equal(frozen, f, err_msg=f"frozen, step {t}")
        np.testing.assert_array_equal(timer[frozen], r[frozen], err_msg=f"timers, step {t}")
