"""Parity at the full workload sizes, in the launch configuration the bench
times: every input generated on the device (bit-identical to the host
generator, checked in test_gpu_synth), the oracle run on sampled
(layer, sequence) instances over every decode step."""
import math

import numpy as np
import pytest

from synth import gen
from tests import _harness as H
from tests._closed_form import ClosedForm, base_trajectory

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2512_11221_amd as A
    A.load()


def test_llama8b_32layer_batch8_ctx32k_sampled():
    """Outputs of two sampled instances against the oracle at every step; the
    token states of all 256 (layer, sequence) instances at the recorded steps,
    bit for bit, against the closed form of the heavy-hitter recipe (no
    recovery fires: theta_H is +inf), which the oracle's own trajectory
    defines."""
    w = gen.llama8b_32layer()
    assert math.isinf(w.entropy_spike) and w.conf_drop <= 0
    s_cold, s_hot = gen.hh_relevance_bounds(w)
    assert s_cold < w.tau - H.MARGIN and s_hot > w.tau + H.MARGIN
    instances = [(0, 0), (31, 7)]
    record = {1, 16, 17, 18, 64, w.steps}
    base = base_trajectory(w.k_soft, w.steps + 1)
    n_end = max(w.prefill) + w.steps
    checked = []

    def check_state(l, b, t, st):
        cf = ClosedForm(w, gen.hh_mask(w, l, b, 0, n_end), base, seq=b)
        count, frozen, timer = cf.state(t)
        assert st["n"] == len(frozen), (l, b, t)
        np.testing.assert_array_equal(st["count"], count, err_msg=f"counts, layer {l} seq {b} step {t}")
        np.testing.assert_array_equal(st["frozen"], frozen, err_msg=f"frozen, layer {l} seq {b} step {t}")
        np.testing.assert_array_equal(st["unfreeze"][frozen] - (t + 1), timer[frozen],
                                      err_msg=f"timers, layer {l} seq {b} step {t}")
        act = np.concatenate([np.nonzero(~frozen)[0], [len(frozen)]])
        np.testing.assert_array_equal(st["active"], act, err_msg=f"list, layer {l} seq {b} step {t}")
        checked.append((l, b, t))

    outs, states, ent = H.run_gpu_device(w, instances, record, check_state=check_state)
    assert len(checked) == w.n_layers * w.batch * len(record)
    inp = H.Inputs(w)
    worst = H.compare_sampled(w, inp, instances, outs, states, record)
    print(f"worst |out - oracle| = {worst:.3e}; states of {w.n_layers * w.batch} instances "
          f"at steps {sorted(record)} match the closed form")
    # entropy of every sequence at every step
    for b in range(w.batch):
        for t in range(1, w.steps + 1, 9):
            e, _ = H.oracle.entropy(inp.logits(b, t))
            assert abs(ent[b][t - 1]["entropy"] - e) <= H.ENTROPY_TOL


def test_ragged_batch64_sampled():
    w = gen.ragged()
    order = np.argsort(w.prefill)
    seqs = [int(order[0]), int(order[len(order) // 2]), int(order[-1])]
    instances = [(0, b) for b in seqs]
    record = {1, 17, 40, w.steps}
    outs, states, ent = H.run_gpu_device(w, instances, record, seqs_for_entropy=seqs)
    inp = H.Inputs(w)
    worst = H.compare_sampled(w, inp, instances, outs, states, record)
    print(f"ragged: prompts {[w.prefill[b] for b in seqs]}, worst |out - oracle| = {worst:.3e}")
