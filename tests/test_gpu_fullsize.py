"""Parity at the full workload sizes, in the launch configuration the bench
times: every input generated on the device (bit-identical to the host
generator, checked in test_gpu_synth), the oracle run on sampled
(layer, sequence) instances over every decode step."""
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


def test_llama8b_32layer_batch8_ctx32k_sampled():
    w = gen.llama8b_32layer()
    instances = [(0, 0), (31, 7)]
    record = {1, 16, 17, 18, 64, w.steps}
    outs, states, ent = H.run_gpu_device(w, instances, record)
    inp = H.Inputs(w)
    worst = H.compare_sampled(w, inp, instances, outs, states, record)
    print(f"worst |out - oracle| = {worst:.3e}")
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
