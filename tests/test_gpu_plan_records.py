"""First-tile records: after every list rebuild a small pass stages, for each
attention workgroup's range, its sequence, first list index, first chunk
length and first positions; the attention kernel compares the record with its
own split and, when they agree, requests its first K/V rows before the
chunk's positions and q have arrived.  The records are used with four or more
layers in resident mode, at the head layouts with one token per wave
iteration (8 KV heads, or 4 with 8 query heads each), while every attention
workgroup has a range: about 32 listed tokens per workgroup and layer, so
some 8k per layer on a 256-CU device.  These runs are sized for that; their
outputs and token states must match the oracle as everywhere else."""
import math

import pytest

from synth import gen
from tests import _harness as H

pytestmark = pytest.mark.gpu

# the benchmark's attention layout, four layers: the records are in use
L4 = dict(n_layers=4, n_q_heads=32, n_kv_heads=8, head_dim=128, dtype="bf16")


@pytest.fixture(scope="module", autouse=True)
def gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2512_11221_amd as A
    A.load()


def _parity(w, inp, modes=None):
    inst = [(l, b) for l in range(w.n_layers) for b in range(w.batch)]
    g, _, _ = H.run_gpu(w, inp, inst, modes)
    o = H.run_oracle(w, inp, inst, modes)
    worst = max(H.compare_instance(g[k], o[k]) for k in inst)
    print(f"{w.name}: worst |out - oracle| = {worst:.3e}")
    return g, o


@pytest.mark.parametrize("scope", ["layer", "token"])
@pytest.mark.parametrize("tau", [-math.inf, math.inf])
def test_ragged_sequences(tau, scope):
    """Five sequences: one without a prompt, one of 40 tokens, three of 3-4k.
    Ranges start among a sequence's cost tokens, straddle two sequences, or
    hold the appended token in their first tile (no record then).  Tau below
    every score keeps every step dense (records in use at every step); above
    every score every out-of-window token is flagged, and as the lists shrink
    some steps have too few tokens for the records and take the plain path."""
    w = gen.Workload(name=f"plan-ragged-{scope}", seed=gen.SEED + 101, batch=5,
                     prefill=[0, 2900, 3100, 40, 4200], steps=24, window_K=16, tau=tau,
                     k_soft=1.0, vocab=64, logit_sigma=1.0, recipe="gauss", scope=scope, **L4)
    _parity(w, H.Inputs(w))


def test_heavy_hitters_freezing():
    """The benchmark's recipe on four layers: heavy hitters attend, the rest
    freeze on Eq. 3's schedule, so the lists (and with them every range's
    first positions) change from step to step."""
    w = gen.Workload(name="plan-hh", seed=gen.SEED + 102, batch=3, prefill=[3000, 2600, 3400],
                     steps=40, window_K=32, tau=0.5, k_soft=2.0, vocab=128256, logit_sigma=3.0,
                     recipe="hh", f_hh=[0.35, 0.3, 0.2], **L4)
    s_cold, s_hot = gen.hh_relevance_bounds(w)
    assert s_cold < w.tau - H.MARGIN and s_hot > w.tau + H.MARGIN
    _parity(w, H.Inputs(w))


def test_forced_recovery():
    """SR, WR and FR forced between steps of heavy freezing: each recovery
    rebuilds long lists from short ones, and the records with them."""
    import paper_2512_11221_amd as A
    w = gen.Workload(name="plan-forced", seed=gen.SEED + 103, batch=3, prefill=[3300, 2700, 3100],
                     steps=36, window_K=16, tau=math.inf, k_soft=0.5, vocab=64, logit_sigma=1.0,
                     recipe="gauss", **L4)
    _parity(w, H.Inputs(w), modes={12: A.SR, 20: A.WR, 27: A.FR, 33: A.SR})


@pytest.mark.parametrize("tau", [-math.inf, math.inf])
def test_wide_query_groups(tau):
    """Four KV heads of eight query heads each: the other layout whose first
    tiles come from the records (half of a KV head's query heads per lane)."""
    w = gen.Workload(name="plan-g8", seed=gen.SEED + 104, n_layers=4, batch=3, n_q_heads=32,
                     n_kv_heads=4, head_dim=128, dtype="bf16", prefill=[2900, 3300, 2500],
                     steps=20, window_K=16, tau=tau, k_soft=1.0, vocab=64, logit_sigma=1.0,
                     recipe="gauss")
    _parity(w, H.Inputs(w))


@pytest.mark.parametrize("layout", [
    dict(n_q_heads=16, n_kv_heads=8, head_dim=128, dtype="f32"),    # 512 B head rows: 2 tokens per wave tile
    dict(n_q_heads=32, n_kv_heads=8, head_dim=64, dtype="bf16"),    # 128 B head rows
    dict(n_q_heads=16, n_kv_heads=8, head_dim=256, dtype="bf16"),   # 512 B head rows, G = 2
])
def test_other_row_sizes(layout):
    """The other row sizes with one token per wave iteration: the tile holds 2
    or 4 tokens per wave, so each wave takes a different part of the record."""
    w = gen.Workload(name="plan-rows", seed=gen.SEED + 105, n_layers=4, batch=3,
                     prefill=[3100, 2800, 3300], steps=12, window_K=16, tau=-math.inf, k_soft=1.0,
                     vocab=64, logit_sigma=1.0, recipe="gauss", **layout)
    _parity(w, H.Inputs(w))
