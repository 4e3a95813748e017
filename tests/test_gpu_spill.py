"""GPU parity in spill mode (frozen KV leaves the device; Sec. 3.2).

The same oracle comparison as the resident-mode tests (states bit for bit,
outputs within the acceptance bound), plus the residency of every position
after every step: a position is held only in the host store exactly while it
is frozen by a freeze of at least spill_min_D steps; the host store holds
every position that was ever released; resident positions own distinct
device rows.  Every restore either takes the token's last device row back
(no other position was written into it since) or copies its rows back from
the host store; outputs that match the oracle after restores show that the
rows came back intact either way.
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
    A.load()
    return torch


def _spill_parity(w, inp, modes=None, with_logits=True, side_delay_us=0):
    instances = [(l, b) for l in range(w.n_layers) for b in range(w.batch)]
    g, mon, stats = H.run_gpu(w, inp, instances, modes, with_logits, side_delay_us=side_delay_us)
    o = H.run_oracle(w, inp, instances, modes, with_logits)
    restores = 0
    for key in instances:
        H.compare_instance(g[key], o[key])
        restores += H.compare_residency(w, g[key], o[key])
    last = stats[-1]
    released = sum(int(np.count_nonzero(g[k][-1]["on_host"])) for k in instances)
    assert last["rows_to_host"] == released           # each token copied out once
    assert last["rows_from_host"] + last["rows_reused"] == restores
    print(f"{w.name}: rows to host {last['rows_to_host']}, restores {restores}, "
          f"releases {last['rows_released']}")
    return g, o, mon, stats


def _flag_all(**kw):
    args = dict(name="spill-flag-all", seed=gen.SEED + 51, n_layers=1, batch=1, n_q_heads=8,
                n_kv_heads=2, head_dim=64, dtype="f32", prefill=[512], steps=64, window_K=32,
                tau=math.inf, k_soft=2.0, vocab=64, logit_sigma=1.0, recipe="gauss",
                spill_min_D=2)
    args.update(kw)
    return gen.Workload(**args)


def test_flag_all_spills_and_restores():
    """Every out-of-window token is flagged each step: the lockstep cohort is
    released and restored again and again."""
    w = _flag_all()
    g, o, _, stats = _spill_parity(w, H.Inputs(w))
    assert stats[-1]["rows_from_host"] + stats[-1]["rows_reused"] > 1000
    assert stats[-1]["rows_released"] > stats[-1]["rows_to_host"]   # rows re-released, not re-copied
    # a row for every position: only new tokens take free rows, so no released
    # row is written over and every restore takes its row back without a copy
    assert stats[-1]["rows_from_host"] == 0


def test_flag_all_tight_rows_copy_and_reuse():
    """The same cohort with just enough device rows: new tokens and restores
    take rows that released tokens left, so some restores copy from the host
    store while others still find their rows intact."""
    w = _flag_all()
    peak = _resident_peak(w, H.Inputs(w))
    assert peak < w.max_ctx, peak
    w = w.replace(device_rows=peak)
    g, o, _, stats = _spill_parity(w, H.Inputs(w))
    assert stats[-1]["rows_from_host"] > 0 and stats[-1]["rows_reused"] > 0


@pytest.mark.parametrize("shape", [
    dict(n_q_heads=32, n_kv_heads=32, head_dim=128, dtype="bf16"),   # four waves share a token
    dict(n_q_heads=64, n_kv_heads=8, head_dim=128, dtype="bf16"),    # G = 8 split in halves
])
def test_flag_all_spill_wide_layouts(shape):
    """Spill mode with the head layouts in which several waves share each token:
    released and restored rows are read through the device-row list."""
    w = _flag_all(name="spill-wide", prefill=[300], steps=40, **shape)
    w = w.replace(device_rows=_resident_peak(w, H.Inputs(w)))
    g, o, _, stats = _spill_parity(w, H.Inputs(w))
    assert stats[-1]["rows_from_host"] > 0
    assert stats[-1]["rows_from_host"] + stats[-1]["rows_reused"] > 100


def _resident_peak(w, inp):
    """Largest number of device rows the run needs: after each step, the
    positions not held only on the host, plus the next token (oracle states)."""
    o = H.run_oracle(w, inp, [(0, 0)])[(0, 0)]
    peak = w.prefill[0] + 1
    for r in o:
        d = np.array([H.oracle.freeze_duration(int(c), w.k_soft) for c in r["count"]])
        host_only = r["frozen"] & (d >= w.spill_min_D)
        peak = max(peak, len(r["frozen"]) - int(host_only.sum()) + 1)
    return peak


def _gauss_spill(**kw):
    w0 = gen.tiny()
    w = gen.tiny(tau=H.score_quantile(w0, 0.6), spill_min_D=2, **kw)
    return w, H.fix_margin(w)


def test_tight_device_rows_reuse_rows():
    """Exactly as many device rows as the run needs at its peak: rows pass
    from released tokens to restored and new ones."""
    w, att = _gauss_spill()
    peak = _resident_peak(w, H.Inputs(w, att))
    assert peak < w.max_ctx, peak              # fewer rows than positions
    w = w.replace(device_rows=peak)
    _spill_parity(w, H.Inputs(w, att))


def test_too_few_device_rows_is_reported():
    import paper_2512_11221_amd as A
    w, att = _gauss_spill()
    peak = _resident_peak(w, H.Inputs(w, att))
    w = w.replace(device_rows=peak - 1)
    with pytest.raises(A.AsrkfError) as e:
        H.run_gpu(w, H.Inputs(w, att), [(0, 0)])
    assert e.value.code == A._lib.ECAPACITY


@pytest.mark.parametrize("spill_min_D", [2, 3])
def test_gaussian_freezing_with_recovery(spill_min_D):
    flat = (40, 50, 51, 60, 61, 62)
    w0 = gen.tiny()
    tau = H.score_quantile(w0, 0.6)
    w = gen.tiny(tau=tau, entropy_spike=6.5, flat_logit_steps=flat, spill_min_D=spill_min_D)
    inp = H.Inputs(w, H.fix_margin(w))
    g, o, mon, stats = _spill_parity(w, inp)
    assert stats[-1]["recoveries"][1:] == [3, 2, 1]


def test_restores_wait_for_a_delayed_side_stream():
    """The side stream that carries the row copies first idles 3 ms every step
    (a test hook), far longer than a step's attention.  Results must not change:
    the next step's attention waits on the copies' events, and the append into
    a reused row waits for that row's copy to the host."""
    import paper_2512_11221_amd as A
    w0 = gen.tiny()
    w = gen.tiny(tau=H.score_quantile(w0, 0.6), spill_min_D=2)
    att = H.fix_margin(w)
    modes = {20: A.SR, 33: A.WR, 47: A.FR}
    # just enough device rows, so that rows change hands and restores copy
    o = H.run_oracle(w, H.Inputs(w, att), [(0, 0)], modes, with_logits=False)[(0, 0)]
    peak = w.prefill[0] + 1
    for r in o:
        d = np.array([H.oracle.freeze_duration(int(c), w.k_soft) for c in r["count"]])
        peak = max(peak, len(r["frozen"]) - int((r["frozen"] & (d >= w.spill_min_D)).sum()) + 1)
    w = w.replace(device_rows=peak)
    g, o, mon, stats = _spill_parity(w, H.Inputs(w, att), modes=modes,
                                     with_logits=False, side_delay_us=3000)
    assert stats[-1]["rows_from_host"] > 0


def test_forced_recovery_modes():
    import paper_2512_11221_amd as A
    w0 = gen.tiny()
    w = gen.tiny(tau=H.score_quantile(w0, 0.6), spill_min_D=2)
    inp = H.Inputs(w, H.fix_margin(w))
    _spill_parity(w, inp, modes={20: A.SR, 33: A.WR, 47: A.FR, 55: A.SR}, with_logits=False)


def test_heavy_hitters_multilayer_ragged():
    w = gen.Workload(name="spill-hh-ragged", seed=gen.SEED + 53, n_layers=2, batch=3,
                     n_q_heads=32, n_kv_heads=8, head_dim=128, dtype="bf16",
                     prefill=[2049, 1, 700], steps=48, window_K=32, tau=0.5, k_soft=2.0,
                     vocab=128256, logit_sigma=3.0, recipe="hh", f_hh=[0.35, 0.3, 0.2],
                     spill_min_D=2)
    _spill_parity(w, H.Inputs(w))


def test_llama8b_one_layer_spill():
    w = gen.llama8b_1layer(spill_min_D=2)
    g, o, mon, stats = _spill_parity(w, H.Inputs(w))
    assert stats[-1]["rows_to_host"] > 1000


def test_too_few_device_rows_long_instance():
    """A long instance (rebuilt in segments) that outgrows its device rows."""
    import paper_2512_11221_amd as A
    w = gen.llama8b_1layer(spill_min_D=2, steps=24, device_rows=8192 + 6)
    with pytest.raises(A.AsrkfError) as e:
        H.run_gpu(w, H.Inputs(w), [(0, 0)], record=lambda t: t % 4 == 0)
    assert e.value.code == A._lib.ECAPACITY


def test_tight_device_rows_long_instance():
    """Device rows just enough for the largest resident set of a long instance."""
    w = gen.llama8b_1layer(spill_min_D=2, steps=40)
    peak = _resident_peak(w, H.Inputs(w))
    assert peak < w.max_ctx, peak
    _spill_parity(w.replace(device_rows=peak), H.Inputs(w))


def test_candidates_inside_window_spill():
    """Freeze candidates inside the window with k = 0.5: a token can freeze for
    two steps in the step that appends it, so rows written by that step's
    attention leave for the host store in the same step and come back."""
    w = _flag_all(name="spill-inside", candidates="inside", k_soft=0.5, window_K=48,
                  prefill=[200], steps=48)
    g, o, _, stats = _spill_parity(w, H.Inputs(w))
    assert stats[-1]["rows_from_host"] + stats[-1]["rows_reused"] > 100
    first = [r for r in o[(0, 0)] if r["t"] == 1][0]
    assert first["frozen"][-1]                 # the token appended at step 1 is frozen at once
