"""The seeded generator: determinism, rounding and the shapes it promises."""
import numpy as np
import pytest

from synth import gen


def test_rows_are_pure_functions_of_their_index():
    w = gen.llama8b_1layer()
    K1, V1 = gen.kv_rows(w, 0, 0, 0, 300)
    K2, V2 = gen.kv_rows(w, 0, 0, 100, 200)
    np.testing.assert_array_equal(K1[100:200], K2)
    np.testing.assert_array_equal(V1[100:200], V2)
    np.testing.assert_array_equal(gen.q_row(w, 0, 0, 7), gen.q_row(w, 0, 0, 7))
    assert not np.array_equal(gen.q_row(w, 0, 0, 7), gen.q_row(w, 0, 0, 8))


def test_bf16_rounding_matches_torch():
    torch = pytest.importorskip("torch")
    x = np.random.default_rng(0).standard_normal(100000).astype(np.float32) * 37.0
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(gen.bf16_bits(x), ref)


def test_gauss_stand_in_moments():
    z = gen.gauss(gen.draw(np.uint64(12345), np.arange(400000, dtype=np.uint64)))
    assert abs(z.mean()) < 0.01 and abs(z.std() - 1.0) < 0.01
    assert np.abs(z).max() <= gen.GAUSS_MAX


def test_heavy_hitter_bounds_hold_on_a_sample():
    w = gen.llama8b_1layer()
    s_cold, s_hot = gen.hh_relevance_bounds(w)
    assert s_cold < 0.499 and s_hot > 0.501
    K, _ = gen.kv_rows(w, 0, 0, 0, 4096)
    hh = gen.hh_mask(w, 0, 0, 0, 4096)
    G = w.group
    for t in (1, 100, 256):
        q = gen.q_row(w, 0, 0, t).astype(np.float64)
        x = np.einsum("hd,nhd->nh", q, K[:, np.arange(w.n_q_heads) // G, :].astype(np.float64))
        s = np.abs(x).mean(1)
        assert s[~hh].max() <= s_cold and s[hh].min() >= s_hot
    assert 0.3 < hh.mean() < 0.4


def test_ragged_workload_ranges():
    w = gen.ragged()
    assert len(w.prefill) == 64
    assert all(2048 <= p <= 32768 for p in w.prefill)
    assert all(0.2 <= f < 0.5 for f in w.f_hh)
