"""The device twin of the input generator writes the host generator's bits."""
import numpy as np
import pytest

from synth import gen

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _host_bits(x, dtype):
    x = np.ascontiguousarray(x, dtype=np.float32)
    return gen.bf16_bits(x).view(np.int16) if dtype == "bf16" else x.view(np.int32)


def _dev_bits(t, dtype):
    import torch
    return t.view(torch.int16 if dtype == "bf16" else torch.int32).cpu().numpy()


@pytest.mark.parametrize("w", [
    gen.llama8b_32layer(),
    gen.ragged(batch=5),
    gen.tiny(flat_logit_steps=(3, 5)),
    gen.Workload(name="g", seed=7, n_layers=2, batch=2, n_q_heads=32, n_kv_heads=8,
                 head_dim=128, dtype="bf16", prefill=[50, 9], steps=6, window_K=4, tau=0.5,
                 k_soft=2.0, vocab=333, logit_sigma=2.0, recipe="gauss"),
], ids=lambda w: w.name)
def test_device_generator_is_bit_identical(torch, w):
    from synth.device import DeviceGen
    dg = DeviceGen(w)
    tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    Hkv, Hq, D = w.n_kv_heads, w.n_q_heads, w.head_dim
    L, B = w.n_layers, w.batch
    for (l, b) in {(0, 0), (L - 1, B - 1), (L // 2, B // 2)}:
        p0, p1 = 3, min(w.prefill[b], 700)
        K = torch.empty((p1 - p0) * Hkv * D, dtype=tdt, device="cuda")
        V = torch.empty_like(K)
        dg.kv_rows(l, b, p0, p1, K, V)
        Kh, Vh = gen.kv_rows(w, l, b, p0, p1)
        np.testing.assert_array_equal(_dev_bits(K, w.dtype), _host_bits(Kh, w.dtype).reshape(-1))
        np.testing.assert_array_equal(_dev_bits(V, w.dtype), _host_bits(Vh, w.dtype).reshape(-1))
    t0, steps = 2, 3
    Q = torch.empty((steps, L, B, Hq, D), dtype=tdt, device="cuda")
    Kn = torch.empty((steps, L, B, Hkv, D), dtype=tdt, device="cuda")
    Vn = torch.empty_like(Kn)
    lg = torch.empty((steps, B, w.vocab), dtype=torch.float32, device="cuda")
    dg.q(t0, steps, Q)
    dg.new_kv(t0, steps, Kn, Vn)
    dg.logits(t0, steps, lg)
    Qd, Knd, Vnd, lgd = (_dev_bits(Q, w.dtype), _dev_bits(Kn, w.dtype), _dev_bits(Vn, w.dtype),
                         lg.cpu().numpy())
    for s in range(steps):
        t = t0 + s
        for (l, b) in {(0, 0), (L - 1, B - 1)}:
            np.testing.assert_array_equal(Qd[s, l, b], _host_bits(gen.q_row(w, l, b, t), w.dtype))
            p = w.prefill[b] + t - 1
            Kh, Vh = gen.kv_rows(w, l, b, p, p + 1)
            np.testing.assert_array_equal(Knd[s, l, b], _host_bits(Kh[0], w.dtype))
            np.testing.assert_array_equal(Vnd[s, l, b], _host_bits(Vh[0], w.dtype))
        for b in range(B):
            np.testing.assert_array_equal(lgd[s, b], gen.logits_row(w, b, t))
