"""The allocation-free decode step (asrkf_decode_step_static) against
asrkf_decode_step: two contexts with the same configuration and inputs, one
stepped with each entry point, must give bitwise the same outputs and token
states.  Run twice in a row, the second time with a smaller input (fewer
sequences, shorter prompts), so the second run finds the first one's partials
in the static array.  A context whose split partials exceed the array is
refused with EINVAL before any work."""
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


def _cfg(A, w):
    return A.make_config(w.n_layers, w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.max_ctx,
                         w.window_K, w.tau, w.k_soft, w.vocab, entropy_spike=w.entropy_spike,
                         conf_drop=w.conf_drop, wr_last_N=w.wr_last_N, dtype=w.dtype)


def _lockstep(w):
    """Step a context through asrkf_decode_step and another through
    asrkf_decode_step_static on the same inputs; compare every step."""
    import torch
    import paper_2512_11221_amd as A
    inp = H.Inputs(w)
    ctxs = [A.asrkf_init(_cfg(A, w)), A.asrkf_init(_cfg(A, w))]
    steps = [A.asrkf_decode_step, A.asrkf_decode_step_static]
    try:
        for ctx in ctxs:
            for l in range(w.n_layers):
                for b in range(w.batch):
                    K, V = inp.prompt(l, b)
                    A.asrkf_prefill(ctx, l, b, H._dev(K, w.dtype), H._dev(V, w.dtype), len(K))
                    torch.cuda.synchronize()
        for t in range(1, w.steps + 1):
            outs = []
            for ctx, step in zip(ctxs, steps):
                out = torch.empty((w.n_layers, w.batch, w.n_q_heads, w.head_dim), device="cuda")
                keep = []
                for l in range(w.n_layers):
                    q = H._dev(np.stack([inp.q(l, b, t) for b in range(w.batch)]), w.dtype)
                    kn = H._dev(np.stack([inp.new_token(l, b, t)[0] for b in range(w.batch)]), w.dtype)
                    vn = H._dev(np.stack([inp.new_token(l, b, t)[1] for b in range(w.batch)]), w.dtype)
                    step(ctx, l, q, kn, vn, out[l])
                    keep += [q, kn, vn]
                lg = H._dev(np.stack([inp.logits(b, t) for b in range(w.batch)]), "f32")
                A.asrkf_restore(ctx, lg, A.AUTO)
                torch.cuda.synchronize()
                outs.append(out.cpu().numpy())
                del keep, lg
            np.testing.assert_array_equal(outs[0], outs[1], err_msg=f"outputs, step {t}")
            for l in range(w.n_layers):
                for b in range(w.batch):
                    sa = A.asrkf_get_state(ctxs[0], l, b, w.max_ctx)
                    sb = A.asrkf_get_state(ctxs[1], l, b, w.max_ctx)
                    for f in ("unfreeze", "count", "frozen", "active"):
                        np.testing.assert_array_equal(sa[f], sb[f], err_msg=f"{f}, step {t}")
        return outs[1]
    finally:
        for ctx in ctxs:
            A.asrkf_destroy(ctx)


def _hh(batch, prefill, steps):
    return gen.Workload(name="no-alloc", seed=gen.SEED + 97, n_layers=2, batch=batch,
                        n_q_heads=32, n_kv_heads=8, head_dim=128, dtype="bf16", prefill=prefill,
                        steps=steps, window_K=16, tau=0.5, k_soft=2.0, vocab=512,
                        logit_sigma=2.0, recipe="hh", f_hh=[0.35] * batch)


def test_static_scratch_matches_decode_step_twice():
    big = _hh(4, [900, 300, 650, 40], 20)
    small = _hh(2, [120, 77], 12)
    _lockstep(big)
    _lockstep(small)


def test_static_scratch_refuses_oversized_partials():
    """64 q heads of 256 at batch 1024 need (grid + 1024) * 64 * 258 * 4 bytes
    of partials, more than the 32 MiB array."""
    import torch
    import paper_2512_11221_amd as A
    from paper_2512_11221_amd import _lib as L
    cfg = A.make_config(1, 1024, 64, 8, 256, 8, 4, 0.5, 2.0, 16, dtype="bf16")
    ctx = A.asrkf_init(cfg)
    try:
        q = torch.zeros((1024, 64, 256), dtype=torch.bfloat16, device="cuda")
        k = torch.zeros((1024, 8, 256), dtype=torch.bfloat16, device="cuda")
        out = torch.empty((1024, 64, 256), device="cuda")
        with pytest.raises(A.AsrkfError) as e:
            A.asrkf_decode_step_static(ctx, 0, q, k, k, out)
        assert e.value.code == L.EINVAL and "static scratch" in str(e.value)
    finally:
        A.asrkf_destroy(ctx)
