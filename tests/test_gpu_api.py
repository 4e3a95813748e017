"""Behaviour of the C ABI on the GPU: call order, capacity, argument checks,
sequences without a prompt, and the statistics it reports."""
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


def _ctx(L=2, B=2, max_ctx=64, **kw):
    import paper_2512_11221_amd as A
    cfg = A.make_config(L, B, 8, 2, 64, max_ctx, 4, 0.5, 2.0, 32, dtype="f32", **kw)
    return A, A.asrkf_init(cfg)


def _io(B=2):
    import torch
    q = torch.zeros((B, 8, 64), device="cuda")
    k = torch.zeros((B, 2, 64), device="cuda")
    out = torch.empty((B, 8, 64), device="cuda")
    return q, k, k.clone(), out


def _code(fn):
    import paper_2512_11221_amd as A
    with pytest.raises(A.AsrkfError) as e:
        fn()
    return e.value.code


def test_layers_out_of_order_and_early_restore():
    A, ctx = _ctx()
    try:
        q, k, v, out = _io()
        assert _code(lambda: A.asrkf_decode_step(ctx, 1, q, k, v, out)) == A._lib.ESTATE
        A.asrkf_decode_step(ctx, 0, q, k, v, out)
        assert _code(lambda: A.asrkf_restore(ctx, None, A.NONE)) == A._lib.ESTATE
        A.asrkf_decode_step(ctx, 1, q, k, v, out)
        assert _code(lambda: A.asrkf_decode_step(ctx, 1, q, k, v, out)) == A._lib.ESTATE
        A.asrkf_restore(ctx, None, A.NONE)
        # prefill is only allowed before the first step
        assert _code(lambda: A.asrkf_prefill(ctx, 0, 0, k, v, 1)) == A._lib.ESTATE
        assert A.asrkf_stats(ctx)["step"] == 1
    finally:
        A.asrkf_destroy(ctx)


def test_capacity_is_reported_before_any_work():
    import torch
    A, ctx = _ctx(L=1, B=1, max_ctx=8)
    try:
        q, k, v, out = _io(1)
        kp = torch.zeros((5, 2, 64), device="cuda")
        A.asrkf_prefill(ctx, 0, 0, kp, kp, 5)
        for _ in range(3):                       # positions 5, 6, 7 fill max_ctx = 8
            A.asrkf_decode_step(ctx, 0, q, k, v, out)
            A.asrkf_restore(ctx, None, A.NONE)
        assert _code(lambda: A.asrkf_decode_step(ctx, 0, q, k, v, out)) == A._lib.ECAPACITY
        st = A.asrkf_stats(ctx)                  # the context is still usable for queries
        assert st["step"] == 3 and st["total_positions"] == 8
    finally:
        A.asrkf_destroy(ctx)


def test_argument_checks():
    import torch
    A, ctx = _ctx()
    try:
        q, k, v, out = _io()
        assert _code(lambda: A.asrkf_decode_step(ctx, 0, None, k, v, out)) == A._lib.EINVAL
        odd = torch.zeros(2 * 8 * 64 + 1, device="cuda")[1:]          # 4-byte offset
        assert _code(lambda: A.asrkf_decode_step(ctx, 0, odd, k, v, out)) == A._lib.EINVAL
        assert _code(lambda: A.asrkf_prefill(ctx, 2, 0, k, v, 1)) == A._lib.EINVAL
        assert _code(lambda: A.asrkf_prefill(ctx, 0, 0, k, v, 64)) == A._lib.EINVAL
        A.asrkf_prefill(ctx, 0, 0, k, v, 1)
        assert _code(lambda: A.asrkf_prefill(ctx, 1, 0, k, v, 2)) == A._lib.EINVAL  # length mismatch
        assert _code(lambda: A.asrkf_restore(ctx, None, 9)) == A._lib.EINVAL
        assert _code(lambda: A.asrkf_get_state(ctx, 0, 5, 64)) == A._lib.EINVAL
    finally:
        A.asrkf_destroy(ctx)


def test_sequence_without_prompt_and_stats():
    """Sequence 1 is never prefilled: its first step attends only its own
    token.  The statistics count every (layer, sequence) position."""
    w = gen.Workload(name="noprompt", seed=gen.SEED + 71, n_layers=2, batch=2, n_q_heads=8,
                     n_kv_heads=2, head_dim=64, dtype="f32", prefill=[40, 0], steps=30,
                     window_K=4, tau=math.inf, k_soft=1.0, vocab=64, logit_sigma=1.0,
                     recipe="gauss")
    inp = H.Inputs(w)
    inst = [(l, b) for l in range(2) for b in range(2)]
    g, _, stats = H.run_gpu(w, inp, inst, with_logits=False)
    o = H.run_oracle(w, inp, inst, with_logits=False)
    for key in inst:
        H.compare_instance(g[key], o[key])
    last = stats[-1]
    n_total = sum(len(o[key][-1]["frozen"]) for key in inst)
    n_active = sum(int((~o[key][-1]["frozen"]).sum()) for key in inst)
    assert last["total_positions"] == n_total
    assert last["active_positions"] == n_active
    assert abs(last["compression"] - (1 - n_active / n_total)) < 1e-12
    attended = sum(len(r["attended"]) for key in inst for r in o[key])
    assert last["attended_total"] == attended


def test_c_program_drives_the_gpu():
    """tests/c_abi/abi_gpu_check.c: a C program with HIP device buffers and no
    Python runs 12 dense steps through the ABI and checks every output against
    its own double-precision attention, plus the statistics."""
    import os
    import subprocess
    here = os.path.dirname(os.path.abspath(__file__))
    exe = os.path.join(here, "c_abi", "abi_gpu_check")
    assert os.path.exists(exe), "build it first: __graft_entry__.build()"
    for src in (os.path.join(here, "c_abi", "abi_gpu_check.c"),
                os.path.join(here, "..", "include", "asrkf.h")):
        # a program built against an older header would pass a struct of the old layout
        assert os.path.getmtime(exe) >= os.path.getmtime(src), \
            f"{exe} is older than {src}: rebuild it with __graft_entry__.build()"
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "C ABI GPU run passed" in r.stdout


def _tiny_freezing(seed_shift=0, **kw):
    w0 = gen.tiny(seed=gen.SEED + 1 + seed_shift)
    w = gen.tiny(seed=gen.SEED + 1 + seed_shift, tau=H.score_quantile(w0, 0.6), **kw)
    return w, H.Inputs(w, H.fix_margin(w))


def test_non_default_stream_gives_the_same_results():
    """Every call queued on a stream of the caller's (torch's current stream
    inside the context manager) gives bitwise the results of the default
    stream."""
    import torch
    w, inp = _tiny_freezing()
    a, _, _ = H.run_gpu(w, inp, [(0, 0)])
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        b, _, _ = H.run_gpu(w, inp, [(0, 0)])
    torch.cuda.synchronize()
    for x, y in zip(a[(0, 0)], b[(0, 0)]):
        np.testing.assert_array_equal(x["out"], y["out"])
        np.testing.assert_array_equal(x["active"], y["active"])


def test_two_contexts_interleaved():
    """Two contexts with different inputs, stepped alternately, each give
    bitwise the outputs of a run alone: the library keeps no state outside a
    context."""
    import torch
    import paper_2512_11221_amd as A
    runs = [_tiny_freezing(0), _tiny_freezing(7)]
    alone = [H.run_gpu(w, inp, [(0, 0)])[0][(0, 0)] for w, inp in runs]
    ctxs = []
    try:
        for w, inp in runs:
            cfg = A.make_config(w.n_layers, w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim,
                                w.max_ctx, w.window_K, w.tau, w.k_soft, w.vocab,
                                entropy_spike=w.entropy_spike, conf_drop=w.conf_drop,
                                wr_last_N=w.wr_last_N, dtype=w.dtype)
            ctx = A.asrkf_init(cfg)
            ctxs.append(ctx)
            K, V = inp.prompt(0, 0)
            A.asrkf_prefill(ctx, 0, 0, H._dev(K, w.dtype), H._dev(V, w.dtype), len(K))
        torch.cuda.synchronize()
        outs = [[], []]
        for t in range(1, runs[0][0].steps + 1):
            for i, (w, inp) in enumerate(runs):
                q = H._dev(inp.q(0, 0, t)[None], w.dtype)
                kn, vn = inp.new_token(0, 0, t)
                out = torch.empty((1, w.n_q_heads, w.head_dim), dtype=torch.float32, device="cuda")
                A.asrkf_decode_step(ctxs[i], 0, q, H._dev(kn[None], w.dtype), H._dev(vn[None], w.dtype), out)
                A.asrkf_restore(ctxs[i], H._dev(inp.logits(0, t)[None], "f32"), A.AUTO)
                torch.cuda.synchronize()
                outs[i].append(out.cpu().numpy()[0])
        for i in range(2):
            for rec, o in zip(alone[i], outs[i]):
                np.testing.assert_array_equal(rec["out"], o)
    finally:
        for ctx in ctxs:
            A.asrkf_destroy(ctx)


def test_attention_timing_per_launch():
    """With timing on, every attention launch records its execution time:
    the series has one positive value per (step, layer), in launch order,
    sums to the reported total, and a stats reset clears it."""
    A, ctx = _ctx(L=2, B=2, max_ctx=64)
    try:
        q, k, v, out = _io()
        A.asrkf_decode_step(ctx, 0, q, k, v, out)      # untimed step
        A.asrkf_decode_step(ctx, 1, q, k, v, out)
        A.asrkf_restore(ctx, None, A.NONE)
        A.asrkf_set_timing(ctx, True)
        for _ in range(3):
            for l in range(2):
                A.asrkf_decode_step(ctx, l, q, k, v, out)
            A.asrkf_restore(ctx, None, A.NONE)
        ms = A.asrkf_timing_series(ctx)
        st = A.asrkf_stats(ctx)
        assert len(ms) == 6 == st["attn_launches"]
        assert (ms > 0).all() and (ms < 1e3).all()
        assert abs(float(ms.astype(np.float64).sum()) - st["attn_kernel_ms"]) <= 1e-6 * max(1.0, st["attn_kernel_ms"])
        A.asrkf_set_timing(ctx, False)
        A.asrkf_decode_step(ctx, 0, q, k, v, out)
        A.asrkf_decode_step(ctx, 1, q, k, v, out)
        A.asrkf_restore(ctx, None, A.NONE)
        assert len(A.asrkf_timing_series(ctx)) == 6
        A.asrkf_stats_reset(ctx)
        assert len(A.asrkf_timing_series(ctx)) == 0
        assert A.asrkf_stats(ctx)["attn_launches"] == 0
    finally:
        A.asrkf_destroy(ctx)


def _config_of(A, w):
    return A.make_config(w.n_layers, w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.max_ctx,
                         w.window_K, w.tau, w.k_soft, w.vocab, entropy_spike=w.entropy_spike,
                         conf_drop=w.conf_drop, wr_last_N=w.wr_last_N, dtype=w.dtype,
                         spill_min_D=w.spill_min_D, device_rows=w.device_rows,
                         history_W=w.history_W, relevance=w.relevance, scope=w.scope,
                         candidates=w.candidates)


@pytest.mark.parametrize("spill", [False, True], ids=["resident", "spill"])
def test_reset_context_runs_like_a_fresh_one(spill):
    """A context that ran another batch (other prompts and lengths, recoveries)
    and was reset runs a workload bit for bit like a fresh context: outputs,
    token states, monitor and counters at every step."""
    import paper_2512_11221_amd as A
    w = gen.Workload(name="reset-hh", seed=gen.SEED + 97, n_layers=2, batch=2, n_q_heads=32,
                     n_kv_heads=8, head_dim=128, dtype="bf16", prefill=[300, 170], steps=24,
                     window_K=16, tau=0.5, k_soft=2.0, vocab=1024, logit_sigma=2.0, recipe="hh",
                     f_hh=[0.35, 0.25], entropy_spike=6.5, flat_logit_steps=(12, 13),
                     spill_min_D=2 if spill else 0)
    s_cold, s_hot = gen.hh_relevance_bounds(w)
    assert s_cold < w.tau - H.MARGIN and s_hot > w.tau + H.MARGIN
    other = w.replace(name="reset-other", seed=gen.SEED + 98, prefill=[120, 250],
                      max_ctx=w.max_ctx, flat_logit_steps=(5, 6, 7))
    inst = [(l, b) for l in range(2) for b in range(2)]
    fresh, mon_f, st_f = H.run_gpu(w, H.Inputs(w), inst)
    ctx = A.asrkf_init(_config_of(A, w))
    try:
        H.run_gpu(other, H.Inputs(other), inst, steps=18, ctx=ctx)
        A.asrkf_set_timing(ctx, True)
        A.asrkf_reset(ctx)
        st0 = A.asrkf_stats(ctx)
        assert st0["step"] == 0 and st0["attended_total"] == 0 and st0["attn_launches"] == 0
        assert st0["recoveries"] == [0, 0, 0, 0] and st0["rr_requests"] == 0
        again, mon_a, st_a = H.run_gpu(w, H.Inputs(w), inst, ctx=ctx)
        assert A.asrkf_stats(ctx)["attn_launches"] == 0          # reset turned timing off
    finally:
        A.asrkf_destroy(ctx)
    for key in inst:
        assert len(fresh[key]) == len(again[key]) == w.steps
        for a, b in zip(fresh[key], again[key]):
            for f in ("out", "unfreeze", "count", "frozen", "active"):
                np.testing.assert_array_equal(a[f], b[f], err_msg=f"{key} step {a['t']} {f}")
    assert mon_f == mon_a
    for a, b in zip(st_f, st_a):
        for k in ("step", "attended_total", "active_positions", "total_positions", "recoveries",
                  "rr_requests", "rows_to_host", "rows_from_host", "rows_reused"):
            assert a[k] == b[k], (k, a[k], b[k])
    o = H.run_oracle(w, H.Inputs(w), inst)
    for key in inst:
        H.compare_instance(fresh[key], o[key])
