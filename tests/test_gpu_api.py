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
    exe = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c_abi", "abi_gpu_check")
    assert os.path.exists(exe), "build it first: __graft_entry__.build()"
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "C ABI GPU run passed" in r.stdout
