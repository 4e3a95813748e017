"""Recovery stress at the LLaMA-3-8B shape: batch 1, context 131072, spill mode.

A planted low-relevance key (a cold token of the heavy-hitter recipe at a
seeded position in the first half of the prompt) is frozen, released to the
host store and restored on its timer for 2000 steps.  At the first step t_s
>= 2001 that leaves it frozen with more than one step to go, the queries turn
to it (cosine 0.9) and the logits go flat, so the entropy trigger fires: Soft
Reset at the end of t_s must bring its rows back from the host store, and at
t_s + 1 the attention output must be its value row.

What is checked, at a size the oracle cannot step through 2000 times:
  * before t_s, the states of every position at sampled steps, bit for bit,
    against the closed form that the heavy-hitter recipe implies: cold tokens
    are flagged at every step they attend once outside the window, hot ones
    never (bounds proved by ``synth.gen.hh_relevance_bounds``), so every cold
    token follows the oracle's single-token trajectory shifted to the step it
    leaves the window;
  * the attention outputs at those steps against the oracle's attention over
    that active set;
  * from t_s - 1 on, the oracle stepped from that state: states and outputs
    at every step, the entropy level, the residency of every position.
"""

import numpy as np
import pytest

import oracle
from synth import gen
from tests import _harness as H
from tests._closed_form import ClosedForm, base_trajectory

pytestmark = pytest.mark.gpu

SWITCH_AFTER = 2000
TAIL = 16


@pytest.fixture(scope="module", autouse=True)
def gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2512_11221_amd as A
    A.load()
    return torch


def _oracle_out(q, K, V, A):
    Kh = np.ascontiguousarray(K[A].transpose(1, 0, 2), dtype=np.float64)
    Vh = np.ascontiguousarray(V[A].transpose(1, 0, 2), dtype=np.float64)
    return oracle.attend_rows(q.astype(np.float64), Kh, Vh)[0]


def _check_out(g, ref, where):
    err = np.abs(g.astype(np.float64) - ref)
    assert err.max() <= H.ATOL, (where, float(err.max()))
    rel = np.linalg.norm(g - ref) / max(np.linalg.norm(ref), 1e-30)
    assert rel <= H.RTOL_NORM, (where, rel)


def _check_state(g, res, t, count, frozen, timer, active):
    n = len(frozen)
    assert g["n"] == n, t
    np.testing.assert_array_equal(g["count"], count, err_msg=f"counts, step {t}")
    np.testing.assert_array_equal(g["frozen"], frozen, err_msg=f"frozen, step {t}")
    np.testing.assert_array_equal(g["unfreeze"][frozen] - (t + 1), timer[frozen],
                                  err_msg=f"remaining timers, step {t}")
    np.testing.assert_array_equal(g["active"], active, err_msg=f"active list, step {t}")
    # spill_min_D = 2 and a freeze of 1 step is a no-op: host-only == frozen
    np.testing.assert_array_equal(res["device_row"] < 0, frozen, err_msg=f"host-only, step {t}")
    assert not (frozen & ~res["on_host"]).any(), t


def test_recovery_stress_ctx131k():
    import torch
    import paper_2512_11221_amd as A
    from synth.device import DeviceGen

    w0 = gen.recovery_stress()
    P, Kw = w0.prefill[0], w0.window_K
    s_cold, s_hot = gen.hh_relevance_bounds(w0)
    assert s_cold < w0.tau - H.MARGIN and s_hot > w0.tau + H.MARGIN

    base = base_trajectory(w0.k_soft, SWITCH_AFTER + 200)
    c_b, f_b, r_b = base
    p_star = gen.plant_position(w0)
    # first step >= 2001 after which the planted token is frozen with remaining > 1
    t_s = next(t for t in range(SWITCH_AFTER + 1, len(f_b)) if f_b[t] and r_b[t] > 1)
    S = t_s + TAIL
    w = w0.replace(steps=S, flat_logit_steps=(t_s,), max_ctx=P + S)
    print(f"planted position {p_star}, switch step {t_s}, steps {S}", flush=True)

    K, V = gen.kv_rows(w, 0, 0, 0, P + S)
    hot = gen.hh_mask(w, 0, 0, 0, P + S)
    assert not hot[p_star]
    cf = ClosedForm(w, hot, base)
    Qp = gen.planted_q_rows(w, K[p_star], t_s, S + 1)          # steps t_s .. S
    ent = [oracle.entropy(gen.logits_row(w, 0, t)) for t in range(1, S + 1)]
    levels, _ = oracle.recovery_schedule(ent, w.entropy_spike, w.conf_drop)
    assert [t for t, lv in enumerate(levels, 1) if lv] == [t_s]
    assert min(abs(h - w.entropy_spike) for h, _ in ent) >= 1e-2

    sample = sorted({1, 16, 17, 18, 19, 500, 1000, t_s - 1})
    record = set(sample) | set(range(t_s - 1, S + 1))

    # ---- GPU run, inputs generated on the device (queries from t_s uploaded)
    tdt = torch.bfloat16
    Hq, Hkv, D = w.n_q_heads, w.n_kv_heads, w.head_dim
    cfg = A.make_config(1, 1, Hq, Hkv, D, w.max_ctx, Kw, w.tau, w.k_soft, w.vocab,
                        entropy_spike=w.entropy_spike, conf_drop=w.conf_drop,
                        wr_last_N=w.wr_last_N, dtype=w.dtype, spill_min_D=w.spill_min_D)
    ctx = A.asrkf_init(cfg)
    gst, gout, glevel = {}, {}, []
    try:
        dg = DeviceGen(w)
        sk = torch.empty(P * Hkv * D, dtype=tdt, device="cuda")
        sv = torch.empty_like(sk)
        dg.kv_rows(0, 0, 0, P, sk, sv)
        A.asrkf_prefill(ctx, 0, 0, sk, sv, P)
        Q = torch.empty((S, 1, 1, Hq, D), dtype=tdt, device="cuda")
        Kn = torch.empty((S, 1, 1, Hkv, D), dtype=tdt, device="cuda")
        Vn = torch.empty_like(Kn)
        LG = torch.empty((S, 1, w.vocab), dtype=torch.float32, device="cuda")
        dg.q(1, S, Q)
        Q[t_s - 1:, 0, 0] = torch.from_numpy(Qp).to(tdt).cuda()
        dg.new_kv(1, S, Kn, Vn)
        dg.logits(1, S, LG)
        out = torch.empty((1, Hq, D), dtype=torch.float32, device="cuda")
        torch.cuda.synchronize()
        del sk, sv
        for t in range(1, S + 1):
            A.asrkf_decode_step(ctx, 0, Q[t - 1, 0], Kn[t - 1, 0], Vn[t - 1, 0], out)
            A.asrkf_restore(ctx, LG[t - 1], A.AUTO)
            glevel.append(A.asrkf_get_seq(ctx, 0)["level"])
            if t in record:
                st = A.asrkf_get_state(ctx, 0, 0, w.max_ctx)
                st["res"] = A.asrkf_get_residency(ctx, 0, 0, w.max_ctx)
                gst[t] = st
                gout[t] = out[0].cpu().numpy()
            if t % 500 == 0:
                print(f"step {t}", flush=True)
        stats = A.asrkf_stats(ctx)
    finally:
        A.asrkf_destroy(ctx)
    assert glevel == levels
    print(f"rows to host {stats['rows_to_host']}, restored from the host {stats['rows_from_host']}, "
          f"taken back intact {stats['rows_reused']}", flush=True)

    # ---- before the switch: closed-form states, oracle attention over them
    def q_of(t):
        return gen.q_row(w, 0, 0, t) if t < t_s else Qp[t - t_s]

    for t in sample:
        cnt, fz, tm = cf.state(t)
        act_next = np.concatenate([np.nonzero(~fz)[0], [P + t]])
        _check_state(gst[t], gst[t]["res"], t, cnt, fz, tm, act_next)
        _check_out(gout[t], _oracle_out(q_of(t), K, V, cf.active(t)), t)
    cnt, fz, tm = cf.state(t_s - 1)
    assert fz[p_star] and tm[p_star] >= 2          # frozen, on the host, 2+ steps to go

    # ---- from t_s - 1 on: the oracle stepped from that state
    n = P + t_s - 1
    inst = oracle.Instance(K[:n], V[:n], Kw, w.tau, w.k_soft, capacity=P + S + 1)
    inst.count[:n], inst.frozen[:n], inst.timer[:n] = cnt, fz, tm
    inst.t = t_s - 1
    for t in range(t_s, S + 1):
        rec = inst.step(q_of(t), K[P + t - 1], V[P + t - 1])
        if levels[t - 1]:
            inst.recover(levels[t - 1], w.wr_last_N)
        timer, count, frozen = inst.state()
        act_next = np.concatenate([np.nonzero(~frozen)[0], [inst.n]])
        _check_state(gst[t], gst[t]["res"], t, count, frozen, timer, act_next)
        _check_out(gout[t], rec.out, t)
        if t == t_s + 1:
            assert p_star in rec.active
            v_star = V[p_star][np.arange(Hq) // w.group]
            assert np.abs(gout[t] - v_star).max() < 0.05
    assert gst[t_s]["res"]["device_row"][p_star] >= 0     # restored from the host store
    assert stats["rows_from_host"] + stats["rows_reused"] > 0 and stats["rows_to_host"] > 0
