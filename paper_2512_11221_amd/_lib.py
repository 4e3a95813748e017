"""ctypes binding of libasrkf.so: the C ABI of include/asrkf.h, same names.

Argument marshalling only.  Every step of the decode path runs in the HIP
kernels of the library; this module converts tensors to device pointers and
status codes to exceptions.  torch is used for device memory and streams.
"""
from __future__ import annotations

import ctypes
import math
import os

HERE = os.path.dirname(os.path.abspath(__file__))
# ASRKF_LIBRARY selects another build of the same library (a sanitizer build)
LIB_PATH = os.environ.get("ASRKF_LIBRARY") or os.path.join(HERE, "libasrkf.so")

OK, EINVAL, ENOMEM, EHIP, ESTATE, ECAPACITY = 0, -1, -2, -3, -4, -5
BF16, F32 = 0, 1
AUTO, SR, WR, FR, NONE = 0, 1, 2, 3, 4
REL_ABS, REL_SOFTMAX = 0, 1
SCOPE_LAYER, SCOPE_TOKEN = 0, 1
CAND_OUTSIDE, CAND_INSIDE = 0, 1
_STATUS = {EINVAL: "EINVAL", ENOMEM: "ENOMEM", EHIP: "EHIP", ESTATE: "ESTATE",
           ECAPACITY: "ECAPACITY"}


class asrkf_config(ctypes.Structure):
    _fields_ = [
        ("n_layers", ctypes.c_int32), ("batch", ctypes.c_int32),
        ("n_q_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32), ("max_ctx", ctypes.c_int32),
        ("window_K", ctypes.c_int32), ("tau", ctypes.c_float), ("k_soft", ctypes.c_float),
        ("vocab", ctypes.c_int32), ("entropy_spike", ctypes.c_float),
        ("conf_drop", ctypes.c_float), ("wr_last_N", ctypes.c_int32),
        ("dtype", ctypes.c_int32), ("spill_min_D", ctypes.c_int32),
        ("device_rows", ctypes.c_int32), ("history_W", ctypes.c_int32),
        ("relevance", ctypes.c_int32), ("scope", ctypes.c_int32),
        ("candidates", ctypes.c_int32), ("debug_margin", ctypes.c_float),
    ]


class asrkf_stats_t(ctypes.Structure):
    _fields_ = [
        ("step", ctypes.c_int64), ("total_positions", ctypes.c_int64),
        ("active_positions", ctypes.c_int64), ("attended_total", ctypes.c_int64),
        ("recoveries", ctypes.c_int64 * 4), ("rr_requests", ctypes.c_int64),
        ("attn_launches", ctypes.c_int64), ("attn_kernel_ms", ctypes.c_double),
        ("compression", ctypes.c_double), ("rows_to_host", ctypes.c_int64),
        ("rows_from_host", ctypes.c_int64), ("rows_released", ctypes.c_int64),
        ("rows_reused", ctypes.c_int64), ("margin_hits", ctypes.c_int64),
    ]

    def as_dict(self):
        d = {k: getattr(self, k) for k, _ in self._fields_}
        d["recoveries"] = list(self.recoveries)
        return d


class AsrkfError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"{_STATUS.get(code, code)}: {msg}")
        self.code = code


_lib = None


def load():
    """Load the built library; raises if it is missing (no fallback path)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
    # torch brings a HIP runtime of its own.  The library must use the same one
    # as the tensors it is given, so torch's is loaded and started first: with
    # the library loaded first, the two runtimes have been seen to disagree
    # (workgroup occupancy reported as zero, torch finding no GPU).
    import torch
    torch.cuda.is_available()
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, F = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float
    sig = {
        "asrkf_init": ([ctypes.POINTER(asrkf_config), ctypes.POINTER(P)], I32),
        "asrkf_prefill": ([P, I32, I32, P, P, I32, P], I32),
        "asrkf_decode_step": ([P, I32, P, P, P, P, P], I32),
        "asrkf_decode_step_static": ([P, I32, P, P, P, P, P], I32),
        "asrkf_restore": ([P, P, I32, P], I32),
        "asrkf_stats": ([P, ctypes.POINTER(asrkf_stats_t)], I32),
        "asrkf_stats_reset": ([P], I32),
        "asrkf_set_timing": ([P, I32], I32),
        "asrkf_timing_series": ([P, P, ctypes.c_int64, P], I32),
        "asrkf_reset": ([P], I32),
        "asrkf_debug_delay_side": ([P, I32], I32),
        "asrkf_get_state": ([P, I32, I32, P, P, P, P, P, P], I32),
        "asrkf_get_seq": ([P, I32, P, P, P, P], I32),
        "asrkf_get_residency": ([P, I32, I32, P, P, P], I32),
        "asrkf_schedule_table": ([F, I32, P], I32),
        "asrkf_destroy": ([P], None),
        "asrkf_last_error": ([], ctypes.c_char_p),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    _lib = lib
    return lib


def _check(code):
    if code != OK:
        raise AsrkfError(code, load().asrkf_last_error().decode())


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if hasattr(x, "data_ptr"):
        return x.data_ptr()
    if hasattr(x, "ctypes"):
        return x.ctypes.data
    raise TypeError(f"cannot take a pointer of {type(x)}")


def _stream(s):
    if s is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(s, int):
        return s
    return s.cuda_stream


def _enum(name, value, names):
    """A string option by name, or an int passed through unchanged (the
    library checks it)."""
    if isinstance(value, int):
        return value
    if value not in names:
        raise ValueError(f"{name} must be one of {sorted(names)}, not {value!r}")
    return names[value]


def make_config(n_layers, batch, n_q_heads, n_kv_heads, head_dim, max_ctx, window_K, tau,
                k_soft, vocab, entropy_spike=math.inf, conf_drop=0.0, wr_last_N=0,
                dtype="bf16", spill_min_D=0, device_rows=0, history_W=0, relevance="abs",
                scope="layer", candidates="outside", debug_margin=0.0):
    return asrkf_config(n_layers, batch, n_q_heads, n_kv_heads, head_dim, max_ctx, window_K,
                        tau, k_soft, vocab, entropy_spike, conf_drop, wr_last_N,
                        _enum("dtype", dtype, {"bf16": BF16, "f32": F32}),
                        spill_min_D, device_rows, history_W,
                        _enum("relevance", relevance, {"abs": REL_ABS, "softmax": REL_SOFTMAX}),
                        _enum("scope", scope, {"layer": SCOPE_LAYER, "token": SCOPE_TOKEN}),
                        _enum("candidates", candidates,
                              {"outside": CAND_OUTSIDE, "inside": CAND_INSIDE}), debug_margin)


def asrkf_init(cfg):
    h = ctypes.c_void_p()
    _check(load().asrkf_init(ctypes.byref(cfg), ctypes.byref(h)))
    return h.value


def asrkf_prefill(ctx, layer, seq, k, v, n_tokens, stream=None):
    _check(load().asrkf_prefill(ctx, layer, seq, _ptr(k), _ptr(v), n_tokens, _stream(stream)))


def asrkf_decode_step(ctx, layer, q, k_new, v_new, out, stream=None):
    _check(load().asrkf_decode_step(ctx, layer, _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(out),
                                    _stream(stream)))


def asrkf_decode_step_static(ctx, layer, q, k_new, v_new, out, stream=None):
    _check(load().asrkf_decode_step_static(ctx, layer, _ptr(q), _ptr(k_new), _ptr(v_new),
                                           _ptr(out), _stream(stream)))


def asrkf_restore(ctx, logits, mode=AUTO, stream=None):
    _check(load().asrkf_restore(ctx, _ptr(logits), mode, _stream(stream)))


def asrkf_stats(ctx):
    st = asrkf_stats_t()
    _check(load().asrkf_stats(ctx, ctypes.byref(st)))
    return st.as_dict()


def asrkf_stats_reset(ctx):
    _check(load().asrkf_stats_reset(ctx))


def asrkf_debug_delay_side(ctx, microseconds):
    _check(load().asrkf_debug_delay_side(ctx, int(microseconds)))


def asrkf_set_timing(ctx, enable):
    _check(load().asrkf_set_timing(ctx, 1 if enable else 0))


def asrkf_reset(ctx):
    _check(load().asrkf_reset(ctx))


def asrkf_timing_series(ctx):
    """Execution times (ms) of the timed attention launches since the last
    stats reset, in launch order, as a numpy float32 array."""
    import numpy as np
    n = ctypes.c_int64()
    _check(load().asrkf_timing_series(ctx, None, 0, ctypes.byref(n)))
    ms = np.zeros(max(1, n.value), np.float32)
    _check(load().asrkf_timing_series(ctx, ms.ctypes.data, n.value, ctypes.byref(n)))
    return ms[:n.value]


def asrkf_get_state(ctx, layer, seq, max_ctx):
    """Returns dict(n, unfreeze, count, frozen, active) as numpy arrays."""
    import numpy as np
    n = ctypes.c_int32()
    na = ctypes.c_int32()
    U = np.zeros(max_ctx + 1, np.int32)
    c = np.zeros(max_ctx + 1, np.int32)
    fr = np.zeros(max_ctx + 1, np.uint8)
    act = np.zeros(max_ctx + 1, np.int32)
    _check(load().asrkf_get_state(ctx, layer, seq, ctypes.addressof(n), U.ctypes.data,
                                  c.ctypes.data, fr.ctypes.data, act.ctypes.data,
                                  ctypes.addressof(na)))
    k = n.value
    return {"n": k, "unfreeze": U[:k].copy(), "count": c[:k].copy(),
            "frozen": fr[:k].astype(bool), "active": act[: na.value].copy()}


def asrkf_get_residency(ctx, layer, seq, max_ctx):
    """Returns dict(n, device_row, on_host) as numpy arrays."""
    import numpy as np
    n = ctypes.c_int32()
    row = np.zeros(max_ctx + 1, np.int32)
    oh = np.zeros(max_ctx + 1, np.uint8)
    _check(load().asrkf_get_residency(ctx, layer, seq, ctypes.addressof(n), row.ctypes.data,
                                      oh.ctypes.data))
    k = n.value
    return {"n": k, "device_row": row[:k].copy(), "on_host": oh[:k].astype(bool)}


def asrkf_get_seq(ctx, seq):
    H, pm = ctypes.c_float(), ctypes.c_float()
    esc, lvl = ctypes.c_int32(), ctypes.c_int32()
    _check(load().asrkf_get_seq(ctx, seq, ctypes.addressof(H), ctypes.addressof(pm),
                                ctypes.addressof(esc), ctypes.addressof(lvl)))
    return {"entropy": H.value, "pmax": pm.value, "escalation": esc.value, "level": lvl.value}


def asrkf_schedule_table(k_soft, n):
    import numpy as np
    out = np.zeros(n, np.int32)
    _check(load().asrkf_schedule_table(k_soft, n, out.ctypes.data))
    return out


def asrkf_destroy(ctx):
    if ctx:
        load().asrkf_destroy(ctx)


def asrkf_last_error():
    return load().asrkf_last_error().decode()
