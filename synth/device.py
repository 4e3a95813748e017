"""ctypes binding of libasrkf_synth.so: the device twin of synth.gen.

Fills the large workloads directly in HBM with the same bits as the host
generator (checked bit for bit by the GPU tests).
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from . import gen

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libasrkf_synth.so")
N_KINDS = 12
MAX_FLAT = 16


class SynthParams(ctypes.Structure):
    _fields_ = [
        ("keys", ctypes.c_void_p), ("hh_thr", ctypes.c_void_p),
        ("L", ctypes.c_int32), ("B", ctypes.c_int32), ("Hq", ctypes.c_int32),
        ("Hkv", ctypes.c_int32), ("D", ctypes.c_int32), ("V", ctypes.c_int32),
        ("recipe", ctypes.c_int32), ("bf16", ctypes.c_int32),
        ("ih_scale", ctypes.c_float), ("sigma", ctypes.c_float), ("flat_sigma", ctypes.c_float),
        ("beta_lo", ctypes.c_float), ("beta_span", ctypes.c_float),
        ("alpha_lo", ctypes.c_float), ("alpha_span", ctypes.c_float),
        ("nonhh_scale", ctypes.c_float), ("q_noise", ctypes.c_float),
        ("n_flat", ctypes.c_int32), ("flat", ctypes.c_int32 * MAX_FLAT),
    ]


_lib = None


def load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(LIB_PATH)
        P, I32, I64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
        lib.synth_kv_rows.argtypes = [P, I32, I32, I64, I64, P, P, P]
        lib.synth_new_kv.argtypes = [P, I32, I32, P, P, P, P]
        lib.synth_q.argtypes = [P, I32, I32, P, P]
        lib.synth_logits.argtypes = [P, I32, I32, P, P]
        for f in (lib.synth_kv_rows, lib.synth_new_kv, lib.synth_q, lib.synth_logits):
            f.restype = I32
        _lib = lib
    return _lib


class DeviceGen:
    """Device generator for one workload (uses torch for the small key tables)."""

    def __init__(self, w):
        import torch
        if len(w.flat_logit_steps) > MAX_FLAT:
            raise ValueError("too many planted flat-logit steps")
        if w.recipe not in ("gauss", "hh"):
            raise ValueError(f"recipe {w.recipe} has no device twin")
        self.w = w
        keys = np.zeros((N_KINDS, w.n_layers, w.batch), dtype=np.uint64)
        for kind in range(N_KINDS):
            for l in range(w.n_layers):
                for b in range(w.batch):
                    keys[kind, l, b] = gen.subkey(w.seed, kind, l, b)
        for b in range(w.batch):
            keys[gen.KIND_LOGIT, 0, b] = gen.subkey(w.seed, gen.KIND_LOGIT, b)
        thr = np.array([int(f * float(1 << 53)) for f in w.f_hh], dtype=np.uint64)
        self._keys = torch.from_numpy(keys.view(np.int64).reshape(-1).copy()).cuda()
        self._thr = torch.from_numpy(thr.view(np.int64).copy()).cuda()
        self.plen = torch.tensor(w.prefill, dtype=torch.int32).cuda()
        p = SynthParams()
        p.keys, p.hh_thr = self._keys.data_ptr(), self._thr.data_ptr()
        p.L, p.B, p.Hq, p.Hkv, p.D, p.V = (w.n_layers, w.batch, w.n_q_heads, w.n_kv_heads,
                                           w.head_dim, w.vocab)
        p.recipe = 1 if w.recipe == "hh" else 0
        p.bf16 = 1 if w.dtype == "bf16" else 0
        p.ih_scale = float(gen.IH_SCALE)
        p.sigma, p.flat_sigma = float(np.float32(w.logit_sigma)), float(np.float32(w.flat_sigma))
        p.beta_lo, p.beta_span = float(gen.HH_BETA_LO), float(gen.HH_BETA_SPAN)
        p.alpha_lo, p.alpha_span = float(gen.HH_ALPHA_LO), float(gen.HH_ALPHA_SPAN)
        p.nonhh_scale, p.q_noise = float(gen.HH_NONHH_AXIS_SCALE), float(gen.HH_Q_NOISE)
        p.n_flat = len(w.flat_logit_steps)
        for i, t in enumerate(w.flat_logit_steps):
            p.flat[i] = t
        self.params = p
        load()

    @staticmethod
    def _stream(stream):
        import torch
        return (stream or torch.cuda.current_stream()).cuda_stream

    def _check(self, rc):
        if rc != 0:
            raise RuntimeError(f"synth launch failed with HIP error {rc}")

    def kv_rows(self, layer, seq, p0, p1, K, V, stream=None):
        """K, V: device tensors of at least (p1-p0)*Hkv*D elements of the storage type."""
        self._check(load().synth_kv_rows(ctypes.byref(self.params), layer, seq, p0, p1 - p0,
                                         K.data_ptr(), V.data_ptr(), self._stream(stream)))

    def new_kv(self, t0, steps, K, V, stream=None):
        """New-token rows of steps t0..t0+steps-1 into [steps][L][B][Hkv][D]."""
        self._check(load().synth_new_kv(ctypes.byref(self.params), t0, steps,
                                        self.plen.data_ptr(), K.data_ptr(), V.data_ptr(),
                                        self._stream(stream)))

    def q(self, t0, steps, Q, stream=None):
        """Queries of steps t0..t0+steps-1 into [steps][L][B][Hq][D]."""
        self._check(load().synth_q(ctypes.byref(self.params), t0, steps, Q.data_ptr(),
                                   self._stream(stream)))

    def logits(self, t0, steps, out, stream=None):
        """Logits after steps t0..t0+steps-1 into [steps][B][V] float32."""
        self._check(load().synth_logits(ctypes.byref(self.params), t0, steps, out.data_ptr(),
                                        self._stream(stream)))
