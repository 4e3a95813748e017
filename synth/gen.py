"""Seeded synthetic inputs for the active-set decode path (host implementation).

Every value is a pure function of (config seed, tensor kind, layer, sequence,
element index), built from a counter-based generator, so that any row of any
tensor can be produced on its own: the oracle regenerates only the instances
it checks, and the device twin (``synth/csrc/synth_gen.hip``) fills the large
workloads in HBM with the identical bits.

This module holds none of the method's arithmetic: it draws numbers, shapes
them into the distributions stated below, and rounds them to the storage
type.  Nothing here scores, freezes, compacts or attends.

Generator: SplitMix64 (Steele, Lea and Flood, OOPSLA 2014), output function
``mix64`` applied to ``key + (ctr + 1) * golden_gamma``.

Normal stand-in: Irwin-Hall with four 16-bit uniforms, centred and scaled to
unit variance.  Its support is bounded (|z| <= 3.4641) and every step is an
exact integer operation followed by one IEEE fp32 multiply, so host and device
agree bit for bit.  bf16 values are made by round-to-nearest-even from fp32.
"""
from __future__ import annotations

import numpy as np

U64 = np.uint64
GAMMA = U64(0x9E3779B97F4A7C15)
M1 = U64(0xBF58476D1CE4E5B9)
M2 = U64(0x94D049BB133111EB)
MASK16 = U64(0xFFFF)

# Irwin-Hall(4) over 16-bit uniforms: mean 4*65535/2, variance (2^32-1)/3.
IH_MEAN = 131070
IH_SCALE = np.float32(1.0 / np.sqrt((2.0 ** 32 - 1.0) / 3.0))
GAUSS_MAX = float(np.float32(IH_MEAN) * IH_SCALE)  # largest |gauss| value

# Tensor kinds (first level of key derivation).
KIND_K, KIND_V, KIND_Q, KIND_LOGIT = 1, 2, 3, 4
KIND_HH, KIND_BETA, KIND_AXIS, KIND_ALPHA = 5, 6, 7, 8
KIND_CTX, KIND_FHH, KIND_PLANT = 9, 10, 11
ATTEMPT_BASE = 1 << 62          # counter offset of re-drawn rows

# Heavy-hitter recipe constants (all exact powers of two where they scale).
HH_BETA_LO, HH_BETA_SPAN = np.float32(8.0), np.float32(56.0)
HH_ALPHA_LO, HH_ALPHA_SPAN = np.float32(0.2), np.float32(0.1)
HH_NONHH_AXIS_SCALE = np.float32(2.0 ** -4)
HH_Q_NOISE = np.float32(2.0 ** -13)


def mix64(z):
    """SplitMix64 output function on uint64 arrays (wrapping arithmetic)."""
    z = np.asarray(z, dtype=U64)
    with np.errstate(over="ignore"):
        z = (z ^ (z >> U64(30))) * M1
        z = (z ^ (z >> U64(27))) * M2
    return z ^ (z >> U64(31))


def draw(key, ctr):
    """Counter-based draw: 64 random bits for (key, ctr)."""
    key = np.asarray(key, dtype=U64)
    ctr = np.asarray(ctr, dtype=U64)
    with np.errstate(over="ignore"):
        return mix64(key + (ctr + U64(1)) * GAMMA)


def subkey(key, *parts):
    k = U64(key)
    for p in parts:
        k = U64(draw(k, U64(p)))
    return k


def gauss(z):
    """Irwin-Hall(4) normal stand-in from 64 random bits, as float32."""
    z = np.asarray(z, dtype=U64)
    s = (z & MASK16) + ((z >> U64(16)) & MASK16) + ((z >> U64(32)) & MASK16) + (z >> U64(48))
    return (s.astype(np.int64) - IH_MEAN).astype(np.float32) * IH_SCALE


def uniform(z):
    """Uniform in [0, 1) with 24 bits, as float32 (exact)."""
    z = np.asarray(z, dtype=U64)
    return (z >> U64(40)).astype(np.float32) * np.float32(2.0 ** -24)


def bf16_bits(x):
    """Round-to-nearest-even fp32 -> bf16, returned as uint16 bits."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_to_f32(bits):
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def round_to(x, dtype):
    """Values as stored: fp32 unchanged, bf16 rounded (returned as fp32 values)."""
    return x.astype(np.float32) if dtype == "f32" else bf16_to_f32(bf16_bits(x))


# --------------------------------------------------------------------------
# Workload descriptors
# --------------------------------------------------------------------------

class Workload:
    """Shapes, method parameters and input recipe of one synthetic workload.

    recipe:
      'gauss'    Q, K, V ~ N(0,1) stand-in (Irwin-Hall) per element.
      'hh'       heavy-hitter keys: per (layer, seq, kv head g) a signed
                 coordinate axis e_{a_g}; a token is a heavy hitter with
                 probability f_hh; its key has +-beta (beta in [8, 64)) on
                 the axis, other keys 2^-4 * z there; the rest of every key
                 and all of V are z.  Queries are sign * alpha (alpha in
                 [0.2, 0.3)) on the group's axis plus 2^-13 * z noise.
                 The relevance of every token then stays provably on one
                 side of tau = 0.5 at every step (see hh_relevance_bounds).
    """

    def __init__(self, name, seed, n_layers, batch, n_q_heads, n_kv_heads, head_dim,
                 dtype, prefill, steps, window_K, tau, k_soft, vocab, logit_sigma,
                 recipe, f_hh=0.0, entropy_spike=float("inf"), conf_drop=0.0,
                 wr_last_N=None, flat_logit_steps=(), flat_sigma=0.1, spill_min_D=0,
                 max_ctx=None, device_rows=0, history_W=0, relevance="abs", scope="layer",
                 candidates="outside"):
        self.name = name
        self.seed = int(seed)
        self.n_layers = int(n_layers)
        self.batch = int(batch)
        self.n_q_heads = int(n_q_heads)
        self.n_kv_heads = int(n_kv_heads)
        self.head_dim = int(head_dim)
        self.dtype = dtype
        self.prefill = [int(p) for p in prefill]
        assert len(self.prefill) == self.batch
        self.steps = int(steps)
        self.window_K = int(window_K)
        self.tau = float(tau)
        self.k_soft = float(k_soft)
        self.vocab = int(vocab)
        self.logit_sigma = float(logit_sigma)
        self.recipe = recipe
        self.f_hh = [float(f) for f in (f_hh if np.ndim(f_hh) else [f_hh] * self.batch)]
        self.entropy_spike = float(entropy_spike)
        self.conf_drop = float(conf_drop)
        self.wr_last_N = int(wr_last_N if wr_last_N is not None else 4 * window_K)
        self.flat_logit_steps = tuple(int(t) for t in flat_logit_steps)
        self.flat_sigma = float(flat_sigma)
        self.spill_min_D = int(spill_min_D)
        self.device_rows = int(device_rows)
        self.history_W = int(history_W)
        self.relevance = relevance              # "abs" (Eq. 2) or "softmax" (attention weight)
        self.scope = scope                      # "layer" or "token"
        self.candidates = candidates            # freeze candidates "outside" or "inside" the window
        self.max_ctx = int(max_ctx if max_ctx is not None else max(self.prefill) + self.steps)

    @property
    def group(self):
        return self.n_q_heads // self.n_kv_heads

    def replace(self, **kw):
        d = dict(self.__dict__)
        d.update(kw)
        return Workload(**d)

    def kv_bytes_per_token(self):
        esz = 2 if self.dtype == "bf16" else 4
        return 2 * self.n_kv_heads * self.head_dim * esz


def _ragged_prefill(seed, batch, lo, hi):
    k = subkey(seed, KIND_CTX)
    z = draw(k, np.arange(batch, dtype=U64))
    return [int(lo + int(v) % (hi - lo + 1)) for v in z]


def _ragged_fhh(seed, batch, lo, hi):
    k = subkey(seed, KIND_FHH)
    u = uniform(draw(k, np.arange(batch, dtype=U64))).astype(np.float64)
    return [float(lo + (hi - lo) * x) for x in u]


SEED = 0x25121122


def tiny(tau=0.5, recipe="gauss", **kw):
    """1 layer, batch 1, 8 q / 2 kv heads, head_dim 64, fp32, prompt 512, 64 steps."""
    args = dict(name="tiny", seed=SEED + 1, n_layers=1, batch=1, n_q_heads=8, n_kv_heads=2,
                head_dim=64, dtype="f32", prefill=[512], steps=64, window_K=32, tau=tau,
                k_soft=2.0, vocab=1024, logit_sigma=2.0, recipe=recipe)
    args.update(kw)
    return Workload(**args)


def llama8b_1layer(**kw):
    """LLaMA-3-8B attention shape, one layer: batch 1, 32/8 heads, d 128, bf16, 8192 + 256."""
    args = dict(name="llama3-8b-1layer", seed=SEED + 2, n_layers=1, batch=1, n_q_heads=32,
                n_kv_heads=8, head_dim=128, dtype="bf16", prefill=[8192], steps=256,
                window_K=128, tau=0.5, k_soft=2.0, vocab=128256, logit_sigma=3.0,
                recipe="hh", f_hh=0.35)
    args.update(kw)
    return Workload(**args)


def llama8b_32layer(**kw):
    """32-layer attention-only decode, batch 8, context 32768, 128 steps, bf16."""
    args = dict(name="llama3-8b-32layer-b8-ctx32k", seed=SEED + 3, n_layers=32, batch=8,
                n_q_heads=32, n_kv_heads=8, head_dim=128, dtype="bf16", prefill=[32768] * 8,
                steps=128, window_K=128, tau=0.5, k_soft=2.0, vocab=128256, logit_sigma=3.0,
                recipe="hh", f_hh=0.35)
    args.update(kw)
    return Workload(**args)


def ragged(**kw):
    """Batch 64, context uniform in [2048, 32768], f_hh uniform in [0.2, 0.5], 64 steps."""
    seed = kw.pop("seed", SEED + 5)
    batch = kw.pop("batch", 64)
    args = dict(name="llama3-8b-ragged-b64", seed=seed, n_layers=1, batch=batch, n_q_heads=32,
                n_kv_heads=8, head_dim=128, dtype="bf16",
                prefill=_ragged_prefill(seed, batch, 2048, 32768), steps=64, window_K=128,
                tau=0.5, k_soft=2.0, vocab=128256, logit_sigma=3.0, recipe="hh",
                f_hh=_ragged_fhh(seed, batch, 0.2, 0.5))
    args.update(kw)
    return Workload(**args)


def recovery_stress(**kw):
    """Recovery stress at the LLaMA-3-8B shape: batch 1, context 131072, spill
    mode (a token frozen for >= 2 steps leaves the device), entropy trigger at
    10 nats.  The caller sets ``steps`` and the planted flat-logit step."""
    args = dict(name="llama3-8b-recovery-ctx131k", seed=SEED + 4, n_layers=1, batch=1,
                n_q_heads=32, n_kv_heads=8, head_dim=128, dtype="bf16", prefill=[131072],
                steps=2016, window_K=128, tau=0.5, k_soft=2.0, vocab=128256, logit_sigma=3.0,
                recipe="hh", f_hh=0.35, entropy_spike=10.0, spill_min_D=2)
    args.update(kw)
    return Workload(**args)


# --------------------------------------------------------------------------
# Tensors
# --------------------------------------------------------------------------

def _keys(w, kind, layer, seq):
    return subkey(w.seed, kind, layer, seq)


def _row_key(key, attempt):
    return key if attempt == 0 else U64(draw(key, U64(ATTEMPT_BASE + int(attempt))))


def hh_axes(w, layer, seq):
    """Per kv head: (axis index, sign) of the heavy-hitter direction."""
    z = draw(_keys(w, KIND_AXIS, layer, seq), np.arange(w.n_kv_heads, dtype=U64))
    axis = (z % U64(w.head_dim)).astype(np.int64)
    sign = np.where(((z >> U64(32)) & U64(1)) == U64(1), -1.0, 1.0).astype(np.float32)
    return axis, sign


def hh_mask(w, layer, seq, p0, p1):
    thr = U64(int(w.f_hh[seq] * float(1 << 53)))
    z = draw(_keys(w, KIND_HH, layer, seq), np.arange(p0, p1, dtype=U64))
    return (z >> U64(11)) < thr


def _gauss_rows(key, p0, p1, width, attempts=None, block=1024):
    n = p1 - p0
    out = np.empty((n, width), dtype=np.float32)
    cols = np.arange(width, dtype=U64)[None, :]
    for r0 in range(p0, p1, block):            # row blocks keep the temporaries small
        r1 = min(p1, r0 + block)
        ctr = np.arange(r0, r1, dtype=U64)[:, None] * U64(width) + cols
        out[r0 - p0:r1 - p0] = gauss(draw(key, ctr))
    if attempts is not None:
        a = np.asarray(attempts[p0:p1])
        for r in np.nonzero(a)[0]:
            ctr = U64(p0 + int(r)) * U64(width) + cols[0]
            out[r] = gauss(draw(_row_key(key, int(a[r])), ctr))
    return out


def kv_rows(w, layer, seq, p0, p1, attempts=None):
    """K and V rows of positions [p0, p1): float32 arrays [n][Hkv][D] holding the
    stored values (bf16-rounded for bf16 workloads).  ``attempts`` (int array over
    positions, optional) re-draws the key rows whose entry is non-zero."""
    Hkv, D = w.n_kv_heads, w.head_dim
    n = p1 - p0
    kk = _keys(w, KIND_K, layer, seq)
    kv = _keys(w, KIND_V, layer, seq)
    K = _gauss_rows(kk, p0, p1, Hkv * D, attempts).reshape(n, Hkv, D)
    V = _gauss_rows(kv, p0, p1, Hkv * D).reshape(n, Hkv, D)
    if w.recipe == "hh":
        axis, sign = hh_axes(w, layer, seq)
        hh = hh_mask(w, layer, seq, p0, p1)
        ctr = (np.arange(p0, p1, dtype=U64)[:, None] * U64(Hkv) + np.arange(Hkv, dtype=U64)[None, :])
        u = uniform(draw(_keys(w, KIND_BETA, layer, seq), ctr))
        beta = (u * HH_BETA_SPAN) + HH_BETA_LO              # two fp32 roundings
        for g in range(Hkv):
            a = axis[g]
            small = K[:, g, a] * HH_NONHH_AXIS_SCALE         # exact
            K[:, g, a] = np.where(hh, sign[g] * beta[:, g], small)
    return round_to(K, w.dtype), round_to(V, w.dtype)


def q_row(w, layer, seq, t):
    """Query of decode step t (1-based): float32 [Hq][D] of stored values."""
    Hq, D, G = w.n_q_heads, w.head_dim, w.group
    key = _keys(w, KIND_Q, layer, seq)
    ctr = U64(t) * U64(Hq * D) + np.arange(Hq * D, dtype=U64)
    q = gauss(draw(key, ctr)).reshape(Hq, D)
    if w.recipe == "hh":
        axis, sign = hh_axes(w, layer, seq)
        ua = uniform(draw(_keys(w, KIND_ALPHA, layer, seq),
                          U64(t) * U64(Hq) + np.arange(Hq, dtype=U64)))
        alpha = (ua * HH_ALPHA_SPAN) + HH_ALPHA_LO
        q = q * HH_Q_NOISE                                    # exact
        for h in range(Hq):
            g = h // G
            q[h, axis[g]] = q[h, axis[g]] + sign[g] * alpha[h]  # one fp32 add
    return round_to(q, w.dtype)


def logits_row(w, seq, t):
    """Next-token logits after step t for sequence seq: float32 [V]."""
    key = subkey(w.seed, KIND_LOGIT, seq)
    ctr = U64(t) * U64(w.vocab) + np.arange(w.vocab, dtype=U64)
    sigma = np.float32(w.flat_sigma if t in w.flat_logit_steps else w.logit_sigma)
    return gauss(draw(key, ctr)) * sigma


def hh_relevance_bounds(w):
    """Proven bounds on the mean-|q.k| relevance under the 'hh' recipe.

    Returns (max over non-heavy-hitter tokens, min over heavy-hitter tokens),
    valid for every step and token: the query is sign*alpha on the axis plus
    noise of at most n = 2^-13 * GAUSS_MAX per coordinate; bf16 rounding moves
    a value by at most 2^-8 of itself.  Off-axis terms are bounded by
    (D-1) * n' * z', the axis term by (alpha + e) * |k_axis|.
    """
    D = w.head_dim
    rnd = 1.0 + 2.0 ** -8
    z = GAUSS_MAX * rnd                                   # |off-axis key entry|
    e1 = GAUSS_MAX * float(HH_Q_NOISE) * rnd              # |off-axis query entry|
    a_lo, a_hi = float(HH_ALPHA_LO) - 1e-6, float(HH_ALPHA_LO + HH_ALPHA_SPAN) + 1e-6
    e_axis = GAUSS_MAX * float(HH_Q_NOISE) + 2.0 ** -8 * (a_hi + e1)
    off = (D - 1) * e1 * z
    small_axis = GAUSS_MAX * float(HH_NONHH_AXIS_SCALE) * rnd
    s_max_cold = (a_hi + e_axis) * small_axis + off
    beta_min = float(HH_BETA_LO) * (1.0 - 2.0 ** -8)
    s_min_hot = (a_lo - e_axis) * beta_min - off
    return s_max_cold, s_min_hot


# --------------------------------------------------------------------------
# Planted key (recovery stress)
# --------------------------------------------------------------------------

PLANT_ALPHA = 24.0        # query norm once the queries turn to the planted key
PLANT_COS = 0.9           # cosine between those queries and the planted key


def plant_position(w, layer=0, seq=0, lo=0, hi=65536):
    """The planted position: the first non-heavy-hitter position at or after a
    seeded uniform draw in [lo, hi)."""
    u = float(uniform(draw(subkey(w.seed, KIND_PLANT, layer, seq), U64(0))))
    p = lo + int(u * (hi - lo))
    hh = hh_mask(w, layer, seq, p, min(w.prefill[seq], p + 4096))
    free = np.nonzero(~hh)[0]
    if len(free) == 0:
        raise ValueError("no non-heavy-hitter position near the draw")
    return p + int(free[0])


def planted_q_rows(w, k_star, t0, t1, layer=0, seq=0):
    """Queries of steps t0..t1-1 aimed at the planted key: per head h,
    alpha * (cos * khat + sqrt(1 - cos^2) * u) with khat the unit key of the
    head's KV group and u a seeded unit vector orthogonal to khat and to the
    group's heavy-hitter axis (so heavy-hitter keys do not compete with the
    planted one).  k_star: [Hkv][D] stored key of the planted position.
    Returns float32 [t1 - t0][Hq][D] of stored (rounded) values."""
    Hq, D, G = w.n_q_heads, w.head_dim, w.group
    kh = np.asarray(k_star, dtype=np.float64)
    kh = kh / np.linalg.norm(kh, axis=1, keepdims=True)
    axis, _ = hh_axes(w, layer, seq)
    key = subkey(w.seed, KIND_PLANT, layer, seq, 1)
    sine = np.sqrt(1.0 - PLANT_COS ** 2)
    out = np.empty((t1 - t0, Hq, D), dtype=np.float32)
    for i, t in enumerate(range(t0, t1)):
        ctr = U64(t) * U64(Hq * D) + np.arange(Hq * D, dtype=U64)
        z = gauss(draw(key, ctr)).astype(np.float64).reshape(Hq, D)
        for h in range(Hq):
            g = h // G
            a = np.zeros(D)
            a[axis[g]] = 1.0
            e = kh[g]
            a = a - (a @ e) * e                      # the axis, made orthogonal to khat
            a /= np.linalg.norm(a)
            u = z[h] - (z[h] @ e) * e - (z[h] @ a) * a
            u /= np.linalg.norm(u)
            out[i, h] = PLANT_ALPHA * (PLANT_COS * e + sine * u)
    return round_to(out, w.dtype)
