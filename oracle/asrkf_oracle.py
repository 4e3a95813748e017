"""CPU oracle of the ASR-KF-EGR decode step.  TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this module.  The GPU library never calls it, and it
shares no code, tables or constants with the GPU library.

Plain, slow NumPy in float64.  Each function cites the passage of the paper
(arXiv 2512.11221) that it follows:

* Eq. 1 (Sec. 3.1)  attention over the cached (here: active) KV pairs;
* Eq. 2 (Sec. 3.2)  relevance s_j = (1/H) sum_h |Q^(h) . K_j^(h)|;
* Eq. 3 (Sec. 3.4)  freeze duration d_j = floor(sqrt(c_j) / k);
* Algorithm 1       order of one generation step: attention over the active
                    cache, relevance of the active tokens, the freeze loop over
                    low-relevance tokens outside the sliding window, then the
                    timer loop over frozen storage, which restores a token when
                    its timer reaches zero;
* Sec. 3.5          rolling re-evaluation (the timer loop);
* Sec. 3.6          entropy-guided staged recovery SR / WR / FR (+ RR flag).

Readings taken where the paper is silent or ambiguous (each is listed in the
design notes with the evidence for it):

* candidates for freezing are active tokens outside the window of the K most
  recent positions, the window including the token appended this step;
* the timer loop also visits tokens frozen earlier in the same step (literal
  statement order of Algorithm 1), so a duration of 1 has no effect;
* relevance uses H = number of query heads; under grouped-query attention head
  h reads KV head floor(h / (Hq/Hkv)); the score is Eq. 2 as printed (no 1/sqrt(d));
* the detection count c_j is cumulative (history window W unbounded) and kept
  across restores;
* entropy is Shannon entropy in nats of softmax(logits), 0 ln 0 = 0;
* optional readings, each selected explicitly: a finite history window W
  for c_j (detections in the last W steps, Eq. 3's text); relevance by
  attention weight (mean over heads of the softmax weights) instead of Eq. 2's
  |q . k|; token-global scope (one token state per sequence shared by all
  layers, relevance averaged over layers) instead of per-(layer, sequence)
  states; freeze candidates taken inside the window of the K most recent
  positions (the wording of Sec. 3.2) instead of outside it.  Which state
  scope the paper means is fixed by no printed value (every flagged token
  gives the same counts in both scopes): parity unpinned for that reading,
  while each scope's own functions are pinned by their reductions;
* recovery (the paper proposes but never evaluates it, so no printed value
  pins it; hand-derived expected states under these readings do):
  a step whose entropy exceeds theta_H (or whose top probability falls below
  theta_p when theta_p > 0) raises the sequence's escalation count by one, a
  calm step resets it; level = min(count, 3) selects SR, WR or FR, a count of
  4 or more also flags RR.  SR restores frozen tokens whose remaining timer
  exceeds 1, WR restores frozen tokens among the last N positions, FR restores
  every frozen token.  Detection counts are kept.
"""
from __future__ import annotations

from fractions import Fraction

import numpy as np

SR, WR, FR = 1, 2, 3


# ---------------------------------------------------------------------------
# Eq. 3: sublinear freeze schedule
# ---------------------------------------------------------------------------

def freeze_duration(c, k_soft):
    """d = floor(sqrt(c) / k) exactly (Eq. 3), with k taken as the exact value
    of the float32 number k_soft.  The largest integer d >= 0 with
    d * k <= sqrt(c), i.e. (d * k)^2 <= c."""
    k = Fraction(float(np.float32(k_soft)))
    if k <= 0:
        raise ValueError("k must be positive")
    d = 0
    while ((d + 1) * k) ** 2 <= c:
        d += 1
    return d


def duration_table(max_count, k_soft):
    """freeze_duration for every count 0..max_count (a lookup for the step)."""
    return np.array([freeze_duration(c, k_soft) for c in range(max_count + 1)], dtype=np.int64)


# ---------------------------------------------------------------------------
# Eq. 1 and Eq. 2
# ---------------------------------------------------------------------------

def attention(q, K, V):
    """Eq. 1 restricted to the given KV rows.

    q: [Hq][D]; K, V: [n][Hkv][D].  Query head h uses KV head h // (Hq/Hkv).
    Returns [Hq][D] float64: softmax(q_h K^T / sqrt(D)) V per head."""
    q = np.asarray(q, dtype=np.float64)
    Hq, D = q.shape
    group = Hq // K.shape[1]
    out = np.zeros((Hq, D))
    for g in range(K.shape[1]):
        Kg = np.ascontiguousarray(K[:, g, :], dtype=np.float64)
        Vg = np.ascontiguousarray(V[:, g, :], dtype=np.float64)
        for h in range(g * group, (g + 1) * group):
            logits = Kg @ q[h] / np.sqrt(D)
            w = np.exp(logits - logits.max())
            out[h] = (w / w.sum()) @ Vg
    return out


def relevance(q, K):
    """Eq. 2: s_j = (1/H) sum_h |q_h . K_j^(h)| for every row j of K, H = Hq."""
    q = np.asarray(q, dtype=np.float64)
    Hq = q.shape[0]
    group = Hq // K.shape[1]
    s = np.zeros(K.shape[0])
    for g in range(K.shape[1]):
        Kg = np.ascontiguousarray(K[:, g, :], dtype=np.float64)
        for h in range(g * group, (g + 1) * group):
            s += np.abs(Kg @ q[h])
    return s / Hq


def relevance_softmax(q, K):
    """Relevance by attention weight: s_j = (1/H) sum_h softmax_j(q_h . K_j^(h) / sqrt(d))
    over the rows of K, H = Hq.  A reading of Eq. 2 under which a token's score
    is the share of attention it receives, averaged over the heads."""
    q = np.asarray(q, dtype=np.float64)
    Hq, D = q.shape
    group = Hq // K.shape[1]
    s = np.zeros(K.shape[0])
    for g in range(K.shape[1]):
        Kg = np.ascontiguousarray(K[:, g, :], dtype=np.float64)
        for h in range(g * group, (g + 1) * group):
            logits = Kg @ q[h] / np.sqrt(D)
            w = np.exp(logits - logits.max())
            s += w / w.sum()
    return s / Hq


def attend_rows(q, Kh, Vh, relevance_kind="abs"):
    """Eq. 1 and the relevance together over rows given per KV head: Kh[g],
    Vh[g] are [n][D] arrays of the same n tokens.  The G query heads of a KV
    head are taken together as one matrix product, so each KV head's rows are
    read once; the results equal attention() and relevance() (or
    relevance_softmax()) up to summation order."""
    q = np.asarray(q, dtype=np.float64)
    Hq, D = q.shape
    group = Hq // len(Kh)
    out = np.zeros((Hq, D))
    s = np.zeros(len(Kh[0]))
    for g in range(len(Kh)):
        Kg = np.asarray(Kh[g], dtype=np.float64)
        Vg = np.asarray(Vh[g], dtype=np.float64)
        heads = slice(g * group, (g + 1) * group)
        X = Kg @ q[heads].T                        # [n][G]: q_h . k_j
        logits = X / np.sqrt(D)
        W = np.exp(logits - logits.max(axis=0))
        W /= W.sum(axis=0)
        for i in range(group):
            s += np.abs(X[:, i]) if relevance_kind == "abs" else W[:, i]
        out[heads] = W.T @ Vg
    return out, s / Hq


# ---------------------------------------------------------------------------
# Sec. 3.6: entropy monitoring and the escalation ladder
# ---------------------------------------------------------------------------

def entropy(logits):
    """Shannon entropy (nats) and top probability of softmax(logits)."""
    x = np.asarray(logits, dtype=np.float64)
    e = np.exp(x - x.max())
    p = e / e.sum()
    nz = p[p > 0]
    return float(-(nz * np.log(nz)).sum()), float(p.max())


def escalate(count, H, pmax, theta_H, theta_p):
    """One step of the SR -> WR -> FR -> RR ladder for one sequence.

    Returns (new count, level applied after this step, RR requested)."""
    spike = (H > theta_H) or (theta_p > 0 and pmax < theta_p)
    count = count + 1 if spike else 0
    return count, min(count, FR), count > FR


# ---------------------------------------------------------------------------
# Algorithm 1 for one (layer, sequence)
# ---------------------------------------------------------------------------

class StepRecord:
    __slots__ = ("out", "active", "scores")

    def __init__(self, out, active, scores):
        self.out = out          # [Hq][D] attention output of this step ([L][Hq][D] token-global)
        self.active = active    # positions attended this step, ascending
        self.scores = scores    # relevance of each attended position


class TokenStates:
    """Per-token detection count c_j, freeze timer d_j and membership of the
    frozen storage F (Algorithm 1 REQUIRE), with the freeze loop, the timer
    loop and the restores of the recovery ladder.

    history_W = 0 counts every detection (c_j cumulative); history_W = W > 0
    counts the detections of the last W steps only (Eq. 3's history window):
    at a detection in step t, c_j = number of detections in steps t-W+1 .. t.

    candidates "outside" takes the freeze candidates among the active tokens
    outside the window of the K most recent positions (Algorithm 1's freeze
    loop); "inside" takes them among the active tokens inside that window (the
    wording of Sec. 3.2, which estimates relevance within the window)."""

    def __init__(self, cap, window_K, tau, k_soft, history_W=0, candidates="outside"):
        if candidates not in ("outside", "inside"):
            raise ValueError(f"candidates must be 'outside' or 'inside', not {candidates!r}")
        self.n = 0
        self.candidates = candidates
        self.t = 0                                      # current step
        self.window_K = int(window_K)
        self.tau = float(tau)
        self.k_soft = float(k_soft)
        self.history_W = int(history_W)
        self.count = np.zeros(cap, dtype=np.int64)      # c_j
        self.timer = np.zeros(cap, dtype=np.int64)      # d_j
        self.frozen = np.zeros(cap, dtype=bool)         # membership of F
        self.detections = [[] for _ in range(cap)] if self.history_W else None
        self._durations = duration_table(64, k_soft)

    def _duration(self, c):
        while c >= len(self._durations):
            self._durations = duration_table(2 * len(self._durations), self.k_soft)
        return self._durations[c]

    def _new_position(self, j):
        self.count[j] = 0
        self.timer[j] = 0
        self.frozen[j] = False

    def active_positions(self):
        return np.nonzero(~self.frozen[: self.n])[0]

    def outside_window(self, j):
        """True when position j is not among the K most recent positions
        (the window includes the token appended this step)."""
        return j < self.n - self.window_K

    def is_candidate(self, j):
        """True when position j may be frozen by the freeze loop."""
        return self.outside_window(j) if self.candidates == "outside" else not self.outside_window(j)

    def detect(self, j):
        """Record a low-relevance detection of j at the current step; returns c_j."""
        if not self.history_W:
            self.count[j] += 1
        else:
            hist = self.detections[j]
            hist.append(self.t)
            self.count[j] = sum(1 for s in hist if s > self.t - self.history_W)
        return self.count[j]

    def freeze_loop(self, A, s):
        """For each candidate j (by default: outside the sliding window) with
        s_j < tau: c_j += 1, d_j = floor(sqrt(c_j)/k), and if d_j > 0 move j
        from A to F."""
        for j, sj in zip(A, s):
            if self.is_candidate(j) and sj < self.tau:
                self.timer[j] = self._duration(self.detect(j))
                if self.timer[j] > 0:
                    self.frozen[j] = True

    def timer_loop(self):
        """For j in F: d_j -= 1, and if d_j <= 0 restore j from F to A."""
        for j in np.nonzero(self.frozen[: self.n])[0]:
            self.timer[j] -= 1
            if self.timer[j] <= 0:
                self.frozen[j] = False

    def recover(self, level, last_N):
        """Staged recovery on this instance (Sec. 3.6), applied after a step."""
        n = self.n
        F = np.nonzero(self.frozen[:n])[0]
        if level == SR:
            sel = F[self.timer[F] > 1]
        elif level == WR:
            sel = F[F >= n - last_N]
        elif level == FR:
            sel = F
        else:
            return
        self.frozen[sel] = False
        self.timer[sel] = 0

    def state(self):
        """(timers, counts, frozen mask) over the n current positions."""
        n = self.n
        return self.timer[:n].copy(), self.count[:n].copy(), self.frozen[:n].copy()


class LayerCache:
    """The cached pairs (K_j, V_j) of one layer of one sequence, KV-head major
    [Hkv][position][D] in float64, and Eq. 1 / the relevance over a subset."""

    def __init__(self, K_prompt, V_prompt, cap, relevance_kind="abs"):
        K_prompt = np.asarray(K_prompt)
        V_prompt = np.asarray(V_prompt)
        P, Hkv, D = K_prompt.shape
        self.K = np.zeros((Hkv, cap, D))
        self.V = np.zeros((Hkv, cap, D))
        self._rows_k = np.empty((Hkv, cap, D))     # the attended rows of one step
        self._rows_v = np.empty((Hkv, cap, D))
        self.K[:, :P] = K_prompt.transpose(1, 0, 2)
        self.V[:, :P] = V_prompt.transpose(1, 0, 2)
        self.relevance_kind = relevance_kind

    def put(self, j, k_new, v_new):
        self.K[:, j] = k_new
        self.V[:, j] = v_new

    def attend(self, q, A):
        """Attn(q, A) and the relevance of every j in A."""
        n = len(A)
        for g in range(self.K.shape[0]):
            np.take(self.K[g], A, axis=0, out=self._rows_k[g, :n], mode="clip")
            np.take(self.V[g], A, axis=0, out=self._rows_v[g, :n], mode="clip")
        return attend_rows(q, self._rows_k[:, :n], self._rows_v[:, :n], self.relevance_kind)


class Instance(TokenStates):
    """Token states of one (layer, sequence): active cache A, frozen storage F,
    per-token detection count c_j and freeze timer d_j (Algorithm 1 REQUIRE).
    relevance_kind "abs" is Eq. 2; "softmax" scores by attention weights."""

    def __init__(self, K_prompt, V_prompt, window_K, tau, k_soft, capacity=None,
                 history_W=0, relevance_kind="abs", candidates="outside"):
        P = len(K_prompt)
        cap = capacity if capacity is not None else P + 4096
        super().__init__(cap, window_K, tau, k_soft, history_W, candidates)
        self.cache = LayerCache(K_prompt, V_prompt, cap, relevance_kind)
        self.K, self.V = self.cache.K, self.cache.V
        self.n = P

    def step(self, q, k_new, v_new):
        """One generation step for this layer (Algorithm 1, freeze and timer loops)."""
        self.t += 1
        j_new = self.n
        self.cache.put(j_new, k_new, v_new)
        self._new_position(j_new)
        self.n += 1
        A = self.active_positions()
        out, s = self.cache.attend(q, A)
        self.freeze_loop(A, s)
        self.timer_loop()
        return StepRecord(out, A, s)


class GlobalInstance(TokenStates):
    """Token-global scope: one set of token states per sequence, shared by
    all layers (a token's KV pair leaves every layer at once, Sec. 3.2).  The
    relevance of a token is the mean of its per-layer relevance (each a mean
    over that layer's heads), i.e. the mean over layers x heads."""

    def __init__(self, K_prompts, V_prompts, window_K, tau, k_soft, capacity=None,
                 history_W=0, relevance_kind="abs", candidates="outside"):
        P = len(K_prompts[0])
        cap = capacity if capacity is not None else P + 4096
        super().__init__(cap, window_K, tau, k_soft, history_W, candidates)
        self.caches = [LayerCache(K, V, cap, relevance_kind) for K, V in zip(K_prompts, V_prompts)]
        self.n = P

    def step(self, qs, k_news, v_news):
        """One generation step of every layer: qs, k_news, v_news indexed by layer."""
        self.t += 1
        j_new = self.n
        for cache, k, v in zip(self.caches, k_news, v_news):
            cache.put(j_new, k, v)
        self._new_position(j_new)
        self.n += 1
        A = self.active_positions()
        outs, s = [], np.zeros(len(A))
        for cache, q in zip(self.caches, qs):
            o, sl = cache.attend(q, A)
            outs.append(o)
            s += sl
        s /= len(self.caches)
        self.freeze_loop(A, s)
        self.timer_loop()
        return StepRecord(np.stack(outs), A, s)


# ---------------------------------------------------------------------------
# Driver
# ---------------------------------------------------------------------------

def recovery_schedule(entropies, theta_H, theta_p, mode=None):
    """Levels applied after each step for one sequence.

    entropies: list of (H, pmax) per step.  mode None = entropy-driven,
    otherwise the level forced at every step (SR/WR/FR, 0 = none).
    Returns (levels, rr_flags)."""
    levels, rr, count = [], [], 0
    for H, pmax in entropies:
        if mode is None:
            count, level, r = escalate(count, H, pmax, theta_H, theta_p)
        else:
            level, r = int(mode), False
        levels.append(level)
        rr.append(r)
    return levels, rr


def run_instance(K_prompt, V_prompt, steps, q_of, kv_of, window_K, tau, k_soft,
                 levels=None, last_N=None, on_step=None):
    """Run one (layer, sequence) instance for ``steps`` decode steps.

    q_of(t) -> [Hq][D]; kv_of(t) -> (k_new, v_new) each [Hkv][D], t = 1..steps.
    levels[t-1]: recovery level applied after step t (0 = none).
    on_step(t, record, instance) is called after each step (after recovery).
    """
    inst = Instance(K_prompt, V_prompt, window_K, tau, k_soft,
                    capacity=len(K_prompt) + steps + 1)
    last_N = 4 * window_K if last_N is None else last_N
    for t in range(1, steps + 1):
        k_new, v_new = kv_of(t)
        rec = inst.step(q_of(t), k_new, v_new)
        if levels is not None and levels[t - 1]:
            inst.recover(levels[t - 1], last_N)
        if on_step is not None:
            on_step(t, rec, inst)
    return inst
