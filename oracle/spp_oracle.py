"""Plain fp64 restatement of one offloaded-MoE decode step with SpecPrefetch.

TEST INFRASTRUCTURE ONLY (see the package docstring): never imported by the
product path.

What is computed, and where the paper defines it:

* native routing, T = Top_K(R(x)) -- Section "Problem Formulation"; the batch
  demand is the union of the per-token sets (same section);
* the adapter, z_hat = B A x, pi_hat = softmax(z_hat), s_e = sum over tokens of
  pi_hat_e -- Section "Expert Prediction Adapter";
* the candidate set C_M = Top_M(s) and the adapter parameter count
  (L-1) r (D+n) -- same section;
* the distillation loss L_pred (KL from the next layer's native routing
  distribution to the adapter's, averaged over tokens and layer pairs) and its
  gradient -- Section "Training Objective";
* the window-aware budget M_max and the prefetch set
  P = Top_{M_max}{ s_e : e not available and not in flight }, issued in
  descending priority, |P| <= M_max -- Section "Window-Aware Prefetch
  Budgeting";
* on-demand loading of every routed expert that is missing at execution, so
  that outputs never depend on prediction -- same section, last paragraph;
* ExpertRecall@M and ReadyRecall -- Section "Experimental Setup",
  "Evaluation Metrics".

Readings where the paper is silent (each listed with its reason in the design
notes): the block prologue (RMS normalisation without a learned scale; an
optional dense stand-in projection in place of attention), SwiGLU experts
combined with gates renormalised over the selected K, the fp32 router-input
and logit precision, the tie rule "lowest expert index wins", the budget
formula M_max = clamp(floor(W / c), 0, n), and a deterministic
least-recently-stamped slot replacement policy.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

EMPTY = -1

# --------------------------------------------------------------------------
# storage <-> values (the oracle's own decoding; inputs arrive as bf16 bit
# patterns or fp32 arrays)
# --------------------------------------------------------------------------


def decode(a: np.ndarray, dtype: str) -> np.ndarray:
    """Stored values as fp64: bf16 bits are the high half of an fp32 pattern."""
    if dtype == "bf16":
        bits = np.asarray(a, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
        return bits.view(np.float32).astype(np.float64)
    return np.asarray(a, dtype=np.float32).astype(np.float64)


def encode(v: np.ndarray, dtype: str) -> np.ndarray:
    """Round fp64 values once to the storage dtype (nearest, ties to even).

    bf16 keeps 8 significant bits: v = m 2^e with 0.5 <= |m| < 1, so the
    rounded value is rint(m 2^8) 2^(e-8) (numpy's rint rounds ties to even).
    Values stay in the normal range here (|v| >= 2^-126 or v == 0).
    """
    v = np.asarray(v, dtype=np.float64)
    if dtype == "bf16":
        m, e = np.frexp(v)
        r = np.ldexp(np.rint(m * 256.0), e - 8)
        return (r.astype(np.float32).view(np.uint32) >> np.uint32(16)).astype(np.uint16)
    return v.astype(np.float32)


def f32(v) -> np.ndarray:
    """Round to fp32 and return the rounded values as fp64."""
    return np.asarray(v, dtype=np.float64).astype(np.float32).astype(np.float64)


# --------------------------------------------------------------------------
# elementary functions
# --------------------------------------------------------------------------


def rms_normalize(v: np.ndarray, eps: float) -> np.ndarray:
    """v / sqrt(mean(v^2) + eps) along the last axis (no learned scale)."""
    v = np.asarray(v, dtype=np.float64)
    return v / np.sqrt(np.mean(v * v, axis=-1, keepdims=True) + eps)


def softmax(v: np.ndarray) -> np.ndarray:
    """softmax along the last axis in fp64."""
    v = np.asarray(v, dtype=np.float64)
    e = np.exp(v - np.max(v, axis=-1, keepdims=True))
    return e / np.sum(e, axis=-1, keepdims=True)


def silu(v: np.ndarray) -> np.ndarray:
    return v / (1.0 + np.exp(-v))


def top_k(values: np.ndarray, k: int) -> np.ndarray:
    """Indices of the k largest values in descending order; the lower index wins a tie."""
    values = np.asarray(values)
    order = np.lexsort((np.arange(values.shape[0]), -values))
    return order[:k].astype(np.int64)


# --------------------------------------------------------------------------
# Section "Problem Formulation": native routing
# --------------------------------------------------------------------------


def router_logits(Wr: np.ndarray, x: np.ndarray) -> np.ndarray:
    """Router logits z = W_r x as fp64 dot products rounded once to fp32 ([B, n])."""
    return f32(np.asarray(x, dtype=np.float64) @ np.asarray(Wr, dtype=np.float64).T)


def route(Wr: np.ndarray, x: np.ndarray, K: int):
    """Native Top-K routing of every token plus its combine weights.

    Returns (T [B,K] int64, g [B,K] fp32 values as fp64, z [B,n] fp32 logits).
    The combine weights are the softmax over all n logits renormalised over
    the K selected experts.
    """
    z = router_logits(Wr, x)
    B = z.shape[0]
    T = np.stack([top_k(z[b], K) for b in range(B)])
    p = softmax(z)
    g = np.empty((B, K))
    for b in range(B):
        sel = p[b, T[b]]
        g[b] = sel / np.sum(sel)
    return T, f32(g), z


def batch_demand(T: np.ndarray) -> List[int]:
    """Union of the per-token native selections, ascending expert index."""
    return sorted(set(int(e) for e in np.asarray(T).ravel()))


# --------------------------------------------------------------------------
# Section "Expert Prediction Adapter"
# --------------------------------------------------------------------------


def adapter_scores(A: np.ndarray, Bm: np.ndarray, x: np.ndarray):
    """Predicted next-layer logits, token distributions and batch priorities.

    z_hat = B (A x) (fp64 products, z_hat rounded to fp32); pi_hat = softmax(z_hat);
    s_e = sum over tokens, in token order, of pi_hat_e, rounded to fp32.
    Returns (z_hat [B,n], pi_hat [B,n], s [n]).
    """
    x = np.asarray(x, dtype=np.float64)
    a = x @ np.asarray(A, dtype=np.float64).T                     # [B, r]
    zhat = f32(a @ np.asarray(Bm, dtype=np.float64).T)            # [B, n]
    pi = softmax(zhat)
    s = np.zeros(zhat.shape[1])
    for b in range(pi.shape[0]):
        s = s + pi[b]
    return zhat, pi, f32(s)


def candidate_set(s: np.ndarray, M: int) -> np.ndarray:
    """C_M = Top_M(s) (model-level candidate set)."""
    return top_k(s, M)


def adapter_param_count(L: int, r: int, D: int, n: int) -> int:
    """Trainable adapter parameters over all adjacent layer pairs: (L-1) r (D+n)."""
    return (L - 1) * r * (D + n)


# --------------------------------------------------------------------------
# Section "Training Objective": adapter distillation
# --------------------------------------------------------------------------


def log_softmax(v: np.ndarray) -> np.ndarray:
    """log softmax along the last axis in fp64 (v minus its log-sum-exp)."""
    v = np.asarray(v, dtype=np.float64)
    m = np.max(v, axis=-1, keepdims=True)
    return v - m - np.log(np.sum(np.exp(v - m), axis=-1, keepdims=True))


def distill_pair_loss(A: np.ndarray, Bm: np.ndarray, X: np.ndarray, Z_next: np.ndarray) -> float:
    """The loss of one adjacent layer pair: the mean over the tokens of
    KL(pi || pi_hat), where pi = softmax(z^{l+1}) is the frozen native router's
    distribution at the next layer (the target) and pi_hat = softmax(B A x^l)
    the adapter's.  KL(p || q) = sum_e p_e (log p_e - log q_e): the target
    distribution weights the log ratio.  X [N, D], Z_next [N, n], fp64."""
    X = np.asarray(X, dtype=np.float64)
    zhat = (X @ np.asarray(A, dtype=np.float64).T) @ np.asarray(Bm, dtype=np.float64).T
    logp = log_softmax(Z_next)
    logq = log_softmax(zhat)
    kl = np.sum(np.exp(logp) * (logp - logq), axis=-1)
    return float(np.mean(kl))


def distill_pair_grad(A: np.ndarray, Bm: np.ndarray, X: np.ndarray, Z_next: np.ndarray):
    """Closed-form gradient of distill_pair_loss with respect to A and B.

    With a = A x and z_hat = B a, the derivative of -sum_e pi_e log pi_hat_e
    with respect to z_hat is pi_hat - pi (pi sums to one), so for the mean over
    N tokens G = (pi_hat - pi) / N [N, n], dL/dB = G^T a [n, r] and
    dL/dA = (G B)^T X [r, D].  Returns (dA, dB) in fp64."""
    X = np.asarray(X, dtype=np.float64)
    A = np.asarray(A, dtype=np.float64)
    Bm = np.asarray(Bm, dtype=np.float64)
    a = X @ A.T
    G = (softmax(a @ Bm.T) - softmax(Z_next)) / X.shape[0]
    return (G @ Bm).T @ X, G.T @ a


def distill_loss(adapters, X_layers, Z_layers) -> float:
    """L_pred: the pair losses averaged over the L-1 adjacent layer pairs.
    adapters[l] = (A^l, B^l) for l = 0..L-2; X_layers[l] the router inputs of
    layer l and Z_layers[l] its native router logits, over the same tokens."""
    L = len(X_layers)
    return float(sum(distill_pair_loss(adapters[l][0], adapters[l][1], X_layers[l], Z_layers[l + 1])
                     for l in range(L - 1)) / (L - 1))


# --------------------------------------------------------------------------
# Section "Window-Aware Prefetch Budgeting"
# --------------------------------------------------------------------------


class BudgetError(ValueError):
    pass


def prefetch_budget(window_us: float, per_expert_cost_us: float, n: int) -> int:
    """Maximum prefetch budget: the number of whole expert transfers that fit in
    the profiled overlap window, clamp(floor(W / c), 0, n).

    A non-positive window gives 0; a non-positive or non-finite cost, or a
    non-finite window, is an error.
    """
    if not (math.isfinite(window_us) and math.isfinite(per_expert_cost_us)) or per_expert_cost_us <= 0:
        raise BudgetError("window and per-expert cost must be finite, cost > 0")
    if n < 0:
        raise BudgetError("n must be >= 0")
    if window_us <= 0:
        return 0
    return int(min(n, math.floor(window_us / per_expert_cost_us)))


def select_prefetch(s: np.ndarray, occupied: Sequence[bool], M_max: int) -> List[int]:
    """P = Top_{M_max}{ s_e : e not available and not in flight }, descending priority.

    An expert whose priority is -inf is not a candidate (the adapter's
    priorities are sums of probabilities and never are; the Naive Prefetch
    scores mark the experts the preceding token did not use that way)."""
    eligible = [e for e in range(len(s)) if not occupied[e] and not (np.isinf(s[e]) and s[e] < 0)]
    if M_max <= 0 or not eligible:
        return []
    vals = np.asarray([s[e] for e in eligible])
    picked = top_k(vals, min(M_max, len(eligible)))
    return [eligible[int(i)] for i in picked]


def naive_scores(prev_T: Optional[np.ndarray], prev_g: Optional[np.ndarray], n: int) -> np.ndarray:
    """Naive Prefetch priorities for a target layer (Table 5): the experts the
    preceding decode step activated there, ranked by their gate mass summed
    over the batch (fp64 in token order, then fp32); -inf for every other
    expert, so only those experts are candidates."""
    acc = np.full(n, -np.inf)
    if prev_T is not None:
        for b in range(prev_T.shape[0]):
            for k in range(prev_T.shape[1]):
                e = int(prev_T[b, k])
                acc[e] = (0.0 if np.isinf(acc[e]) else acc[e]) + float(prev_g[b, k])
    return acc.astype(np.float32)


# --------------------------------------------------------------------------
# Available set of one layer: a logical slot table with deterministic
# least-recently-stamped replacement (the paper leaves replacement open)
# --------------------------------------------------------------------------


class SlotCache:
    """S accelerator slots of one layer; each holds one expert (or is EMPTY).

    Every slot carries the stamp of the last decode step that used or filled
    it.  Replacement rules:

    * on-demand load of a missing expert: the lowest-index EMPTY slot, else the
      slot with the smallest (stamp, slot index) whose expert is not needed by
      the current batch, else (when the batch needs more distinct experts than
      there are slots) the lowest-index slot whose expert already ran in an
      earlier round of this step.  A step runs in rounds: load missing experts
      in ascending order while a victim exists, then run every needed expert
      that is resident and has not run yet; repeat until all have run.  With
      at most S distinct needed experts there is a single round;
    * prefetch: the lowest-index EMPTY slot, else the smallest (stamp, slot
      index) among slots stamped before the current step; prefetching stops
      when no such slot is left;
    * after the on-demand loads of a step, every slot holding a needed expert
      takes the step's stamp; a prefetched slot takes the step's stamp.
    """

    def __init__(self, S: int, n: int, resident: Optional[Sequence[int]] = None):
        if S <= 0:
            raise ValueError("S must be positive")
        self.S, self.n = S, n
        self.expert = np.full(S, EMPTY, dtype=np.int64)
        self.stamp = np.zeros(S, dtype=np.int64)
        if resident is not None:
            if len(resident) > S or len(set(resident)) != len(resident):
                raise ValueError("bad resident list")
            for j, e in enumerate(resident):
                self.expert[j] = int(e)

    def occupied(self) -> np.ndarray:
        occ = np.zeros(self.n, dtype=bool)
        for e in self.expert:
            if e != EMPTY:
                occ[e] = True
        return occ

    def slot_of(self, e: int) -> int:
        hit = np.nonzero(self.expert == e)[0]
        return int(hit[0]) if hit.size else EMPTY

    def _victim(self, allowed) -> int:
        empties = [j for j in range(self.S) if self.expert[j] == EMPTY]
        if empties:
            return empties[0]
        cands = [(int(self.stamp[j]), j) for j in range(self.S) if allowed(j)]
        return min(cands)[1] if cands else EMPTY

    def _round_victim(self, need, ran) -> int:
        v = self._victim(lambda j: int(self.expert[j]) not in need)
        if v != EMPTY:
            return v
        done = [j for j in range(self.S) if int(self.expert[j]) in ran]
        return done[0] if done else EMPTY

    def on_demand(self, needed: Sequence[int], tau: int):
        """Load every needed expert that is not present, in rounds; returns
        [(expert, slot, evicted)].  self.rounds lists the experts run in each
        round and self.run_slot maps each needed expert to the slot it ran from."""
        need = set(int(e) for e in needed)
        occ = self.occupied()
        pending = [e for e in sorted(need) if not occ[e]]
        loads, ran = [], set()
        self.rounds, self.run_slot = [], {}
        while True:
            while pending:
                v = self._round_victim(need, ran)
                if v == EMPTY:
                    break
                e = pending.pop(0)
                loads.append((e, v, int(self.expert[v])))
                self.expert[v] = e
            run = sorted(int(self.expert[j]) for j in range(self.S)
                         if int(self.expert[j]) in need and int(self.expert[j]) not in ran)
            if not run and pending:
                raise AssertionError("no progress: no victim and nothing to run")
            for e in run:
                self.run_slot[e] = self.slot_of(e)
            ran |= set(run)
            self.rounds.append(run)
            if not pending:
                break
        for j in range(self.S):
            if int(self.expert[j]) in need:
                self.stamp[j] = tau
        return loads

    def prefetch(self, ordered: Sequence[int], tau: int):
        """Place experts in the given order; returns [(expert, slot, evicted)]."""
        placed = []
        for e in ordered:
            v = self._victim(lambda j: self.stamp[j] < tau)
            if v == EMPTY:
                break
            placed.append((int(e), v, int(self.expert[v])))
            self.expert[v] = int(e)
            self.stamp[v] = tau
        return placed


# --------------------------------------------------------------------------
# routed SwiGLU experts (the FFN the native router executes)
# --------------------------------------------------------------------------


def expert_ffn(Wg: np.ndarray, Wu: np.ndarray, Wd: np.ndarray, x: np.ndarray) -> np.ndarray:
    """Wd (silu(Wg x) * (Wu x)) in fp64 for one token x [D], or row by row for
    the tokens of x [m, D] (one matrix product per weight; every row is the
    one-token value)."""
    x = np.asarray(x, dtype=np.float64)
    Wg, Wu, Wd = (np.asarray(w, dtype=np.float64) for w in (Wg, Wu, Wd))
    if x.ndim == 1:
        return Wd @ (silu(Wg @ x) * (Wu @ x))
    return (silu(x @ Wg.T) * (x @ Wu.T)) @ Wd.T


# --------------------------------------------------------------------------
# weights as the oracle sees them
# --------------------------------------------------------------------------


def q4_decode_expert(gq, gs, uq, us, dq, ds):
    """Values of a 4-bit expert: w = scale * (q - 8), one scale per 32
    consecutive elements along D (gate and up rows, and each down column).
    Returns (gate [I,D], up [I,D], down [D,I]) in fp64."""
    def rows(q, sc):
        return np.repeat(sc.astype(np.float64), 32, axis=1) * (q.astype(np.float64) - 8.0)
    Wd = np.repeat(ds.astype(np.float64), 32, axis=1).T * (dq.astype(np.float64) - 8.0)
    return rows(gq, gs), rows(uq, us), Wd


class OracleWeights:
    """Decoded (fp64-valued) weights of a workload, regenerated from its seeds.

    Expert matrices are kept decoded as fp64 (exact for bf16, fp32 and 4-bit
    storage) in a bounded cache.  ``adapter_override(l) -> (A, B)`` replaces
    the seeded adapters (values, not storage) for special-case tests.
    """

    def __init__(self, cfg, cache_experts: int = 48, adapter_override=None):
        import workload.gen as gen  # seeded inputs only
        self.cfg, self.gen = cfg, gen
        self._cache: Dict[Tuple[int, int], tuple] = {}
        self._order: List[Tuple[int, int]] = []
        self._cap = cache_experts
        self._router: Dict[int, np.ndarray] = {}
        self._adapter: Dict[int, tuple] = {}
        self._proj: Dict[int, np.ndarray] = {}
        self._shared: Dict[Tuple[int, int], tuple] = {}
        self.adapter_override = adapter_override

    def _dec(self, a):
        return decode(a, self.cfg.dtype)

    def router(self, l: int) -> np.ndarray:
        if l not in self._router:
            self._router[l] = decode(self.gen.router_weight(self.cfg, l), self.cfg.dtype)
        return self._router[l]

    def adapter(self, l: int):
        if self.adapter_override is not None:
            return self.adapter_override(l)
        if l not in self._adapter:
            A, B = self.gen.adapter_weights(self.cfg, l)
            self._adapter[l] = (decode(A, self.cfg.dtype), decode(B, self.cfg.dtype))
        return self._adapter[l]

    def proj(self, l: int) -> np.ndarray:
        if l not in self._proj:
            self._proj[l] = decode(self.gen.proj_weight(self.cfg, l), self.cfg.dtype)
        return self._proj[l]

    def expert(self, l: int, e: int):
        key = (self.cfg.expert_layer(l), e)   # tied layers share their expert weights
        if key in self._cache:
            return self._cache[key]
        if self.cfg.codec == "q4":
            w = q4_decode_expert(*self.gen.expert_weights_q4(self.cfg, l, e))
        else:
            w = tuple(self._dec(a) for a in self.gen.expert_weights(self.cfg, l, e))
        self._cache[key] = w
        self._order.append(key)
        if len(self._order) > self._cap:
            del self._cache[self._order.pop(0)]
        return w

    def warm(self, threads: int = 16):
        """Decode every expert of the offload tier ahead of time (in threads)."""
        from concurrent.futures import ThreadPoolExecutor
        self._cap = max(self._cap, self.cfg.host_layers * self.cfg.n + 8)
        with ThreadPoolExecutor(max_workers=threads) as ex:
            list(ex.map(lambda le: self.expert(*le),
                        [(l, e) for l in range(self.cfg.host_layers) for e in range(self.cfg.n)]))

    def shared(self, l: int, j: int):
        key = (l, j)
        if key not in self._shared:
            if self.cfg.codec == "q4":
                self._shared[key] = q4_decode_expert(*self.gen.shared_expert_weights_q4(self.cfg, l, j))
            else:
                self._shared[key] = tuple(self._dec(a) for a in self.gen.shared_expert_weights(self.cfg, l, j))
        return self._shared[key]


# --------------------------------------------------------------------------
# one layer and the decode loop
# --------------------------------------------------------------------------


@dataclass
class LayerStep:
    t: int
    l: int
    tau: int
    x: np.ndarray                 # router input [B, D] (fp64)
    z: np.ndarray                 # router logits [B, n] (fp32 values)
    T: np.ndarray                 # native selection [B, K]
    g: np.ndarray                 # combine weights [B, K] (fp32 values)
    ready: np.ndarray             # per token |T_b cap available| before on-demand loads
    loads: list                   # on-demand loads [(expert, slot, evicted)]
    table_after_demand: np.ndarray
    s: Optional[np.ndarray] = None          # priorities for layer l+1 (fp32 values)
    zhat: Optional[np.ndarray] = None
    P: list = field(default_factory=list)   # prefetch placements for layer l+1 [(expert, slot, evicted)]
    next_table_after_prefetch: Optional[np.ndarray] = None
    next_stamps_after_prefetch: Optional[np.ndarray] = None
    stamps_after_demand: Optional[np.ndarray] = None
    h_out: Optional[np.ndarray] = None      # stored output [B, D] (storage dtype)
    recall: Optional[Dict[int, np.ndarray]] = None   # M -> per token |T_b cap C_M| (prediction made at l-1)
    demand: Optional[Dict[int, int]] = None          # M -> |Top_M(s) minus available(l+1)| at prediction time


def layer_prologue(cfg, W: OracleWeights, l: int, h: np.ndarray):
    """u = h + P_l rms(h) with the stand-in projection, else u = h; x = rms(u)."""
    h = np.asarray(h, dtype=np.float64)
    if cfg.has_proj:
        u = h + rms_normalize(h, cfg.rms_eps) @ W.proj(l).T
    else:
        u = h
    return u, rms_normalize(u, cfg.rms_eps)


def moe_output(cfg, W: OracleWeights, l: int, cache: SlotCache, u, x, T, g):
    """h'_b = u_b + sum_k g_bk FFN_{T_bk}(x_b) (+ shared experts with weight 1),
    accumulated for each token in k order.  An expert must have run from a slot
    (the round structure of the on-demand step decides which slot held it at its
    turn).  FFN_e(x_b) is evaluated for all tokens routed to e at once (one
    matrix product per weight of e, each row the one-token value)."""
    B = x.shape[0]
    ffn = {}
    for e in sorted(set(int(v) for v in np.asarray(T).ravel())):
        if cache.run_slot.get(e, EMPTY) == EMPTY:
            raise AssertionError("executed expert was never resident")
        rows = [b for b in range(B) if e in T[b]]
        Y = expert_ffn(*W.expert(l, e), x[rows])
        for i, b in enumerate(rows):
            ffn[(b, e)] = Y[i]
    shared = [expert_ffn(*W.shared(l, j), x) for j in range(cfg.n_shared)]
    y = np.zeros((B, cfg.D))
    for b in range(B):
        for k in range(T.shape[1]):
            y[b] += g[b, k] * ffn[(b, int(T[b, k]))]
        for j in range(cfg.n_shared):
            y[b] += shared[j][b]
    return u + y


@dataclass
class DecodeResult:
    steps: List[LayerStep]
    ready_recall: float            # mean over target layers 1..L-1 (next-layer coverage)
    layer0_hit_rate: float
    expert_recall: Dict[int, float]
    loads: int
    prefetched: int
    prefetch_used: int
    demand_exceeds: Dict[int, float]
    outputs: List[np.ndarray]      # stored h after the last layer, per token


def run_decode(cfg, W: OracleWeights, h0: np.ndarray, M_max: int, S: Optional[int] = None,
               resident: Optional[Sequence[int]] = None, tokens: Optional[int] = None,
               keep_x: bool = False, policy: str = "adapter") -> DecodeResult:
    """Decode ``tokens`` steps through all L layers.

    M_max < 0: no prediction at all (OFF); M_max == 0: prediction without
    transfers (PRED0); M_max > 0: prediction and budgeted prefetch.
    policy "adapter": priorities from the layer's adapter (SpecPrefetch);
    "naive": the preceding step's experts of the target layer (Naive
    Prefetch, Table 5; no adapter runs and no ExpertRecall is scored).
    ``h0`` holds the stored layer-0 hidden states [tokens, B, D].
    Decode step t, layer l has stamp tau = t L + l + 1.
    """
    L, n, K = cfg.L, cfg.n, cfg.K
    S = cfg.S if S is None else S
    resident = list(range(min(S, n))) if resident is None else list(resident)
    caches = [SlotCache(S, n, resident) for _ in range(L)]
    Ms = sorted(set(m for m in (max(1, K // 2), K, K + 2) if m <= n))
    predicted: List[Optional[Dict[int, np.ndarray]]] = [None] * L
    pending: List[set] = [set() for _ in range(L)]
    steps: List[LayerStep] = []
    outputs = []
    tau = 0
    nT = h0.shape[0] if tokens is None else tokens
    ready_sum, ready_cnt, hit0_sum, hit0_cnt = 0.0, 0, 0.0, 0
    recall_sum = {m: 0.0 for m in Ms}
    recall_cnt = 0
    n_loads = n_pref = n_used = 0
    demand_events = {m: 0 for m in Ms}
    n_events = 0
    prev_route: List[Optional[tuple]] = [None] * L   # (T, g) of each layer at its last step
    for t in range(nT):
        h = decode(h0[t], cfg.dtype)
        for l in range(L):
            tau += 1
            u, x = layer_prologue(cfg, W, l, h)
            T, g, z = route(W.router(l), x, K)
            need = batch_demand(T)
            cache = caches[l]
            occ = cache.occupied()
            ready = np.array([sum(int(occ[e]) for e in T[b]) for b in range(T.shape[0])])
            if l >= 1:
                ready_sum += float(np.sum(ready)) / K
                ready_cnt += T.shape[0]
            else:
                hit0_sum += float(np.sum(ready)) / K
                hit0_cnt += T.shape[0]
            recall = None
            if predicted[l] is not None:
                recall = {m: np.array([len(set(T[b].tolist()) & set(predicted[l][m].tolist()))
                                       for b in range(T.shape[0])]) for m in Ms}
                for m in Ms:
                    recall_sum[m] += float(np.sum(recall[m])) / K
                recall_cnt += T.shape[0]
            n_used += len(pending[l] & set(need))
            pending[l] = set()
            loads = cache.on_demand(need, tau)
            n_loads += len(loads)
            step = LayerStep(t=t, l=l, tau=tau, x=x if keep_x else None, z=z, T=T, g=g, ready=ready,
                             loads=loads, table_after_demand=cache.expert.copy(),
                             stamps_after_demand=cache.stamp.copy(), recall=recall)
            predicted[l] = None
            if l < L - 1 and M_max >= 0:
                nxt = caches[l + 1]
                occ_next = nxt.occupied()
                if policy == "naive":
                    prev = prev_route[l + 1]
                    s = naive_scores(prev[0] if prev else None, prev[1] if prev else None, n)
                    step.s = s
                else:
                    A, Bm = W.adapter(l)
                    zhat, _, s = adapter_scores(A, Bm, x)
                    step.s, step.zhat = s, zhat
                    predicted[l + 1] = {m: candidate_set(s, m) for m in Ms}
                    step.demand = {m: int(sum(1 for e in predicted[l + 1][m] if not occ_next[e])) for m in Ms}
                    for m in Ms:
                        demand_events[m] += int(step.demand[m] > max(M_max, 0))
                    n_events += 1
                if M_max > 0:
                    P = select_prefetch(s, occ_next, M_max)
                    step.P = nxt.prefetch(P, tau)
                    n_pref += len(step.P)
                    pending[l + 1] = set(e for e, _, _ in step.P)
                step.next_table_after_prefetch = nxt.expert.copy()
                step.next_stamps_after_prefetch = nxt.stamp.copy()
            hout = moe_output(cfg, W, l, cache, u, x, T, g)
            step.h_out = encode(hout, cfg.dtype)
            h = decode(step.h_out, cfg.dtype)
            prev_route[l] = (T, g)
            steps.append(step)
        outputs.append(step.h_out)
    return DecodeResult(
        steps=steps,
        ready_recall=ready_sum / ready_cnt if ready_cnt else float("nan"),
        layer0_hit_rate=hit0_sum / hit0_cnt if hit0_cnt else float("nan"),
        expert_recall={m: (recall_sum[m] / recall_cnt if recall_cnt else float("nan")) for m in Ms},
        loads=n_loads, prefetched=n_pref, prefetch_used=n_used,
        demand_exceeds={m: (demand_events[m] / n_events if n_events else float("nan")) for m in Ms},
        outputs=outputs)


def layer_step(cfg, W: OracleWeights, l: int, h_stored: np.ndarray, cache: SlotCache,
               next_cache: Optional[SlotCache], tau: int, M_max: int, policy: str = "adapter",
               next_prev: Optional[tuple] = None):
    """One layer in isolation from given state (the lock-step parity unit).

    Mutates ``cache`` / ``next_cache`` exactly as the decode loop does and
    returns the LayerStep record (x kept).  ``next_prev``: (T, g) of layer
    l+1 at the preceding step, for the "naive" policy.
    """
    K = cfg.K
    u, x = layer_prologue(cfg, W, l, decode(h_stored, cfg.dtype))
    T, g, z = route(W.router(l), x, K)
    need = batch_demand(T)
    occ = cache.occupied()
    ready = np.array([sum(int(occ[e]) for e in T[b]) for b in range(T.shape[0])])
    loads = cache.on_demand(need, tau)
    step = LayerStep(t=-1, l=l, tau=tau, x=x, z=z, T=T, g=g, ready=ready, loads=loads,
                     table_after_demand=cache.expert.copy(), stamps_after_demand=cache.stamp.copy())
    if l < cfg.L - 1 and M_max >= 0:
        if policy == "naive":
            s = naive_scores(next_prev[0] if next_prev else None, next_prev[1] if next_prev else None, cfg.n)
            step.s = s
        else:
            A, Bm = W.adapter(l)
            zhat, _, s = adapter_scores(A, Bm, x)
            step.s, step.zhat = s, zhat
        if M_max > 0 and next_cache is not None:
            P = select_prefetch(s, next_cache.occupied(), M_max)
            step.P = next_cache.prefetch(P, tau)
        if next_cache is not None:
            step.next_table_after_prefetch = next_cache.expert.copy()
            step.next_stamps_after_prefetch = next_cache.stamp.copy()
    step.h_out = encode(moe_output(cfg, W, l, cache, u, x, T, g), cfg.dtype)
    return step
