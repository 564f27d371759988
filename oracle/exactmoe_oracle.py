"""Plain CPU oracle for the ExactMoE fused W4A16 routed-expert layer.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this module; only the test-suite, the package smoke check and the
benchmark's CPU-baseline leg use it.  It shares no code with the HIP library:
it never sees the packed record layout, only plain arrays.

Every function follows the paper ("Every Expert Counts: ExactMoE for
Memory-Efficient W4A16 Inference") and says which passage it restates.
Floating point is fp64 unless the paper fixes a precision; the readings taken
where the paper is silent are listed in each docstring.  Every function here
is pinned by the CPU tests (closed forms, brute force, invariants); none is
"parity unpinned".

Arrays:  bf16 tensors are passed as float32 arrays holding the bf16 values
exactly (bf16 is a subset of fp32).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

GROUP = 128  # quantization group along the input dimension (Sec. 3.2)


# --------------------------------------------------------------------------
# Sec. 3.2, Eq. 3: symmetric group-128 INT4 quantization
# --------------------------------------------------------------------------
class ScaleRangeError(ValueError):
    """A group's scale max|W|/7 does not fit in an FP16 scale (Sec. 3.2 stores FP16 scales)."""


def quantize_matrix(w: np.ndarray):
    """Quantize one expert matrix W[N, K] per (row, 128-wide input group).

    Sec. 3.2, Eq. 3: s = max_{j in g} |W_ij| / 7, q = clip(round(W/s), -8, 7),
    reference W_hat = s * q; an all-zero group gets s = 0 and q = 0.
    Scales are stored as FP16 (Sec. 3.2, Sec. 3.3).

    Readings where the paper is silent:
      * the absmax and the division are done in fp32 (IEEE, round-to-nearest);
      * "round" is round-half-to-even;
      * q is computed from the fp32 scale, then the scale is rounded to FP16
        (the text computes s and q first and packs FP16 scales afterwards);
      * a scale that underflows to FP16 zero also zeroes its codes, so that
        W_hat = s16 * q stays the reference;
      * a scale that overflows FP16 is an error.
    Returns (q int8 [N, K], s16 float16 [N, K/128]).
    """
    w = np.asarray(w, dtype=np.float32)
    n, k = w.shape
    if k % GROUP:
        raise ValueError("input dimension must be a multiple of 128")
    g = w.reshape(n, k // GROUP, GROUP)
    amax = np.max(np.abs(g), axis=2)                      # fp32, exact
    s32 = (amax / np.float32(7.0)).astype(np.float32)      # IEEE fp32 divide
    with np.errstate(divide="ignore", invalid="ignore"):
        ratio = (g / s32[:, :, None]).astype(np.float32)   # IEEE fp32 divide
    q = np.clip(np.rint(ratio), -8, 7)
    q = np.where(amax[:, :, None] == 0, 0, q)              # zero group (Sec. 3.2)
    with np.errstate(over="ignore"):
        s16 = s32.astype(np.float16)                       # RNE to FP16
    if not np.all(np.isfinite(s16)):
        raise ScaleRangeError("group scale overflows FP16")
    q = np.where((s16 == 0)[:, :, None], 0, q)
    return q.reshape(n, k).astype(np.int8), s16


def dequantize_matrix(q: np.ndarray, s16: np.ndarray) -> np.ndarray:
    """W_hat = s * q (Sec. 3.2), in fp64; the product is exact."""
    n, k = q.shape
    s = np.repeat(s16.astype(np.float64), GROUP, axis=1)
    return s * q.astype(np.float64)


@dataclass
class QuantizedExpert:
    """One routed expert's quantized projections (Sec. 3.2, Eq. 2 shapes).

    gate, up: [d_ff, d_model] (N = d_ff, K = d_model); down: [d_model, d_ff].
    """
    q_gate: np.ndarray
    s_gate: np.ndarray
    q_up: np.ndarray
    s_up: np.ndarray
    q_down: np.ndarray
    s_down: np.ndarray
    _hat: dict = field(default_factory=dict, repr=False)

    def w_hat(self, name: str) -> np.ndarray:
        if name not in self._hat:
            q = getattr(self, "q_" + name)
            s = getattr(self, "s_" + name)
            self._hat[name] = dequantize_matrix(q, s)
        return self._hat[name]


def quantize_expert(w_gate, w_up, w_down) -> QuantizedExpert:
    """Quantize the three projections of one expert independently (Sec. 3.2)."""
    qg, sg = quantize_matrix(w_gate)
    qu, su = quantize_matrix(w_up)
    qd, sd = quantize_matrix(w_down)
    return QuantizedExpert(qg, sg, qu, su, qd, sd)


def packed_pool_bytes(n_params: int) -> float:
    """Eq. 4: M_W4 ~= P_expert * (4/8 + 16/(128*8)) bytes."""
    return n_params * (4 / 8 + 16 / (128 * 8))


# --------------------------------------------------------------------------
# Sec. 3.1, Eq. 1: router logits, top-k, mixture weights
# --------------------------------------------------------------------------
def router_logits(h: np.ndarray, w_router: np.ndarray) -> np.ndarray:
    """z_t = W_r h_t (Eq. 1) for all tokens: h [T, d], W_r [E, d] -> z [T, E].

    The paper keeps the router in BF16 without fixing the logit precision.
    Reading: bf16 inputs, products and sum in fp64, one rounding to fp32.
    """
    z = np.asarray(h, np.float64) @ np.asarray(w_router, np.float64).T
    return z.astype(np.float32)


def topk_experts(z: np.ndarray, k: int) -> np.ndarray:
    """S_t = TopK(z_t, k) (Eq. 1), listed in rank order.

    Rank order is logit descending; equal logits rank the lower expert index
    first (the paper gives no tie rule).  z [T, E] fp32 -> ids [T, k] int32.
    """
    t_count, e_count = z.shape
    ids = np.empty((t_count, k), dtype=np.int32)
    idx = np.arange(e_count)
    for t in range(t_count):
        order = np.lexsort((idx, -z[t].astype(np.float64)))  # primary: -z
        ids[t] = order[:k]
    return ids


def mixture_weights(z: np.ndarray, ids: np.ndarray, renormalize: bool) -> np.ndarray:
    """Router-derived mixture weights p_{t,e} (Sec. 3.1).

    The paper only says "router-derived".  Reading (the workload's stated
    rule): softmax over all E logits, keep the selected experts' values and,
    when renormalize is set, divide them by their sum.  fp64, stored fp32.
    """
    z64 = z.astype(np.float64)
    ex = np.exp(z64 - z64.max(axis=1, keepdims=True))
    probs = ex / ex.sum(axis=1, keepdims=True)
    p = np.take_along_axis(probs, ids.astype(np.int64), axis=1)
    if renormalize:
        p = p / p.sum(axis=1, keepdims=True)
    return p.astype(np.float32)


# --------------------------------------------------------------------------
# Fig. 1 / Sec. 3.4: grouping tokens by selected expert
# --------------------------------------------------------------------------
@dataclass
class Grouping:
    counts: np.ndarray        # [E] pairs routed to each expert
    offsets: np.ndarray       # [E+1] exclusive prefix sum of counts
    sorted_pairs: np.ndarray  # [P] pair ids pi = t*k + j, grouped by expert
    active: np.ndarray        # ascending ids of experts with counts > 0


def group_by_expert(ids: np.ndarray, n_experts: int) -> Grouping:
    """Group the T*k (token, rank) pairs by their selected expert.

    Pair index pi = t*k + j with j the rank.  Within one expert the pairs stay
    in ascending pi order (a stable sort); the paper only states that tokens
    are grouped by selected expert.
    """
    flat = ids.reshape(-1).astype(np.int64)
    counts = np.bincount(flat, minlength=n_experts).astype(np.int32)
    offsets = np.zeros(n_experts + 1, dtype=np.int32)
    offsets[1:] = np.cumsum(counts)
    sorted_pairs = np.argsort(flat, kind="stable").astype(np.int32)
    active = np.nonzero(counts)[0].astype(np.int32)
    return Grouping(counts, offsets, sorted_pairs, active)


# --------------------------------------------------------------------------
# Sec. 3.4: waves of at most C experts
# --------------------------------------------------------------------------
def plan_waves(active, resident, capacity: int, overlap: bool = False):
    """Partition the active expert set into waves of at most C experts.

    The paper fixes only the size bound.  Reading: experts already resident
    at layer entry come first (ascending id), then the others (ascending id),
    cut into consecutive chunks of C.  Returns a list of lists of expert ids.

    overlap (a second reading, for filling slots while the previous wave
    computes): Sec. 3.3 lets a slot be refilled once its preceding
    computation has finished, so a wave whose misses all land in slots the
    previous wave does not use can be filled while that wave computes.  When
    the active set does not fit in the C slots at once, the chunks then hold
    at most max(1, C // 2) experts; under the LRU rule of SlotCache the
    previous wave's slots carry the newest stamps, so with at most C // 2
    experts per wave every miss takes a slot outside the previous wave.  A set
    that fits stays one wave of up to C.
    """
    resident = set(int(e) for e in resident)
    act = [int(e) for e in sorted(int(x) for x in active)]
    order = [e for e in act if e in resident] + [e for e in act if e not in resident]
    size = capacity
    if overlap and len(order) > capacity:
        size = max(1, capacity // 2)
    return [order[i:i + size] for i in range(0, len(order), size)]


# --------------------------------------------------------------------------
# Sec. 3.3: per-layer slot cache with LRU replacement
# --------------------------------------------------------------------------
class SlotCache:
    """C-slot cache with a global-to-slot map and one recency stamp per slot.

    Sec. 3.3: resident wave experts are hits; missing ones replace the
    least-recently-used slots that the current wave does not protect.
    Readings: the clock ticks once per wave and stamps every slot the wave
    uses; the victim is the unprotected slot with the smallest (stamp, slot
    index), where an empty slot has stamp -1; misses are placed in ascending
    expert id order; the cache starts empty.  When C = E every expert is
    preloaded into slot e and no accounting happens (Sec. 3.3).
    """

    def __init__(self, n_experts: int, capacity: int, record_bytes: int = 0):
        self.n_experts = n_experts
        self.capacity = capacity
        self.record_bytes = record_bytes
        self.slot_of = [-1] * n_experts
        self.expert_of = [-1] * capacity
        self.stamp = [-1] * capacity
        self.clock = 0
        self.hits = 0
        self.misses = 0
        self.h2d_bytes = 0
        self.resident_all = False

    def preload_all(self):
        if self.capacity != self.n_experts:
            raise ValueError("full residency needs C = E")
        self.slot_of = list(range(self.n_experts))
        self.expert_of = list(range(self.n_experts))
        self.resident_all = True

    def resident(self):
        return [e for e in range(self.n_experts) if self.slot_of[e] >= 0]

    def map_wave(self, wave):
        """Return (slot_map [E] with -1 for experts outside the wave, fills)."""
        if self.resident_all:
            slot_map = [-1] * self.n_experts
            for e in wave:
                slot_map[e] = e
            return slot_map, []
        self.clock += 1
        protected = set()
        for e in wave:
            s = self.slot_of[e]
            if s >= 0:
                self.hits += 1
                protected.add(s)
                self.stamp[s] = self.clock
        fills = []
        for e in sorted(wave):
            if self.slot_of[e] >= 0:
                continue
            free = [s for s in range(self.capacity) if s not in protected]
            victim = min(free, key=lambda s: (self.stamp[s], s))
            old = self.expert_of[victim]
            if old >= 0:
                self.slot_of[old] = -1
            self.expert_of[victim] = e
            self.slot_of[e] = victim
            self.stamp[victim] = self.clock
            protected.add(victim)
            self.misses += 1
            self.h2d_bytes += self.record_bytes
            fills.append((e, victim))
        slot_map = [-1] * self.n_experts
        for e in wave:
            slot_map[e] = self.slot_of[e]
        return slot_map, fills


# --------------------------------------------------------------------------
# Sec. 3.1, Eq. 2: the sparse block output
# --------------------------------------------------------------------------
def silu(x: np.ndarray) -> np.ndarray:
    """phi of Eq. 2; SwiGLU experts use SiLU, x / (1 + exp(-x))."""
    return x / (1.0 + np.exp(-x))


def expert_mlp(expert: QuantizedExpert, h_t: np.ndarray) -> np.ndarray:
    """W_d [phi(W_g h) * (W_u h)] on the dequantized weights (Eq. 2), fp64."""
    h = np.asarray(h_t, np.float64)
    g = expert.w_hat("gate") @ h
    u = expert.w_hat("up") @ h
    return expert.w_hat("down") @ (silu(g) * u)


@dataclass
class Routing:
    logits: np.ndarray   # [T, E] fp32
    ids: np.ndarray      # [T, k] int32, rank order
    weights: np.ndarray  # [T, k] fp32


def route(h, w_router, k: int, renormalize: bool = True, logits_override=None) -> Routing:
    """Eq. 1 plus the mixture weights; an explicit logit matrix may replace W_r h."""
    if logits_override is not None:
        z = np.asarray(logits_override, np.float32)
    else:
        z = router_logits(h, w_router)
    ids = topk_experts(z, k)
    return Routing(z, ids, mixture_weights(z, ids, renormalize))


def moe_forward(h, experts, routing: Routing, tokens=None, wave=None) -> np.ndarray:
    """y_t = sum_{e in S_t} p_{t,e} * expert_e(h_t) (Eq. 2), fp64.

    `tokens` restricts the computation to those token rows (for sampled checks
    at full size).  `wave` restricts the sum to experts in that set without
    renormalizing the weights: Sec. 3.4 recovers Eq. 2 by adding the disjoint
    wave contributions.  The sum runs in rank order.
    """
    h = np.asarray(h, np.float64)
    rows = range(h.shape[0]) if tokens is None else tokens
    wave_set = None if wave is None else set(int(e) for e in wave)
    d = h.shape[1]
    y = np.zeros((len(rows), d), dtype=np.float64)
    for r, t in enumerate(rows):
        for j in range(routing.ids.shape[1]):
            e = int(routing.ids[t, j])
            if wave_set is not None and e not in wave_set:
                continue
            y[r] += float(routing.weights[t, j]) * expert_mlp(experts[e], h[t])
    return y


def pair_outputs(h, experts, routing: Routing, pairs) -> np.ndarray:
    """o_pi = expert_{id_pi}(h_t) for the listed pair ids pi = t*k + j (Eq. 2 summands)."""
    k = routing.ids.shape[1]
    h = np.asarray(h, np.float64)
    out = np.zeros((len(pairs), h.shape[1]))
    for r, pi in enumerate(pairs):
        t, j = divmod(int(pi), k)
        out[r] = expert_mlp(experts[int(routing.ids[t, j])], h[t])
    return out
