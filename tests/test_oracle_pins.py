"""Pins for the CPU oracle: closed forms, brute force and invariants.

Each test checks the oracle against something other than itself: exact
rational arithmetic, enumeration, a textbook characterisation, or a figure
the paper prints.  A plausible mistake (a dropped term, a wrong index, a
transposed operand, a wrong rounding mode) fails at least one of them.
"""
import itertools
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle as O
from paper_2608_15383_amd.inputs import (f32_to_bf16_bits, bf16_bits_to_f32, make_layer,
                                          LayerShape, zipf_gumbel_logits, spread_logits)
from tests._exact import fraction_of, fp32_round, round_half_even

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def bf16(x):
    return bf16_bits_to_f32(f32_to_bf16_bits(np.asarray(x, np.float32)))


# ---------------------------------------------------------------- quantize
def test_bf16_rounding_is_nearest_even():
    # 1 + 2^-8 is halfway between bf16 1.0 and 1 + 2^-7: ties go to the even mantissa.
    vals = np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 2 ** -8), 1 + 2 ** -9], np.float32)
    got = bf16(vals)
    assert list(got) == [1.0, 1 + 2 ** -6, -1.0, 1.0]


def test_quantize_zero_group_is_zero():
    w = np.zeros((2, 256), np.float32)
    w[1, 128:] = bf16(np.linspace(-1, 1, 128))
    q, s = O.quantize_matrix(w)
    assert s[0, 0] == 0 and s[0, 1] == 0 and s[1, 0] == 0
    assert np.all(q[0] == 0) and np.all(q[1, :128] == 0)
    assert s[1, 1] != 0


def test_quantize_single_nonzero_is_plus_minus_seven():
    w = np.zeros((2, 128), np.float32)
    w[0, 37] = 0.3125
    w[1, 5] = -0.0078125
    q, s = O.quantize_matrix(w)
    assert q[0, 37] == 7 and q[1, 5] == -7
    assert np.count_nonzero(q) == 2
    assert s[0, 0] == np.float16(np.float32(0.3125) / np.float32(7))
    assert s[1, 0] == np.float16(np.float32(0.0078125) / np.float32(7))


def test_quantize_ramp_reproduces_codes():
    c = 2.0 ** -7
    w = np.zeros((1, 128), np.float32)
    w[0, :15] = [c * j for j in range(-7, 8)]
    q, s = O.quantize_matrix(w)
    assert list(q[0, :15]) == list(range(-7, 8))
    assert s[0, 0] == np.float16(c)


def _brute_codes(row):
    """Exact rational quantization of one 128-group: argmin over all 16 codes."""
    amax = max(abs(fraction_of(x)) for x in row)
    if amax == 0:
        return [0] * len(row), Fraction(0)
    s32 = fraction_of(fp32_round(amax / 7))
    out = []
    for x in row:
        r = fraction_of(fp32_round(fraction_of(x) / s32))
        best = None
        for code in range(-8, 8):
            dist = abs(r - code)
            if best is None or dist < best[0] or (dist == best[0] and code % 2 == 0):
                best = (dist, code)
        out.append(best[1])
    return out, s32


def test_quantize_matches_brute_force_argmin():
    rng = np.random.default_rng(11)
    w = bf16(rng.standard_normal((6, 256)).astype(np.float32) * 0.02)
    # force exact .5 quotients: amax = 7*2^-6, entries at (2m+1)/2 * 2^-6
    w[5, :128] = 0
    w[5, 0] = 7 * 2 ** -6
    w[5, 1:8] = [(2 * m + 1) / 2 * 2 ** -6 for m in range(7)]
    w[5, 8:15] = [-(2 * m + 1) / 2 * 2 ** -6 for m in range(7)]
    q, s = O.quantize_matrix(w)
    for i in range(w.shape[0]):
        for g in range(2):
            codes, s32 = _brute_codes(w[i, 128 * g:128 * (g + 1)])
            assert list(q[i, 128 * g:128 * (g + 1)]) == codes, (i, g)
            assert s[i, g] == np.float16(np.float32(float(s32)))
    # half-way quotients went to the even neighbour
    assert list(q[5, 1:8]) == [round_half_even(Fraction(2 * m + 1, 2)) for m in range(7)]
    assert list(q[5, 1:8]) == [0, 2, 2, 4, 4, 6, 6]


def test_quantize_invariants_and_roundtrip_bound():
    rng = np.random.default_rng(5)
    w = bf16(rng.standard_normal((64, 512)).astype(np.float32) * 0.02)
    q, s16 = O.quantize_matrix(w)
    qn, _ = O.quantize_matrix(-w)
    assert np.array_equal(qn, -q)                        # odd symmetry
    assert q.min() >= -7 and q.max() <= 7                # -8 is never produced
    g = q.reshape(64, 4, 128)
    assert np.all(np.max(np.abs(g), axis=2) == 7)        # every nonzero group reaches 7
    wg = w.reshape(64, 4, 128).astype(np.float64)
    s32 = (np.max(np.abs(w.reshape(64, 4, 128)), axis=2) / np.float32(7)).astype(np.float64)
    err32 = np.abs(wg - s32[:, :, None] * g)
    assert np.all(err32 <= s32[:, :, None] * (0.5 + 2 ** -20))
    what = O.dequantize_matrix(q, s16).reshape(64, 4, 128)
    bound = s32 * (0.5 + 7 * 2 ** -11) * (1 + 2 ** -20)
    assert np.all(np.abs(wg - what) <= bound[:, :, None])


def test_quantize_tiny_scale_zeroes_codes_and_huge_scale_is_an_error():
    w = np.zeros((1, 128), np.float32)
    w[0, 0] = 1e-45                                     # fp16 scale underflows to 0
    q, s = O.quantize_matrix(w)
    assert s[0, 0] == 0 and np.all(q == 0)
    w[0, 0] = 1e6                                       # 1e6/7 > 65504
    with pytest.raises(O.ScaleRangeError):
        O.quantize_matrix(w)


def test_eq4_pool_size_matches_paper():
    fig = json.load(open(os.path.join(GOLDEN, "paper_figures.json")))
    m = fig["olmoe_shape"]
    n_params = m["layers"] * m["n_experts"] * 3 * m["d_model"] * m["d_ff"]
    assert abs(n_params / 1e9 - m["routed_params_billion"]) < 0.005
    gib = O.packed_pool_bytes(n_params) / 2 ** 30
    assert abs(gib - fig["packed_pool"]["pool_gib"]) < 0.005


# ---------------------------------------------------------------- router
def test_router_logits_are_correctly_rounded_exact_sums():
    rng = np.random.default_rng(3)
    h = bf16(rng.standard_normal((3, 128)).astype(np.float32))
    wr = bf16(rng.standard_normal((5, 128)).astype(np.float32) * 0.02)
    z = O.router_logits(h, wr)
    assert z.dtype == np.float32
    for t in range(3):
        for e in range(5):
            exact = sum(fraction_of(a) * fraction_of(b) for a, b in zip(h[t], wr[e]))
            assert z[t, e] == fp32_round(exact), (t, e)


def test_router_one_hot_token_reads_one_column():
    wr = bf16(np.random.default_rng(1).standard_normal((6, 128)).astype(np.float32))
    h = np.zeros((1, 128), np.float32)
    h[0, 17] = 2.0
    assert np.array_equal(O.router_logits(h, wr)[0], (2.0 * wr[:, 17]).astype(np.float32))


# ---------------------------------------------------------------- top-k
def test_topk_is_max_sum_subset_by_enumeration():
    rng = np.random.default_rng(7)
    for trial in range(40):
        e, k = 8, 2 + trial % 3
        z = rng.integers(-3, 4, size=(1, e)).astype(np.float32)   # many ties
        ids = O.topk_experts(z, k)[0]
        best = None
        for sub in itertools.combinations(range(e), k):           # lexicographic order
            val = sum(float(z[0, i]) for i in sub)
            if best is None or val > best[0]:
                best = (val, sub)
        assert sorted(ids.tolist()) == list(best[1])
        # rank order: descending logit, lower index first on ties
        keys = [(-float(z[0, i]), int(i)) for i in ids]
        assert keys == sorted(keys)


def test_topk_strictly_decreasing_and_ties():
    z = np.array([[5, 4, 3, 2, 1, 0]], np.float32)
    assert O.topk_experts(z, 3).tolist() == [[0, 1, 2]]
    z = np.array([[1, 1, 1, 1]], np.float32)
    assert O.topk_experts(z, 2).tolist() == [[0, 1]]
    z = np.array([[0, 2, 1, 2]], np.float32)
    assert O.topk_experts(z, 3).tolist() == [[1, 3, 2]]


# ---------------------------------------------------------------- weights
def test_mixture_weights_closed_form():
    rng = np.random.default_rng(9)
    z = rng.standard_normal((5, 8)).astype(np.float32)
    ids = O.topk_experts(z, 3)
    p = O.mixture_weights(z, ids, True)
    for t in range(5):
        sel = [float(z[t, i]) for i in ids[t]]
        m = max(sel)
        den = sum(math.exp(v - m) for v in sel)
        for j in range(3):
            assert abs(p[t, j] - math.exp(sel[j] - m) / den) <= 2e-7
        assert abs(float(np.sum(p[t], dtype=np.float64)) - 1.0) < 1e-6
    pf = O.mixture_weights(z, ids, False)
    for t in range(5):
        full = [math.exp(float(v)) for v in z[t]]
        for j in range(3):
            assert abs(pf[t, j] - full[ids[t, j]] / sum(full)) <= 2e-7


def test_mixture_weights_special_cases():
    z = np.zeros((2, 6), np.float32)
    ids = O.topk_experts(z, 4)
    assert np.allclose(O.mixture_weights(z, ids, True), 0.25, atol=0, rtol=0)
    z = np.random.default_rng(0).standard_normal((3, 6)).astype(np.float32)
    assert np.all(O.mixture_weights(z, O.topk_experts(z, 1), True) == 1.0)
    pk = O.mixture_weights(z, O.topk_experts(z, 6), False)
    assert np.allclose(pk.sum(axis=1), 1.0, atol=1e-6)


# ---------------------------------------------------------------- grouping
def test_grouping_matches_python_stable_sort():
    rng = np.random.default_rng(4)
    for e, t, k in [(8, 16, 2), (64, 37, 8), (5, 1, 3)]:
        ids = np.stack([rng.choice(e, size=k, replace=False) for _ in range(t)]).astype(np.int32)
        gr = O.group_by_expert(ids, e)
        flat = ids.reshape(-1).tolist()
        assert gr.sorted_pairs.tolist() == sorted(range(len(flat)), key=lambda pi: flat[pi])
        assert gr.counts.tolist() == [flat.count(x) for x in range(e)]
        assert gr.offsets[0] == 0 and gr.offsets[-1] == t * k
        assert gr.active.tolist() == sorted(set(flat))
        for x in range(e):
            seg = gr.sorted_pairs[gr.offsets[x]:gr.offsets[x + 1]]
            assert all(flat[pi] == x for pi in seg)


# ---------------------------------------------------------------- waves
def test_waves_partition_active_set():
    rng = np.random.default_rng(2)
    for _ in range(50):
        e = 64
        c = int(rng.integers(8, 33))
        active = np.sort(rng.choice(e, size=int(rng.integers(1, 65)), replace=False))
        resident = rng.choice(e, size=int(rng.integers(0, c + 1)), replace=False)
        waves = O.plan_waves(active, resident, c)
        assert len(waves) == -(-len(active) // c)
        flat = [x for w in waves for x in w]
        assert sorted(flat) == active.tolist() and len(flat) == len(set(flat))
        assert all(1 <= len(w) <= c for w in waves)
        res = set(resident.tolist())
        n_res = sum(1 for x in flat if x in res)
        assert all(x in res for x in flat[:n_res])        # resident experts first


def test_overlap_waves_partition_active_set():
    """Overlap reading: a set that fits stays one wave; a larger one is cut into
    the fewest chunks of at most max(1, C // 2), resident experts first."""
    rng = np.random.default_rng(21)
    for _ in range(200):
        e = 64
        c = int(rng.integers(1, 33))
        active = np.sort(rng.choice(e, size=int(rng.integers(1, 65)), replace=False))
        resident = rng.choice(e, size=int(rng.integers(0, c + 1)), replace=False)
        waves = O.plan_waves(active, resident, c, overlap=True)
        size = c if len(active) <= c else max(1, c // 2)
        assert len(waves) == -(-len(active) // size)
        flat = [x for w in waves for x in w]
        assert flat == [x for w in O.plan_waves(active, resident, size) for x in w]
        assert sorted(flat) == active.tolist() and len(flat) == len(set(flat))
        assert all(1 <= len(w) <= size for w in waves)
    assert O.plan_waves(range(10), [], 4, overlap=True) == [[0, 1], [2, 3], [4, 5], [6, 7], [8, 9]]
    assert O.plan_waves(range(4), [], 4, overlap=True) == [[0, 1, 2, 3]]


def _previous_wave_slots_refilled(capacity, calls, rng, overlap):
    """Run random layer calls through a SlotCache; count fills that land in a
    slot the call's previous wave used (such a fill must wait for that wave)."""
    e = 64
    cache = O.SlotCache(e, capacity)
    clashes = 0
    for _ in range(calls):
        active = np.sort(rng.choice(e, size=int(rng.integers(1, e + 1)), replace=False))
        prev_slots = set()
        for w in O.plan_waves(active, cache.resident(), capacity, overlap=overlap):
            sm, fills = cache.map_wave(w)
            clashes += sum(1 for _, s in fills if s in prev_slots)
            prev_slots = {sm[x] for x in w}
    return clashes


def test_overlap_waves_never_refill_the_previous_waves_slots():
    """With overlap waves and C >= 2, no miss of a wave takes a slot that the
    call's previous wave used, under the unchanged LRU rule; with full-size
    waves such refills do occur (so the check has teeth)."""
    rng = np.random.default_rng(22)
    for c in (2, 3, 5, 8, 16, 32):
        assert _previous_wave_slots_refilled(c, 60, rng, overlap=True) == 0, c
    assert _previous_wave_slots_refilled(16, 20, rng, overlap=False) > 0


# ---------------------------------------------------------------- LRU
def _stack_distances(seq):
    """Mattson stack distance of each reference (inf for a first reference)."""
    out, stack = [], []
    for x in seq:
        if x in stack:
            out.append(stack.index(x) + 1)
            stack.remove(x)
        else:
            out.append(math.inf)
        stack.insert(0, x)
    return out


def test_lru_single_expert_waves_hit_iff_stack_distance_within_capacity():
    rng = np.random.default_rng(8)
    for c in (1, 2, 3, 5):
        seq = rng.integers(0, 9, size=200).tolist()
        cache = O.SlotCache(9, c, record_bytes=10)
        hits = []
        for x in seq:
            before = cache.hits
            cache.map_wave([x])
            hits.append(cache.hits > before)
        dist = _stack_distances(seq)
        assert hits == [d <= c for d in dist]
        assert cache.h2d_bytes == 10 * cache.misses


def test_lru_worked_example():
    cache = O.SlotCache(4, 2, record_bytes=1)
    assert cache.map_wave([0])[1] == [(0, 0)]
    assert cache.map_wave([1])[1] == [(1, 1)]
    sm, fills = cache.map_wave([2])          # evicts expert 0 (older stamp), slot 0
    assert fills == [(2, 0)] and sm == [-1, -1, 0, -1]
    sm, fills = cache.map_wave([1, 3])       # 1 hits and is protected; 3 takes slot 0
    assert fills == [(3, 0)] and sm == [-1, 1, -1, 0]
    assert (cache.hits, cache.misses) == (1, 4)


def test_lru_multi_expert_wave_invariants():
    rng = np.random.default_rng(12)
    e, c = 16, 6
    cache = O.SlotCache(e, c)
    last_use = {}
    for step in range(300):
        wave = sorted(rng.choice(e, size=int(rng.integers(1, c + 1)), replace=False).tolist())
        before = dict((x, s) for x, s in enumerate(cache.slot_of) if s >= 0)
        h0, m0 = cache.hits, cache.misses
        sm, fills = cache.map_wave(wave)
        assert cache.hits - h0 == sum(1 for x in wave if x in before)
        assert cache.misses - m0 == len(fills)
        slots = [sm[x] for x in wave]
        assert len(set(slots)) == len(slots) and all(0 <= s < c for s in slots)
        assert all(sm[x] == -1 for x in range(e) if x not in wave)
        hit_slots = {before[x] for x in wave if x in before}
        evicted = [x for x in before if cache.slot_of[x] < 0]
        for x in evicted:
            assert before[x] not in hit_slots                   # protected slots survive
            others = [y for y in before if y not in wave and y not in evicted]
            assert all(last_use[x] <= last_use[y] for y in others)  # LRU victim
        for x in wave:
            last_use[x] = step


def test_table1_h2d_is_misses_times_record_size():
    """Table 1's H2D column equals (1 - hit) x accesses x the packed record size (within 1.5%)."""
    fig = json.load(open(os.path.join(GOLDEN, "paper_figures.json")))
    m = fig["olmoe_shape"]
    params_per_expert = 3 * m["d_model"] * m["d_ff"]
    record = O.packed_pool_bytes(params_per_expert)
    accesses = fig["capacity_table"]["generated_tokens"] * m["layers"] * m["top_k"]
    for row in fig["capacity_table"]["rows"]:
        pred = (1 - row["hit_rate_pct"] / 100) * accesses * record / 2 ** 30
        assert abs(pred / row["h2d_gib"] - 1) < 0.015, row


# ---------------------------------------------------------------- expert MLP / forward
def _scalar_forward(h, experts, k, wr, renorm=True):
    """Eq. 1-2 written with scalar loops (tiny sizes only)."""
    t_count, d = h.shape
    e_count = wr.shape[0]
    y = [[0.0] * d for _ in range(t_count)]
    for t in range(t_count):
        z = []
        for e in range(e_count):
            acc = Fraction(0)
            for i in range(d):
                acc += fraction_of(h[t, i]) * fraction_of(wr[e, i])
            z.append(float(fp32_round(acc)))
        order = sorted(range(e_count), key=lambda e: (-z[e], e))[:k]
        mx = max(z)
        if renorm:
            den = sum(math.exp(z[e] - mx) for e in order)
        else:
            den = sum(math.exp(v - mx) for v in z)
        for e in order:
            p = float(np.float32(math.exp(z[e] - mx) / den))
            ex = experts[e]
            wg, wu, wd = ex.w_hat("gate"), ex.w_hat("up"), ex.w_hat("down")
            f = wg.shape[0]
            a = []
            for n in range(f):
                g = sum(wg[n, i] * float(h[t, i]) for i in range(d))
                u = sum(wu[n, i] * float(h[t, i]) for i in range(d))
                a.append(g / (1 + math.exp(-g)) * u)
            for i in range(d):
                y[t][i] += p * sum(wd[i, n] * a[n] for n in range(f))
    return np.array(y)


def _tiny_layer(e=4, k=2, t=3, d=256, f=128, seed=21):
    lay = make_layer(LayerShape(d, f, e, k), t, seed)
    experts = [O.quantize_expert(lay.f32("w_gate")[i], lay.f32("w_up")[i], lay.f32("w_down")[i])
               for i in range(e)]
    return lay, experts


def test_forward_matches_scalar_loops():
    lay, experts = _tiny_layer(t=2)
    h, wr = lay.f32("h"), lay.f32("w_router")
    r = O.route(h, wr, 2)
    y = O.moe_forward(h, experts, r)
    ref = _scalar_forward(h, experts, 2, wr)
    assert np.allclose(y, ref, rtol=1e-10, atol=1e-12)


def test_single_expert_top1_is_plain_swiglu_mlp():
    lay, experts = _tiny_layer(e=1, k=1, t=3)
    h, wr = lay.f32("h"), lay.f32("w_router")
    r = O.route(h, wr, 1)
    assert np.all(r.weights == 1.0) and np.all(r.ids == 0)
    y = O.moe_forward(h, experts, r)
    ex = experts[0]
    for t in range(3):
        g = ex.w_hat("gate") @ h[t].astype(np.float64)
        u = ex.w_hat("up") @ h[t].astype(np.float64)
        assert np.allclose(y[t], ex.w_hat("down") @ (g * u / (1 + np.exp(-g))), rtol=1e-12)


def test_all_experts_selected_is_dense_softmax_mixture():
    lay, experts = _tiny_layer(e=4, k=4, t=3)
    h, wr = lay.f32("h"), lay.f32("w_router")
    r = O.route(h, wr, 4, renormalize=True)
    y = O.moe_forward(h, experts, r)
    z = O.router_logits(h, wr).astype(np.float64)
    for t in range(3):
        gate = np.exp(z[t] - z[t].max())
        gate /= gate.sum()
        dense = sum(gate[e] * O.expert_mlp(experts[e], h[t]) for e in range(4))
        assert np.allclose(y[t], dense, rtol=1e-6, atol=1e-9)


def test_zero_tokens_and_permutation_equivariance():
    lay, experts = _tiny_layer(t=4)
    h, wr = lay.f32("h"), lay.f32("w_router")
    y0 = O.moe_forward(np.zeros_like(h), experts, O.route(np.zeros_like(h), wr, 2))
    assert np.all(y0 == 0)
    perm = np.array([2, 0, 3, 1])
    y = O.moe_forward(h, experts, O.route(h, wr, 2))
    yp = O.moe_forward(h[perm], experts, O.route(h[perm], wr, 2))
    assert np.allclose(yp, y[perm], rtol=1e-12, atol=0)


def test_waves_sum_to_single_wave_result():
    lay, experts = _tiny_layer(e=4, k=2, t=4)
    h, wr = lay.f32("h"), lay.f32("w_router")
    r = O.route(h, wr, 2)
    full = O.moe_forward(h, experts, r)
    gr = O.group_by_expert(r.ids, 4)
    waves = O.plan_waves(gr.active, [], 2)
    parts = sum(O.moe_forward(h, experts, r, wave=w) for w in waves)
    assert np.allclose(parts, full, rtol=1e-12, atol=1e-15)
    pairs = O.pair_outputs(h, experts, r, range(8))
    comb = np.array([sum(float(r.weights[t, j]) * pairs[t * 2 + j] for j in range(2)) for t in range(4)])
    assert np.allclose(comb, full, rtol=1e-12, atol=1e-15)


def test_synthetic_logit_generators_have_the_stated_structure():
    z = spread_logits(16, 64, 8, 40, seed=2)
    ids = O.topk_experts(z, 8)
    assert len(set(ids.reshape(-1).tolist())) == 40
    rng = np.random.default_rng(0)
    perm = rng.permutation(64)
    zz = zipf_gumbel_logits(4096, 64, 1.1, perm, rng)
    top1 = np.argmax(zz, axis=1)
    freq = np.bincount(top1, minlength=64)
    assert freq[perm[0]] == freq.max()                 # rank-1 expert is the most popular
