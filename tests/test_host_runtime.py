"""Host-side library tests (no GPU): exported symbols, shape checks, record
size, pack/unpack, wave planning and the LRU slot map against the oracle."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle as O
from paper_2608_15383_amd import api
from paper_2608_15383_amd._lib import (lib, EMOE_ESHAPE, EMOE_ECAPACITY, EMOE_EINVAL,
                                       ExactMoEError)
from paper_2608_15383_amd.inputs import make_layer, LayerShape, bf16_bits_to_f32

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_symbols():
    inc = os.path.join(ROOT, "include")
    text = "".join(open(os.path.join(inc, f)).read() for f in sorted(os.listdir(inc)) if f.endswith(".h"))
    return sorted(set(re.findall(r"(?:int32_t|size_t|char\*)\s+(emoe_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    names = declared_symbols()
    assert len(names) >= 18
    h = lib()
    for n in names:
        assert hasattr(h, n), n
    assert set(names) == set(api._lib.SIGNATURES), "binding and header disagree"


def test_dims_validation():
    assert lib().emoe_check_dims(ctypes.byref(api.dims(2048, 1024, 64, 8))) == 0
    for bad in [(100, 1024, 64, 8), (2048, 1000, 64, 8), (2048, 1024, 0, 1), (2048, 1024, 300, 8),
                (2048, 1024, 64, 0), (2048, 1024, 4, 5)]:
        assert lib().emoe_check_dims(ctypes.byref(api.dims(*bad))) == EMOE_ESHAPE, bad
    assert api.expert_record_bytes(api.dims(100, 128, 4, 2)) == 0


def test_record_bytes_is_eq4_without_padding():
    for d, f in [(2048, 1024), (256, 128), (128, 384)]:
        params = 3 * d * f
        assert api.expert_record_bytes(api.dims(d, f, 8, 2)) == params * (4 / 8 + 16 / (128 * 8))
    assert api.expert_record_bytes(api.dims(2048, 1024, 64, 8)) == 3_244_032


def test_workspace_layout_is_disjoint_and_aligned():
    dm = api.dims(2048, 1024, 64, 8)
    for t in (0, 1, 16, 2048):
        L = api.workspace_layout(dm, t)
        fields = [L.logits, L.topk_ids, L.topk_w, L.counts, L.offsets, L.sorted_pairs, L.active,
                  L.n_active, L.tile_offsets, L.act, L.pair_out, L.total]
        assert all(a % 256 == 0 for a in fields)
        assert fields == sorted(fields)
        assert L.pair_out + t * 8 * 2048 * 4 <= L.total
        assert api.workspace_bytes(dm, t) == L.total


def test_pack_unpack_round_trip_and_oracle_codes():
    dm = api.dims(256, 128, 2, 1)
    rng = np.random.default_rng(0)
    q = {n: rng.integers(-8, 8, size=s).astype(np.int8)
         for n, s in [("q_gate", (128, 256)), ("q_up", (128, 256)), ("q_down", (256, 128))]}
    s = {n: rng.integers(0, 2 ** 15, size=sh).astype(np.uint16)
         for n, sh in [("s_gate", (128, 2)), ("s_up", (128, 2)), ("s_down", (256, 1))]}
    rec = api.pack_expert(dm, q["q_gate"], s["s_gate"], q["q_up"], s["s_up"], q["q_down"], s["s_down"])
    assert rec.nbytes == api.expert_record_bytes(dm)
    out = api.unpack_expert(dm, rec)
    for k in q:
        assert np.array_equal(out[k], q[k]), k
    for k in s:
        assert np.array_equal(out[k], s[k]), k
    with pytest.raises(ExactMoEError):
        bad = q["q_down"].copy()
        bad[0, 0] = 9
        api.pack_expert(dm, q["q_gate"], s["s_gate"], q["q_up"], s["s_up"], bad, s["s_down"])


@pytest.mark.parametrize("overlap", [False, True])
def test_plan_waves_and_slot_maps_match_oracle(overlap):
    rng = np.random.default_rng(1)
    for e, c, k in [(64, 16, 8), (8, 2, 2), (16, 5, 3), (32, 32, 4), (16, 1, 1)]:
        dm = api.dims(128, 128, e, k)
        cache = api.Cache(dm, c)
        cache.set_wave_overlap(overlap)
        ref = O.SlotCache(e, c, record_bytes=api.expert_record_bytes(dm))
        stats = api.Stats()
        for step in range(60):
            counts = np.zeros(e, np.int32)
            act = rng.choice(e, size=int(rng.integers(1, e + 1)), replace=False)
            counts[act] = rng.integers(1, 5, size=len(act))
            waves = cache.plan_waves(counts)
            assert waves == O.plan_waves(np.nonzero(counts)[0], ref.resident(), c, overlap)
            for w in waves:
                sm, fills = cache.build_slot_map(w, stats)
                rsm, rfills = ref.map_wave(w)
                assert sm.tolist() == rsm and fills == rfills
            so, eo, st = cache.state()
            assert so.tolist() == ref.slot_of and eo.tolist() == ref.expert_of
            assert st.tolist() == ref.stamp
        assert (stats.hits, stats.misses, stats.h2d_bytes) == (ref.hits, ref.misses, ref.h2d_bytes)
        cache.close()


def test_cache_argument_errors():
    dm = api.dims(128, 128, 8, 2)
    with pytest.raises(ExactMoEError) as ei:
        api.Cache(dm, 1)
    assert ei.value.status == EMOE_ECAPACITY
    with pytest.raises(ExactMoEError) as ei:
        api.Cache(dm, 9)
    assert ei.value.status == EMOE_ECAPACITY
    cache = api.Cache(dm, 2)
    with pytest.raises(ExactMoEError) as ei:
        cache.build_slot_map([0, 1, 2])
    assert ei.value.status == EMOE_ECAPACITY
    with pytest.raises(ExactMoEError) as ei:
        cache.build_slot_map([3, 3])
    assert ei.value.status == EMOE_EINVAL
    with pytest.raises(ExactMoEError) as ei:
        cache.build_slot_map([8])
    assert ei.value.status == EMOE_EINVAL
    assert cache.state()[0].tolist() == [-1] * 8    # failed calls change nothing
    cache.close()


# ------------------------------------------------------------ fused decode plan
def _fused_plan(dm, tokens, cap):
    plan = (ctypes.c_int32 * 9)()
    work = (ctypes.c_int32 * (3 * 1024))()
    rc = lib().emoe_debug_fused_plan(ctypes.byref(dm), tokens, cap, plan, work, 1024)
    if rc != 0:
        return rc, None, None
    keys = ("n_router", "n_gate", "n_work", "ppi", "down_r", "tail_r", "lag", "tail_pairs", "gw")
    p = dict(zip(keys, list(plan)))
    w = np.frombuffer(work, dtype=np.int32)[:3 * p["n_work"]].reshape(-1, 3)
    return rc, p, w


def _check_fused_assignment(d, f, E, k, T, cap):
    """Every (pair, output row block) of the down projection is computed by
    exactly one worker; a worker reads an activation row only from gate/up
    workers of lower index, and a combining worker (last pair of a token)
    reads the token's other outputs only from workers of lower index."""
    dm = api.dims(d, f, E, k)
    rc, p, w = _fused_plan(dm, T, cap)
    if rc != 0:
        assert rc == EMOE_ESHAPE
        return None
    P, n_rb = T * k, d // 16
    chunks = -(-(f // 16) // p["ppi"])
    assert p["n_gate"] == P * chunks
    assert p["n_router"] + p["n_work"] <= min(cap, 1024)
    assert 1 <= p["lag"] <= p["tail_pairs"] <= P
    producer = {}
    for wk, (q, rb0, nu) in enumerate(w):
        blk = p["n_router"] + wk
        if nu == 0:
            continue
        assert 0 <= q < P and 0 <= rb0 and rb0 + nu <= n_rb
        if wk < p["n_gate"]:
            assert q == wk // chunks - p["lag"] and q < P - p["tail_pairs"]
        else:
            assert q >= P - p["tail_pairs"]
        # The activation row of pair q comes from gate/up workers of pair q.
        assert p["n_router"] + (q + 1) * chunks - 1 < blk, (wk, q)
        for r in range(rb0, rb0 + nu):
            assert (q, r) not in producer, (q, r)
            producer[(q, r)] = blk
    assert len(producer) == P * n_rb
    for (q, r), blk in producer.items():
        if q % k == k - 1:
            for j in range(q - (k - 1), q):
                assert producer[(j, r)] < blk, (q, j, r)
    return p


@pytest.mark.parametrize("d,f,E,k", [(2048, 1024, 64, 8), (256, 128, 8, 2), (384, 256, 6, 3),
                                     (256, 384, 1, 1), (128, 128, 200, 8), (2048, 2048, 8, 4),
                                     (512, 1536, 8, 2), (4096, 4096, 64, 8)])
@pytest.mark.parametrize("T", [1, 2, 3, 4])
@pytest.mark.parametrize("cap", [768, 512, 1024, 300])
def test_fused_decode_work_assignment(d, f, E, k, T, cap):
    _check_fused_assignment(d, f, E, k, T, cap)


def test_fused_decode_plan_at_olmoe_shape():
    """One token: 64 one-expert router items, 512 one-pair gate/up items, a
    down lag of two pairs and 192 tail workers for the last three pairs;
    four tokens: 32 router items, items of four row-block pairs and 128 tail
    workers for the last two pairs."""
    p1 = _check_fused_assignment(2048, 1024, 64, 8, 1, 768)
    assert (p1["n_router"], p1["n_gate"], p1["n_work"], p1["ppi"], p1["down_r"], p1["tail_r"],
            p1["lag"], p1["tail_pairs"], p1["gw"]) == (64, 512, 704, 1, 2, 2, 2, 3, 2)
    p4 = _check_fused_assignment(2048, 1024, 64, 8, 4, 768)
    assert (p4["n_router"], p4["n_gate"], p4["n_work"], p4["ppi"], p4["down_r"], p4["tail_r"],
            p4["lag"], p4["tail_pairs"]) == (32, 512, 640, 4, 8, 2, 2, 2)


def test_fused_decode_plan_rejections():
    dm = api.dims(2048, 1024, 64, 8)
    for T in (0, 5):
        assert _fused_plan(dm, T, 768)[0] == EMOE_ESHAPE
    assert _fused_plan(dm, 1, 0)[0] == EMOE_EINVAL
    assert _fused_plan(dm, 1, 100)[0] == EMOE_ESHAPE  # the grid does not fit
    plan = (ctypes.c_int32 * 9)()
    assert lib().emoe_debug_fused_plan(ctypes.byref(dm), 1, 768, None, None, 0) == EMOE_EINVAL
    assert lib().emoe_debug_fused_plan(ctypes.byref(dm), 1, 768, plan, None, 4) == EMOE_EINVAL
