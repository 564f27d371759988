"""Host-forced failure and race tests of the slot cache (Sec. 3.3, Sec. 3.4).

Every condition is forced from the host, so every kernel still exits normally:
  * a slot copy is made to fail on the host before it is enqueued
    (emoe_test_fail_copy_after): the call must return EMOE_EHIP, leave the
    failing wave's slots empty and every other slot as it was, and the next
    call must compute on correct records;
  * a bounded spin kernel is enqueued before each wave's projections
    (emoe_test_set_wave_delay): a fill that did not wait for the slot's
    completion event would overwrite records still being read, so the
    multi-wave result must still equal the single-wave one bit for bit.
"""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2608_15383_amd import api
from paper_2608_15383_amd._lib import EMOE_EHIP, ExactMoEError
from paper_2608_15383_amd.inputs import OLMOE, make_layer, spread_logits
from tests._gpu import Layer, LazyExperts, assert_close_rel, dims_of

pytestmark = pytest.mark.gpu

T, C = 16, 16


@pytest.fixture(scope="module")
def olmoe16():
    lay = make_layer(OLMOE, T, seed=3)
    layer = Layer(dims_of(OLMOE), lay, T)
    host = torch.empty(layer.bank.numel(), dtype=torch.uint8, pin_memory=True)
    host.copy_(layer.bank)
    torch.cuda.synchronize()
    return lay, layer, host


def _new_cache(layer, host):
    slots = torch.zeros(C * api.expert_record_bytes(layer.dm), dtype=torch.uint8, device="cuda:0")
    return api.Cache(layer.dm, C, slot_bank=slots, host_bank=host), slots


def _active(z):
    return O.group_by_expert(O.topk_experts(z, 8), 64).active


def _slot_records_match_host(cache, slots, host):
    """Every occupied slot holds exactly its expert's record from the host bank."""
    rec = api.expert_record_bytes(cache.dims)
    _, eo, _ = cache.state()
    s_np, h_np = slots.cpu().numpy(), host.numpy()
    for s, e in enumerate(eo.tolist()):
        if e >= 0:
            assert np.array_equal(s_np[s * rec:(s + 1) * rec], h_np[e * rec:(e + 1) * rec]), (s, e)


def test_forward_fill_failure_leaves_no_stale_slot(olmoe16):
    lay, layer, host = olmoe16
    rng = np.random.default_rng(5)
    z1 = spread_logits(T, 64, 8, 48, seed=2)
    z2 = np.ascontiguousarray(z1[:, rng.permutation(64)])   # another 48-expert active set
    cache, slots = _new_cache(layer, host)
    ref = O.SlotCache(64, C, api.expert_record_bytes(layer.dm))
    try:
        layer.forward(lay.h, logits=z1, cache=cache)            # cold call, no failure
        for w in O.plan_waves(_active(z1), ref.resident(), C):
            ref.map_wave(w)
        # The second call's waves: fail the 4th copy of its second wave.
        waves = O.plan_waves(_active(z2), ref.resident(), C)
        assert len(waves) == 3
        _, fills0 = ref.map_wave(waves[0])
        before = (list(ref.expert_of), list(ref.stamp), ref.clock)
        _, fills1 = ref.map_wave(waves[1])
        assert len(fills1) >= 4
        api.test_fail_copy_after(len(fills0) + 3)
        with pytest.raises(ExactMoEError) as ei:
            layer.forward(lay.h, logits=z2, cache=cache)
        assert ei.value.status == EMOE_EHIP
        api.test_fail_copy_after(-1)
        failed = {s for _, s in fills1}
        so, eo, st = cache.state()
        for s in range(C):
            if s in failed:
                assert (eo[s], st[s]) == (-1, -1), s
            else:
                assert (eo[s], st[s]) == (before[0][s], before[1][s]), s
        for e in range(64):
            assert so[e] == (eo.tolist().index(e) if e in eo.tolist() else -1), e
        torch.cuda.synchronize()
        _slot_records_match_host(cache, slots, host)
        # The next call refills what it needs and matches the resident call.
        st_next = api.Stats()
        y = layer.forward(lay.h, logits=z2, cache=cache, stats=st_next)
        assert st_next.misses >= len(failed)
        y_res = layer.forward(lay.h, logits=z2)
        assert np.array_equal(y, y_res)
        ref_y = O.moe_forward(lay.f32("h"), LazyExperts(lay), O.route(lay.f32("h"), None, 8,
                                                                      logits_override=z2))
        assert_close_rel(y, ref_y, "after a failed fill")
        _slot_records_match_host(cache, slots, host)
    finally:
        api.test_fail_copy_after(-1)
        cache.close()


def test_fill_slots_failure_vacates_listed_slots(olmoe16):
    _, layer, host = olmoe16
    cache, slots = _new_cache(layer, host)
    try:
        _, fills = cache.build_slot_map(list(range(8)))
        assert len(fills) == 8
        api.test_fail_copy_after(2)
        with pytest.raises(ExactMoEError) as ei:
            cache.fill_slots(fills)
        assert ei.value.status == EMOE_EHIP
        api.test_fail_copy_after(-1)
        so, eo, st = cache.state()
        for e, s in fills:
            assert so[e] == -1 and eo[s] == -1 and st[s] == -1
        _, again = cache.build_slot_map(list(range(8)))   # all misses again
        assert sorted(again) == sorted(fills)
        cache.fill_slots(again)
        torch.cuda.synchronize()
        _slot_records_match_host(cache, slots, host)
    finally:
        api.test_fail_copy_after(-1)
        cache.close()


@pytest.mark.parametrize("path,sequential", [(api.EMOE_PATH_GEMV, False),
                                             (api.EMOE_PATH_GEMV, True),
                                             (api.EMOE_PATH_MFMA, False)])
def test_slot_reuse_waits_for_the_wave_reading_it(olmoe16, path, sequential):
    """64 active experts through 16 slots: every slot is refilled by each of
    the 4 waves while a 400 us spin holds back the previous wave's reads."""
    lay, layer, host = olmoe16
    z = spread_logits(T, 64, 8, 64, seed=2)
    y1 = layer.forward(lay.h, logits=z, path=path)
    cache, slots = _new_cache(layer, host)
    try:
        cache.set_wave_delay(400)
        for state in ("cold", "warm"):
            st = api.Stats()
            y = layer.forward(lay.h, logits=z, cache=cache, stats=st, path=path,
                              sequential=sequential)
            assert st.waves == 4 and st.misses == (64 if state == "cold" else 48), state
            assert np.array_equal(y, y1), state
        cache.set_wave_delay(0)
        _slot_records_match_host(cache, slots, host)
    finally:
        cache.close()


@pytest.mark.parametrize("distinct,path", [(24, api.EMOE_PATH_GEMV), (40, api.EMOE_PATH_GEMV),
                                           (64, api.EMOE_PATH_GEMV), (64, api.EMOE_PATH_MFMA)])
def test_overlap_waves_equal_single_wave(olmoe16, distinct, path):
    """Waves of C/2 (fills overlapping the previous wave's computation, with a
    200 us spin widening that window): the result equals the resident
    single-wave call bit for bit, and waves, hits, misses and the cache state
    follow the oracle's overlap plan."""
    lay, layer, host = olmoe16
    z = spread_logits(T, 64, 8, distinct, seed=6)
    y1 = layer.forward(lay.h, logits=z, path=path)
    cache, slots = _new_cache(layer, host)
    ref = O.SlotCache(64, C, api.expert_record_bytes(layer.dm))
    try:
        cache.set_wave_overlap(True)
        cache.set_wave_delay(200)
        for call in range(2):
            st = api.Stats()
            y = layer.forward(lay.h, logits=z, cache=cache, stats=st, path=path)
            waves = O.plan_waves(_active(z), ref.resident(), C, overlap=True)
            h0, m0 = ref.hits, ref.misses
            for w in waves:
                ref.map_wave(w)
            assert st.waves == len(waves) and max(len(w) for w in waves) <= C // 2
            assert (st.hits, st.misses) == (ref.hits - h0, ref.misses - m0)
            so, eo, stamp = cache.state()
            assert so.tolist() == ref.slot_of and eo.tolist() == ref.expert_of
            assert stamp.tolist() == ref.stamp
            assert np.array_equal(y, y1), call
        cache.set_wave_delay(0)
        _slot_records_match_host(cache, slots, host)
    finally:
        cache.close()
