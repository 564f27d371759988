"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Integer results (codes, scales, top-k ids, grouping, slot maps, counters) are
compared bit for bit; layer outputs within max|err| <= 2e-2 * max|ref|; a
multi-wave call must equal the single-wave call bit for bit.
"""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2608_15383_amd import api
from paper_2608_15383_amd._lib import EMOE_ERANGE, EMOE_ESHAPE, ExactMoEError
from paper_2608_15383_amd.inputs import (LayerInputs, LayerShape, OLMOE, TINY, bf16_bits_to_f32,
                                          f32_to_bf16_bits, make_layer, spread_logits)
from tests._gpu import TOL, Layer, LazyExperts, dev, host_bits, quantize, rel_err

pytestmark = pytest.mark.gpu

GEMV, MFMA, MIXED = api.EMOE_PATH_GEMV, api.EMOE_PATH_MFMA, api.EMOE_PATH_MIXED


def dims_of(shape: LayerShape):
    return api.dims(shape.d_model, shape.d_ff, shape.n_experts, shape.top_k)


def oracle_y(lay, experts, k, logits=None, tokens=None, renormalize=True):
    h = lay.f32("h")
    r = O.route(h, lay.f32("w_router"), k, renormalize, logits)
    return O.moe_forward(h, experts, r, tokens=tokens), r


def assert_close(y, ref, label=""):
    mx, mean = rel_err(y, ref)
    print(f"{label}: max|err|/max|ref| = {mx:.3e}, mean rel = {mean:.3e}", flush=True)
    assert mx <= TOL, (label, mx)


# ------------------------------------------------------------------ quantization
def _check_codes(dm, lay, bank, experts):
    rec_bytes = api.expert_record_bytes(dm)
    host = bank.cpu().numpy()
    for i, e in enumerate(experts):
        got = api.unpack_expert(dm, host[i * rec_bytes:(i + 1) * rec_bytes])
        for name, w in (("gate", lay.w_gate[e]), ("up", lay.w_up[e]), ("down", lay.w_down[e])):
            q, s = O.quantize_matrix(bf16_bits_to_f32(w))
            assert np.array_equal(got["q_" + name], q), (e, name)
            assert np.array_equal(got["s_" + name], s.view(np.uint16)), (e, name)


def test_quantize_bit_exact_with_special_groups():
    dm = dims_of(TINY)
    lay = make_layer(TINY, 4, seed=0)
    g = bf16_bits_to_f32(lay.w_gate).copy()
    g[0, 0, :128] = 0.0                                   # zero group
    g[0, 1, :128] = 0.0
    g[0, 1, 77] = -0.3125                                 # single nonzero
    g[0, 2, :128] = 0.0
    g[0, 2, :15] = [2.0 ** -7 * j for j in range(-7, 8)]  # ramp
    g[0, 3, :128] = 0.0
    g[0, 3, 0] = 7 * 2 ** -6                              # half-way quotients
    g[0, 3, 1:8] = [(2 * m + 1) / 2 * 2 ** -6 for m in range(7)]
    g[1, 0, :128] = 0.0
    g[1, 0, 5] = 2.0 ** -126                              # scale underflows FP16
    g[1, 1, :128] *= 1e-4                                 # subnormal FP16 scales
    lay.w_gate = f32_to_bf16_bits(g)
    bank = quantize(dm, lay)
    _check_codes(dm, lay, bank, range(TINY.n_experts))


def test_quantize_bit_exact_olmoe_shape():
    lay = make_layer(OLMOE, 1, seed=5, n_experts_drawn=2)
    dm = dims_of(OLMOE)
    bank = quantize(dm, lay)
    _check_codes(dm, lay, bank, [0, 1])


def test_quantize_scale_overflow_is_an_error():
    lay = make_layer(TINY, 1, seed=0, n_experts_drawn=1)
    w = bf16_bits_to_f32(lay.w_down).copy()
    w[0, 3, 7] = 1.0e6
    lay.w_down = f32_to_bf16_bits(w)
    with pytest.raises(ExactMoEError) as ei:
        quantize(dims_of(TINY), lay)
    assert ei.value.status == EMOE_ERANGE


# ------------------------------------------------------------------ routing
def _route(dm, h_bits, wr_bits, logits=None, renormalize=True):
    t, e, k = h_bits.shape[0], dm.n_experts, dm.top_k
    i32 = dict(dtype=torch.int32, device="cuda:0")
    out = dict(logits=torch.zeros((max(t, 1), e), dtype=torch.float32, device="cuda:0"),
               ids=torch.zeros(max(t * k, 1), **i32), w=torch.zeros(max(t * k, 1), dtype=torch.float32,
                                                                    device="cuda:0"),
               counts=torch.zeros(e, **i32), offsets=torch.zeros(e + 1, **i32),
               sorted=torch.zeros(max(t * k, 1), **i32), active=torch.zeros(e, **i32),
               n_active=torch.zeros(1, **i32))
    lo = None if logits is None else dev(np.asarray(logits, np.float32))
    api.route(dm, t, dev(h_bits), dev(wr_bits), lo, renormalize, out["logits"], out["ids"],
              out["w"], out["counts"], out["offsets"], out["sorted"], out["active"], out["n_active"])
    torch.cuda.synchronize()
    return {k_: v.cpu().numpy() for k_, v in out.items()}


def _check_route(dm, got, h, wr, logits=None, renormalize=True):
    t, k = h.shape[0], dm.top_k
    r = O.route(bf16_bits_to_f32(h), bf16_bits_to_f32(wr), k, renormalize, logits)
    if logits is None:
        assert np.array_equal(got["logits"][:t].view(np.uint32), r.logits.view(np.uint32))
    assert np.array_equal(got["ids"][:t * k].reshape(t, k), r.ids)
    ulp = np.abs(got["w"][:t * k].view(np.int32).astype(np.int64)
                 - r.weights.reshape(-1).view(np.int32).astype(np.int64))
    assert ulp.max(initial=0) <= 4
    gr = O.group_by_expert(r.ids, dm.n_experts)
    assert np.array_equal(got["counts"], gr.counts)
    assert np.array_equal(got["offsets"], gr.offsets)
    assert np.array_equal(got["sorted"][:t * k], gr.sorted_pairs)
    assert got["n_active"][0] == len(gr.active)
    assert np.array_equal(got["active"][:len(gr.active)], gr.active)


@pytest.mark.parametrize("shape,tokens", [(TINY, 16), (OLMOE, 1), (OLMOE, 16), (OLMOE, 2048),
                                          (LayerShape(384, 128, 200, 6), 37)])
def test_route_and_grouping_bit_exact(shape, tokens):
    lay = make_layer(shape, tokens, seed=7, n_experts_drawn=0)
    dm = dims_of(shape)
    got = _route(dm, lay.h, lay.w_router)
    _check_route(dm, got, lay.h, lay.w_router)


def test_route_override_ties_and_no_renormalize():
    dm = api.dims(256, 128, 16, 4)
    rng = np.random.default_rng(3)
    z = rng.integers(-2, 3, size=(50, 16)).astype(np.float32)   # many exact ties
    z[3] = -0.0
    z[4, ::2] = 0.0
    lay = make_layer(LayerShape(256, 128, 16, 4), 50, seed=3, n_experts_drawn=0)
    for renorm in (True, False):
        got = _route(dm, lay.h, lay.w_router, logits=z, renormalize=renorm)
        _check_route(dm, got, lay.h, lay.w_router, logits=z, renormalize=renorm)


def test_route_zero_tokens():
    dm = dims_of(TINY)
    lay = make_layer(TINY, 0, seed=1, n_experts_drawn=0)
    got = _route(dm, lay.h, lay.w_router)
    assert got["counts"].sum() == 0 and got["n_active"][0] == 0 and np.all(got["offsets"] == 0)


# ------------------------------------------------------------------ layer, small shapes
@pytest.mark.parametrize("path", [GEMV, MFMA])
def test_forward_tiny_config(path):
    lay = make_layer(TINY, 16, seed=0)
    layer = Layer(dims_of(TINY), lay, 16)
    y = layer.forward(lay.h, path=path)
    ref, r = oracle_y(lay, LazyExperts(lay), TINY.top_k)
    assert_close(y, ref, f"tiny path={path}")
    po = layer.pair_out(32, mfma=path == MFMA)
    assert_close(po, O.pair_outputs(lay.f32("h"), LazyExperts(lay), r, range(32)), "tiny pairs")


@pytest.mark.parametrize("shape,tokens", [(LayerShape(384, 256, 6, 3), 7),
                                          (LayerShape(256, 384, 1, 1), 5),
                                          (LayerShape(128, 128, 4, 4), 9),
                                          (LayerShape(640, 128, 12, 2), 70)])
@pytest.mark.parametrize("path", [GEMV, MFMA])
def test_forward_ragged_and_degenerate_shapes(shape, tokens, path):
    lay = make_layer(shape, tokens, seed=11)
    layer = Layer(dims_of(shape), lay, tokens)
    y = layer.forward(lay.h, path=path)
    ref, _ = oracle_y(lay, LazyExperts(lay), shape.top_k)
    assert_close(y, ref, f"{shape} T={tokens} path={path}")


def _random_cases(n, seed, max_tokens=80):
    """Seeded layer shapes within the documented limits: d_model, d_ff in
    128 .. 1024, 1 .. 96 experts, top_k up to 16, 1 .. max_tokens tokens, and a
    slot capacity between top_k and E."""
    rng = np.random.default_rng(seed)
    cases = []
    for _ in range(n):
        d, f = 128 * int(rng.integers(1, 9)), 128 * int(rng.integers(1, 9))
        e = int(rng.integers(1, 97))
        k = int(rng.integers(1, min(e, 16) + 1))
        t = int(rng.integers(1, max_tokens + 1))
        cases.append((LayerShape(d, f, e, k), t, int(rng.integers(k, e + 1))))
    return cases


@pytest.mark.parametrize("shape,tokens,capacity",
                         _random_cases(10, 41) + _random_cases(6, 43, max_tokens=4)
                         + _random_cases(6, 107, max_tokens=300))
def test_random_shapes_every_path(shape, tokens, capacity):
    """Each path against the oracle on seeded random shapes; through a cache of
    `capacity` slots (several waves when the call touches more experts) each
    path equals its resident call bit for bit, and so does the sequential path.
    With at most 4 tokens the resident default call is the fused decode launch
    where it fits."""
    lay = make_layer(shape, tokens, seed=shape.d_model + shape.n_experts + tokens)
    layer = Layer(dims_of(shape), lay, tokens)
    ref, _ = oracle_y(lay, LazyExperts(lay), shape.top_k)
    resident = {}
    for path in (GEMV, MFMA, api.EMOE_PATH_AUTO):
        st = api.Stats()
        resident[path] = layer.forward(lay.h, path=path, stats=st)
        assert_close(resident[path], ref, f"{shape} T={tokens} path={path}")
    k, f, d = shape.top_k, shape.d_ff, shape.d_model
    fused = (tokens <= 4 and tokens * k <= 32 and f <= 2048 and d <= 4096
             and tokens * d * 2 <= 32768 and tokens * k * f // 2 <= 32 * 2048)
    assert (st.kernel_launches == 1) == fused
    dm = layer.dm
    slots = torch.zeros(capacity * api.expert_record_bytes(dm), dtype=torch.uint8, device="cuda:0")
    cache = api.Cache(dm, capacity, slot_bank=slots, host_bank=_host_bank(layer))
    resident[MIXED] = layer.forward(lay.h, path=MIXED)
    for path in (GEMV, MFMA, MIXED):
        assert np.array_equal(layer.forward(lay.h, path=path, cache=cache), resident[path]), path
    assert np.array_equal(layer.forward(lay.h, path=GEMV, cache=cache, sequential=True),
                          resident[GEMV])
    cache.close()


@pytest.mark.parametrize("shape", [LayerShape(8192, 256, 3, 2), LayerShape(256, 8192, 3, 2)])
def test_mfma_at_its_group_limit(shape):
    """64 input groups (d_model or d_ff = 8192), the most the MFMA path's
    per-tile bias table holds, against the oracle on a ragged token count."""
    lay = make_layer(shape, 70, seed=17)
    layer = Layer(dims_of(shape), lay, 70)
    y = layer.forward(lay.h, path=MFMA)
    ref, _ = oracle_y(lay, LazyExperts(lay), shape.top_k)
    assert_close(y, ref, f"{shape} MFMA")


def test_mfma_past_its_group_limit_is_a_shape_error():
    """65 groups: an explicit MFMA request fails with EMOE_ESHAPE; the automatic
    choice takes the GEMV path and still matches the oracle."""
    shape = LayerShape(8320, 128, 2, 1)
    lay = make_layer(shape, 9, seed=18)
    layer = Layer(dims_of(shape), lay, 9)
    with pytest.raises(ExactMoEError) as ei:
        layer.forward(lay.h, path=MFMA)
    assert ei.value.status == EMOE_ESHAPE
    y = layer.forward(lay.h)
    ref, _ = oracle_y(lay, LazyExperts(lay), shape.top_k)
    assert_close(y, ref, f"{shape} automatic path")


@pytest.mark.parametrize("shape,tokens", [(LayerShape(128, 128, 200, 5), 300),
                                          (LayerShape(128, 128, 64, 8), 2048),
                                          (LayerShape(128, 128, 64, 4), 700),
                                          (LayerShape(128, 128, 96, 16), 101)])
def test_forward_grouping_of_large_calls_bit_exact(shape, tokens):
    """Calls above 1024 pairs group over many workgroups (per-chunk counts, then
    a stable placement); the arrays must equal the oracle's grouping.  With
    top_k dividing 64 the top-k launch also counts the chunks (64 / top_k
    tokens per workgroup; the last chunk ragged here), otherwise a separate
    launch does.  The
    MFMA row-tile prefix sum counts the experts on the MFMA kernels: all of
    them on the MFMA path, those with at least EMOE_MIXED_MFMA_ROWS rows on the
    mixed path, none on the GEMV path."""
    lay = make_layer(shape, tokens, seed=5)
    layer = Layer(dims_of(shape), lay, tokens)
    E, P = shape.n_experts, tokens * shape.top_k
    r = O.route(lay.f32("h"), lay.f32("w_router"), shape.top_k)
    gr = O.group_by_expert(r.ids, E)
    for path, min_rows in ((GEMV, P + 1), (MFMA, 1), (MIXED, api.EMOE_MIXED_MFMA_ROWS)):
        layer.forward(lay.h, path=path)
        assert np.array_equal(layer.ws_array("topk_ids", P, np.int32).reshape(tokens, -1), r.ids)
        assert np.array_equal(layer.ws_array("counts", E, np.int32), gr.counts)
        assert np.array_equal(layer.ws_array("offsets", E + 1, np.int32), gr.offsets)
        assert np.array_equal(layer.ws_array("sorted_pairs", P, np.int32), gr.sorted_pairs)
        assert layer.ws_array("n_active", 1, np.int32)[0] == len(gr.active)
        assert np.array_equal(layer.ws_array("active", len(gr.active), np.int32), gr.active)
        per = np.where(gr.counts >= min_rows, -(-gr.counts // 64), 0)
        tiles = np.concatenate([[0], np.cumsum(per)])
        assert np.array_equal(layer.ws_array("tile_offsets", E + 1, np.int32), tiles), path


@pytest.mark.parametrize("path", [GEMV, MFMA])
def test_token_group_sizes_1_to_128(path):
    """Token-group sizes 1..128 routed to one expert (the paper's kernel-test range)."""
    shape = LayerShape(256, 256, 4, 1)
    lay = make_layer(shape, 128, seed=13)
    layer = Layer(dims_of(shape), lay, 128)
    experts = LazyExperts(lay)
    for m in (1, 2, 3, 15, 16, 17, 63, 64, 65, 127, 128):
        z = np.zeros((128, 4), np.float32)
        z[:, 0] = 1.0
        z[:m, 0] = 0.0
        z[:m, 2] = 1.0                    # the first m tokens go to expert 2
        y = layer.forward(lay.h, logits=z, path=path)
        ref, _ = oracle_y(lay, experts, 1, logits=z)
        assert_close(y, ref, f"group size {m} path={path}")


def test_zero_tokens_forward():
    lay = make_layer(TINY, 0, seed=0)
    layer = Layer(dims_of(TINY), lay, 1)
    st = api.Stats()
    h = torch.zeros((0, 256), dtype=torch.int16, device="cuda:0")
    api.moe_forward(layer.cache, h, layer.wr, torch.empty_like(h), layer.ws, stats=st)
    assert st.layer_calls == 1 and st.kernel_launches == 0


# ------------------------------------------------------------------ OLMoE shapes
@pytest.fixture(scope="module")
def olmoe():
    lay = make_layer(OLMOE, 2048, seed=3)
    layer = Layer(dims_of(OLMOE), lay, 2048)
    return lay, layer, LazyExperts(lay)


def _sub(lay, tokens):
    return LayerInputs(lay.shape, lay.w_gate, lay.w_up, lay.w_down, lay.w_router, lay.h[:tokens])


def test_decode_token_full_size(olmoe):
    lay, layer, experts = olmoe
    for t in (0, 1, 2):
        one = _sub(lay, 2048)
        one.h = lay.h[t:t + 1]
        y = layer.forward(one.h)
        ref, _ = oracle_y(one, experts, 8)
        assert_close(y, ref, f"decode token {t}")


def _host_bank(layer):
    host = torch.empty(layer.bank.numel(), dtype=torch.uint8, pin_memory=True)
    host.copy_(layer.bank)
    torch.cuda.synchronize()
    return host


@pytest.mark.parametrize("distinct", [40, 48, 56, 64])
def test_multi_wave_equals_single_wave(olmoe, distinct):
    """16 tokens touching `distinct` experts through a 16-slot cache (3-4 waves)."""
    lay, layer, experts = olmoe
    dm = layer.dm
    sub = _sub(lay, 16)
    z = spread_logits(16, 64, 8, distinct, seed=2)
    y1 = layer.forward(sub.h, logits=z)
    po1 = layer.ws_array("pair_out", 128 * 2048, np.float32)

    host = _host_bank(layer)
    slots = torch.zeros(16 * api.expert_record_bytes(dm), dtype=torch.uint8, device="cuda:0")
    cache = api.Cache(dm, 16, slot_bank=slots, host_bank=host)
    ref_cache = O.SlotCache(64, 16, api.expert_record_bytes(dm))
    for call in range(2):   # cold, then warm with the same active set
        st = api.Stats()
        y = layer.forward(sub.h, logits=z, cache=cache, stats=st)
        assert np.array_equal(y, y1)
        assert np.array_equal(layer.ws_array("pair_out", 128 * 2048, np.float32), po1)
        ids = O.topk_experts(z, 8)
        active = O.group_by_expert(ids, 64).active
        waves = O.plan_waves(active, ref_cache.resident(), 16)
        h0, m0 = ref_cache.hits, ref_cache.misses
        for w in waves:
            ref_cache.map_wave(w)
        assert st.waves == len(waves) == -(-distinct // 16)
        assert (st.hits, st.misses) == (ref_cache.hits - h0, ref_cache.misses - m0)
        assert st.h2d_bytes == st.misses * api.expert_record_bytes(dm)
        assert st.grouped_gemm_calls == 2 * len(waves)
        so, eo, _ = cache.state()
        assert so.tolist() == ref_cache.slot_of and eo.tolist() == ref_cache.expert_of
    ys = layer.forward(sub.h, logits=z, cache=cache, sequential=True)
    assert np.array_equal(ys, y1)
    ref, _ = oracle_y(sub, experts, 8, logits=z)
    assert_close(y1, ref, f"16 tokens, {distinct} experts")
    cache.close()


def test_skewed_multi_wave_with_hot_experts(olmoe):
    """64 tokens under Zipf(1.1) routing through a 16-slot cache: popular
    experts hold dozens of rows, which the GEMV kernels split into row chunks
    across workgroups; the multi-wave result equals the single-wave one bit
    for bit and matches the oracle."""
    from paper_2608_15383_amd.inputs import zipf_gumbel_logits
    lay, layer, experts = olmoe
    dm = layer.dm
    sub = _sub(lay, 64)
    rng = np.random.default_rng(11)
    z = zipf_gumbel_logits(64, 64, 1.1, rng.permutation(64), rng).astype(np.float32)
    counts = np.bincount(O.topk_experts(z, 8).ravel(), minlength=64)
    assert counts.max() > 16          # several row chunks for one expert
    y1 = layer.forward(sub.h, logits=z, path=GEMV)
    host = _host_bank(layer)
    slots = torch.zeros(16 * api.expert_record_bytes(dm), dtype=torch.uint8, device="cuda:0")
    cache = api.Cache(dm, 16, slot_bank=slots, host_bank=host)
    for call in range(2):
        st = api.Stats()
        y = layer.forward(sub.h, logits=z, cache=cache, stats=st, path=GEMV)
        assert st.waves >= 3
        assert np.array_equal(y, y1)
    ys = layer.forward(sub.h, logits=z, cache=cache, sequential=True, path=GEMV)
    assert np.array_equal(ys, y1)
    cache.close()
    ref, _ = oracle_y(_sub(lay, 8), experts, 8, logits=z[:8])
    assert_close(y1[:8], ref, "Zipf batch, first 8 tokens")


def test_mfma_multi_wave_equals_single_wave(olmoe):
    """The MFMA path through a 16-slot cache (4 waves over all 64 experts, 256
    tokens): every wave's grouped launches skip the row tiles of experts
    outside the wave, and the result equals the single-wave call bit for bit."""
    lay, layer, experts = olmoe
    dm = layer.dm
    sub = _sub(lay, 256)
    y1 = layer.forward(sub.h, path=MFMA)
    host = _host_bank(layer)
    slots = torch.zeros(16 * api.expert_record_bytes(dm), dtype=torch.uint8, device="cuda:0")
    cache = api.Cache(dm, 16, slot_bank=slots, host_bank=host)
    st = api.Stats()
    y = layer.forward(sub.h, cache=cache, stats=st, path=MFMA)
    cache.close()
    assert st.waves == 4
    assert np.array_equal(y, y1)
    ref, _ = oracle_y(sub, experts, 8, tokens=[0, 255])
    assert_close(y[[0, 255]], ref, "MFMA multi-wave")
    experts.cache.clear()


def test_mixed_path_takes_each_expert_by_its_rows(olmoe):
    """128 tokens under Zipf(1.1) routing: experts with at least
    EMOE_MIXED_MFMA_ROWS rows run on the MFMA kernels, the rest on the GEMV
    kernels.  Each pair's fp32 output equals, bit for bit, its own path's:
    rounded to bf16 it is the all-MFMA call's output for the first kind, and
    it is the all-GEMV call's output for the second.  A 16-slot cache
    (several waves) and the sequential path give the same bits; y matches
    the oracle, and AUTO (the all-MFMA call here) equals the MFMA path."""
    from paper_2608_15383_amd.inputs import zipf_gumbel_logits
    lay, layer, experts = olmoe
    dm = layer.dm
    T, k, d = 128, 8, 2048
    sub = _sub(lay, T)
    rng = np.random.default_rng(12)
    z = zipf_gumbel_logits(T, 64, 1.1, rng.permutation(64), rng).astype(np.float32)
    ids = O.topk_experts(z, k)
    counts = np.bincount(ids.ravel(), minlength=64)
    big = counts >= api.EMOE_MIXED_MFMA_ROWS
    assert big.sum() >= 4 and ((counts > 0) & ~big).sum() >= 4   # both kinds present
    y_gemv = layer.forward(sub.h, logits=z, path=GEMV)
    po_gemv = layer.pair_out(T * k, mfma=False)
    y_mfma = layer.forward(sub.h, logits=z, path=MFMA)
    po_mfma = layer.ws_array("pair_out", T * k * d, np.uint16).reshape(T * k, d)
    st = api.Stats()
    y = layer.forward(sub.h, logits=z, path=MIXED, stats=st)
    # top-k and grouping, the row sums of h, both kinds of both projections, combine
    assert st.kernel_launches == 2 + 1 + 4 + 1
    po = layer.pair_out(T * k, mfma=False)
    on_mfma = big[ids.ravel()]
    assert np.array_equal(f32_to_bf16_bits(po[on_mfma]), po_mfma[on_mfma])
    assert np.array_equal(po[~on_mfma], po_gemv[~on_mfma])
    assert np.array_equal(layer.forward(sub.h, logits=z), y_mfma)     # AUTO
    host = _host_bank(layer)
    slots = torch.zeros(16 * api.expert_record_bytes(dm), dtype=torch.uint8, device="cuda:0")
    cache = api.Cache(dm, 16, slot_bank=slots, host_bank=host)
    st = api.Stats()
    assert np.array_equal(layer.forward(sub.h, logits=z, path=MIXED, cache=cache, stats=st), y)
    assert st.waves >= 3
    assert np.array_equal(layer.forward(sub.h, logits=z, path=MIXED, cache=cache,
                                        sequential=True), y)
    cache.close()
    rows = [int(np.argmax(on_mfma.reshape(T, k).any(1))), int(np.argmin(on_mfma.reshape(T, k).all(1)))]
    ref, _ = oracle_y(sub, experts, k, logits=z, tokens=rows)
    assert_close(y[rows], ref, "mixed path")
    assert_close(y, y_gemv.astype(np.float64), "mixed vs GEMV path")
    experts.cache.clear()


def test_mixed_path_without_large_experts_is_the_gemv_path():
    """Below EMOE_MIXED_MFMA_ROWS rows per expert the mixed path runs the GEMV
    kernels only: the same bits as the GEMV path."""
    shape = LayerShape(512, 256, 16, 4)
    lay = make_layer(shape, 12, seed=5)
    layer = Layer(dims_of(shape), lay, 12)
    y = layer.forward(lay.h, path=MIXED)
    assert np.array_equal(y, layer.forward(lay.h, path=GEMV))
    ref, _ = oracle_y(lay, LazyExperts(lay), 4)
    assert_close(y, ref, "mixed, small experts")


def test_global_to_slot_map_permutation(olmoe):
    """Experts placed in permuted slots give the identical output (map preflight)."""
    lay, layer, _ = olmoe
    dm = layer.dm
    sub = _sub(lay, 16)
    y_res = layer.forward(sub.h)
    host = _host_bank(layer)
    slots = torch.zeros(64 * api.expert_record_bytes(dm), dtype=torch.uint8, device="cuda:0")
    cache = api.Cache(dm, 64, slot_bank=slots, host_bank=host)
    order = np.random.default_rng(0).permutation(64)
    for chunk in np.array_split(order, 8):   # warm the slots in a scrambled order
        sm, fills = cache.build_slot_map(sorted(chunk.tolist()))
        cache.fill_slots(fills)
    torch.cuda.synchronize()
    so, _, _ = cache.state()
    assert sorted(so.tolist()) == list(range(64)) and so.tolist() != list(range(64))
    y = layer.forward(sub.h, cache=cache)
    assert np.array_equal(y, y_res)
    cache.close()


def test_prefill_full_size_sampled(olmoe):
    lay, layer, experts = olmoe
    y = layer.forward(lay.h)                       # AUTO -> MFMA at 16,384 pairs
    r = O.route(lay.f32("h"), lay.f32("w_router"), 8)
    gr = O.group_by_expert(r.ids, 64)
    assert np.array_equal(layer.ws_array("counts", 64, np.int32), gr.counts)
    assert np.array_equal(layer.ws_array("sorted_pairs", 16384, np.int32), gr.sorted_pairs)
    po = layer.pair_out(16384, mfma=True)
    for e in (int(gr.active[0]), int(gr.active[31]), int(gr.active[-1])):
        seg = gr.sorted_pairs[gr.offsets[e]:gr.offsets[e + 1]]
        pick = np.concatenate([seg[:3], seg[63:66], seg[-3:]])  # head, tile edge, ragged tail
        assert_close(po[pick], O.pair_outputs(lay.f32("h"), experts, r, pick), f"prefill expert {e}")
    toks = [0, 1000, 2047]
    ref = O.moe_forward(lay.f32("h"), experts, r, tokens=toks)
    assert_close(y[toks], ref, "prefill tokens")
    experts.cache.clear()


def test_prefill_full_size_whole_expert_and_every_row(olmoe):
    """T = 2048 at full size: every pair of the busiest expert (all of its
    64-row tiles, the ragged last one included) against the oracle, and all
    2048 output rows against the GEMV path's."""
    lay, layer, experts = olmoe
    y = layer.forward(lay.h, path=MFMA)
    r = O.route(lay.f32("h"), lay.f32("w_router"), 8)
    gr = O.group_by_expert(r.ids, 64)
    e = int(np.argmax(gr.counts))
    seg = gr.sorted_pairs[gr.offsets[e]:gr.offsets[e + 1]]
    assert len(seg) > 4 * 64
    po = layer.pair_out(16384, mfma=True)
    assert_close(po[seg], O.pair_outputs(lay.f32("h"), experts, r, seg), f"all pairs of expert {e}")
    y_g = layer.forward(lay.h, path=GEMV)
    assert_close(y, y_g.astype(np.float64), "T=2048 MFMA vs GEMV, every row")
    experts.cache.clear()


def test_prefill_paths_agree(olmoe):
    lay, layer, experts = olmoe
    sub = _sub(lay, 256)
    y_g = layer.forward(sub.h, path=GEMV)
    y_m = layer.forward(sub.h, path=MFMA)
    ref, _ = oracle_y(sub, experts, 8, tokens=[0, 128, 255])
    assert_close(y_g[[0, 128, 255]], ref, "256 tokens GEMV")
    assert_close(y_m[[0, 128, 255]], ref, "256 tokens MFMA")
    assert_close(y_m, y_g.astype(np.float64), "MFMA vs GEMV")
    experts.cache.clear()


# ------------------------------------------------------------------ fused decode launch
@pytest.mark.parametrize("shape,tokens", [(TINY, 1), (TINY, 4), (LayerShape(384, 256, 6, 3), 3),
                                          (LayerShape(256, 384, 1, 1), 1),
                                          (LayerShape(128, 128, 200, 8), 4), (OLMOE, 2),
                                          (OLMOE, 4), (LayerShape(2048, 2048, 8, 4), 1),
                                          (LayerShape(2048, 2048, 8, 4), 4),
                                          (LayerShape(512, 1536, 8, 2), 3)])
def test_fused_decode_matches_unfused_bitwise(shape, tokens):
    """The single-launch decode layer equals the per-kernel path bit for bit:
    one- and several-pair items, one and two router items per expert quad, and
    two and four down input groups per wavefront (d_ff above 1024)."""
    lay = make_layer(shape, tokens, seed=17)
    layer = Layer(dims_of(shape), lay, tokens)
    st = api.Stats()
    y_f = layer.forward(lay.h, stats=st)
    # Fused when it fits: the token rows in 32 KB of LDS, at most four down
    # input groups per wavefront, the handed-over words in the cache.
    fits = (shape.d_ff <= 2048 and shape.d_model <= 4096 and tokens * shape.d_model * 2 <= 32768
            and tokens * shape.top_k * shape.d_ff // 2 <= 32 * 2048)
    assert (st.kernel_launches == 1) == fits
    po_f = layer.ws_array("pair_out", tokens * shape.top_k * shape.d_model, np.float32)
    y_s = layer.forward(lay.h, sequential=True)          # per-expert launches, unfused kernels
    po_s = layer.ws_array("pair_out", tokens * shape.top_k * shape.d_model, np.float32)
    assert np.array_equal(y_f, y_s) and np.array_equal(po_f, po_s)
    ref, _ = oracle_y(lay, LazyExperts(lay), shape.top_k)
    assert_close(y_f, ref, f"fused {shape} T={tokens}")
    assert layer.cache.sync_timeouts() == 0


def test_fused_decode_repeated_calls_and_override():
    """Back-to-back fused launches reuse the cache's counters; override logits work."""
    lay = make_layer(OLMOE, 4, seed=19)
    layer = Layer(dims_of(OLMOE), lay, 4)
    experts = LazyExperts(lay)
    z = spread_logits(4, 64, 8, 32, seed=5)
    for rep in range(3):
        for t in (1, 2, 4):
            sub = _sub(lay, t)
            y = layer.forward(sub.h, logits=z[:t])
            ys = layer.forward(sub.h, logits=z[:t], sequential=True)
            assert np.array_equal(y, ys), (rep, t)
    ref, _ = oracle_y(_sub(lay, 4), experts, 8, logits=z)
    assert_close(y, ref, "fused with override")
    assert layer.cache.sync_timeouts() == 0


@pytest.mark.parametrize("shape,tokens", [(OLMOE, 1), (OLMOE, 4), (LayerShape(384, 256, 6, 3), 3),
                                          (TINY, 16)])
def test_forward_without_renormalization(shape, tokens):
    """Mixture weights as the softmax over all E logits (renormalize = 0): every
    path against the oracle, and the default call (the fused decode launch at up
    to 4 tokens) bit for bit against the per-kernel path."""
    lay = make_layer(shape, tokens, seed=37)
    layer = Layer(dims_of(shape), lay, tokens)
    ref, _ = oracle_y(lay, LazyExperts(lay), shape.top_k, renormalize=False)
    for path in (GEMV, MFMA, MIXED, api.EMOE_PATH_AUTO):
        y = layer.forward(lay.h, path=path, renormalize=False)
        assert_close(y, ref, f"{shape} T={tokens} path={path} without renormalization")
    y_seq = layer.forward(lay.h, renormalize=False, sequential=True)
    assert np.array_equal(layer.forward(lay.h, renormalize=False), y_seq)


@pytest.mark.parametrize("shape,tokens", [(TINY, 1), (OLMOE, 1), (OLMOE, 4)])
def test_fused_decode_waits_that_give_up(shape, tokens):
    """Bounded waits of the fused decode launch, forced from the host to give up
    (emoe_test_set_decode_waits: the readers wait for a tag no writer uses, 8
    polls each): every workgroup still exits, every output is NaN and the
    timeouts are counted.  With the normal waits restored, the next calls equal
    the per-kernel path bit for bit and count no timeout."""
    lay = make_layer(shape, tokens, seed=31)
    layer = Layer(dims_of(shape), lay, tokens)
    y_ref = layer.forward(lay.h, sequential=True)
    layer.cache.set_decode_waits(8, unmatched=True)
    st = api.Stats()
    y_bad = layer.forward(lay.h, stats=st)
    assert st.kernel_launches == 1
    assert np.isnan(y_bad).all()
    gave_up = layer.cache.sync_timeouts()
    assert gave_up > 0
    layer.cache.set_decode_waits()
    for _ in range(3):
        assert np.array_equal(layer.forward(lay.h), y_ref)
    assert layer.cache.sync_timeouts() == gave_up


@pytest.mark.parametrize("tokens,path,launches,override",
                         [(1, api.EMOE_PATH_AUTO, 1, False), (2, api.EMOE_PATH_AUTO, 1, False),
                          (3, api.EMOE_PATH_AUTO, 1, True),
                          (8, GEMV, None, False), (48, MFMA, None, False)])
def test_resident_layer_replays_from_a_captured_graph(tokens, path, launches, override):
    """A fully resident layer call captured into a HIP graph replays correctly,
    replay after replay: the fused decode launch (1-3 tokens) takes its hand-over
    epoch from device memory, not from its launch arguments.  Eager calls run
    between the replays; every replay equals the eager call on the same input
    bit for bit."""
    lay = make_layer(OLMOE, tokens, seed=23)
    layer = Layer(dims_of(OLMOE), lay, tokens)
    rng = np.random.default_rng(29)
    hs = [f32_to_bf16_bits(rng.standard_normal((tokens, OLMOE.d_model)).astype(np.float32))
          for _ in range(3)]
    h = dev(hs[0])
    y = torch.empty_like(h)
    z = spread_logits(tokens, 64, 8, 16, seed=5) if override else None
    lo = dev(z) if override else None
    st = api.Stats()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):   # first call outside the capture
        api.moe_forward(layer.cache, h, layer.wr, y, layer.ws, logits_override=lo, path=path,
                        stats=st)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    assert launches is None or st.kernel_launches == launches
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        api.moe_forward(layer.cache, h, layer.wr, y, layer.ws, logits_override=lo, path=path)
    torch.cuda.synchronize()
    for rep in range(3):
        for i, hb in enumerate(hs):
            expect = layer.forward(hb, logits=z, path=path)
            h.copy_(dev(hb))
            graph.replay()
            torch.cuda.synchronize()
            got = bf16_bits_to_f32(host_bits(y))
            assert np.array_equal(got, expect), (rep, i)
    last = LayerInputs(lay.shape, lay.w_gate, lay.w_up, lay.w_down, lay.w_router, hs[-1])
    ref, _ = oracle_y(last, LazyExperts(lay), OLMOE.top_k, logits=z)
    assert_close(got, ref, f"graph replay T={tokens}")
    assert layer.cache.sync_timeouts() == 0
