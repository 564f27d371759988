"""The no-allocation layer call (emoe_moe_forward_noalloc) through the C ABI.

Its output must equal emoe_moe_forward's (caller workspace) bit for bit, on
two calls in a row, the second with a smaller input, on every execution path:
the fused decode launch, the GEMV and MFMA paths of a resident layer, and a
16-slot cache (several waves).  Sizes past the library's scratch are refused.
"""
import numpy as np
import pytest
import torch

from paper_2608_15383_amd import api
from paper_2608_15383_amd._lib import EMOE_EINVAL, EMOE_NOALLOC_SCRATCH_BYTES, ExactMoEError
from paper_2608_15383_amd.inputs import OLMOE, make_layer, spread_logits
from tests._gpu import Layer, dev, dims_of, host_bits

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def olmoe():
    lay = make_layer(OLMOE, 300, seed=31)
    layer = Layer(dims_of(OLMOE), lay, 300)
    return lay, layer


def _both(layer, cache, h_bits, path=api.EMOE_PATH_AUTO, logits=None):
    """(y from emoe_moe_forward, y from emoe_moe_forward_noalloc), bf16 bits."""
    h = dev(h_bits)
    lo = None if logits is None else dev(np.asarray(logits, np.float32))
    y_ws, y_na = torch.full_like(h, -1), torch.full_like(h, -1)
    st_ws, st_na = api.Stats(), api.Stats()
    api.moe_forward(cache, h, layer.wr, y_ws, layer.ws, logits_override=lo, path=path, stats=st_ws)
    api.moe_forward_noalloc(cache, h, layer.wr, y_na, logits_override=lo, path=path, stats=st_na)
    torch.cuda.synchronize()
    assert st_na.kernel_launches == st_ws.kernel_launches and st_na.waves == st_ws.waves
    return host_bits(y_ws), host_bits(y_na)


@pytest.mark.parametrize("path,tokens", [(api.EMOE_PATH_AUTO, (4, 1)),      # fused decode
                                         (api.EMOE_PATH_GEMV, (64, 9)),
                                         (api.EMOE_PATH_MFMA, (300, 70))])
def test_noalloc_equals_workspace_call_resident(olmoe, path, tokens):
    lay, layer = olmoe
    for t in tokens:                       # the second call is smaller
        y_ws, y_na = _both(layer, layer.cache, lay.h[:t], path)
        assert np.array_equal(y_ws, y_na), (path, t)


def test_noalloc_equals_workspace_call_through_a_small_cache(olmoe):
    lay, layer = olmoe
    host = torch.empty(layer.bank.numel(), dtype=torch.uint8, pin_memory=True)
    host.copy_(layer.bank)
    torch.cuda.synchronize()
    dm = layer.dm
    slots = torch.zeros(16 * api.expert_record_bytes(dm), dtype=torch.uint8, device="cuda:0")
    cache = api.Cache(dm, 16, slot_bank=slots, host_bank=host)
    try:
        for t, d in ((16, 56), (8, 40)):
            z = spread_logits(t, 64, 8, d, seed=4)
            y_ws, y_na = _both(layer, cache, lay.h[:t], logits=z)
            assert np.array_equal(y_ws, y_na), t
    finally:
        cache.close()


def test_noalloc_refuses_sizes_past_its_scratch(olmoe):
    lay, layer = olmoe
    dm = layer.dm
    t = 1
    while api.workspace_bytes(dm, t) <= EMOE_NOALLOC_SCRATCH_BYTES:
        t *= 2
    h = torch.zeros((t, dm.d_model), dtype=torch.int16, device="cuda:0")
    y = torch.full_like(h, 7)
    with pytest.raises(ExactMoEError) as ei:
        api.moe_forward_noalloc(layer.cache, h, layer.wr, y)
    assert ei.value.status == EMOE_EINVAL and "scratch" in str(ei.value)
    torch.cuda.synchronize()
    assert bool((y == 7).all())            # nothing was enqueued
