"""GPU checks of the adapter load pipeline: host-packed slabs loaded with an
asynchronous copy give the same outputs, bit for bit, as adapters loaded
through bdlora_load_adapter; a load on a side stream overlapped with forward
calls on other slots is correct once ordered by an event."""
import numpy as np
import pytest

import workloads as wl
from workloads.gpu import DeviceLayer, device_to_float, load_adapters, make_pool
from oracle import bdlora

pytestmark = pytest.mark.gpu
TOL = 1e-2


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    import paper_2510_23346_amd as bd
    bd.lib()
    return torch


def _spec(T, ids, ranks, seed):
    return wl.custom_workload("load", wl.tiny_projs(), T, ranks, ids=ids, seed=seed)


@pytest.mark.parametrize("T", [48, 200])
def test_packed_load_equals_device_packed_load(torch_cuda, T):
    # slot 0 loaded by bdlora_load_adapter, slot 1 with the same adapter from
    # a host-packed slab: rows with the same X and id 0 / id 1 match bit for bit
    torch = torch_cuda
    rng = np.random.default_rng(T)
    ids = np.tile([0, 1], T // 2)
    spec = _spec(T, ids, [16, 16], 5)
    layer = wl.draw_layer(spec, slots=[0])
    for pi in layer.projs:                       # rows 2i and 2i+1 share their X
        pi.X_bits[1::2] = pi.X_bits[0::2]
        pi.X[1::2] = pi.X[0::2]
    pool = make_pool(spec, max_tokens=T)
    ad = layer.adapters[0]
    pool.load_adapter(0, ad.rank, ad.scale, ad.A_bits, ad.B_bits)
    slab = torch.empty(pool.slot_bytes, dtype=torch.uint8).pin_memory()
    pool.pack_adapter_host(ad.rank, ad.A_bits, ad.B_bits, out=slab)
    pool.load_adapter_packed(1, ad.rank, ad.scale, slab)
    torch.cuda.synchronize()
    dl = DeviceLayer(layer)
    pool.forward_layer(list(range(len(spec.projs))), dl.X, dl.W, dl.out, dl.ids)
    torch.cuda.synchronize()
    for y in dl.outputs():
        assert np.array_equal(y[0::2].view(np.uint32), y[1::2].view(np.uint32))
    layer.adapters[1] = layer.adapters[0]        # slot 1 holds the same adapter
    refs = bdlora.layer_forward(layer)
    for y, r in zip(dl.outputs(), refs):
        assert bdlora.rel_errors(y, r)["pointwise"] <= TOL
    pool.close()


def test_async_load_on_a_side_stream(torch_cuda):
    # adapters 0, 1 resident; adapter 2 arrives from a pinned slab on a side
    # stream while forwards on slots 0 / 1 run on the main stream; after an
    # event the batch that uses slot 2 matches the oracle
    torch = torch_cuda
    T = 64
    rng = np.random.default_rng(2)
    ids_a = rng.integers(-1, 2, size=T)
    ids_b = rng.integers(-1, 3, size=T)
    spec = _spec(T, ids_b, [8, 16, 24], 9)
    layer = wl.draw_layer(spec, slots=[0, 1, 2])
    pool = make_pool(spec, max_tokens=T)
    load_adapters(pool, spec, [0, 1], cache=layer.adapters)
    ad = layer.adapters[2]
    slab = torch.empty(pool.slot_bytes, dtype=torch.uint8).pin_memory()
    pool.pack_adapter_host(ad.rank, ad.A_bits, ad.B_bits, out=slab)
    dl = DeviceLayer(layer)
    projs = list(range(len(spec.projs)))
    main = torch.cuda.current_stream()
    side = torch.cuda.Stream()
    ids_a_d = torch.from_numpy(ids_a.astype(np.int32)).cuda()
    outs_a = [torch.empty_like(o) for o in dl.out]
    with torch.cuda.stream(side):
        pool.load_adapter_packed(2, ad.rank, ad.scale, slab, stream=side)
        done = torch.cuda.Event()
        done.record(side)
    for _ in range(3):                          # other slots keep running meanwhile
        pool.forward_layer(projs, dl.X, dl.W, outs_a, ids_a_d, stream=main)
    main.wait_event(done)
    pool.forward_layer(projs, dl.X, dl.W, dl.out, dl.ids, stream=main)
    torch.cuda.synchronize()
    for y, r in zip(dl.outputs(), bdlora.layer_forward(layer)):
        assert bdlora.rel_errors(y, r)["pointwise"] <= TOL
    assert pool.device_error() == 0
    pool.close()


def test_pageable_slab_and_errors(torch_cuda):
    torch = torch_cuda
    import paper_2510_23346_amd as bd
    T = 16
    ids = np.zeros(T, dtype=np.int32)
    spec = _spec(T, ids, [8], 3)
    layer = wl.draw_layer(spec, slots=[0])
    pool = make_pool(spec, max_tokens=T)
    ad = layer.adapters[0]
    slab = pool.pack_adapter_host(ad.rank, ad.A_bits, ad.B_bits)        # numpy, pageable
    assert slab.nbytes == pool.slot_bytes
    pool.load_adapter_packed(0, ad.rank, ad.scale, slab)
    torch.cuda.synchronize()
    dl = DeviceLayer(layer)
    pool.forward_layer(list(range(len(spec.projs))), dl.X, dl.W, dl.out, dl.ids)
    torch.cuda.synchronize()
    for y, r in zip(dl.outputs(), bdlora.layer_forward(layer)):
        assert bdlora.rel_errors(y, r)["pointwise"] <= TOL
    with pytest.raises(bd.BDLoRAError):
        pool.load_adapter_packed(5, 8, 1.0, slab)                 # slot out of range
    with pytest.raises(bd.BDLoRAError):
        pool.load_adapter_packed(0, 9, 1.0, slab)                 # rank above max_rank
    with pytest.raises(bd.BDLoRAError):
        pool.load_adapter_packed(0, 8, float("nan"), slab)
    bad = [[a.copy() for a in row] for row in ad.A_bits]
    bad[0][0][3, 1] = 0x7FC0                                      # NaN in A
    with pytest.raises(bd.BDLoRAError):
        pool.pack_adapter_host(ad.rank, bad, ad.B_bits)
    with pytest.raises(ValueError):
        pool.load_adapter_packed(0, 8, 1.0, slab[:100])
    pool.close()


def test_batched_load_into_consecutive_slots(torch_cuda):
    # three adapters of different ranks, packed back to back and loaded with
    # one copy into slots 4..6; a batch naming them matches the oracle
    torch = torch_cuda
    T = 40
    rng = np.random.default_rng(6)
    ranks = [8, 3, 16, 1, 24, 5, 12]
    ids = rng.choice([-1, 4, 5, 6], size=T)
    spec = _spec(T, ids, ranks, 12)
    layer = wl.draw_layer(spec, slots=[4, 5, 6])
    pool = make_pool(spec, max_tokens=T)
    sb = pool.slot_bytes
    slabs = torch.empty(3 * sb, dtype=torch.uint8).pin_memory()
    for i, a in enumerate((4, 5, 6)):
        ad = layer.adapters[a]
        pool.pack_adapter_host(ad.rank, ad.A_bits, ad.B_bits, out=slabs[i * sb:(i + 1) * sb])
    pool.load_adapters_packed(4, [ranks[a] for a in (4, 5, 6)], [layer.adapters[a].scale for a in (4, 5, 6)],
                              slabs)
    dl = DeviceLayer(layer)
    pool.forward_layer(list(range(len(spec.projs))), dl.X, dl.W, dl.out, dl.ids)
    torch.cuda.synchronize()
    for y, r in zip(dl.outputs(), bdlora.layer_forward(layer)):
        assert bdlora.rel_errors(y, r)["pointwise"] <= TOL
    import paper_2510_23346_amd as bd
    with pytest.raises(bd.BDLoRAError):
        pool.load_adapters_packed(6, [8, 8], [1.0, 1.0], slabs)        # slot 7 is out of range
    pool.close()
