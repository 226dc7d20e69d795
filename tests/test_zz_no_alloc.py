"""The allocation-free decode entry point (bdlora_forward_layer_static)
against bdlora_forward_layer: the same kernels on the library's static
scratch instead of the pool's workspace must give the same bits, call after
call (the second with a smaller batch, the array keeping the first call's
contents), eagerly and replayed from a captured graph, without allocating
device memory; sizes past the array are refused."""
import ctypes

import numpy as np
import pytest

import workloads as wl
from workloads.gpu import DeviceLayer, device_to_float, load_adapters, make_pool

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    import paper_2510_23346_amd as bd
    bd.lib()
    return torch


def _bits(outs):
    return [device_to_float(o).view(np.uint32).copy() for o in outs]


def _fresh(torch, outs):
    return [torch.full_like(o, float("nan")) for o in outs]


def test_static_forward_equals_layer_forward_twice(torch_cuda):
    # the 8B decode layer shard (64 tokens, 32 adapters, Zipf ids), then a
    # smaller batch (its first 12 tokens, other ids) on the same array; at 12
    # tokens the plan runs inside the decode launch
    torch = torch_cuda
    spec = wl.workload(1)
    slots = list(range(spec.n_slots))
    layer = wl.draw_layer(spec, slots=slots)
    pool = make_pool(spec)
    load_adapters(pool, spec, slots, cache=layer.adapters)
    projs = list(range(len(spec.projs)))
    dl = DeviceLayer(layer)
    ref = _fresh(torch, dl.out)
    pool.forward_layer(projs, dl.X, dl.W, ref, dl.ids)            # also loads the kernels
    torch.cuda.synchronize()
    free0 = torch.cuda.mem_get_info()[0]
    got = _fresh(torch, dl.out)
    pool.forward_layer_static(projs, dl.X, dl.W, got, dl.ids)
    torch.cuda.synchronize()
    for p, (a, b) in enumerate(zip(_bits(ref), _bits(got))):
        assert np.array_equal(a, b), f"first call, projection {p}"
    # second call: 12 tokens with their own ids
    T2 = 12
    ids2 = torch.from_numpy(np.array([(7 * t) % spec.n_slots - (t % 6 == 0) * (1 + (7 * t) % spec.n_slots)
                                      for t in range(T2)], np.int32)).cuda()
    X2 = [x[:T2].contiguous() for x in dl.X]
    ref2 = [torch.full((T2, o.shape[1]), float("nan"), dtype=o.dtype, device="cuda") for o in dl.out]
    got2 = _fresh(torch, ref2)
    pool.forward_layer_static(projs, X2, dl.W, got2, ids2)
    torch.cuda.synchronize()
    free1 = torch.cuda.mem_get_info()[0]
    pool.forward_layer(projs, X2, dl.W, ref2, ids2)
    torch.cuda.synchronize()
    for p, (a, b) in enumerate(zip(_bits(ref2), _bits(got2))):
        assert np.array_equal(a, b), f"second call, projection {p}"
    assert free1 >= free0 - (2 << 20), "the static forward allocated device memory"
    assert pool.device_error() == 0
    pool.close()


def test_static_forward_segments_and_graph_replay(torch_cuda):
    torch = torch_cuda
    import paper_2510_23346_amd as bd
    T = 37
    ranks = [8, 16, 3, 0, 24]
    ids = np.repeat(np.array([2, -1, 0, 4, 1, 0], np.int32), [5, 3, 9, 7, 10, 3])
    spec = wl.custom_workload("static-seg", wl.tiny_projs(), T, ranks, ids=ids, seed=31)
    layer = wl.draw_layer(spec, slots=range(len(ranks)))
    pool = make_pool(spec)
    load_adapters(pool, spec, range(len(ranks)), cache=layer.adapters)
    projs = list(range(len(spec.projs)))
    dl = DeviceLayer(layer)
    ref = _fresh(torch, dl.out)
    pool.forward_layer(projs, dl.X, dl.W, ref, dl.ids)
    got = _fresh(torch, dl.out)
    pool.forward_layer_static(projs, dl.X, dl.W, got, None, segs=bd.Segments.from_ids(ids))
    torch.cuda.synchronize()
    want = _bits(ref)
    for p, (a, b) in enumerate(zip(want, _bits(got))):
        assert np.array_equal(a, b), f"segments, projection {p}"
    # captured once, replayed with eager forwards of another batch between
    g = torch.cuda.CUDAGraph()
    cap = _fresh(torch, dl.out)
    with torch.cuda.graph(g, stream=torch.cuda.Stream()):
        pool.forward_layer_static(projs, dl.X, dl.W, cap, dl.ids, stream=torch.cuda.current_stream())
    torch.cuda.synchronize()
    other = _fresh(torch, dl.out)
    for rep in range(3):
        for o in cap:
            o.fill_(float("nan"))
        pool.forward_layer_static(projs, [x[:9] for x in dl.X], dl.W, [o[:9] for o in other], dl.ids[:9])
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for p, (a, b) in enumerate(zip(want, _bits(cap))):
            assert np.array_equal(a, b), f"replay {rep}, projection {p}"
    assert pool.device_error() == 0
    pool.close()


def test_static_forward_refuses_what_does_not_fit(torch_cuda):
    torch = torch_cuda
    import paper_2510_23346_amd as bd
    # a batch above the decode size
    spec = wl.custom_workload("static-big", wl.tiny_projs(), 80, [8], seed=2)
    layer = wl.draw_layer(spec, slots=[0])
    pool = make_pool(spec)
    load_adapters(pool, spec, [0], cache=layer.adapters)
    dl = DeviceLayer(layer)
    with pytest.raises(bd.BDLoRAError) as e:
        pool.forward_layer_static([0], dl.X[:1], dl.W[:1], dl.out[:1], dl.ids)
    assert e.value.code == -4
    pool.close()
    # eight projections of d_in 8192 and 16384 outputs at 64 tokens need
    # more than the array holds (packed activations 8 MiB, partial tiles
    # about 40 MiB); refused before anything is launched (the weight, input
    # and output pointers all name one zeroed buffer that must stay zero)
    projs = [wl.ProjSpec(f"p{i}", "column", 8192, (16384,)) for i in range(8)]
    pool = bd.Pool(projs, 4, 16, 64)
    buf = torch.zeros(8192 * 8192, dtype=torch.bfloat16, device="cuda")
    ids = torch.zeros(64, dtype=torch.int32, device="cuda") - 1
    L = bd.lib()
    n = 8
    pr = (ctypes.c_int32 * n)(*range(n))
    ptrs = (ctypes.c_void_p * n)(*([buf.data_ptr()] * n))
    rc = L.bdlora_forward_layer_static(pool.handle, n, pr, ptrs, ptrs, ptrs, ids.data_ptr(), None, 64,
                                       torch.cuda.current_stream().cuda_stream)
    assert rc == -4 and "static scratch" in L.bdlora_last_error().decode()
    torch.cuda.synchronize()
    assert torch.count_nonzero(buf).item() == 0                     # nothing ran
    pool.close()
