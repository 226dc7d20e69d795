"""The segments form of the forward (a batch given as runs of tokens that
share an adapter: heterogeneous batching of Sec. 2, prefill requests as
contiguous runs), the pool's byte budget, the graph-capture bound of the
decode launches, and decode batches on the smallest projections.

The segments form must give the same bits as the per-token ids form for the
same batch on every launch sequence, and both must match the oracle."""
import ctypes
import dataclasses

import numpy as np
import pytest

import workloads as wl
from workloads.gpu import DeviceLayer, device_to_float, load_adapters, make_pool
from oracle import bdlora, plan as oplan

pytestmark = pytest.mark.gpu
TOL = 1e-2
RANKS = [8, 16, 0, 24, 5, 32]


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    import paper_2510_23346_amd as bd
    bd.lib()
    return torch


def _bits(outs):
    return [device_to_float(o).view(np.uint32).copy() for o in outs]


def _runs_ids(T, seed, n_slots):
    # requests of random lengths, each naming one adapter (or none)
    rng = np.random.default_rng(seed)
    ids, t = [], 0
    while t < T:
        L = int(rng.integers(1, max(2, T // 4)))
        ids += [int(rng.integers(-1, n_slots))] * min(L, T - t)
        t += L
    return np.asarray(ids, np.int32)


@pytest.mark.parametrize("T,path", [(5, "decode"), (64, "decode"), (100, "tile64"), (300, "large"),
                                    (1100, "large")])
def test_segments_equal_ids_and_oracle(torch_cuda, T, path):
    torch = torch_cuda
    import paper_2510_23346_amd as bd
    ids = _runs_ids(T, T, len(RANKS))
    sg = bd.Segments.from_ids(ids)
    assert sg.n_seg <= bd.MAX_SEGMENTS
    assert list(zip(sg.start.tolist(), sg.len.tolist(), sg.slot.tolist())) == [tuple(r) for r in oplan.segments(ids)]
    spec = wl.custom_workload(f"seg-{T}", wl.tiny_projs(), T, RANKS, ids=ids, seed=50 + T)
    layer = wl.draw_layer(spec, slots=range(len(RANKS)))
    pool = make_pool(spec)
    load_adapters(pool, spec, range(len(RANKS)), cache=layer.adapters)
    projs = list(range(len(spec.projs)))
    a = DeviceLayer(layer)
    pool.forward_layer(projs, a.X, a.W, a.out, a.ids)
    torch.cuda.synchronize()
    assert pool.last_path() == path
    b = DeviceLayer(layer)
    pool.forward_layer(projs, b.X, b.W, b.out, None, segs=sg)
    torch.cuda.synchronize()
    assert pool.last_path() == path
    for p, (x, y) in enumerate(zip(_bits(a.out), _bits(b.out))):
        assert np.array_equal(x, y), f"T={T} projection {p}: segments and ids forms differ"
    refs = bdlora.layer_forward(layer)
    for p, y in enumerate(b.outputs()):
        e = bdlora.rel_errors(y, refs[p])
        assert e["pointwise"] <= TOL, (T, p, e)
    # one projection through forward_shard (its own launch geometry), the
    # segments given as a plain id list, against the ids form of the call
    o1 = torch.full_like(b.out[0], float("nan"))
    o2 = torch.full_like(b.out[0], float("nan"))
    pool.forward_shard(0, b.X[0], b.W[0], a.ids, o1)
    pool.forward_shard(0, b.X[0], b.W[0], None, o2, segs=ids.tolist())
    torch.cuda.synchronize()
    assert np.array_equal(device_to_float(o1).view(np.uint32), device_to_float(o2).view(np.uint32))
    assert pool.device_error() == 0
    pool.close()


def test_prefill_workload_segments_equal_ids(torch_cuda):
    # the sorted 8 x 512 prefill batch of the 8B layer shard, as 8 segments
    torch = torch_cuda
    import paper_2510_23346_amd as bd
    spec = wl.workload(2)
    layer = wl.draw_layer(spec, slots=range(spec.n_slots))
    pool = make_pool(spec)
    load_adapters(pool, spec, range(spec.n_slots), cache=layer.adapters)
    projs = list(range(len(spec.projs)))
    sg = bd.Segments([512 * i for i in range(8)], [512] * 8, list(range(8)))
    a, b = DeviceLayer(layer), DeviceLayer(layer)
    pool.forward_layer(projs, a.X, a.W, a.out, a.ids)
    pool.forward_layer(projs, b.X, b.W, b.out, None, segs=sg)
    torch.cuda.synchronize()
    for x, y in zip(_bits(a.out), _bits(b.out)):
        assert np.array_equal(x, y)
    pool.close()


def test_mlp_segments_equal_ids(torch_cuda):
    torch = torch_cuda
    import paper_2510_23346_amd as bd
    for T in (33, 200):
        ids = _runs_ids(T, 7 * T, 3)
        spec = wl.custom_workload(f"mlpseg-{T}", wl.tiny_mlp_projs(), T, [8, 16, 4], ids=ids, seed=T)
        layer = wl.draw_layer(spec, slots=range(3))
        pool = make_pool(spec)
        load_adapters(pool, spec, range(3), cache=layer.adapters)
        dl = DeviceLayer(layer)
        o1 = torch.full((T, 160), float("nan"), dtype=torch.bfloat16, device="cuda")
        o2 = torch.full_like(o1, float("nan"))
        pool.forward_mlp(bd.ACT_SILU_MUL, [0, 1], 2, dl.X[0], dl.W[:2], dl.W[2], o1, dl.ids)
        pool.forward_mlp(bd.ACT_SILU_MUL, [0, 1], 2, dl.X[0], dl.W[:2], dl.W[2], o2, None,
                         segs=bd.Segments.from_ids(ids))
        torch.cuda.synchronize()
        assert np.array_equal(device_to_float(o1).view(np.uint32), device_to_float(o2).view(np.uint32))
        pool.close()


def test_segment_errors_enqueue_nothing(torch_cuda):
    torch = torch_cuda
    import paper_2510_23346_amd as bd
    T = 40
    spec = wl.custom_workload("segerr", wl.tiny_projs(), T, [8, 8, 8], seed=9)
    layer = wl.draw_layer(spec, slots=[0, 1, 2])
    pool = make_pool(spec)
    load_adapters(pool, spec, [0, 1], cache=layer.adapters)          # slot 2 stays empty
    dl = DeviceLayer(layer)
    cases = [
        (bd.Segments([0, 20], [20, 20], [0, 2]), -3),                  # names an empty slot
        (bd.Segments([0, 20], [20, 20], [0, 7]), -3),                  # out of range
        (bd.Segments([0, 20], [20, 20], [0, -2]), -3),                 # below -1
        (bd.Segments([0, 21], [20, 19], [0, 1]), -1),                  # a gap
        (bd.Segments([0, 20], [20, 19], [0, 1]), -1),                  # does not reach T
        (bd.Segments([0, 20], [20, 0], [0, 1]), -1),                   # empty segment
    ]
    for sg, code in cases:
        with pytest.raises(bd.BDLoRAError) as e:
            pool.forward_shard(0, dl.X[0], dl.W[0], None, dl.out[0], T=T, segs=sg)
        assert e.value.code == code
    torch.cuda.synchronize()
    assert np.all(np.isnan(device_to_float(dl.out[0])))                 # nothing ran
    # both forms, or neither, through the C ABI directly
    L = bd.lib()
    pr = (ctypes.c_int32 * 1)(0)
    xs = (ctypes.c_void_p * 1)(dl.X[0].data_ptr())
    ws = (ctypes.c_void_p * 1)(dl.W[0].data_ptr())
    os_ = (ctypes.c_void_p * 1)(dl.out[0].data_ptr())
    sg = bd.Segments([0], [T], [0])
    s = torch.cuda.current_stream().cuda_stream
    assert L.bdlora_forward_layer(pool.handle, 1, pr, xs, ws, os_, dl.ids.data_ptr(), sg.ref(), T, s) == -1
    assert L.bdlora_forward_layer(pool.handle, 1, pr, xs, ws, os_, None, None, T, s) == -1
    pool.close()


def test_pool_byte_budget_sizes_the_slots(torch_cuda):
    import paper_2510_23346_amd as bd
    projs = wl.tiny_projs()
    per = bd.layout_slot_bytes(projs, 16)
    pool = bd.Pool(projs, 0, 16, 32, pool_bytes=5 * per + per // 2)
    assert pool.max_slots == 5 and pool.slot_bytes == per
    pool.close()
    pool = bd.Pool(projs, 3, 16, 32, pool_bytes=3 * per)
    assert pool.max_slots == 3
    pool.close()


@pytest.mark.parametrize("T", [24, 10])
def test_captured_decode_bounds_adapters_loaded_later(torch_cuda, T):
    # A decode forward captured while 2 adapters were loaded replays with ids
    # that use 4: the adapters past the bound (slots 2 and 3, ascending slot
    # order) get the base output and the device error flag is raised; the
    # others stay exact.  The segments form has no such bound.  At 10 tokens
    # the plan runs inside the decode launch.
    torch = torch_cuda
    import paper_2510_23346_amd as bd
    ranks = [8, 16, 8, 16, 8, 8]
    ids0 = np.array([[0, 1, -1][t % 3] for t in range(T)], np.int32)
    ids1 = np.array([[0, 1, 2, 3, -1][t % 5] for t in range(T)], np.int32)
    spec = wl.custom_workload("capbound", wl.tiny_projs(), T, ranks, ids=ids0, seed=21)
    layer = wl.draw_layer(spec, slots=range(len(ranks)))
    pool = make_pool(spec)
    load_adapters(pool, spec, [0, 1], cache=layer.adapters)
    projs = list(range(len(spec.projs)))
    dl = DeviceLayer(layer)
    pool.forward_layer(projs, dl.X, dl.W, dl.out, dl.ids)
    torch.cuda.synchronize()
    assert pool.last_path() == "decode" and pool.device_error() == 0
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=torch.cuda.Stream()):
        pool.forward_layer(projs, dl.X, dl.W, dl.out, dl.ids, stream=torch.cuda.current_stream())
    torch.cuda.synchronize()
    load_adapters(pool, spec, [2, 3], cache=layer.adapters)
    dl.ids.copy_(torch.from_numpy(ids1).cuda())
    for o in dl.out:
        o.fill_(float("nan"))
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    assert pool.device_error() == 1
    capped = dataclasses.replace(layer, ids=np.where(ids1 >= 2, -1, ids1).astype(np.int32))
    refs = bdlora.layer_forward(capped)
    for p, y in enumerate(dl.outputs()):
        e = bdlora.rel_errors(y, refs[p])
        assert e["pointwise"] <= TOL, (p, e)
    # eager calls now see 4 loaded adapters, and the segments form its own count
    full = dataclasses.replace(layer, ids=ids1)
    refs = bdlora.layer_forward(full)
    for form in ("ids", "segs"):
        for o in dl.out:
            o.fill_(float("nan"))
        if form == "ids":
            pool.forward_layer(projs, dl.X, dl.W, dl.out, dl.ids)
        else:
            pool.forward_layer(projs, dl.X, dl.W, dl.out, None, segs=bd.Segments.from_ids(ids1))
        torch.cuda.synchronize()
        for p, y in enumerate(dl.outputs()):
            e = bdlora.rel_errors(y, refs[p])
            assert e["pointwise"] <= TOL, (form, p, e)
    assert pool.device_error() == 0
    pool.close()


@pytest.mark.parametrize("d_in,n_out", [(32, 16), (64, 16), (32, 48), (96, 32)])
@pytest.mark.parametrize("T", [1, 9, 64])
def test_decode_on_the_smallest_projections(torch_cuda, d_in, n_out, T):
    # fewer than 4 weight k-step blocks: the decode launch runs one workgroup
    torch = torch_cuda
    projs = [wl.ProjSpec("p", "column", d_in, (n_out,))]
    rng = np.random.default_rng(d_in + n_out + T)
    ids = rng.integers(-1, 3, size=T)
    spec = wl.custom_workload(f"small-{d_in}-{n_out}-{T}", projs, T, [8, 16, 3], ids=ids, seed=T)
    layer = wl.draw_layer(spec, slots=range(3))
    pool = make_pool(spec)
    load_adapters(pool, spec, range(3), cache=layer.adapters)
    dl = DeviceLayer(layer)
    pool.forward_layer([0], dl.X, dl.W, dl.out, dl.ids)
    torch.cuda.synchronize()
    assert pool.last_path() == "decode"
    e = bdlora.rel_errors(dl.outputs()[0], bdlora.layer_forward(layer)[0])
    assert e["pointwise"] <= TOL, e
    pool.close()
