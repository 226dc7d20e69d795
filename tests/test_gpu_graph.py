"""Forwards captured in a HIP graph replay to the eager result.

`bench.py` times forwards captured into HIP graphs, and the medium-batch
path forks the shrink onto a pool-owned side stream inside each forward, so
the capture must record that branch and its join.  Each case captures one
forward, replays the graph several times with eager forwards of other
inputs and synchronizations between the replays, and checks every replay
against the eager output bit for bit (the kernels are deterministic).  The
cases cover the decode launches, the 64-row kernel, the medium-batch path
with its side stream, and the large tiles.
"""
import dataclasses

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


@pytest.mark.parametrize("model,T,path", [("llama-3.1-8b", 64, "decode"), ("llama-3.1-8b", 16, "decode"),
                                          ("llama-3.1-8b", 100, "tile64"),
                                          ("llama-3.1-70b", 200, "medium"), ("llama-3.1-8b", 300, "large")])
def test_graph_replays_match_eager(torch_cuda, model, T, path):
    torch = torch_cuda
    ranks = [16, 8, 32, 16, 16, 8]
    base = wl.workload(3) if model == "llama-3.1-70b" else wl.workload(1)
    spec = dataclasses.replace(base, name=f"graph-{model}-{T}", T=T, n_slots=len(ranks), ranks=ranks,
                               scales=[2.0, 1.0, 0.5, 1.5, 1.0, 0.75], seed=900 + T)
    ids = wl.draw_ids(spec)
    slots = list(range(len(ranks)))
    layer = wl.draw_layer(spec, slots=slots)
    pool = make_pool(spec, max_tokens=T)
    load_adapters(pool, spec, slots, cache=layer.adapters)
    dl = DeviceLayer(layer)                      # captured inputs
    other = DeviceLayer(wl.draw_layer(dataclasses.replace(spec, seed=spec.seed + 1), slots=slots))
    projs = list(range(len(spec.projs)))

    pool.forward_layer(projs, dl.X, dl.W, dl.out, dl.ids)
    torch.cuda.synchronize()
    assert pool.last_path() == path
    want = _bits(dl.out)

    side = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        pool.forward_layer(projs, dl.X, dl.W, dl.out, dl.ids, stream=torch.cuda.current_stream())
    torch.cuda.synchronize()
    for rep in range(4):
        for o in dl.out:
            o.zero_()
        # eager work on other inputs between the replays
        pool.forward_layer(projs, other.X, other.W, other.out, other.ids)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = _bits(dl.out)
        for p in projs:
            assert np.array_equal(got[p], want[p]), f"{model} T={T} replay {rep} projection {p}"
    assert pool.device_error() == 0
    pool.close()
