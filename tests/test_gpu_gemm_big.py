"""GPU parity of the large-tile (256 x 256) prefill base GEMM with the fused
expand, against the fp64 oracle.

Batches above 256 tokens with bf16 base weights take that kernel; when a
batch has too few tiles to fill the chip, long-K tiles are split into
k-ranges whose fp32 partials a fix-up launch adds (the small shapes above
256 tokens here are all split; the full-size prefill workloads in
test_gpu_parity are not).  On the same shapes, 65 tokens take the
medium-batch launches and 130 the 64-row kernel.  The
projections here are wider than one 256-column tile, with a ragged column
tail, slice boundaries inside a tile, and more row tiles than one with a
ragged row tail, so that the clamped edge blocks, the per-64-row octet lists
and the slice lookup of the expand are all exercised.  Ranks go up to 64
(eight octets per adapter) and a 64-row block holds many adapters, so the
expand loop runs several passes.  One case repeats a forward five times
with the caches flushed before each (the k-step waits with operands arriving
slowly from memory).  Error rule as in test_gpu_parity.
"""
import numpy as np
import pytest

import workloads as wl
from workloads.gpu import DeviceLayer, device_to_float, load_adapters, make_pool
from oracle import bdlora

pytestmark = pytest.mark.gpu
TOL = 1e-2

RANKS = [0, 1, 8, 16, 24, 33, 64, 5, 40, 12, 56, 32]


def _projs():
    return [
        wl.ProjSpec("qkv", "column", 128, (272, 256, 16)),   # 544 columns: 3 tiles, slices cut tiles
        wl.ProjSpec("o", "row", 160, (528,)),                 # 528 columns, K of 5 k-steps
        wl.ProjSpec("up", "column", 96, (256,)),              # exactly one tile wide
    ]


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    import paper_2510_23346_amd as bd
    bd.lib()
    return torch


@pytest.mark.parametrize("T,kind", [(65, "uniform"), (130, "segments"), (257, "uniform"), (520, "uniform"), (777, "segments")])
def test_big_tile_parity(torch_cuda, T, kind):
    torch = torch_cuda
    rng = np.random.default_rng(1000 + T)
    if kind == "segments":
        # contiguous runs of one adapter, as in sorted prefill batches
        cuts = np.sort(rng.choice(np.arange(1, T), size=9, replace=False))
        ids = np.zeros(T, np.int64)
        for i, (a, b) in enumerate(zip(np.r_[0, cuts], np.r_[cuts, T])):
            ids[a:b] = rng.integers(-1, len(RANKS)) if i % 3 else i % len(RANKS)
    else:
        ids = rng.integers(-1, len(RANKS), size=T)
    spec = wl.custom_workload(f"big-{T}", _projs(), T, RANKS,
                              scales=[0.5 + 0.125 * i for i in range(len(RANKS))], ids=ids, seed=T)
    layer = wl.draw_layer(spec, slots=range(len(RANKS)))
    pool = make_pool(spec, max_tokens=T)
    load_adapters(pool, spec, range(len(RANKS)), cache=layer.adapters)
    dl = DeviceLayer(layer)
    pool.forward_layer(list(range(len(spec.projs))), dl.X, dl.W, dl.out, dl.ids)
    torch.cuda.synchronize()
    ys = dl.outputs()
    ids_none = torch.full_like(dl.ids, -1)
    base = [torch.empty_like(o) for o in dl.out]
    pool.forward_layer(list(range(len(spec.projs))), dl.X, dl.W, base, ids_none)
    torch.cuda.synchronize()
    yb = [device_to_float(o) for o in base]
    refs = bdlora.layer_forward(layer)
    for p, pi in enumerate(layer.projs):
        rbase = pi.X.astype(np.float64) @ pi.W.astype(np.float64)
        e = bdlora.rel_errors(ys[p], refs[p])
        assert e["pointwise"] <= TOL, f"T={T} {pi.spec.name}: {e}"
        assert bdlora.rel_errors(yb[p], rbase)["pointwise"] <= TOL, f"T={T} {pi.spec.name} base"
        d = bdlora.delta_errors(ys[p], yb[p], refs[p], rbase)
        assert d <= TOL, f"T={T} {pi.spec.name}: LoRA-term error {d}"
        # rows without an adapter carry the base product only, bit for bit
        none = np.asarray(ids) < 0
        assert np.array_equal(ys[p][none], yb[p][none])
    assert pool.device_error() == 0
    pool.close()


@pytest.mark.parametrize("T,case", [(300, "none"), (300, "one"), (8500, "uniform")])
def test_big_tile_edge_batches(torch_cuda, T, case):
    """No token with an adapter (empty octet lists, every row after the
    adapted ones), one adapter for every token, and a batch above the plan's
    LDS token limit (8192: the plan reads ids back from HBM)."""
    torch = torch_cuda
    rng = np.random.default_rng(7 + T)
    ranks = [16, 8, 32]
    if case == "none":
        ids = np.full(T, -1)
    elif case == "one":
        ids = np.full(T, 2)
    else:
        ids = rng.integers(-1, len(ranks), size=T)
    projs = [wl.ProjSpec("qkv", "column", 64, (32, 16, 16)), wl.ProjSpec("o", "row", 32, (48,))]
    spec = wl.custom_workload(f"edge-{case}-{T}", projs, T, ranks, scales=[1.5, 0.5, 2.0], ids=ids, seed=T)
    layer = wl.draw_layer(spec, slots=range(len(ranks)))
    pool = make_pool(spec, max_tokens=T)
    load_adapters(pool, spec, range(len(ranks)), cache=layer.adapters)
    dl = DeviceLayer(layer)
    pool.forward_layer(list(range(len(spec.projs))), dl.X, dl.W, dl.out, dl.ids)
    torch.cuda.synchronize()
    ys = dl.outputs()
    refs = bdlora.layer_forward(layer)
    for p, pi in enumerate(layer.projs):
        e = bdlora.rel_errors(ys[p], refs[p])
        assert e["pointwise"] <= TOL, f"{case} T={T} {pi.spec.name}: {e}"
    assert pool.device_error() == 0
    pool.close()


def _projs_k64():
    return [
        wl.ProjSpec("qkv", "column", 128, (272, 256, 16)),
        wl.ProjSpec("o", "row", 192, (528,)),                 # K of 6 k-steps
        wl.ProjSpec("up", "column", 256, (256,)),
    ]


def test_big_tile_parity_cold_caches(torch_cuda):
    """The large tiles' k-step waits with activations and weights arriving
    slowly from memory: every K a multiple of 64, so the launch and its
    shrink read the caller's row-major X; the caches are flushed (1 GiB
    written) before each of five forwards of a 520-token batch, and every
    forward matches the oracle."""
    torch = torch_cuda
    T = 520
    rng = np.random.default_rng(7520)
    ids = rng.integers(-1, len(RANKS), size=T)
    spec = wl.custom_workload("big-cold-520", _projs_k64(), T, RANKS,
                              scales=[0.5 + 0.125 * i for i in range(len(RANKS))], ids=ids, seed=T)
    layer = wl.draw_layer(spec, slots=range(len(RANKS)))
    pool = make_pool(spec, max_tokens=T)
    load_adapters(pool, spec, range(len(RANKS)), cache=layer.adapters)
    dl = DeviceLayer(layer)
    refs = bdlora.layer_forward(layer)
    flush = torch.empty(1 << 29, dtype=torch.float16, device="cuda")
    projs = list(range(len(spec.projs)))
    for it in range(5):
        for o in dl.out:
            o.fill_(float("nan"))
        flush.fill_(it)
        pool.forward_layer(projs, dl.X, dl.W, dl.out, dl.ids)
        torch.cuda.synchronize()
        assert pool.last_path() == "large"
        ys = dl.outputs()
        for p, pi in enumerate(layer.projs):
            e = bdlora.rel_errors(ys[p], refs[p])
            assert e["pointwise"] <= TOL, f"run {it} {pi.spec.name}: {e}"
    assert pool.device_error() == 0
    pool.close()
