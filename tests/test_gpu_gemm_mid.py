"""GPU parity of the medium-batch base GEMM against the fp64 oracle.

Batches of 65..256 tokens over bf16 layers whose weight is large against the
fp32 partials (the Llama-3.1-70B layer shard at TP 8) take the medium-batch
launches:
- a main launch holds every row of the batch in one tile, so each weight
  fragment is read once; long-K tiles are split into k-ranges, and each item
  stores an fp32 partial;
- an epilogue adds each output's partials in range order, plus the expand
  of the token's own adapter.
Rows run in the plan's adapter order, so the main launch gathers activation
rows and the epilogue scatters output rows.

Covered here:
- the 70B shard at batch sizes on both sides of the tile-height switch
  (8 and 16 row blocks, ragged row tails);
- a variant with ragged column tails and qkv slice boundaries inside
  256-column tiles, with ranks from 1 to 64 (the expand's loop past 16
  ranks);
- edge batches: no adapted token, and one rank-64 adapter for every token;
- five forwards with the caches flushed before each (the k-step wait of the
  main launch with activations arriving slowly from memory);
- the path each shape takes (the rule that keeps small layers with few
  adapters on the 64-row kernel).
Every case checks that the path ran (pool.last_path()).  The error rule is
as in test_gpu_parity.
"""
import dataclasses

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


def _run(torch, spec, slots):
    """Forward the layer with its ids and with no adapter; return outputs,
    base-only outputs, the layer and the path taken."""
    layer = wl.draw_layer(spec, slots=slots)
    pool = make_pool(spec, max_tokens=spec.T)
    load_adapters(pool, spec, slots, cache=layer.adapters)
    dl = DeviceLayer(layer)
    projs = list(range(len(spec.projs)))
    pool.forward_layer(projs, dl.X, dl.W, dl.out, dl.ids)
    torch.cuda.synchronize()
    path = pool.last_path()
    ys = dl.outputs()
    base = [torch.empty_like(o) for o in dl.out]
    pool.forward_layer(projs, dl.X, dl.W, base, torch.full_like(dl.ids, -1))
    torch.cuda.synchronize()
    assert pool.last_path() == path
    yb = [device_to_float(o) for o in base]
    assert pool.device_error() == 0
    pool.close()
    return layer, ys, yb, path


def _check_all(layer, ids, ys, yb, what):
    refs = bdlora.layer_forward(layer)
    none = np.asarray(ids) < 0
    for p, pi in enumerate(layer.projs):
        rbase = pi.X.astype(np.float64) @ pi.W.astype(np.float64)
        e = bdlora.rel_errors(ys[p], refs[p])
        assert e["pointwise"] <= TOL, f"{what} {pi.spec.name}: {e}"
        assert bdlora.rel_errors(yb[p], rbase)["pointwise"] <= TOL, f"{what} {pi.spec.name} base"
        d = bdlora.delta_errors(ys[p], yb[p], refs[p], rbase)
        assert d <= TOL, f"{what} {pi.spec.name}: LoRA-term error {d}"
        # rows without an adapter carry the base product only, bit for bit
        assert np.array_equal(ys[p][none], yb[p][none]), f"{what} {pi.spec.name}: unadapted rows"


@pytest.mark.parametrize("T", [65, 128, 129, 200])
def test_medium_parity_70b_shard(torch_cuda, T):
    """The 70B layer shard (128 resident rank-16 adapters, Zipf ids) at
    batch sizes below the full 256-token workload, which test_gpu_parity
    covers."""
    spec = dataclasses.replace(wl.workload(3), name=f"70b-layer-T{T}", T=T, seed=300 + T)
    ids = wl.draw_ids(spec)
    active = sorted(int(s) for s in np.unique(ids) if s >= 0)
    layer, ys, yb, path = _run(torch_cuda, spec, active)
    assert path == "medium", f"T={T}: the batch took the {path} path"
    _check_all(layer, ids, ys, yb, f"T={T}")


@pytest.mark.parametrize("T", [100, 256])
def test_medium_parity_8b_shard_many_adapters(torch_cuda, T):
    """The 8B layer shard with 32 resident rank-16 adapters and Zipf ids:
    too small for the byte rule, but at most 8 tokens per loaded adapter,
    so the medium path runs its long shrink beside the base product."""
    spec = dataclasses.replace(wl.workload(1), name=f"8b-layer-T{T}", T=T, seed=800 + T)
    ids = wl.draw_ids(spec)
    active = sorted(int(s) for s in np.unique(ids) if s >= 0)
    layer, ys, yb, path = _run(torch_cuda, spec, list(range(spec.n_slots)))
    assert path == "medium", f"T={T}: the batch took the {path} path"
    _check_all(layer, ids, ys, yb, f"8b T={T}")
    assert len(active) > 8


def _ragged_projs():
    return [
        wl.ProjSpec("qkv", "column", 8192, (1008, 144, 128)),   # slice boundaries inside 256-column tiles
        wl.ProjSpec("o", "row", 1024, (8192,)),
        wl.ProjSpec("gate", "column", 8192, (3600,)),           # 14 tiles + a 16-column tail
        wl.ProjSpec("up", "column", 8192, (3584,)),
        wl.ProjSpec("down", "row", 3584, (8208,)),              # 32 tiles + a 16-column tail
    ]


RANKS = [16, 8, 32, 64, 1, 33, 24, 5]


@pytest.mark.parametrize("T", [100, 200])
def test_medium_ragged_columns_and_ranks(torch_cuda, T):
    rng = np.random.default_rng(4000 + T)
    ids = rng.integers(-1, len(RANKS), size=T)
    spec = wl.custom_workload(f"mid-ragged-{T}", _ragged_projs(), T, RANKS,
                              scales=[0.5 + 0.25 * i for i in range(len(RANKS))], ids=ids, seed=T)
    layer, ys, yb, path = _run(torch_cuda, spec, list(range(len(RANKS))))
    assert path == "medium", f"T={T}: the batch took the {path} path"
    _check_all(layer, ids, ys, yb, f"ragged T={T}")


@pytest.mark.parametrize("T,case", [(256, "none"), (100, "one"), (256, "one")])
def test_medium_edge_batches(torch_cuda, T, case):
    """No adapted token (every row after the adapted ones, none), and one
    rank-64 adapter for every token (a single adapter group)."""
    ranks = [16, 64]
    ids = np.full(T, -1) if case == "none" else np.full(T, 1)
    spec = wl.custom_workload(f"mid-{case}-{T}", wl.model_projs("llama-3.1-70b", 8), T, ranks,
                              scales=[1.5, 0.75], ids=ids, seed=5 + T)
    layer, ys, yb, path = _run(torch_cuda, spec, [0, 1])
    assert path == "medium", f"{case} T={T}: the batch took the {path} path"
    _check_all(layer, ids, ys, yb, f"{case} T={T}")


def _small_projs():
    return [
        wl.ProjSpec("qkv", "column", 128, (272, 256, 16)),
        wl.ProjSpec("o", "row", 160, (528,)),                 # K of 5 k-steps
        wl.ProjSpec("up", "column", 96, (256,)),
    ]


def test_medium_parity_cold_caches(torch_cuda):
    """The main launch's k-step wait must hold when the activations arrive
    slowly from memory: the caches are flushed (1 GiB written) before each
    of five forwards of a 65-token batch over small projections and twelve
    adapters, and every forward matches the oracle.  (A form whose wait
    counted copies into LDS together with loads into registers gave wrong
    outputs in about half of such runs.)"""
    torch = torch_cuda
    ranks = [0, 1, 8, 16, 24, 33, 64, 5, 40, 12, 56, 32]
    T = 65
    rng = np.random.default_rng(1000 + T)
    ids = rng.integers(-1, len(ranks), size=T)
    spec = wl.custom_workload("mid-cold-65", _small_projs(), T, ranks,
                              scales=[0.5 + 0.125 * i for i in range(len(ranks))], ids=ids, seed=T)
    layer = wl.draw_layer(spec, slots=range(len(ranks)))
    pool = make_pool(spec, max_tokens=T)
    load_adapters(pool, spec, range(len(ranks)), cache=layer.adapters)
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
        assert pool.last_path() == "medium"
        ys = dl.outputs()
        for p, pi in enumerate(layer.projs):
            e = bdlora.rel_errors(ys[p], refs[p])
            assert e["pointwise"] <= TOL, f"run {it} {pi.spec.name}: {e}"
    assert pool.device_error() == 0
    pool.close()


@pytest.mark.parametrize("model,T,n_slots,path", [
    ("llama-3.1-8b", 64, 2, "decode"), ("llama-3.1-70b", 65, 2, "medium"), ("llama-3.1-70b", 256, 2, "medium"),
    ("llama-3.1-70b", 257, 2, "large"), ("llama-3.1-8b", 100, 2, "tile64"), ("llama-3.1-8b", 256, 2, "tile64"),
    ("llama-3.1-8b", 128, 32, "medium"), ("llama-3.1-8b", 256, 32, "medium")])
def test_path_choice(torch_cuda, model, T, n_slots, path):
    """The launch sequence each batch takes: decode up to 64 tokens, the
    medium-batch launches for the 70B shard up to 256; for the 8B shard
    (whose weight is too small against the partials of a chip-filling split)
    the 64-row kernel, unless the batch spreads over many adapters (at most
    8 tokens per loaded adapter), whose long shrink the medium path runs
    beside the base product; the large tiles above 256.  Outputs are checked
    on a few rows against the oracle."""
    torch = torch_cuda
    ranks = [16, 8] * (n_slots // 2)
    rng = np.random.default_rng(T)
    ids = rng.integers(-1, len(ranks), size=T)
    spec = wl.custom_workload(f"path-{model}-{T}-{n_slots}", wl.model_projs(model, 8), T, ranks,
                              scales=[2.0, 1.0] * (n_slots // 2), ids=ids, seed=T)
    layer = wl.draw_layer(spec, slots=range(n_slots))
    pool = make_pool(spec, max_tokens=T)
    load_adapters(pool, spec, range(n_slots), cache=layer.adapters)
    dl = DeviceLayer(layer)
    pool.forward_layer(list(range(len(spec.projs))), dl.X, dl.W, dl.out, dl.ids)
    torch.cuda.synchronize()
    assert pool.last_path() == path
    rows = np.array(sorted({0, T // 3, T - 1}))
    refs = bdlora.layer_forward_rows(layer, rows)
    ys = dl.outputs()
    for p, pi in enumerate(layer.projs):
        e = bdlora.rel_errors(ys[p][rows], refs[p])
        assert e["pointwise"] <= TOL, f"{model} T={T} {pi.spec.name}: {e}"
    assert pool.device_error() == 0
    pool.close()
