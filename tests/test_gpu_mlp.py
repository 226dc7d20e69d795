"""GPU parity of the BD-LoRA MLP shard (Alg. 1) through the C ABI against the
fp64 MLP oracle.  Same error rule as the projection parity tests: every
element |y - ref| <= 1e-2 * max(|ref|, rms(ref)); the oracle holds the
intermediate in bf16 like the GPU path."""
import numpy as np
import pytest

import paper_2510_23346_amd as bd
import workloads as wl
from workloads.gpu import DeviceLayer, device_to_float, load_adapters, make_pool
from oracle import bdlora, mlp

pytestmark = pytest.mark.gpu
TOL = 1e-2
RANKS = [0, 4, 8, 16, 24, 5]
ACTS = {"none": (bd.ACT_NONE, [0]), "silu_mul": (bd.ACT_SILU_MUL, [0, 1])}


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    bd.lib()
    return torch


def _setup(T, seed, act_name):
    rng = np.random.default_rng(seed)
    ids = rng.integers(-1, len(RANKS), size=T)
    spec = wl.custom_workload(f"mlp-{T}", wl.tiny_mlp_projs(), T, RANKS,
                              scales=[0.5 + 0.3 * i for i in range(len(RANKS))], ids=ids, seed=seed)
    layer = wl.draw_layer(spec, slots=range(len(RANKS)))
    pool = make_pool(spec, max_tokens=T)
    load_adapters(pool, spec, range(len(RANKS)), cache=layer.adapters)
    return spec, layer, pool


def _run_mlp(torch, pool, dl, act, first, T):
    out = torch.empty((T, 160), dtype=torch.bfloat16, device="cuda")
    pool.forward_mlp(act, first, 2, dl.X[0], [dl.W[p] for p in first], dl.W[2], out, dl.ids)
    torch.cuda.synchronize()
    return device_to_float(out)


@pytest.mark.parametrize("act_name", ["none", "silu_mul"])
@pytest.mark.parametrize("T", [1, 16, 24, 37, 64, 100, 300])
def test_mlp_parity(torch_cuda, T, act_name):
    torch = torch_cuda
    spec, layer, pool = _setup(T, 100 + T, act_name)
    act, first = ACTS[act_name]
    dl = DeviceLayer(layer)
    y = _run_mlp(torch, pool, dl, act, first, T)
    _, ref = mlp.mlp_layer_forward(layer, first, 2, act_name)
    e = bdlora.rel_errors(y, ref)
    assert e["pointwise"] <= TOL, f"T={T} act={act_name}: {e}"
    assert pool.device_error() == 0
    pool.close()


@pytest.mark.parametrize("T", [12, 40, 200])
def test_mlp_equals_layer_calls_and_is_deterministic(torch_cuda, T):
    # act=none: H is the bf16 output of the first projection either way, so
    # the MLP entry point must reproduce, bit for bit, forward_layer on the
    # first projection followed by forward_shard on the down projection.
    # silu_mul: two calls give identical bits.
    torch = torch_cuda
    spec, layer, pool = _setup(T, 7 + T, "silu_mul")
    dl = DeviceLayer(layer)
    y1 = _run_mlp(torch, pool, dl, bd.ACT_SILU_MUL, [0, 1], T)
    y2 = _run_mlp(torch, pool, dl, bd.ACT_SILU_MUL, [0, 1], T)
    assert np.array_equal(y1.view(np.uint32), y2.view(np.uint32))
    y_none = _run_mlp(torch, pool, dl, bd.ACT_NONE, [0], T)
    g = torch.empty((T, 224), dtype=torch.bfloat16, device="cuda")
    pool.forward_layer([0], [dl.X[0]], [dl.W[0]], [g], dl.ids)
    out = torch.empty((T, 160), dtype=torch.bfloat16, device="cuda")
    pool.forward_shard(2, g, dl.W[2], dl.ids, out)
    torch.cuda.synchronize()
    assert np.array_equal(y_none.view(np.uint32), device_to_float(out).view(np.uint32))
    pool.close()


def test_mlp_8b_shapes_decode(torch_cuda):
    # Llama-3.1-8B MLP shard at 1/8 tensor parallelism: gate/up 4096 -> 1792,
    # down 1792 -> 4096, 64 decode tokens, 32 adapters of rank 16
    torch = torch_cuda
    projs = [p for p in wl.model_projs("llama-3.1-8b", 8) if p.name in ("gate", "up", "down")]
    T = 64
    rng = np.random.default_rng(8)
    ids = rng.integers(-1, 32, size=T)
    spec = wl.custom_workload("mlp-8b", projs, T, [16] * 32, ids=ids, seed=8)
    layer = wl.draw_layer(spec, slots=range(32))
    pool = make_pool(spec)
    load_adapters(pool, spec, range(32), cache=layer.adapters)
    dl = DeviceLayer(layer)
    out = torch.empty((T, 4096), dtype=torch.bfloat16, device="cuda")
    pool.forward_mlp(bd.ACT_SILU_MUL, [0, 1], 2, dl.X[0], [dl.W[0], dl.W[1]], dl.W[2], out, dl.ids)
    torch.cuda.synchronize()
    _, ref = mlp.mlp_layer_forward(layer, [0, 1], 2, "silu_mul")
    e = bdlora.rel_errors(device_to_float(out), ref)
    assert e["pointwise"] <= TOL, e
    pool.close()


@pytest.mark.parametrize("T", [72, 128])
def test_mlp_70b_shapes_medium_batch(torch_cuda, T):
    # Llama-3.1-70B MLP shard at 1/8 tensor parallelism: gate/up 8192 -> 3584,
    # down 3584 -> 8192.  At these batch sizes gate and up (117 MB of weight)
    # take the medium-batch launches, whose epilogue pairs gate's and up's
    # column tiles and writes H = silu(gate) * up once, in bf16, as down's
    # packed input; then down runs on its own path.
    torch = torch_cuda
    projs = [p for p in wl.model_projs("llama-3.1-70b", 8) if p.name in ("gate", "up", "down")]
    rng = np.random.default_rng(70 + T)
    ranks = [16, 8, 32, 16]
    ids = rng.integers(-1, len(ranks), size=T)
    spec = wl.custom_workload(f"mlp-70b-{T}", projs, T, ranks, scales=[2.0, 1.0, 0.5, 1.5], ids=ids, seed=70 + T)
    layer = wl.draw_layer(spec, slots=range(len(ranks)))
    pool = make_pool(spec, max_tokens=T)
    load_adapters(pool, spec, range(len(ranks)), cache=layer.adapters)
    dl = DeviceLayer(layer)
    # gate and up on their own take the medium-batch path
    g = [torch.empty((T, 3584), dtype=torch.bfloat16, device="cuda") for _ in range(2)]
    pool.forward_layer([0, 1], [dl.X[0], dl.X[0]], [dl.W[0], dl.W[1]], g, dl.ids)
    torch.cuda.synchronize()
    assert pool.last_path() == "medium"
    out = torch.empty((T, 8192), dtype=torch.bfloat16, device="cuda")
    pool.forward_mlp(bd.ACT_SILU_MUL, [0, 1], 2, dl.X[0], [dl.W[0], dl.W[1]], dl.W[2], out, dl.ids)
    torch.cuda.synchronize()
    _, ref = mlp.mlp_layer_forward(layer, [0, 1], 2, "silu_mul")
    e = bdlora.rel_errors(device_to_float(out), ref)
    assert e["pointwise"] <= TOL, f"T={T}: {e}"
    assert pool.device_error() == 0
    pool.close()


def test_mlp_argument_errors(torch_cuda):
    torch = torch_cuda
    spec, layer, pool = _setup(8, 3, "silu_mul")
    dl = DeviceLayer(layer)
    out = torch.empty((8, 160), dtype=torch.bfloat16, device="cuda")
    L = bd.lib()
    import ctypes
    ws = (ctypes.c_void_p * 2)(dl.W[0].data_ptr(), dl.W[1].data_ptr())

    def call(act, first, down):
        pr = (ctypes.c_int32 * 2)(*first, *([0] * (2 - len(first))))
        return L.bdlora_forward_mlp(pool._h, act, pr, down, dl.X[0].data_ptr(), ws, dl.W[2].data_ptr(),
                                    out.data_ptr(), dl.ids.data_ptr(), None, 8, None)
    assert call(bd.ACT_SILU_MUL, [0, 1], 2) == 0
    torch.cuda.synchronize()
    assert call(7, [0, 1], 2) == -1                  # unknown act
    assert call(bd.ACT_SILU_MUL, [0, 0], 2) == -1    # gate listed twice
    assert call(bd.ACT_SILU_MUL, [0, 2], 2) == -1    # down listed as up
    assert call(bd.ACT_NONE, [2], 0) == -1           # a row projection first
    assert call(bd.ACT_NONE, [0], 1) == -4           # gate's width is not up's d_in
    assert call(bd.ACT_NONE, [0], 5) == -1           # index out of range
    pool.close()


@pytest.mark.parametrize("act_name", ["silu_mul", "none"])
@pytest.mark.parametrize("T", [300, 600])
def test_mlp_8b_shapes_prefill_large_tiles(torch_cuda, T, act_name):
    # Llama-3.1-8B MLP shard at 1/8 TP above one 256-row tile: gate and up
    # take the large tiles, paired (each workgroup holds 128 gate and the
    # same 128 up columns), and their epilogue writes H once in bf16; runs of
    # requests sharing an adapter, as in prefill
    torch = torch_cuda
    projs = [p for p in wl.model_projs("llama-3.1-8b", 8) if p.name in ("gate", "up", "down")]
    rng = np.random.default_rng(T)
    ranks = [16, 32, 8, 16, 64, 24]
    ids = np.repeat(rng.integers(-1, len(ranks), size=T // 50 + 1), 50)[:T]
    spec = wl.custom_workload(f"mlp-8b-{T}", projs, T, ranks, ids=ids, seed=T + 3)
    layer = wl.draw_layer(spec, slots=range(len(ranks)))
    pool = make_pool(spec)
    load_adapters(pool, spec, range(len(ranks)), cache=layer.adapters)
    dl = DeviceLayer(layer)
    g = [torch.empty((T, 1792), dtype=torch.bfloat16, device="cuda") for _ in range(2)]
    pool.forward_layer([0, 1], [dl.X[0], dl.X[0]], [dl.W[0], dl.W[1]], g, dl.ids)
    torch.cuda.synchronize()
    assert pool.last_path() == "large"
    act, first = ACTS[act_name]
    out = torch.full((T, 4096), float("nan"), dtype=torch.bfloat16, device="cuda")
    pool.forward_mlp(act, first, 2, dl.X[0], [dl.W[p] for p in first], dl.W[2], out, dl.ids)
    torch.cuda.synchronize()
    _, ref = mlp.mlp_layer_forward(layer, first, 2, act_name)
    e = bdlora.rel_errors(device_to_float(out), ref)
    assert e["pointwise"] <= TOL, f"T={T} act={act_name}: {e}"
    # the same batch as segments: the same bits
    out2 = torch.full_like(out, float("nan"))
    pool.forward_mlp(act, first, 2, dl.X[0], [dl.W[p] for p in first], dl.W[2], out2, None,
                     segs=bd.Segments.from_ids(ids))
    torch.cuda.synchronize()
    assert np.array_equal(device_to_float(out).view(np.uint32), device_to_float(out2).view(np.uint32))
    assert pool.device_error() == 0
    pool.close()
