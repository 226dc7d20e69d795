"""GPU parity of the INT4 base weight (weight-only quantized base, Sec. 5.2)
through the C ABI against the fp64 oracle on the same stored nibbles and
scales.  Same error rule as the bf16 parity tests."""
import numpy as np
import pytest

import workloads as wl
from workloads.gpu import DeviceLayer, bits_to_device, device_to_float, load_adapters, make_pool
from oracle import bdlora, quant

pytestmark = pytest.mark.gpu
TOL = 1e-2
RANKS = [0, 1, 3, 8, 16, 24, 5, 32]


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    import paper_2510_23346_amd as bd
    bd.lib()
    return torch


def int4_projs():
    """Small INT4-compatible projections: d_in a multiple of 128, outputs a
    multiple of 64 (q/k/v slices of 128 + 64 + 64)."""
    return [
        wl.ProjSpec("qkv", "column", 256, (128, 64, 64)),
        wl.ProjSpec("o", "row", 128, (192,)),
        wl.ProjSpec("up", "column", 384, (320,)),
    ]


def _layer(T, seed, ranks=RANKS, projs=None):
    rng = np.random.default_rng(seed)
    ids = rng.integers(-1, len(ranks), size=T)
    spec = wl.custom_workload(f"int4-{T}", projs or int4_projs(), T, ranks,
                              scales=[0.5 + 0.25 * i for i in range(len(ranks))], ids=ids, seed=seed,
                              weight_format="int4_g128")
    layer = wl.draw_layer(spec, slots=range(len(ranks)))
    pool = make_pool(spec, max_tokens=T)
    load_adapters(pool, spec, range(len(ranks)), cache=layer.adapters)
    return spec, layer, pool


def _run(torch, spec, layer, pool, ids=None):
    dl = DeviceLayer(layer)
    outs = dl.out
    if ids is not None:
        outs = [torch.empty_like(o) for o in dl.out]
    pool.forward_layer(list(range(len(spec.projs))), dl.X, dl.W, outs, dl.ids if ids is None else ids)
    torch.cuda.synchronize()
    return dl, [device_to_float(o) for o in outs]


@pytest.mark.parametrize("T", [1, 16, 24, 37, 64, 100, 300])
def test_int4_parity(torch_cuda, T):
    torch = torch_cuda
    spec, layer, pool = _layer(T, 40 + T)
    dl, ys = _run(torch, spec, layer, pool)
    _, yb = _run(torch, spec, layer, pool, ids=torch.full_like(dl.ids, -1))
    refs = quant.layer_forward_w4(layer)
    for p, pi in enumerate(layer.projs):
        rb = pi.X.astype(np.float64) @ quant.dequantize(pi.Wq, pi.Ws_bits, pi.spec.d_in)
        e = bdlora.rel_errors(ys[p], refs[p])
        assert e["pointwise"] <= TOL, f"T={T} {pi.spec.name}: {e}"
        assert bdlora.rel_errors(yb[p], rb)["pointwise"] <= TOL, f"T={T} {pi.spec.name} base"
        assert bdlora.delta_errors(ys[p], yb[p], refs[p], rb) <= TOL
    assert pool.device_error() == 0
    pool.close()


def _int4_layout(q: np.ndarray, s: np.ndarray) -> np.ndarray:
    """The packed INT4 buffer as the header documents it, built on the host."""
    N, K = q.shape[0], 2 * q.shape[1]
    nib = np.empty((N, K), dtype=np.uint32)
    nib[:, 0::2] = q & 15
    nib[:, 1::2] = q >> 4
    KS = K // 32
    words = np.zeros((N // 16, KS, 64), dtype=np.uint32)
    for lane in range(64):
        n = np.arange(N // 16)[:, None] * 16 + lane % 16
        for i in range(8):
            k = np.arange(KS)[None, :] * 32 + 8 * (lane // 16) + i
            words[:, :, lane] |= nib[n, k] << np.uint32(4 * (i // 2) + 16 * (i % 2))
    G = K // 128
    sc = s.reshape(N // 16, 16, G).transpose(0, 2, 1).reshape(-1)
    return np.concatenate([words.reshape(-1).view(np.uint8), sc.astype(np.uint16).view(np.uint8)])


@pytest.mark.parametrize("N,K", [(64, 128), (192, 384)])
def test_pack_int4_layout_bit_exact(torch_cuda, N, K):
    torch = torch_cuda
    import paper_2510_23346_amd as bd
    rng = np.random.default_rng(N + K)
    q = rng.integers(0, 256, size=(N, K // 2), dtype=np.uint8)
    s = rng.integers(0, 1 << 16, size=(N, K // 128), dtype=np.uint16)
    P = bd.pack_weight_int4(torch.from_numpy(q).cuda(), bits_to_device(s))
    torch.cuda.synchronize()
    got = P.cpu().numpy()
    assert got.size == bd.packed_weight_bytes(bd.WEIGHT_INT4_G128, N, K)
    assert np.array_equal(got, _int4_layout(q, s))
    with pytest.raises(ValueError):
        bd.pack_weight_int4(torch.from_numpy(q[:48]).cuda(), bits_to_device(s[:48]))      # N % 64
    # the library's own checks: N % 64, K % 128, null pointers
    qd, sd = torch.from_numpy(q).cuda(), bits_to_device(s)
    L = bd.lib()
    assert L.bdlora_pack_weight_int4(qd.data_ptr(), sd.data_ptr(), P.data_ptr(), 48, K, None) == -4
    assert L.bdlora_pack_weight_int4(qd.data_ptr(), sd.data_ptr(), P.data_ptr(), N, K - 64, None) == -4
    assert L.bdlora_pack_weight_int4(None, sd.data_ptr(), P.data_ptr(), N, K, None) == -1


def test_int4_decode_and_prefill_agree(torch_cuda):
    # the same rows through the decode launches (T = 64) and through the
    # prefill launches (the first 64 of T = 200): both within tolerance of the
    # oracle and of each other
    torch = torch_cuda
    spec, layer, pool = _layer(200, 9)
    dl = DeviceLayer(layer)
    projs = list(range(len(spec.projs)))
    pool.forward_layer(projs, dl.X, dl.W, dl.out, dl.ids)
    small = [torch.empty((64, o.shape[1]), dtype=o.dtype, device=o.device) for o in dl.out]
    pool.forward_layer(projs, [x[:64] for x in dl.X], dl.W, small, dl.ids[:64])
    torch.cuda.synchronize()
    refs = quant.layer_forward_w4(layer, rows=np.arange(64))
    for p in projs:
        a, b = device_to_float(dl.out[p])[:64], device_to_float(small[p])
        assert bdlora.rel_errors(a, refs[p])["pointwise"] <= TOL
        assert bdlora.rel_errors(b, refs[p])["pointwise"] <= TOL
    pool.close()


def test_int4_8b_layer_decode(torch_cuda):
    # Llama-3.1-8B decoder-layer shard at 1/8 TP with an INT4 base: 64 decode
    # tokens, 32 adapters of rank 16, Zipf ids (the default benchmark
    # workload with a quantized base)
    torch = torch_cuda
    s1 = wl.workload(1)
    spec = wl.WorkloadSpec(s1.name + "-int4", s1.model, s1.tp, s1.projs, s1.T, s1.n_slots, s1.ranks,
                           s1.scales, s1.ids_kind, s1.seed, weight_format="int4_g128")
    # every slot loaded, as the benchmark does (same launch geometry)
    slots = list(range(spec.n_slots))
    layer = wl.draw_layer(spec, slots=slots)
    pool = make_pool(spec)
    load_adapters(pool, spec, slots, cache=layer.adapters)
    dl, ys = _run(torch, spec, layer, pool)
    refs = quant.layer_forward_w4(layer)
    # the LoRA term alone: the base-only forward (every id -1) against the
    # oracle's product with the decoded INT4 weight
    base = [torch.full_like(o, float("nan")) for o in dl.out]
    pool.forward_layer(list(range(len(spec.projs))), dl.X, dl.W, base, torch.full_like(dl.ids, -1))
    torch.cuda.synchronize()
    for p, pi in enumerate(layer.projs):
        e = bdlora.rel_errors(ys[p], refs[p])
        assert e["pointwise"] <= TOL, f"{pi.spec.name}: {e}"
        Wd = quant.dequantize(pi.Wq, pi.Ws_bits, pi.spec.d_in)
        rbase = pi.X.astype(np.float64) @ Wd
        d = bdlora.delta_errors(ys[p], device_to_float(base[p]), refs[p], rbase)
        assert d <= TOL, f"{pi.spec.name}: LoRA-term error {d}"
    assert pool.device_error() == 0
    pool.close()


def test_int4_mlp(torch_cuda):
    # the MLP entry point with INT4 gate / up / down
    torch = torch_cuda
    import paper_2510_23346_amd as bd
    from oracle import mlp
    # down's d_in (the intermediate width) must be a multiple of 128 for INT4
    projs = [wl.ProjSpec("gate", "column", 256, (256,)), wl.ProjSpec("up", "column", 256, (256,)),
             wl.ProjSpec("down", "row", 256, (128,))]
    for T in (24, 130):
        spec, layer, pool = _layer(T, 70 + T, ranks=[8, 16, 4], projs=projs)
        dl = DeviceLayer(layer)
        out = torch.empty((T, 128), dtype=torch.bfloat16, device="cuda")
        pool.forward_mlp(bd.ACT_SILU_MUL, [0, 1], 2, dl.X[0], [dl.W[0], dl.W[1]], dl.W[2], out, dl.ids)
        torch.cuda.synchronize()
        ad = lambda p: {s: (a.scale, a.A[p], a.B[p]) for s, a in layer.adapters.items()}
        X = layer.projs[0].X
        Wd = [quant.dequantize(pi.Wq, pi.Ws_bits, pi.spec.d_in) for pi in layer.projs]
        _, ref = mlp.mlp_shard_forward(X, [(Wd[0], ad(0)), (Wd[1], ad(1))], (Wd[2], ad(2)), layer.ids, "silu_mul")
        e = bdlora.rel_errors(device_to_float(out), ref)
        assert e["pointwise"] <= TOL, f"T={T}: {e}"
        pool.close()
