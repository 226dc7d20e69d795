"""GPU parity: the HIP path through the C ABI against the fp64 oracle.

Error rule (bf16 inputs, fp32 accumulation, bf16 output): every element must
satisfy |y - ref| <= 1e-2 * max(|ref|, rms(ref)).  The LoRA term alone
(y - y_base against ref - ref_base) is held to the same rule with the full
output's rms as floor, after allowing the two bf16 output roundings the
difference of two GPU outputs carries (2^-8 (|y| + |y_base|)).  Integer plan
results are compared exactly.
"""
import dataclasses

import numpy as np
import pytest

import workloads as wl
from workloads.gpu import DeviceLayer, device_to_float, load_adapters, make_pool
from oracle import bdlora, plan as oplan

pytestmark = pytest.mark.gpu
TOL = 1e-2


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    import paper_2510_23346_amd as bd
    bd.lib()                                   # loud failure if the library is missing
    return torch


def _run_layer(torch, spec, layer, pool, T=None):
    dl = DeviceLayer(layer, T=T)
    pool.forward_layer(list(range(len(spec.projs))), dl.X, dl.W, dl.out, dl.ids)
    torch.cuda.synchronize()
    return dl, dl.outputs()


def _base_only(torch, spec, dl, pool):
    ids_none = torch.full_like(dl.ids, -1)
    outs = [torch.full_like(o, float("nan")) for o in dl.out]
    pool.forward_layer(list(range(len(spec.projs))), dl.X, dl.W, outs, ids_none)
    torch.cuda.synchronize()
    return [device_to_float(o) for o in outs]


def _check(y, ref, y_base=None, ref_base=None, what=""):
    e = bdlora.rel_errors(y, ref)
    assert e["pointwise"] <= TOL, f"{what}: {e}"
    if y_base is not None:
        d = bdlora.delta_errors(y, y_base, ref, ref_base)
        assert d <= TOL, f"{what}: LoRA-term error {d}"
    return e


def _oracle_base(layer, rows=None):
    outs = []
    for pi in layer.projs:
        X = pi.X if rows is None else pi.X[rows]
        outs.append(X.astype(np.float64) @ pi.W.astype(np.float64))
    return outs


# ---------------------------------------------------------------------------
# small shapes: several tiles, ragged tails, odd ranks, id -1, rank 0
# ---------------------------------------------------------------------------

TINY_RANKS = [0, 1, 3, 8, 16, 24, 5, 32]


@pytest.mark.parametrize("T", [1, 5, 16, 24, 37, 64, 100, 300, 700])
def test_tiny_parity(torch_cuda, T):
    torch = torch_cuda
    rng = np.random.default_rng(T)
    ids = rng.integers(-1, len(TINY_RANKS), size=T)
    spec = wl.custom_workload(f"tiny-{T}", wl.tiny_projs(), T, TINY_RANKS,
                              scales=[0.5 + 0.25 * i for i in range(len(TINY_RANKS))], ids=ids, seed=T)
    layer = wl.draw_layer(spec, slots=range(len(TINY_RANKS)))
    pool = make_pool(spec, max_tokens=T)
    load_adapters(pool, spec, range(len(TINY_RANKS)), cache=layer.adapters)
    dl, ys = _run_layer(torch, spec, layer, pool)
    yb = _base_only(torch, spec, dl, pool)
    refs = bdlora.layer_forward(layer)
    rb = _oracle_base(layer)
    for p in range(len(spec.projs)):
        _check(ys[p], refs[p], yb[p], rb[p], what=f"T={T} proj={spec.projs[p].name}")
    assert pool.device_error() == 0
    pool.close()


def test_consecutive_batches_on_one_pool(torch_cuda):
    """Two adapted batches of different sizes through one pool (the shrink's
    unit counter, the plan tables and the partial workspaces are reused):
    each matches the oracle on every row.  Rows are computed independently,
    so the first 300 rows of the 700-token forward are the smaller batch's
    reference."""
    torch = torch_cuda
    T = 700
    rng = np.random.default_rng(77)
    ids = rng.integers(-1, len(TINY_RANKS), size=T)
    spec = wl.custom_workload("two-batches", wl.tiny_projs(), T, TINY_RANKS,
                              scales=[0.5 + 0.25 * i for i in range(len(TINY_RANKS))], ids=ids, seed=77)
    layer = wl.draw_layer(spec, slots=range(len(TINY_RANKS)))
    pool = make_pool(spec, max_tokens=T)
    load_adapters(pool, spec, range(len(TINY_RANKS)), cache=layer.adapters)
    refs = bdlora.layer_forward(layer)
    for t in (T, 300, T):
        _, ys = _run_layer(torch, spec, layer, pool, T=t)
        for p in range(len(spec.projs)):
            _check(ys[p], refs[p][:t], what=f"T={t} proj={spec.projs[p].name}")
    assert pool.device_error() == 0
    pool.close()


def test_base_only_rows_equal_no_adapter_rows(torch_cuda):
    torch = torch_cuda
    T = 48
    ids = np.array([(-1 if t % 3 == 0 else (0 if t % 3 == 1 else 1)) for t in range(T)])
    spec = wl.custom_workload("r0", wl.tiny_projs(), T, [0, 8], ids=ids, seed=3)
    layer = wl.draw_layer(spec, slots=[0, 1])
    pool = make_pool(spec)
    load_adapters(pool, spec, [0, 1], cache=layer.adapters)
    dl, ys = _run_layer(torch, spec, layer, pool)
    yb = _base_only(torch, spec, dl, pool)
    for p in range(len(spec.projs)):
        rows = np.nonzero(ids <= 0)[0]          # id -1 and the rank-0 adapter
        assert np.array_equal(ys[p][rows], yb[p][rows])     # value equality (+0 == -0)
        _check(yb[p], _oracle_base(layer)[p], what="base only")
    pool.close()


def test_decode_path_is_deterministic(torch_cuda):
    torch = torch_cuda
    T = 40
    spec = wl.custom_workload("det-dec", wl.tiny_projs(), T, [8, 16, 4], seed=6)
    layer = wl.draw_layer(spec, slots=[0, 1, 2])
    pool = make_pool(spec)
    load_adapters(pool, spec, [0, 1, 2], cache=layer.adapters)
    _, y1 = _run_layer(torch, spec, layer, pool)
    _, y2 = _run_layer(torch, spec, layer, pool)
    for a, b in zip(y1, y2):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    pool.close()


def test_deterministic_and_shard_equals_layer(torch_cuda):
    torch = torch_cuda
    T = 70
    spec = wl.custom_workload("det", wl.tiny_projs(), T, [8, 16, 4], seed=5)
    layer = wl.draw_layer(spec, slots=[0, 1, 2])
    pool = make_pool(spec)
    load_adapters(pool, spec, [0, 1, 2], cache=layer.adapters)
    dl, y1 = _run_layer(torch, spec, layer, pool)
    _, y2 = _run_layer(torch, spec, layer, pool)
    for a, b in zip(y1, y2):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    for p in range(len(spec.projs)):
        o = torch.empty_like(dl.out[p])
        pool.forward_shard(p, dl.X[p], dl.W[p], dl.ids, o)
        torch.cuda.synchronize()
        assert np.array_equal(device_to_float(o).view(np.uint32), y1[p].view(np.uint32))
    pool.close()


# ---------------------------------------------------------------------------
# plan: bit-exact against the host plan and the oracle; error flag
# ---------------------------------------------------------------------------

# kinds: "uniform" ids over the pool; "runs": requests of 100 tokens sharing
# an adapter, then 150 scattered decode tokens (prefill + decode batches).
# The cases cover the plan's placement by all waves (batches over 1024
# tokens with at most 256 adapters in pools of at most 4096 slots; chunks of
# one and of many adapters), its single-wave fallback (more adapters, or a
# larger pool) and the per-token count of smaller batches.
@pytest.mark.parametrize("T,n_slots,kind", [(1, 4, "uniform"), (64, 32, "uniform"), (333, 20, "uniform"),
                                            (4288, 512, "uniform"), (4288, 128, "uniform"), (4288, 512, "runs"),
                                            (1500, 4200, "runs"), (8192, 300, "runs")])
def test_plan_device_bit_exact(torch_cuda, T, n_slots, kind):
    torch = torch_cuda
    import paper_2510_23346_amd as bd
    rng = np.random.default_rng(T + n_slots)
    if kind == "uniform":
        ids = rng.integers(-1, n_slots, size=T).astype(np.int32)
    else:
        ids = np.concatenate([np.repeat(rng.integers(-1, n_slots, size=T // 100 + 1), 100)[:T - 150],
                              rng.integers(-1, n_slots, size=150)]).astype(np.int32)
    ids[::17] = n_slots + 3                  # out of range
    ids[1::29] = -7                          # negative, not -1
    unloaded = {1, n_slots - 1}
    projs = [("column", 64, (16,))]
    pool = bd.Pool(projs, n_slots, 8, T)
    z = np.zeros((64, 2), np.uint16)
    zb = np.zeros((2, 16), np.uint16)
    for s in range(n_slots):
        if s not in unloaded:
            pool.load_adapter(s, 2, 1.0, [[z]], [[zb]])
    loaded = pool.loaded.copy()
    ids_d = torch.from_numpy(ids).cuda()
    G = min(T, n_slots)
    vid = torch.empty(T, dtype=torch.int32, device="cuda")
    perm = torch.empty(T, dtype=torch.int32, device="cuda")
    gs, gst, gc = (torch.empty(G, dtype=torch.int32, device="cuda") for _ in range(3))
    ng = torch.zeros(1, dtype=torch.int32, device="cuda")
    pool.plan_device(ids_d, vid, gs, gst, gc, perm, ng)
    torch.cuda.synchronize()
    ovid, oerr = oplan.validate(ids, loaded)
    otab, operm = oplan.groups(ovid)
    n = int(ng.item())
    assert np.array_equal(vid.cpu().numpy(), ovid)
    assert n == len(otab)
    got = list(zip(gs.cpu().numpy()[:n].tolist(), gst.cpu().numpy()[:n].tolist(), gc.cpu().numpy()[:n].tolist()))
    assert got == [tuple(x) for x in otab]
    assert np.array_equal(perm.cpu().numpy()[:len(operm)], operm)
    rc, hvid, htab, hperm = bd.build_plan(loaded, ids)
    assert rc == (-3 if oerr else 0)
    assert np.array_equal(hvid, ovid) and htab == [tuple(x) for x in otab] and np.array_equal(hperm, operm)
    assert pool.device_error() == int(oerr)
    assert pool.device_error() == 0          # cleared by the read
    pool.close()


@pytest.mark.parametrize("T", [40, 12])
def test_invalid_ids_are_base_only_and_flagged(torch_cuda, T):
    # 12 tokens: batches of at most 16 plan inside the decode launch itself
    torch = torch_cuda
    ids = np.array([t % 4 for t in range(T)])
    ids[5] = 99
    ids[6] = 3                                # slot 3 will be unloaded
    spec = wl.custom_workload("bad", wl.tiny_projs(), T, [8, 8, 8, 8], ids=ids, seed=7)
    layer = wl.draw_layer(spec, slots=[0, 1, 2, 3])
    pool = make_pool(spec)
    load_adapters(pool, spec, [0, 1, 2, 3], cache=layer.adapters)
    pool.unload_adapter(3)
    dl, ys = _run_layer(torch, spec, layer, pool)
    assert pool.device_error() == 1
    vid, _ = oplan.validate(ids, pool.loaded)
    layer.ids = vid
    refs = bdlora.layer_forward(layer)
    for p in range(len(spec.projs)):
        _check(ys[p], refs[p], what="invalid ids")
    pool.close()


@pytest.mark.parametrize("T", [60, 14])
@pytest.mark.parametrize("n_slots", [64, 150])
def test_decode_plan_pool_sizes(torch_cuda, n_slots, T):
    # decode batches plan in one wave: pools of up to 64 slots keep the slot
    # tables in lanes (slot 63 is the mask's top bit), larger pools take the
    # per-pass minimum; unloaded and out-of-range ids must read as -1.  At 14
    # tokens the plan runs inside the decode launch, at 60 in its own launch
    torch = torch_cuda
    rng = np.random.default_rng(n_slots)
    loaded = sorted(set(rng.choice(n_slots, size=min(40, n_slots - 1), replace=False).tolist()) | {0, n_slots - 1})
    ids = rng.choice(loaded, size=T)
    ids[:4] = [n_slots - 1, 0, -1, n_slots - 1]
    ids[7] = n_slots + 5                       # out of range
    unloaded = [s for s in range(n_slots) if s not in loaded][0]
    ids[9] = unloaded
    ranks = [8 if s % 3 else 16 for s in range(n_slots)]
    spec = wl.custom_workload(f"pool{n_slots}", wl.tiny_projs(), T, ranks, ids=ids, seed=n_slots)
    layer = wl.draw_layer(spec, slots=loaded)
    pool = make_pool(spec)
    load_adapters(pool, spec, loaded, cache=layer.adapters)
    dl, ys = _run_layer(torch, spec, layer, pool)
    assert pool.device_error() == 1
    vid, _ = oplan.validate(ids, pool.loaded)
    layer.ids = vid
    refs = bdlora.layer_forward(layer)
    for p in range(len(spec.projs)):
        _check(ys[p], refs[p], what=f"pool {n_slots} proj {spec.projs[p].name}")
    pool.close()


def _fragment_layout(W):
    """Reference of the packed weight layout: 16-row blocks x 32-wide k-steps,
    element [(rb*KS + ks)*512 + lane*8 + i] = W[16 rb + lane%16][32 ks + 8 (lane//16) + i]."""
    N, K = W.shape
    KS = K // 32
    out = np.empty(N * K, W.dtype)
    for rb in range(N // 16):
        for ks in range(KS):
            for lane in range(64):
                base = (rb * KS + ks) * 512 + lane * 8
                out[base:base + 8] = W[16 * rb + lane % 16, 32 * ks + 8 * (lane // 16): 32 * ks + 8 * (lane // 16) + 8]
    return out


@pytest.mark.parametrize("N,K", [(16, 32), (48, 96), (80, 256)])
def test_pack_weight_layout_bit_exact(torch_cuda, N, K):
    torch = torch_cuda
    import paper_2510_23346_amd as bd
    rng = np.random.default_rng(N + K)
    W = rng.integers(0, 1 << 16, size=(N, K), dtype=np.uint16)
    Wd = torch.from_numpy(W.view(np.int16)).cuda()
    P = bd.pack_weight(Wd)
    torch.cuda.synchronize()
    got = P.cpu().numpy().view(np.uint16).reshape(-1)
    assert np.array_equal(got, _fragment_layout(W))
    with pytest.raises(bd.BDLoRAError):
        bd.pack_weight(Wd[:, :K - 8].contiguous())                               # K not a multiple of 32


def test_empty_batch_and_errors(torch_cuda):
    torch = torch_cuda
    import paper_2510_23346_amd as bd
    spec = wl.custom_workload("err", wl.tiny_projs(), 8, [8], seed=1)
    layer = wl.draw_layer(spec, slots=[0])
    pool = make_pool(spec)
    load_adapters(pool, spec, [0], cache=layer.adapters)
    dl = DeviceLayer(layer)
    e = torch.empty((0, spec.projs[0].d_out), dtype=torch.bfloat16, device="cuda")
    pool.forward_shard(0, dl.X[0][:0], dl.W[0], dl.ids[:0], e, T=0)
    xp, wp, op = dl.X[0].data_ptr(), dl.W[0].data_ptr(), dl.out[0].data_ptr()
    with pytest.raises(bd.BDLoRAError) as e:
        pool.forward_shard(0, xp, wp, dl.ids, op, T=9)                          # T > max_tokens
    assert e.value.code == -4
    with pytest.raises(bd.BDLoRAError) as e:
        pool.forward_shard(5, xp, wp, dl.ids, op, T=8)                          # no such projection
    assert e.value.code == -1
    with pytest.raises(bd.BDLoRAError) as e:
        pool.forward_shard(0, xp + 2, wp, dl.ids, op, T=8)                      # misaligned X
    assert e.value.code == -1
    with pytest.raises(ValueError):
        pool.forward_shard(0, dl.X[0], dl.W[0], dl.ids, dl.out[0], T=9)         # binding shape check
    A9 = [[np.zeros((ps.d_in, 9), np.uint16) for _ in ps.slices] for ps in spec.projs]
    B9 = [[np.zeros((9, n), np.uint16) for n in ps.slices] for ps in spec.projs]
    with pytest.raises(bd.BDLoRAError) as e:
        pool.load_adapter(0, 9, 1.0, A9, B9)                                    # rank > max_rank
    assert e.value.code == -1
    bad = [[a.copy() for a in row] for row in layer.adapters[0].A_bits]
    bad[0][0][0, 0] = 0x7FC0                                                    # NaN
    with pytest.raises(bd.BDLoRAError):
        pool.load_adapter(0, 8, 1.0, bad, layer.adapters[0].B_bits)
    pool.close()


# ---------------------------------------------------------------------------
# the N shards of one layer, run one after another on one GPU (Sec. 3)
# ---------------------------------------------------------------------------

def test_all_shards_reassemble_the_unsharded_layer(torch_cuda):
    torch = torch_cuda
    import paper_2510_23346_amd as bd
    from workloads import bf16_round
    rng = np.random.default_rng(42)
    N, S, d, di, r_tot = 4, 24, 128, 256, 32
    bf = lambda shape, sc: bf16_round(rng.standard_normal(shape).astype(np.float32) * sc)
    Xb, X = bf((S, d), 1.0)
    W1b, W1 = bf((d, di), d ** -0.5)            # column layer d -> di
    A1b, A1 = bf((d, r_tot), d ** -0.5)
    B1b, B1 = bf((r_tot // N, di), (r_tot // N) ** -0.5)     # compact block-diagonal B
    W2b, W2 = bf((di, d), di ** -0.5)           # row layer di -> d
    A2b, A2 = bf((di, r_tot // N), di ** -0.5)               # compact block-diagonal A
    B2b, B2 = bf((r_tot, d), (r_tot // N) ** -0.5)
    gamma = 2.0
    ids = torch.zeros(S, dtype=torch.int32, device="cuda")
    col_parts, row_sum = [], np.zeros((S, d))
    Y1 = np.zeros((S, di), np.float32)
    for i, ((a1, b1), (a1b, b1b)) in enumerate(zip(bdlora.column_shards(A1, B1, N),
                                                 bdlora.column_shards(A1b, B1b, N))):
        n_s = di // N
        pool = bd.Pool([("column", d, (n_s,))], 1, r_tot // N, S)
        pool.load_adapter(0, r_tot // N, gamma, [[np.ascontiguousarray(a1b)]], [[np.ascontiguousarray(b1b)]])
        Xd = torch.from_numpy(Xb.view(np.int16)).cuda().view(torch.bfloat16)
        Wd = bd.pack_weight(torch.from_numpy(np.ascontiguousarray(W1b[:, i * n_s:(i + 1) * n_s].T).view(np.int16)).cuda().view(torch.bfloat16))
        out = torch.empty((S, n_s), dtype=torch.bfloat16, device="cuda")
        pool.forward_shard(0, Xd, Wd, ids, out)
        torch.cuda.synchronize()
        col_parts.append(device_to_float(out))
        pool.close()
    y_col = np.concatenate(col_parts, axis=1)
    _check(y_col, bdlora.column_full(X, W1, A1, B1, N, gamma), what="column shards")
    for i, ((a2, b2), (a2b, b2b)) in enumerate(zip(bdlora.row_shards(A2, B2, N), bdlora.row_shards(A2b, B2b, N))):
        k_s = di // N
        pool = bd.Pool([("row", k_s, (d,))], 1, r_tot // N, S)
        pool.load_adapter(0, r_tot // N, gamma, [[np.ascontiguousarray(a2b)]], [[np.ascontiguousarray(b2b)]])
        Xs = np.ascontiguousarray(bf16_round(y_col[:, i * k_s:(i + 1) * k_s])[0])
        Xd = torch.from_numpy(Xs.view(np.int16)).cuda().view(torch.bfloat16)
        Wd = bd.pack_weight(torch.from_numpy(np.ascontiguousarray(W2b[i * k_s:(i + 1) * k_s, :].T).view(np.int16)).cuda().view(torch.bfloat16))
        out = torch.empty((S, d), dtype=torch.bfloat16, device="cuda")
        pool.forward_shard(0, Xd, Wd, ids, out)
        torch.cuda.synchronize()
        row_sum += device_to_float(out)
        pool.close()
    Y1r = bf16_round(y_col)[1]
    _check(row_sum, bdlora.row_full(Y1r, W2, A2, B2, N, gamma), what="row partial sum")


# ---------------------------------------------------------------------------
# the five benchmark workloads at full size
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("index", [0, 1, 2, 3, 4])
def test_workload_parity(torch_cuda, index):
    # the resident set bench.py loads (every slot of the pool, config 4's 512
    # included), so the launch geometry checked here is the one it times;
    # every row of every output is compared with the oracle
    torch = torch_cuda
    spec = wl.workload(index)
    ids = wl.draw_ids(spec)
    slots = list(range(spec.n_slots))
    layer = wl.draw_layer(spec, slots=slots)
    pool = make_pool(spec)
    load_adapters(pool, spec, slots, cache=layer.adapters)
    dl, ys = _run_layer(torch, spec, layer, pool)
    yb = _base_only(torch, spec, dl, pool)
    refs = bdlora.layer_forward(layer)
    rbase = _oracle_base(layer)
    for p in range(len(spec.projs)):
        _check(ys[p], refs[p], yb[p], rbase[p], what=f"{spec.name} {spec.projs[p].name}")
    assert pool.device_error() == 0
    pool.close()


@pytest.mark.parametrize("index", [5, 6])
def test_decode_variants_parity(torch_cuda, index):
    # the 8B decode layer with an INT4 base (5) and with ranks alternating 8
    # and 64 in slots sized for 64 (6: a rank-8 adapter streams its own A^T
    # blocks only), every slot loaded as in the benchmark, every row compared
    torch = torch_cuda
    from oracle import quant
    spec = wl.workload(index)
    slots = list(range(spec.n_slots))
    layer = wl.draw_layer(spec, slots=slots)
    pool = make_pool(spec)
    load_adapters(pool, spec, slots, cache=layer.adapters)
    dl, ys = _run_layer(torch, spec, layer, pool)
    assert pool.last_path() == "decode"
    yb = _base_only(torch, spec, dl, pool)
    if spec.weight_format == "int4_g128":
        refs = quant.layer_forward_w4(layer)
        rbase = [pi.X.astype(np.float64) @ quant.dequantize(pi.Wq, pi.Ws_bits, pi.spec.d_in) for pi in layer.projs]
    else:
        refs = bdlora.layer_forward(layer)
        rbase = _oracle_base(layer)
    for p in range(len(spec.projs)):
        _check(ys[p], refs[p], yb[p], rbase[p], what=f"{spec.name} {spec.projs[p].name}")
    assert pool.device_error() == 0
    pool.close()


@pytest.mark.parametrize("model,T,in_main", [("llama-3.1-8b", 32, True), ("llama-3.1-70b", 24, True),
                                             ("llama-3.1-70b", 32, False), ("llama-3.1-70b", 17, True)])
def test_decode_plan_in_main_boundary(torch_cuda, model, T, in_main):
    # decode batches of two row blocks plan inside the K-split launch while
    # their activations stay small (the 8B layer shard at 32 tokens, the 70B
    # one up to about 26) and take the plan launch above that; both forms
    # are compared with the oracle on every row
    torch = torch_cuda
    import paper_2510_23346_amd as bd
    ranks = [16, 8, 32, 64, 16, 8]
    base = wl.workload(3) if model == "llama-3.1-70b" else wl.workload(1)
    spec = dataclasses.replace(base, name=f"boundary-{model}-{T}", T=T, n_slots=len(ranks), ranks=ranks,
                               scales=[2.0, 1.0, 0.5, 1.5, 1.0, 0.75], seed=700 + T)
    assert bd.decode_plans_in_main(T, [p.d_in for p in spec.projs]) == in_main
    slots = list(range(len(ranks)))
    layer = wl.draw_layer(spec, slots=slots)
    pool = make_pool(spec, max_tokens=T)
    load_adapters(pool, spec, slots, cache=layer.adapters)
    dl, ys = _run_layer(torch, spec, layer, pool)
    assert pool.last_path() == "decode"
    yb = _base_only(torch, spec, dl, pool)
    refs = bdlora.layer_forward(layer)
    rbase = _oracle_base(layer)
    for p in range(len(spec.projs)):
        _check(ys[p], refs[p], yb[p], rbase[p], what=f"{spec.name} {spec.projs[p].name}")
    assert pool.device_error() == 0
    pool.close()


def test_mixed_rank_decode_small_shapes(torch_cuda):
    # own-rank blocks on shapes where weight and adapter blocks share groups
    # (N / 16 not a multiple of 4) and adapters of ranks 1..64 sit in slots
    # sized for 64; several batches on one pool, some ids unused or -1
    torch = torch_cuda
    ranks = [64, 1, 8, 0, 24, 64, 3, 16, 40, 8]
    for T, seed in ((64, 1), (17, 2), (40, 3)):
        rng = np.random.default_rng(seed)
        ids = rng.integers(-1, len(ranks), size=T)
        spec = wl.custom_workload(f"mixed-{T}", wl.tiny_projs(), T, ranks, ids=ids, seed=seed)
        layer = wl.draw_layer(spec, slots=range(len(ranks)))
        pool = make_pool(spec)
        load_adapters(pool, spec, range(len(ranks)), cache=layer.adapters)
        dl, ys = _run_layer(torch, spec, layer, pool)
        yb = _base_only(torch, spec, dl, pool)
        refs = bdlora.layer_forward(layer)
        rb = _oracle_base(layer)
        for p in range(len(spec.projs)):
            _check(ys[p], refs[p], yb[p], rb[p], what=f"mixed T={T} {spec.projs[p].name}")
        assert pool.device_error() == 0
        pool.close()
