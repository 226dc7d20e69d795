"""CPU checks of the C ABI library: it loads, exports every function the
header declares, and its pure host functions (plan, sizing, element counts)
agree with the oracle.  No GPU call is made here."""
import ctypes
import itertools
import os
import re

import numpy as np
import pytest

import paper_2510_23346_amd as bd
import workloads as wl
from oracle import costs, plan as oplan

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(bd.lib_path()):
        from paper_2510_23346_amd.build import build
        build()
    return bd.lib()


def _header_functions():
    text = open(os.path.join(ROOT, "include", "bdlora.h")).read()
    return sorted(set(re.findall(r"^\s*(?:int|int64_t|size_t|const char\s*\*)\s+(bdlora_\w+)\s*\(", text, re.M)))


def test_exports_every_declared_function(L):
    names = _header_functions()
    assert len(names) >= 15
    for n in names:
        assert hasattr(L, n), n
    assert sorted(bd.HEADER_FUNCTIONS) == names


def test_binding_constants_match_header():
    text = open(os.path.join(ROOT, "include", "bdlora.h")).read()
    macros = dict(re.findall(r"^#define (BDLORA_\w+)\s+\(?(-?\d+)\)?", text, re.M))
    assert int(macros["BDLORA_DECODE_MAX_T"]) == bd.DECODE_MAX_T
    assert int(macros["BDLORA_DECODE_PLAN_IN_MAIN_T"]) == bd.DECODE_PLAN_IN_MAIN_T
    assert int(macros["BDLORA_DECODE_PLAN_IN_MAIN_BYTES"]) == bd.DECODE_PLAN_IN_MAIN_BYTES
    assert (int(macros["BDLORA_ACT_NONE"]), int(macros["BDLORA_ACT_SILU_MUL"])) == (bd.ACT_NONE, bd.ACT_SILU_MUL)
    assert int(macros["BDLORA_MAX_SLICES"]) == bd.MAX_SLICES
    assert (int(macros["BDLORA_COLUMN"]), int(macros["BDLORA_ROW"])) == (bd.COLUMN, bd.ROW)
    assert (int(macros["BDLORA_WEIGHT_BF16"]), int(macros["BDLORA_WEIGHT_INT4_G128"])) == \
        (bd.WEIGHT_BF16, bd.WEIGHT_INT4_G128)
    for code, name in bd.STATUS.items():
        assert int(macros["BDLORA_" + ("OK" if code == 0 else "ERR_" + name)]) == code
    for code, name in bd.PATHS.items():
        if code:
            assert int(macros["BDLORA_PATH_" + ("TILE64" if name == "tile64" else name.upper())]) == code


def test_adapter_elems_reproduce_paper_counts(L):
    # per-shard elements x N shards x layers = the paper's BD-LoRA counts
    for model, tp, r_total, mill in [("llama-3.1-8b", 8, 32, 36.2), ("llama-3.1-8b", 8, 512, 578.8),
                                     ("llama-3.1-70b", 8, 512, 2883.6), ("llama-3.2-1b", 4, 32, 11.1)]:
        m = wl.MODELS[model]
        per_shard = bd.adapter_elems(wl.model_projs(model, tp), r_total // tp)
        assert abs(per_shard * tp * m.n_layers / 1e6 - mill) <= 0.05
        assert per_shard * tp * m.n_layers == costs.bd_model_params(m.d_h, m.d_i, m.d_kv, m.n_layers, r_total, tp)


def test_pool_size(L):
    projs = wl.model_projs("llama-3.1-8b", 8)
    slab, ws = bd.pool_size(projs, 32, 16, 64)
    per_slot = slab // 32
    assert slab % 32 == 0 and per_slot * 32 == slab
    assert per_slot >= 2 * bd.adapter_elems(projs, 16)          # padded layout holds the adapter
    assert per_slot <= 2 * bd.adapter_elems(projs, 16) * 1.01 + 32 * 256
    assert ws > 0
    slab4, _ = bd.pool_size(wl.model_projs("llama-3.1-70b", 8), 512, 64, 4288)
    assert slab4 > 4e9                                           # 512 slots at rank 64


@pytest.mark.parametrize("bad", [
    [("column", 48, (16,))],          # d_in not a multiple of 32
    [("column", 64, (24,))],          # slice not a multiple of 16
    [("column", 64, (16, 16, 16, 16, 16))],
])
def test_shape_errors(L, bad):
    with pytest.raises((bd.BDLoRAError, ValueError)):
        bd.pool_size(bad, 4, 8, 16)


def test_argument_errors(L):
    # the path query validates its pointers without touching a device
    v = ctypes.c_int32(7)
    assert L.bdlora_last_path(None, ctypes.byref(v)) == -1 and v.value == 7
    with pytest.raises(bd.BDLoRAError) as e:
        bd.pool_size([("column", 64, (16,))], 0, 8, 16)
    assert e.value.code == -1
    with pytest.raises(bd.BDLoRAError):
        bd.pool_size([("column", 64, (16,))], 4, 129, 16)
    assert "max_rank" in bd.lib().bdlora_last_error().decode()


def test_host_plan_exhaustive(L):
    loaded = np.array([1, 0, 1], np.int32)
    for T in range(0, 6):
        for ids in itertools.product([-2, -1, 0, 1, 2, 3], repeat=T) if T <= 3 else \
                [np.random.default_rng(T * 100 + k).integers(-2, 4, size=T) for k in range(200)]:
            ids = np.asarray(ids, np.int32)
            rc, vid, groups, perm = bd.build_plan(loaded, ids)
            ovid, oerr = oplan.validate(ids, loaded)
            otab, operm = oplan.groups(ovid)
            assert rc == (-3 if oerr else 0)
            assert np.array_equal(vid, ovid)
            assert groups == [tuple(x) for x in otab]
            assert np.array_equal(perm, operm)


def test_host_plan_large(L):
    rng = np.random.default_rng(1)
    loaded = (rng.random(512) < 0.9).astype(np.int32)
    ids = rng.integers(-1, 520, size=5000).astype(np.int32)
    rc, vid, groups, perm = bd.build_plan(loaded, ids)
    ovid, oerr = oplan.validate(ids, loaded)
    otab, operm = oplan.groups(ovid)
    assert groups == [tuple(x) for x in otab] and np.array_equal(perm, operm)
    assert rc == -3 and oerr


def test_no_gpu_means_a_loud_error(L):
    try:
        import torch
        has_gpu = torch.cuda.is_available()
    except Exception:
        has_gpu = False
    if has_gpu:
        pytest.skip("a GPU is present")
    with pytest.raises(bd.BDLoRAError) as e:
        bd.Pool([("column", 64, (16,))], 4, 8, 16)
    assert e.value.code in (-6, -5)


def test_packed_weight_bytes(L):
    # bf16: 2 bytes per element; INT4: half a byte per element plus one bf16
    # scale per 128 inputs of each column
    assert bd.packed_weight_bytes(bd.WEIGHT_BF16, 1792, 4096) == 1792 * 4096 * 2
    assert bd.packed_weight_bytes(bd.WEIGHT_INT4_G128, 1792, 4096) == 1792 * 4096 // 2 + 1792 * 32 * 2
    assert bd.packed_weight_bytes(bd.WEIGHT_INT4_G128, 4096, 512) == 4096 * 256 + 4096 * 4 * 2
    # shapes the format does not take, and unknown formats
    assert bd.packed_weight_bytes(bd.WEIGHT_INT4_G128, 48, 4096) == 0       # N % 64
    assert bd.packed_weight_bytes(bd.WEIGHT_INT4_G128, 64, 96) == 0         # K % 128
    assert bd.packed_weight_bytes(bd.WEIGHT_BF16, 24, 64) == 0
    assert bd.packed_weight_bytes(7, 64, 128) == 0


def test_int4_descriptor_validation(L):
    ok = [("column", 256, (64,))]
    assert bd.pool_size(ok, 4, 8, 16)[0] > 0
    import ctypes
    arr, _ = bd._descs(ok, bd.WEIGHT_INT4_G128)
    a, b = ctypes.c_int64(), ctypes.c_int64()
    assert L.bdlora_pool_size(arr, 1, 4, 8, 16, ctypes.byref(a), ctypes.byref(b)) == 0
    for projs in ([("column", 96, (64,))], [("column", 256, (48,))]):        # K % 128, N % 64
        arr, _ = bd._descs(projs, bd.WEIGHT_INT4_G128)
        assert L.bdlora_pool_size(arr, 1, 4, 8, 16, ctypes.byref(a), ctypes.byref(b)) == -4
    arr, _ = bd._descs(ok, 5)
    assert L.bdlora_pool_size(arr, 1, 4, 8, 16, ctypes.byref(a), ctypes.byref(b)) == -1


def test_segment_constant_matches_header():
    text = open(os.path.join(ROOT, "include", "bdlora.h")).read()
    macros = dict(re.findall(r"^#define (BDLORA_\w+)\s+\(?(-?\d+)\)?", text, re.M))
    assert int(macros["BDLORA_MAX_SEGMENTS"]) == bd.MAX_SEGMENTS


@pytest.mark.parametrize("T", [0, 1, 7, 40])
def test_segments_from_ids_are_the_oracle_runs(L, T):
    rng = np.random.default_rng(T)
    ids = np.repeat(rng.integers(-1, 5, size=T), rng.integers(1, 4, size=T))[:T]
    sg = bd.Segments.from_ids(ids)
    runs = oplan.segments(ids)
    assert sg.n_seg == len(runs) and sg.T == T
    assert list(zip(sg.start.tolist(), sg.len.tolist(), sg.slot.tolist())) == [tuple(r) for r in runs]


def _slot_layout_reference(projs, max_rank, rank, A, B):
    """The pool's documented slot layout, written out element by element:
    per projection, A^T_cat (row s*r8 + j = column j of slice s's A, rows
    padded to 16) in 1 KB fragments, element [(rb*KS + ks)*512 + lane*8 + i]
    = A^T_cat[16 rb + lane%16][32 ks + 8 (lane//16) + i], then B^T_cat
    [N x r8] row-major (row n = column n of its slice's B), each region
    starting at a multiple of 128 elements."""
    r8max = max(8, (max_rank + 7) // 8 * 8)
    r8 = (rank + 7) // 8 * 8
    regions, off = [], 0
    up = lambda v, m: (v + m - 1) // m * m
    for kind, d_in, slices in projs:
        S, N, KS = len(slices), sum(slices), d_in // 32
        a_off = off
        off = up(off + up(S * r8max, 16) * d_in, 128)
        b_off = off
        off = up(off + N * r8max, 128)
        regions.append((a_off, b_off))
    out = np.zeros(off, np.uint16)
    for p, (kind, d_in, slices) in enumerate(projs):
        a_off, b_off = regions[p]
        KS = d_in // 32
        for s, n_s in enumerate(slices):
            for j in range(rank):
                row = s * r8 + j
                rb, lr = divmod(row, 16)
                for k in range(d_in):
                    ks, w = divmod(k, 32)
                    lane = lr + 16 * (w // 8)
                    out[a_off + (rb * KS + ks) * 512 + lane * 8 + w % 8] = A[p][s][k, j]
            col0 = sum(slices[:s])
            for j in range(rank):
                for n in range(n_s):
                    out[b_off + (col0 + n) * r8 + j] = B[p][s][j, n]
    return out


@pytest.mark.parametrize("max_rank,rank", [(8, 3), (16, 16), (24, 9), (16, 0)])
def test_host_packer_writes_the_documented_slot_layout(L, max_rank, rank):
    projs = [("column", 64, (32, 16, 16)), ("row", 32, (48,))]
    rng = np.random.default_rng(max_rank * 10 + rank)
    A = [[rng.integers(1, 1 << 14, size=(d, rank), dtype=np.uint16) for _ in sl] for _, d, sl in projs]
    B = [[rng.integers(1, 1 << 14, size=(rank, n), dtype=np.uint16) for n in sl] for _, _, sl in projs]
    nbytes = bd.layout_slot_bytes(projs, max_rank)
    assert nbytes == bd.pool_size(projs, 3, max_rank, 16)[0] // 3
    slab = bd.pack_adapter_layout(projs, max_rank, rank, A, B)
    assert slab.nbytes == nbytes
    ref = _slot_layout_reference(projs, max_rank, rank, A, B)
    assert np.array_equal(slab.view(np.uint16), ref)


def test_host_packer_errors(L):
    projs = [("column", 64, (16,))]
    A = [[np.zeros((64, 4), np.uint16)]]
    B = [[np.zeros((4, 16), np.uint16)]]
    with pytest.raises(bd.BDLoRAError) as e:
        bd.pack_adapter_layout(projs, 2, 4, A, B)                 # rank > max_rank
    assert e.value.code == -1
    A[0][0][3, 1] = 0x7F80                                        # +inf
    with pytest.raises(bd.BDLoRAError) as e:
        bd.pack_adapter_layout(projs, 8, 4, A, B)
    assert e.value.code == -1 and "non-finite" in str(e.value)


def test_pool_byte_budget_is_checked_before_any_device_work(L):
    # a budget that holds no slot, or fewer slots than asked for, is OOM;
    # both are decided on the host (no device is needed to fail)
    projs = [("column", 256, (64,))]
    per = bd.layout_slot_bytes(projs, 16)
    with pytest.raises(bd.BDLoRAError) as e:
        bd.Pool(projs, 0, 16, 32, pool_bytes=per - 1)
    assert e.value.code == -2
    with pytest.raises(bd.BDLoRAError) as e:
        bd.Pool(projs, 8, 16, 32, pool_bytes=8 * per - 1)
    assert e.value.code == -2 and "pool_bytes" in str(e.value)
    with pytest.raises(bd.BDLoRAError) as e:
        bd.Pool(projs, 8, 16, 32, pool_bytes=-5)
    assert e.value.code == -1
