"""Pins for the oracle's cost model (CPU only): the paper's printed parameter
counts, the parameter ratios quoted in its abstract, the equal-parameter rank
of App. A, and element counts of drawn adapters."""
import os

import numpy as np
import pytest

from oracle import costs
import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "param_counts.txt")


def _golden_rows():
    rows = []
    with open(GOLDEN) as f:
        for line in f:
            if not line.strip() or line.startswith("#"):
                continue
            model, meth, tp, rank, mill = line.split()[:5]
            rows.append((model, meth, int(tp), int(rank), float(mill)))
    return rows


def _count(model, meth, tp, rank):
    m = wl.MODELS[model]
    if meth == "bd":
        return costs.bd_model_params(m.d_h, m.d_i, m.d_kv, m.n_layers, rank, tp)
    return costs.lora_model_params(m.d_h, m.d_i, m.d_kv, m.n_layers, rank)


@pytest.mark.parametrize("row", _golden_rows(), ids=lambda r: "-".join(map(str, r[:4])))
def test_printed_parameter_counts(row):
    model, meth, tp, rank, mill = row
    assert abs(_count(model, meth, tp, rank) / 1e6 - mill) <= 0.05 + 1e-9


def test_golden_file_is_complete():
    assert len(_golden_rows()) == 43


@pytest.mark.parametrize("model,bd_rank,lora_rank,ratio", [
    # abstract / App. F.1: parameter ratios of the compared configurations
    ("llama-3.1-8b", 256, 128, 0.86), ("llama-3.1-8b", 256, 64, 1.73),
    ("llama-3.1-70b", 512, 256, 0.87), ("llama-3.1-70b", 512, 128, 1.74),
])
def test_parameter_ratios_quoted_in_abstract(model, bd_rank, lora_rank, ratio):
    r = _count(model, "bd", 8, bd_rank) / _count(model, "lora", 0, lora_rank)
    assert abs(r - ratio) < 0.005


@pytest.mark.parametrize("d_h,d_i,N", [(4096, 14336, 8), (8192, 28672, 8), (4096, 14336, 4)])
def test_equal_parameter_rank(d_h, d_i, N):
    r = 64
    rp = costs.equal_param_rank(r, d_h, d_i, N)
    s = costs.mlp_cost_table("s-lora", 7, d_h, d_i, r, N)["sum"]
    b = costs.mlp_cost_table("bd-lora", 7, d_h, d_i, rp, N)["sum"]
    assert abs(s["params"] - b["params"]) < 1e-6 * s["params"]
    assert abs(s["ops"] - b["ops"]) < 1e-6 * s["ops"]
    # r < r' < r (1 + d_I/d_H)
    assert r < rp < r * (1 + d_i / d_h)


def test_equal_parameter_rank_for_llama_is_about_3_13():
    for name in ("llama-3.1-8b", "llama-3.1-70b"):
        m = wl.MODELS[name]
        assert abs(costs.equal_param_rank(1.0, m.d_h, m.d_i, 8) - 3.1304) < 1e-3


@pytest.mark.parametrize("method", ["s-lora", "bd-lora"])
def test_cost_table_sum_rows(method):
    # each row's ops are 2 S #params; the rows add up to the printed sum row
    S, d_h, d_i, r, N = 5, 64, 224, 16, 8
    t = costs.mlp_cost_table(method, S, d_h, d_i, r, N)
    for k in ("A1", "B1", "A2", "B2"):
        assert t[k]["ops"] == 2 * S * t[k]["params"]
    if method == "s-lora":
        params = 2 * (d_h + d_i) * r / N
        out = 2 * S * (r / N + d_i / N + d_h / N + r)
    else:
        params = 2 * (d_h + d_i / N) * r / N
        out = 2 * S * (2 * r / N + d_i / N + d_h)
    assert abs(t["sum"]["params"] - params) < 1e-9
    assert abs(t["sum"]["ops"] - 4 * S * params / 2) < 1e-9
    assert abs(t["sum"]["out"] - out) < 1e-9


def test_shard_params_match_drawn_adapter_elements():
    spec = wl.workload(1)
    ad = wl.draw_adapter(spec, 0)
    m = wl.MODELS["llama-3.1-8b"]
    lin = {n: (k, di, do) for n, k, di, do in costs.llama_linears(m.d_h, m.d_i, m.d_kv)}
    r_total = spec.ranks[0] * 8
    names = [["q", "k", "v"], ["o"], ["gate"], ["up"], ["down"]]
    for p, pnames in enumerate(names):
        for j, n in enumerate(pnames):
            k, di, do = lin[n]
            drawn = ad.A[p][j].size + ad.B[p][j].size
            assert drawn == costs.bd_shard_params(k, di, do, r_total, 8)


def test_batch_bytes_and_flops_by_brute_count():
    spec = wl.custom_workload("t", wl.tiny_projs(), T=5, ranks=[4, 8, 0], ids=[0, 1, 0, -1, 2])
    lay = wl.draw_layer(spec)
    active = sorted(set(int(a) for a in lay.ids if a >= 0))
    elems = 0
    for p, pi in enumerate(lay.projs):
        elems += pi.W.size + pi.X.size + pi.X.shape[0] * pi.spec.d_out
        for s in active:
            elems += sum(a.size for a in lay.adapters[s].A[p]) + sum(b.size for b in lay.adapters[s].B[p])
    assert costs.batch_bytes(spec.projs, spec.T, [spec.ranks[s] for s in active]) == 2 * elems
    # flops: 2 per multiply-add of the base and of each token's own (X A) B
    fl = 0
    for pi in lay.projs:
        fl += 2 * pi.X.shape[0] * pi.spec.d_in * pi.spec.d_out
        for a in lay.ids:
            if a >= 0:
                r = spec.ranks[a]
                fl += 2 * sum(pi.spec.d_in * r + r * n for n in pi.spec.slices)
    rk = [spec.ranks[a] if a >= 0 else 0 for a in lay.ids]
    assert costs.batch_flops(spec.projs, rk) == fl
