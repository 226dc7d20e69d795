#!/usr/bin/env python3
"""Benchmark of the BD-LoRA layer-shard forward on one MI355X.

A step is one forward of a whole decoder-layer shard (all its projections:
plan, shrink, base product, expand) over one batch of synthetic tokens,
through the library's C ABI.  Default workload: Llama-3.1-8B layer
shard at 1/8 tensor parallelism, 64 decode tokens, 32 resident adapters of
rank 16, adapter ids Zipf(1.0).

Timing: steps are captured into HIP graphs, each graph one pass over R
rotated copies of every input (weights, adapter pool, activations, outputs)
whose footprint exceeds twice the 256 MB Infinity Cache, so the data comes
from HBM.  The K timed steps are bracketed by torch.cuda.synchronize(); the
reported time is the wall clock over them.

Prints one JSON line (rank 0).
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, published
MFMA_BF16_PEAK_TFS = 2500.0    # MI355X dense bf16 matrix, published
MALL_BYTES = 256 << 20


def base_weight_bytes(spec, p):
    """Bytes of one projection's base weight: bf16, or INT4 nibbles plus one
    bf16 scale per 128 inputs of each output column."""
    n = sum(p.slices)
    if spec.weight_format == "int4_g128":
        return p.d_in * n // 2 + n * (p.d_in // 128) * 2
    return 2 * p.d_in * n


def algorithmic_bytes(spec, ids, ranks):
    """Per-step bytes the method must move (bf16 = 2 bytes), split by launch.

    Returns (main, expand, active): ``main`` is what the shrink and base
    product must read, i.e. every base weight once, X once per projection and
    the A factor of every adapter some token uses; ``expand`` is the B factor
    of every such adapter plus the output written once.
    """
    active = sorted({int(a) for a in ids if a >= 0})
    T = len(ids)
    m = e = 0
    for p in spec.projs:
        n = sum(p.slices)
        m += base_weight_bytes(spec, p) + 2 * T * p.d_in
        e += 2 * T * n
        for a in active:
            r = ranks[a]
            m += 2 * len(p.slices) * p.d_in * r
            e += 2 * r * n
    return m, e, len(active)


def algorithmic_flops(spec, ids, ranks):
    T = len(ids)
    g = s = 0
    for p in spec.projs:
        n = sum(p.slices)
        g += 2 * T * p.d_in * n
        for a in ids:
            if a >= 0:
                r = ranks[a]
                g += 2 * r * n
                s += 2 * len(p.slices) * p.d_in * r
    return g, s


KERNEL_SOURCES = ("bdl_prep.hip", "bdl_decode.hip", "bdl_kernels.hip", "bdl_gemm.hip", "bdl_device.h",
                  "bdl_launch.h", "bdl_api.cpp")


def kernel_source_hash():
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2510_23346_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def committed_traffic(kernel, workload_name):
    """HBM bytes per launch of ``kernel`` from the committed rocprofv3
    counter summary of this workload, if it was taken on the current kernel
    sources (else None: the counters are stale or absent)."""
    import re
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload_name}.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    mh = re.search(r"first 16 hex\): `([0-9a-f]{16})`", text)
    mt = re.search(r"traffic_bytes_per_launch: (\d+)", text)
    if not mh or not mt or mh.group(1) != kernel_source_hash():
        return None
    return int(mt.group(1))


def cpu_baseline(spec, layer, seconds):
    """Time the oracle (fp64 numpy) on this host: whole steps until
    ``seconds`` have passed."""
    from oracle import bdlora, quant
    forward = quant.layer_forward_w4 if spec.weight_format == "int4_g128" else bdlora.layer_forward
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    forward(layer)                                  # warm-up
    n = 0
    t0 = time.perf_counter()
    while True:
        forward(layer)
        n += 1
        el = time.perf_counter() - t0
        if el >= seconds:
            break
    return {
        "value": spec.T * n / el,
        "unit": "tokens/s",
        "cores": int(threads),
        "kind": "oracle",
        "sample": f"{n} full steps of the same workload ({spec.T} tokens x {len(spec.projs)} "
                  f"projections), fp64 numpy, {el:.1f} s",
    }


def adapter_load_bench(args):
    """Adapter load pipeline on the default layer shard (Llama-3.1-8B, 1/8
    TP, 5 projections): per-adapter load time against its parameter count,
    and decode steps whose adapters are not cached (every step loads the
    adapters its batch uses before its forward), with the loads serialized
    before the forward or overlapped with the previous step's forward on a
    second stream.  Prints one JSON line."""
    import numpy as np
    import torch

    import paper_2510_23346_amd as bd
    import workloads as wl
    from workloads.gpu import DeviceLayer

    base = wl.workload(1)
    projs = list(range(len(base.projs)))
    out = {"metric": "adapter load", "workload": base.name, "loads": []}
    # 1. load time per adapter against its parameter count
    for r in (8, 16, 32, 64):
        spec = wl.WorkloadSpec(f"load-r{r}", base.model, base.tp, base.projs, base.T, 64, [r] * 64,
                               [2.0] * 64, "uniform", 11)
        pool = bd.Pool(spec.projs, 64, r, spec.T)
        ad = wl.draw_adapter(spec, 0)
        params = bd.adapter_elems(spec.projs, r)
        slab = torch.empty(pool.slot_bytes, dtype=torch.uint8).pin_memory()
        pool.pack_adapter_host(r, ad.A_bits, ad.B_bits, out=slab)
        s = torch.cuda.Stream()
        n = 64
        for i in range(4):
            pool.load_adapter_packed(i, r, 2.0, slab, stream=s)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(n):
            pool.load_adapter_packed(i % 64, r, 2.0, slab, stream=s)
        torch.cuda.synchronize()
        t_packed = (time.perf_counter() - t0) / n
        t0 = time.perf_counter()
        for i in range(8):
            pool.load_adapter(i, r, 2.0, ad.A_bits, ad.B_bits)
        t_sync = (time.perf_counter() - t0) / 8
        many = torch.empty(16 * pool.slot_bytes, dtype=torch.uint8).pin_memory()
        for i in range(16):
            many[i * pool.slot_bytes:(i + 1) * pool.slot_bytes].copy_(slab)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(8):
            pool.load_adapters_packed(16 * (i % 4), [r] * 16, [2.0] * 16, many, stream=s)
        torch.cuda.synchronize()
        t_batch = (time.perf_counter() - t0) / (8 * 16)
        out["loads"].append({"rank": r, "params": params, "bytes": 2 * params,
                             "packed_pinned_us": round(t_packed * 1e6, 1),
                             "packed_GBps": round(2 * params / t_packed / 1e9, 1),
                             "slot_bytes": pool.slot_bytes,
                             "packed_batch16_us_per_adapter": round(t_batch * 1e6, 1),
                             "packed_batch16_GBps": round(pool.slot_bytes / t_batch / 1e9, 1),
                             "paper_layout_sync_us": round(t_sync * 1e6, 1)})
        pool.close()
    # 2. no adapter cache: each decode step loads its batch's adapters first,
    # back to back into consecutive slots with one copy (slot i of a half
    # holds the batch's i-th adapter)
    spec = base
    ids = wl.draw_ids(spec)
    active = sorted(int(a) for a in np.unique(ids) if a >= 0)
    layer = wl.draw_layer(spec, slots=active)
    nS = len(active)
    pool = bd.Pool(spec.projs, 2 * nS, max(spec.ranks), spec.T)     # two halves of slots
    sb = pool.slot_bytes
    slabs = torch.empty(nS * sb, dtype=torch.uint8).pin_memory()
    for i, a in enumerate(active):
        ad = layer.adapters[a]
        pool.pack_adapter_host(ad.rank, ad.A_bits, ad.B_bits, out=slabs[i * sb:(i + 1) * sb])
    ranks = [spec.ranks[a] for a in active]
    scales = [spec.scales[a] for a in active]
    dl = DeviceLayer(layer)
    pos = np.full(spec.n_slots, -1, np.int64)
    pos[active] = np.arange(nS)
    local = torch.from_numpy(np.where(ids >= 0, pos[np.maximum(ids, 0)], -1).astype(np.int32)).cuda()
    ids_half = [local, torch.where(local >= 0, local + nS, local)]
    main, side = torch.cuda.current_stream(), torch.cuda.Stream()

    def load_step(half, stream):
        pool.load_adapters_packed(half * nS, ranks, scales, slabs, stream=stream)

    K = 50
    for h in (0, 1):
        load_step(h, main)
    pool.forward_layer(projs, dl.X, dl.W, dl.out, ids_half[0], stream=main)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(K):
        pool.forward_layer(projs, dl.X, dl.W, dl.out, ids_half[0], stream=main)
    torch.cuda.synchronize()
    t_fwd = (time.perf_counter() - t0) / K
    t0 = time.perf_counter()
    for i in range(K):
        load_step(0, main)
        pool.forward_layer(projs, dl.X, dl.W, dl.out, ids_half[0], stream=main)
    torch.cuda.synchronize()
    t_serial = (time.perf_counter() - t0) / K
    # overlapped: the loads of step i+1 go to the other half of the slots on
    # the side stream while step i runs; each forward waits for its loads
    loaded = [torch.cuda.Event() for _ in range(2)]
    freed = [torch.cuda.Event() for _ in range(2)]
    for h in (0, 1):
        freed[h].record(main)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    side.wait_event(freed[0])
    load_step(0, side)
    loaded[0].record(side)
    for i in range(K):
        h = i % 2
        side.wait_event(freed[1 - h])
        load_step(1 - h, side)
        loaded[1 - h].record(side)
        main.wait_event(loaded[h])
        pool.forward_layer(projs, dl.X, dl.W, dl.out, ids_half[h], stream=main)
        freed[h].record(main)
    torch.cuda.synchronize()
    t_overlap = (time.perf_counter() - t0) / K
    # the load alone
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(K):
        load_step(i % 2, main)
    torch.cuda.synchronize()
    t_load = (time.perf_counter() - t0) / K
    pool.close()
    out["no_cache_decode"] = {
        "tokens": spec.T, "adapters_loaded_per_step": len(active),
        "bytes_loaded_per_step": int(nS * sb),
        "load_only_us": round(t_load * 1e6, 1), "load_GBps": round(nS * sb / t_load / 1e9, 1),
        "forward_only_us": round(t_fwd * 1e6, 1), "load_then_forward_us": round(t_serial * 1e6, 1),
        "overlapped_us": round(t_overlap * 1e6, 1), "timing": "eager launches, host clock"}
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=1000)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--workload", type=int, default=1,
                    help="workload index 0..5 (default 1; 5 = workload 1 with an INT4 base)")
    ap.add_argument("--rotate", type=int, default=0, help="input copies to rotate (0 = auto)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--eager", action="store_true", help="time eager launches instead of graphs")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="before the benchmark, run 3 plain device copies of MIB MiB (untimed), "
                         "a known-size reference for hardware byte counters")
    ap.add_argument("--adapter-load", action="store_true",
                    help="measure the adapter load pipeline instead (one JSON line of its own)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this build runs one GPU's shard only; --gpus {args.gpus} is not supported "
              "(the multi-GPU path is a design note, not built)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2510_23346_amd as bd
    import workloads as wl
    from workloads.gpu import DeviceLayer, load_adapters, make_pool

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    bd.lib()
    if args.adapter_load:
        adapter_load_bench(args)
        return
    if args.copy_calibration:
        n = args.copy_calibration << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    spec = wl.workload(args.workload)
    ids_np = wl.draw_ids(spec)
    resident = list(range(spec.n_slots)) if spec.n_slots <= 128 else sorted(
        int(s) for s in np.unique(ids_np) if s >= 0)
    layer = wl.draw_layer(spec, slots=resident)
    m_bytes, e_bytes, n_active = algorithmic_bytes(spec, ids_np, spec.ranks)
    g_flops, s_flops = algorithmic_flops(spec, ids_np, spec.ranks)
    step_bytes = m_bytes + e_bytes
    decode = spec.T <= bd.DECODE_MAX_T

    # rotated copies: each is a pool with the same adapters plus its own tensors
    pool0 = make_pool(spec)
    load_adapters(pool0, spec, resident, cache=layer.adapters)
    set_bytes = step_bytes + pool0.bytes
    R = args.rotate or max(2, math.ceil(2 * MALL_BYTES / max(1, step_bytes)))
    R = min(R, 16)
    sets = []
    for i in range(R):
        pool = pool0 if i == 0 else make_pool(spec)
        if i:
            load_adapters(pool, spec, resident, cache=layer.adapters)
        sets.append((pool, DeviceLayer(layer)))
    projs = list(range(len(spec.projs)))
    stream = torch.cuda.current_stream()

    def step(i):
        pool, dl = sets[i % R]
        pool.forward_layer(projs, dl.X, dl.W, dl.out, dl.ids, stream=stream)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    # graphs: one per pass over the R copies, plus one for a remainder
    K = args.steps
    graphs = []
    if not args.eager:
        def capture(n):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=torch.cuda.Stream()):
                s = torch.cuda.current_stream()
                for i in range(n):
                    pool, dl = sets[i % R]
                    pool.forward_layer(projs, dl.X, dl.W, dl.out, dl.ids, stream=s)
            return g
        full, rem = divmod(K, R)
        g_full = capture(R) if full else None
        g_rem = capture(rem) if rem else None
        for _ in range(2):
            if g_full:
                g_full.replay()
        torch.cuda.synchronize()
        plan = [g_full] * full + ([g_rem] if g_rem else [])
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    if args.eager:
        for i in range(K):
            step(i)
    else:
        for g in plan:
            g.replay()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_per_step = (t1 - t0) * 1e3 / K

    # per-kernel durations with HIP events on the launch stream (eager)
    n_prof = max(R, min(K, 400))
    per_pool = math.ceil(n_prof / R)
    for pool, _ in sets:
        pool.profile_begin(per_pool)
    for i in range(per_pool * R):
        step(i)
    torch.cuda.synchronize()
    path = sets[0][0].last_path()
    sums, cnt = [0.0, 0.0, 0.0, 0.0], 0
    for pool, _ in sets:
        ms, n = pool.profile_end()
        for k in range(4):
            sums[k] += ms[k] * n
        cnt += n
    k_ms = [s / max(1, cnt) for s in sums]
    if decode:
        # decode launches: prep (plan + packing), main (K-split shrink and
        # base partials), epilogue (partial sums + expand); main moves the
        # weights and dominates
        names = ("prep", "main", "epilogue")
        dom, dom_name = 1, "bdl::dec_main_kernel"
        achieved = m_bytes / (k_ms[dom] * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4)}
    elif path == "medium":
        # medium batches: prep, shrink, base product of all rows per tile
        # (fp32 partials), epilogue (partials + expand).  The main launch
        # streams the base weight once; at about 240 flops per byte it sits
        # below the MFMA/HBM ridge, so its bound is HBM: the weight and X
        # once per projection
        names = ("prep", "shrink", "gemm", "epilogue")
        dom, dom_name = 2, "bdl::gemm_mid_kernel"
        mid_bytes = sum(base_weight_bytes(spec, p) + 2 * spec.T * p.d_in for p in spec.projs)
        achieved = mid_bytes / (k_ms[dom] * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4)}
    else:
        names = ("prep", "shrink", "gemm")
        # the library's base GEMM: the 256 x 256 LDS-staged kernel for bf16
        # weights above 256 tokens, the 64-row kernel otherwise
        dom, dom_name = 2, "bdl::gemm_big_kernel" if path == "large" else "bdl::gemm_kernel"
        achieved = g_flops / (k_ms[dom] * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": MFMA_BF16_PEAK_TFS,
                "unit": "TFLOP/s", "frac": round(achieved / MFMA_BF16_PEAK_TFS, 4)}
    roof["traffic"] = committed_traffic(dom_name.split("::")[1], spec.name)
    roof["kernel"] = dom_name
    roof["kernel_ms"] = round(k_ms[dom], 5)
    roof["algorithmic"] = m_bytes if decode else (mid_bytes if path == "medium" else g_flops)

    out = {
        "metric": "tokens/s per layer-shard",
        "value": round(spec.T / (ms_per_step * 1e-3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": spec.name,
            "description": spec.description,
            "tokens": spec.T,
            "projections": [p.name for p in spec.projs],
            "adapters_resident": len(resident),
            "adapters_active": n_active,
            "ranks": sorted(set(spec.ranks)),
            "base_weight": spec.weight_format,
            "parallelism": "one tensor-parallel shard (1 of 8) on one GPU",
            "timing": "eager launches" if args.eager else f"HIP graphs over {R} rotated input copies",
        },
        "step_hbm": {
            "algorithmic_bytes": step_bytes,
            "GB/s": round(step_bytes / (ms_per_step * 1e-3) / 1e9, 1),
            "frac": round(step_bytes / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        },
        "step_flops": g_flops + s_flops,
        "kernel_ms": {nm: round(v, 5) for nm, v in zip(names, k_ms)},
        "roofline": roof,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(spec, layer, args.cpu_seconds)
    for pool, _ in sets:
        pool.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
