"""Seeded synthetic inputs for the BD-LoRA shard forward.

This module is shared by the tests, the benchmark and the oracle harness.  It
only draws random numbers, rounds them to bfloat16 and describes workload
shapes; it performs none of the arithmetic of the method itself (no products,
no slicing of adapters into shards, no sums).

Shapes follow the tensor-parallel layout of the paper (Sec. 2, Megatron-style
sharding; Sec. 3 / Fig. 3 for the BD-LoRA factors; Alg. 1 and Alg. 2 for the
per-device shapes):

* column-parallel projections (q/k/v, gate, up): local input ``d_in`` is the
  full hidden size, local output is ``d_out / N``; the shard's adapter is
  ``A_s`` of shape ``[d_in, r_s]`` and ``B_s`` of shape ``[r_s, d_out / N]``.
* row-parallel projections (o, down): local input is ``d_in / N``, output is
  the full ``d_out``; ``A_s`` is ``[d_in / N, r_s]``, ``B_s`` is ``[r_s, d_out]``.

q, k and v are one projection call with three slices, each with an adapter of
its own (the parameter counts of the paper's Table on fine-tuning scores only
come out with separate adapters per linear layer).

Value distributions: ``X ~ N(0, 1)``; ``W_s`` and ``A_s`` ~ ``N(0, 1/d_in)``
where ``d_in`` is the projection's local input size; ``B_s ~ N(0, 1/r_s)``.
The second argument of ``N`` is the variance.  Every value is rounded to
bfloat16 (round to nearest, ties to even) and handed to both the oracle (as
float) and the GPU path (as raw 16-bit patterns).
"""
from __future__ import annotations

import os
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

__all__ = [
    "ModelShape", "ProjSpec", "WorkloadSpec", "Adapter", "ProjInputs", "LayerInputs",
    "MODELS", "model_projs", "bf16_round", "bf16_bits_to_float", "finite_zipf_probs",
    "workload", "WORKLOADS", "draw_layer", "draw_adapter", "draw_ids", "draw_proj",
    "tiny_projs",
]


# --------------------------------------------------------------------------
# bfloat16 helpers (input preparation only)
# --------------------------------------------------------------------------

def bf16_round(x: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Round ``x`` to bfloat16 with round-to-nearest-even.

    Returns ``(bits, values)``: ``bits`` is a uint16 array of the bfloat16
    patterns and ``values`` a float32 array holding exactly those numbers.
    Inputs are finite; NaN/Inf are never generated here.
    """
    f = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    u = f.view(np.uint32)
    # u + 0x7FFF + lsb stays below 2**32 for every finite input
    r = (u >> np.uint32(16)) & np.uint32(1)
    r += np.uint32(0x7FFF)
    r += u
    r >>= np.uint32(16)
    bits = r.astype(np.uint16)
    r <<= np.uint32(16)
    return bits, r.view(np.float32)


def bf16_bits_to_float(bits: np.ndarray) -> np.ndarray:
    b = np.ascontiguousarray(np.asarray(bits, dtype=np.uint16))
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def finite_zipf_probs(n: int, alpha: float = 1.0) -> np.ndarray:
    """Finite Zipf law over ranks 1..n: ``p_k`` proportional to ``k**-alpha``."""
    k = np.arange(1, n + 1, dtype=np.float64)
    w = k ** (-float(alpha))
    return w / w.sum()


# --------------------------------------------------------------------------
# model and projection shapes
# --------------------------------------------------------------------------

@dataclass(frozen=True)
class ModelShape:
    name: str
    d_h: int          # hidden size
    d_i: int          # MLP intermediate size
    n_layers: int
    n_kv_heads: int
    head_dim: int

    @property
    def d_kv(self) -> int:
        return self.n_kv_heads * self.head_dim


# Public Llama configurations.  The paper states d_H and d_I of Llama-3.1-8B
# (Appendix A); the others reproduce its parameter counts exactly.
MODELS: Dict[str, ModelShape] = {
    "llama-3.2-1b": ModelShape("llama-3.2-1b", 2048, 8192, 16, 8, 64),
    "llama-3.1-8b": ModelShape("llama-3.1-8b", 4096, 14336, 32, 8, 128),
    "llama-3.1-70b": ModelShape("llama-3.1-70b", 8192, 28672, 80, 8, 128),
}


@dataclass(frozen=True)
class ProjSpec:
    """One projection call on one shard.

    ``kind`` is ``"column"`` or ``"row"``; ``d_in`` is the local input size
    (K); ``slices`` are the per-slice local output widths (q, k, v for the
    attention input projection, a single slice otherwise).
    """
    name: str
    kind: str
    d_in: int
    slices: Tuple[int, ...]

    @property
    def d_out(self) -> int:
        return int(sum(self.slices))


def model_projs(model: str, tp: int) -> List[ProjSpec]:
    """The five projection calls of one decoder layer on one shard of ``tp``."""
    m = MODELS[model]
    for d in (m.d_h, m.d_i, m.d_kv):
        if d % tp:
            raise ValueError(f"{model}: dimension {d} not divisible by TP={tp}")
    return [
        ProjSpec("qkv", "column", m.d_h, (m.d_h // tp, m.d_kv // tp, m.d_kv // tp)),
        ProjSpec("o", "row", m.d_h // tp, (m.d_h,)),
        ProjSpec("gate", "column", m.d_h, (m.d_i // tp,)),
        ProjSpec("up", "column", m.d_h, (m.d_i // tp,)),
        ProjSpec("down", "row", m.d_i // tp, (m.d_h,)),
    ]


def tiny_mlp_projs() -> List[ProjSpec]:
    """A small MLP shard for the MLP parity tests: gate and up (column), down
    (row), the intermediate width a multiple of 32 and of 16."""
    return [
        ProjSpec("gate", "column", 320, (224,)),
        ProjSpec("up", "column", 320, (224,)),
        ProjSpec("down", "row", 224, (160,)),
    ]


def tiny_projs() -> List[ProjSpec]:
    """Small projections used by parity tests: several tiles and ragged shapes."""
    return [
        ProjSpec("qkv", "column", 256, (64, 32, 48)),
        ProjSpec("o", "row", 96, (160,)),
        ProjSpec("up", "column", 320, (208,)),
    ]


# --------------------------------------------------------------------------
# workloads (the five benchmark configurations plus generic test cases)
# --------------------------------------------------------------------------

@dataclass
class WorkloadSpec:
    name: str
    model: Optional[str]
    tp: int
    projs: List[ProjSpec]
    T: int
    n_slots: int
    ranks: List[int]                  # per slot
    scales: List[float]               # per slot
    ids_kind: str                     # "uniform", "zipf", "segments", "mixed"
    seed: int
    zipf_alpha: float = 1.0
    segments: Tuple[int, ...] = ()    # prefill request lengths (segments/mixed)
    n_decode: int = 0                 # decode tokens after the segments (mixed)
    n_active: int = 0                 # active slot count (mixed)
    weight_format: str = "bf16"       # base weight: "bf16" or "int4_g128"
    description: str = ""
    extra: Dict[str, object] = field(default_factory=dict)


def _ranks_uniform(seed: int, n: int, choices: Sequence[int]) -> List[int]:
    rng = np.random.default_rng([seed, 7])
    return [int(c) for c in rng.choice(np.asarray(choices), size=n)]


def workload(index: int) -> WorkloadSpec:
    """The five benchmark workloads (one tensor-parallel shard at TP=8)."""
    if index == 0:
        m = MODELS["llama-3.1-8b"]
        projs = [ProjSpec("up", "column", m.d_h, (m.d_i // 8,))]
        return WorkloadSpec(
            "8b-up-decode-T16", "llama-3.1-8b", 8, projs, T=16, n_slots=4,
            ranks=[8] * 4, scales=[2.0] * 4, ids_kind="uniform", seed=0,
            description="Llama-3.1-8B up_proj shard (1/8 TP), 16 decode tokens, "
                        "4 adapters r_s=8, ids uniform over 4")
    if index == 1:
        return WorkloadSpec(
            "8b-layer-decode-T64", "llama-3.1-8b", 8, model_projs("llama-3.1-8b", 8),
            T=64, n_slots=32, ranks=[16] * 32, scales=[2.0] * 32, ids_kind="zipf",
            seed=1, description="Llama-3.1-8B decoder-layer shard (1/8 TP), 64 decode "
                                "tokens, 32 adapters r_s=16, ids Zipf(1.0)")
    if index == 2:
        return WorkloadSpec(
            "8b-layer-prefill-8x512", "llama-3.1-8b", 8, model_projs("llama-3.1-8b", 8),
            T=4096, n_slots=8, ranks=[32] * 8, scales=[2.0] * 8, ids_kind="segments",
            seed=2, segments=(512,) * 8,
            description="Llama-3.1-8B layer shard, prefill 8 requests x 512 tokens "
                        "sorted by adapter, 8 adapters r_s=32")
    if index == 3:
        return WorkloadSpec(
            "70b-layer-decode-T256", "llama-3.1-70b", 8, model_projs("llama-3.1-70b", 8),
            T=256, n_slots=128, ranks=[16] * 128, scales=[2.0] * 128, ids_kind="zipf",
            seed=3, description="Llama-3.1-70B decoder-layer shard (1/8 TP), 256 decode "
                                "tokens, 128 adapters r_s=16, ids Zipf(1.0)")
    if index == 4:
        return WorkloadSpec(
            "70b-layer-mixed-4x1024+192", "llama-3.1-70b", 8, model_projs("llama-3.1-70b", 8),
            T=4 * 1024 + 192, n_slots=512, ranks=_ranks_uniform(4, 512, (8, 16, 32, 64)),
            scales=[2.0] * 512, ids_kind="mixed", seed=4, segments=(1024,) * 4,
            n_decode=192, n_active=64,
            description="Llama-3.1-70B layer shard, 4 prefill requests x 1024 tokens "
                        "plus 192 decode tokens, 512-adapter pool, r_s in {8,16,32,64}, "
                        "64 active adapters")
    if index == 5:
        w = workload(1)
        return WorkloadSpec(
            "8b-layer-decode-T64-int4", w.model, w.tp, w.projs, w.T, w.n_slots, w.ranks, w.scales,
            w.ids_kind, w.seed, weight_format="int4_g128",
            description="workload 1 (Llama-3.1-8B layer shard, 64 decode tokens, 32 adapters "
                        "r_s=16, Zipf ids) with an INT4 base (one bf16 scale per 128 inputs)")
    if index == 6:
        w = workload(1)
        return WorkloadSpec(
            "8b-layer-decode-T64-r8r64", w.model, w.tp, w.projs, w.T, w.n_slots,
            [8 if s % 2 == 0 else 64 for s in range(w.n_slots)], w.scales, w.ids_kind, 6,
            description="Llama-3.1-8B layer shard, 64 decode tokens, 32 adapters whose ranks "
                        "alternate 8 and 64 (slots sized for rank 64), Zipf ids")
    raise KeyError(index)


WORKLOADS = [workload(i) for i in range(5)]


# --------------------------------------------------------------------------
# drawing the arrays
# --------------------------------------------------------------------------

@dataclass
class Adapter:
    """One adapter for one layer shard: per projection, per slice, the paper-
    layout factors ``A [d_in, r]`` and ``B [r, slice_out]`` (bf16 bits and
    float values)."""
    slot: int
    rank: int
    scale: float
    A_bits: List[List[np.ndarray]]
    B_bits: List[List[np.ndarray]]
    A: List[List[np.ndarray]]
    B: List[List[np.ndarray]]


@dataclass
class ProjInputs:
    spec: ProjSpec
    X_bits: np.ndarray    # uint16 [T, d_in]
    X: np.ndarray         # float32 [T, d_in]
    W_bits: np.ndarray    # uint16 [d_in, d_out]  (paper layout: X @ W)
    W: np.ndarray         # float32 [d_in, d_out]
    # INT4 base (weight_format "int4_g128"): nibbles q + 8, two per byte,
    # [d_out, d_in / 2], and bf16 scales [d_out, d_in / 128]
    Wq: Optional[np.ndarray] = None
    Ws_bits: Optional[np.ndarray] = None


def quantize_int4_g128(W: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Round-to-nearest symmetric INT4 quantization of a paper-layout weight
    ``W [d_in, d_out]`` in groups of 128 input channels: the scale of a group
    is the bf16 value nearest to max|W| / 7 (1 for an all-zero group), the
    stored nibble ``clip(rint(W / scale), -8, 7) + 8``.  Returns
    ``(qbytes [d_out, d_in / 2] uint8, scale_bits [d_out, d_in / 128])``;
    input preparation only (the oracle decodes the stored values itself)."""
    W = np.asarray(W, dtype=np.float32)
    K, N = W.shape
    if K % 128:
        raise ValueError("d_in must be a multiple of 128")
    g = np.abs(W.T.reshape(N, K // 128, 128)).max(axis=2) / np.float32(7.0)
    g = np.where(g > 0, g, np.float32(1.0)).astype(np.float32)
    s_bits, s = bf16_round(g)
    q = np.clip(np.rint(W.T / np.repeat(s, 128, axis=1)), -8, 7).astype(np.int64) + 8
    qbytes = (q[:, 0::2] | (q[:, 1::2] << 4)).astype(np.uint8)
    return np.ascontiguousarray(qbytes), np.ascontiguousarray(s_bits)


@dataclass
class LayerInputs:
    spec: WorkloadSpec
    ids: np.ndarray                      # int32 [T]; -1 means "no adapter"
    projs: List[ProjInputs]
    adapters: Dict[int, Adapter]


def _normal_bf16(rng: np.random.Generator, shape, var: float):
    x = rng.standard_normal(size=shape, dtype=np.float32) * np.float32(np.sqrt(var))
    return bf16_round(x)


def draw_ids(spec: WorkloadSpec) -> np.ndarray:
    rng = np.random.default_rng([spec.seed, 0])
    T, n = spec.T, spec.n_slots
    if spec.ids_kind == "uniform":
        ids = rng.integers(0, n, size=T)
    elif spec.ids_kind == "zipf":
        p = finite_zipf_probs(n, spec.zipf_alpha)
        ids = rng.choice(n, size=T, p=p)          # rank k -> slot k-1
    elif spec.ids_kind == "segments":
        if sum(spec.segments) != T:
            raise ValueError("segment lengths do not add up to T")
        ids = np.concatenate([np.full(L, i) for i, L in enumerate(spec.segments)])
    elif spec.ids_kind == "mixed":
        active = np.sort(rng.choice(n, size=spec.n_active, replace=False))
        seg_ids = rng.choice(active, size=len(spec.segments))
        dec_ids = rng.choice(active, size=spec.n_decode)
        ids = np.concatenate([np.full(L, s) for L, s in zip(spec.segments, seg_ids)]
                             + [dec_ids])
        if ids.size != T:
            raise ValueError("mixed workload size mismatch")
    elif spec.ids_kind == "explicit":
        ids = np.asarray(spec.extra["ids"])
    else:
        raise ValueError(spec.ids_kind)
    return np.ascontiguousarray(ids.astype(np.int32))


def draw_proj(spec: WorkloadSpec, p: int, T: Optional[int] = None) -> ProjInputs:
    ps = spec.projs[p]
    T = spec.T if T is None else T
    rng = np.random.default_rng([spec.seed, 1, p])
    Xb, X = _normal_bf16(rng, (T, ps.d_in), 1.0)
    Wb, W = _normal_bf16(rng, (ps.d_in, ps.d_out), 1.0 / ps.d_in)
    if spec.weight_format == "int4_g128":
        q, sb = quantize_int4_g128(W)
        return ProjInputs(ps, Xb, X, Wb, W, q, sb)
    if spec.weight_format != "bf16":
        raise ValueError(spec.weight_format)
    return ProjInputs(ps, Xb, X, Wb, W)


def draw_adapter(spec: WorkloadSpec, slot: int) -> Adapter:
    r = int(spec.ranks[slot])
    rng = np.random.default_rng([spec.seed, 2, slot])
    Ab, A, Bb, B = [], [], [], []
    for ps in spec.projs:
        ab_l, a_l, bb_l, b_l = [], [], [], []
        for n_out in ps.slices:
            ab, a = _normal_bf16(rng, (ps.d_in, r), 1.0 / ps.d_in)
            bb, b = _normal_bf16(rng, (r, n_out), 1.0 / max(r, 1))
            ab_l.append(ab); a_l.append(a); bb_l.append(bb); b_l.append(b)
        Ab.append(ab_l); A.append(a_l); Bb.append(bb_l); B.append(b_l)
    return Adapter(slot, r, float(spec.scales[slot]), Ab, Bb, A, B)


def draw_adapters(spec: WorkloadSpec, slots: Sequence[int]) -> Dict[int, Adapter]:
    """The adapters of ``slots``, drawn on a few threads (each slot has its
    own random stream, so the result does not depend on the order)."""
    slots = [int(s) for s in slots]
    if len(slots) <= 4:
        return {s: draw_adapter(spec, s) for s in slots}
    from concurrent.futures import ThreadPoolExecutor
    workers = max(1, min(16, len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else 4))
    with ThreadPoolExecutor(max_workers=workers) as ex:
        drawn = list(ex.map(lambda s: draw_adapter(spec, s), slots))
    return dict(zip(slots, drawn))


def draw_layer(spec: WorkloadSpec, slots: Optional[Sequence[int]] = None) -> LayerInputs:
    """Draw ids, per-projection X and W, and the adapters of ``slots``
    (default: every slot that some token uses)."""
    ids = draw_ids(spec)
    projs = [draw_proj(spec, p) for p in range(len(spec.projs))]
    if slots is None:
        slots = sorted(int(s) for s in np.unique(ids) if s >= 0)
    return LayerInputs(spec, ids, projs, draw_adapters(spec, slots))


def custom_workload(name: str, projs: List[ProjSpec], T: int, ranks: Sequence[int],
                    scales: Optional[Sequence[float]] = None, ids=None, seed: int = 0,
                    ids_kind: str = "uniform", weight_format: str = "bf16") -> WorkloadSpec:
    """A generic test workload; ``ids`` may be given explicitly."""
    n = len(ranks)
    sc = list(scales) if scales is not None else [2.0] * n
    kind = "explicit" if ids is not None else ids_kind
    extra = {"ids": np.asarray(ids, dtype=np.int32)} if ids is not None else {}
    return WorkloadSpec(name, None, 0, list(projs), T=T, n_slots=n, ranks=list(ranks),
                        scales=sc, ids_kind=kind, seed=seed, extra=extra,
                        weight_format=weight_format)


__all__.append("custom_workload")
__all__.append("draw_adapters")
__all__.append("quantize_int4_g128")
__all__.append("tiny_mlp_projs")
