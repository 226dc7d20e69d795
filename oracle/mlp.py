"""BD-LoRA MLP shard forward (Alg. 1) in float64 -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s CPU baseline
may use this package; the GPU path never does.

Alg. 1 (App. B), on device i:

    Y1 = X W1 + (X A1) B1        first projection, column-parallel, B1 block-diagonal
    Y2 = Y1 W2 + (Y1 A2) B2      second projection, row-parallel, A2 block-diagonal

followed by the base model's all-reduce over devices.  Alg. 1 writes the two
projections back to back.  The Llama MLPs the paper serves (Sec. 4) put a
gated activation between them: two column projections ``gate`` and ``up``
(each with its own BD-LoRA adapter, as the paper's parameter counts require) and
``H = silu(gate) * up`` feeding the row projection ``down``.  Both forms are
here: ``act="none"`` (H = Y1, Alg. 1 as written) and ``act="silu_mul"``.

The intermediate H is held in bfloat16 (round to nearest, ties to even), as
the GPU path stores it between the two projections; ``round_h=False`` keeps
it in float64 (used by the pins).

Pins (tests/test_oracle_mlp.py): a Python-loop evaluation on tiny inputs;
the sum of the N shards' outputs equals the unsharded MLP with block-
diagonal factors (the claim of Alg. 1 that only the final all-reduce
communicates); rank 0 reduces to two plain matrix products; silu against
the logistic function of scipy; the bf16 rounding against hand-computed
values.
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from .bdlora import ProjAdapter, shard_forward

ACTS = ("none", "silu_mul")


def silu(x: np.ndarray) -> np.ndarray:
    """x * sigmoid(x) = x / (1 + exp(-x)), float64."""
    x = np.asarray(x, dtype=np.float64)
    return x / (1.0 + np.exp(-x))


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Nearest bfloat16 value (8 significant bits, ties to even) of float64
    ``x``, returned as float64.  Finite normal-range inputs (zero kept)."""
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)                  # x = m 2^e, 0.5 <= |m| < 1
    q = np.rint(m * 256.0)              # 8 significant bits, half to even
    return np.ldexp(q / 256.0, e)


def mlp_shard_forward(X: np.ndarray, first: Sequence[Tuple[np.ndarray, Dict[int, ProjAdapter]]],
                      down: Tuple[np.ndarray, Dict[int, ProjAdapter]], ids: Sequence[int],
                      act: str = "silu_mul", round_h: bool = True) -> Tuple[np.ndarray, np.ndarray]:
    """One device's share of the MLP of Alg. 1 for a heterogeneous batch.

    ``first``: ``[(W1, adapters)]`` for ``act="none"`` or ``[(W_gate,
    adapters), (W_up, adapters)]`` for ``act="silu_mul"``; weights in the
    paper orientation ``[d_in, d_out]``, adapters as in
    :func:`oracle.bdlora.shard_forward` (one slice).  ``down = (W2,
    adapters)``.  Returns ``(H, Y2)``: the intermediate ``[S, d_I/N]`` and the
    device's partial output ``[S, d_out]`` (float64).
    """
    if act not in ACTS:
        raise ValueError(f"act must be one of {ACTS}")
    if len(first) != (1 if act == "none" else 2):
        raise ValueError("act='none' takes one first projection, 'silu_mul' two (gate, up)")
    ys = [shard_forward(X, W, ids, ad, [W.shape[1]]) for W, ad in first]
    H = ys[0] if act == "none" else silu(ys[0]) * ys[1]
    if round_h:
        H = round_bf16(H)
    W2, ad2 = down
    return H, shard_forward(H, W2, ids, ad2, [W2.shape[1]])


def mlp_brute_force(X, first, down, ids, act: str) -> np.ndarray:
    """``Y2`` of :func:`mlp_shard_forward` with ``round_h=False``, written
    out with Python loops (tiny inputs only)."""
    X = np.asarray(X, dtype=np.float64)
    S, d_in = X.shape

    def proj(Xm, W, ad):
        W = np.asarray(W, dtype=np.float64)
        n_in, n_out = W.shape
        Y = [[0.0] * n_out for _ in range(len(Xm))]
        for t in range(len(Xm)):
            for n in range(n_out):
                Y[t][n] = sum(Xm[t][k] * W[k, n] for k in range(n_in))
            a = int(ids[t])
            if a >= 0:
                gamma, A_l, B_l = ad[a]
                A = np.asarray(A_l[0], dtype=np.float64)
                B = np.asarray(B_l[0], dtype=np.float64)
                z = [sum(Xm[t][k] * A[k, j] for k in range(n_in)) for j in range(A.shape[1])]
                for n in range(n_out):
                    Y[t][n] += gamma * sum(z[j] * B[j, n] for j in range(A.shape[1]))
        return Y

    Xm = [[float(v) for v in row] for row in X]
    ys = [proj(Xm, W, ad) for W, ad in first]
    if act == "none":
        H = ys[0]
    else:
        H = [[g / (1.0 + math.exp(-g)) * u for g, u in zip(rg, ru)] for rg, ru in zip(ys[0], ys[1])]
    W2, ad2 = down
    return np.asarray(proj(H, W2, ad2), dtype=np.float64)


def mlp_layer_forward(layer, first: Sequence[int], down_idx: int, act: str,
                      rows: Optional[Sequence[int]] = None) -> Tuple[np.ndarray, np.ndarray]:
    """:func:`mlp_shard_forward` on a drawn layer (``workloads.LayerInputs``):
    the first projections' ``X`` (they share one input) and weights, the down
    projection's weights and every projection's adapters."""
    def ad(p):
        return {s: (a.scale, a.A[p], a.B[p]) for s, a in layer.adapters.items()}
    X = layer.projs[first[0]].X
    ids = layer.ids
    if rows is not None:
        rows = np.asarray(rows, dtype=np.int64)
        X, ids = X[rows], ids[rows]
    return mlp_shard_forward(X, [(layer.projs[p].W, ad(p)) for p in first],
                             (layer.projs[down_idx].W, ad(down_idx)), ids, act)
