"""BD-LoRA shard forward in float64 -- TEST INFRASTRUCTURE ONLY (see package doc).

The parity reference is the float64 evaluation.  ``shard_forward`` and the
layer helpers also take ``dtype=np.float32``: the same steps in single
precision, the plain fp32 CPU implementation whose speed the benchmark
reports as its CPU baseline.

Notation follows the paper.  ``X`` is ``[S, d_in]`` (S tokens), base weights
are in the paper's orientation ``W [d_in, d_out]`` so the base product is
``X W``; a LoRA adapter is ``A [d_in, r]``, ``B [r, d_out]`` with scale
``gamma`` (the rsLoRA parametrisation ``gamma * A B`` of Sec. 2).

What is computed, per shard i (Alg. 2, single column-parallel layer; Alg. 1
for the row-parallel second projection of an MLP):

    Y_base    = X W^(i)
    Z         = X A^(i)
    Y_adapter = Z B^(i)
    Y_local   = Y_base + gamma * Y_adapter

For a heterogeneous batch each token uses its own adapter (unmerged multi-LoRA
serving, Sec. 1 and Sec. 2 on S-LoRA): the oracle groups tokens by adapter id
and runs the steps above once per group, products taken as ``(X A) B``.
Tokens with id -1 get the base product only.

Pins (tests/test_oracle_*.py):
  * brute-force triple loops on tiny inputs (definition written out);
  * concatenated column shards equal the unsharded product with a
    block-diagonal B (Sec. 3 display equation, Fig. 3);
  * summed row partials equal the unsharded product with a block-diagonal A
    (Sec. 3, Alg. 1 final all-reduce);
  * a single-adapter batch equals the merged weight W + gamma A B (Sec. 1);
  * rank 0 / id -1 reduces to np.matmul of the base (Sec. 1, unmerged form);
  * each shard is an independent rank r/N LoRA of its weight shard (Sec. 3,
    alternative interpretation; App. B);
  * linearity in gamma; token-permutation equivariance.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from . import plan as _plan

# adapter for one projection: (gamma, [A per slice], [B per slice])
ProjAdapter = Tuple[float, List[np.ndarray], List[np.ndarray]]


def _f64(a) -> np.ndarray:
    return np.asarray(a, dtype=np.float64)


# --------------------------------------------------------------------------
# one shard, one projection call
# --------------------------------------------------------------------------

def shard_forward(X: np.ndarray, W: np.ndarray, ids: Sequence[int],
                  adapters: Dict[int, ProjAdapter], slices: Sequence[int],
                  dtype=np.float64) -> np.ndarray:
    """One projection on one shard for a heterogeneous batch (Alg. 2 / Alg. 1).

    ``X [S, d_in]``; ``W [d_in, sum(slices)]`` (paper orientation); ``ids[S]``
    are adapter ids (-1: none); ``adapters[slot] = (gamma, A_list, B_list)``
    where slice ``j`` has ``A_j [d_in, r]`` and ``B_j [r, slices[j]]``.  The
    output of slice ``j`` occupies columns ``sum(slices[:j]) ...`` (for the
    attention input projection: ``[q_s | k_s | v_s]``).  Returns
    ``[S, sum(slices)]`` in ``dtype`` (float64 unless asked otherwise).
    """
    X = np.asarray(X, dtype=dtype)
    W = np.asarray(W, dtype=dtype)
    ids = np.asarray(ids, dtype=np.int64)
    S, d_in = X.shape
    if W.shape != (d_in, int(sum(slices))):
        raise ValueError(f"W shape {W.shape} does not match d_in={d_in}, slices={slices}")
    if ids.shape != (S,):
        raise ValueError("ids must have one entry per token")
    # Y_base = X W  (base model contribution)
    Y = X @ W
    groups = _plan.group_rows(ids)
    for slot, rows in groups:
        if slot < 0:
            continue                                   # no adapter: base only
        gamma, A_list, B_list = adapters[slot]
        Xg = X[rows]
        col = 0
        for j, n_out in enumerate(slices):
            A = np.asarray(A_list[j], dtype=dtype)
            B = np.asarray(B_list[j], dtype=dtype)
            if A.shape[0] != d_in or B.shape[1] != n_out or A.shape[1] != B.shape[0]:
                raise ValueError(f"adapter {slot} slice {j}: bad shapes {A.shape} {B.shape}")
            Z = Xg @ A                                 # local adapter projection
            Y_adapter = Z @ B                          # expand
            Y[rows, col:col + n_out] += dtype(gamma) * Y_adapter
            col += n_out
    return Y


def layer_forward(layer, dtype=np.float64) -> List[np.ndarray]:
    """All projection calls of a drawn layer (``workloads.LayerInputs``).

    Each projection uses its own ``X`` and ``W`` (the inputs are independent
    synthetic tensors), the shared per-token ids and the shared adapters.
    Returns outputs (in ``dtype``) in the paper orientation ``[S, d_out_s]``.
    """
    outs = []
    for p, pi in enumerate(layer.projs):
        ad = {s: (a.scale, a.A[p], a.B[p]) for s, a in layer.adapters.items()}
        outs.append(shard_forward(pi.X, pi.W, layer.ids, ad, pi.spec.slices, dtype))
    return outs


def layer_forward_rows(layer, rows: Sequence[int], dtype=np.float64) -> List[np.ndarray]:
    """Like :func:`layer_forward` but only for the token rows ``rows``
    (each output row depends on its own token only)."""
    rows = np.asarray(rows, dtype=np.int64)
    outs = []
    for p, pi in enumerate(layer.projs):
        ad = {s: (a.scale, a.A[p], a.B[p]) for s, a in layer.adapters.items()}
        outs.append(shard_forward(pi.X[rows], pi.W, layer.ids[rows], ad, pi.spec.slices, dtype))
    return outs


# --------------------------------------------------------------------------
# brute force (tiny inputs only): the definition written out as loops
# --------------------------------------------------------------------------

def brute_force(X, W, ids, adapters: Dict[int, ProjAdapter], slices) -> np.ndarray:
    """Y[t, n] = sum_k X[t,k] W[k,n] + gamma_a * sum_j (sum_k X[t,k] A_a[k,j]) B_a[j,n]
    with a = ids[t], evaluated with Python loops in float64."""
    X = [[float(v) for v in row] for row in _f64(X)]
    W = [[float(v) for v in row] for row in _f64(W)]
    S = len(X)
    d_in = len(X[0]) if S else len(W)
    d_out = int(sum(slices))
    Y = [[0.0] * d_out for _ in range(S)]
    for t in range(S):
        for n in range(d_out):
            acc = 0.0
            for k in range(d_in):
                acc += X[t][k] * W[k][n]
            Y[t][n] = acc
        a = int(ids[t])
        if a < 0:
            continue
        gamma, A_list, B_list = adapters[a]
        col = 0
        for j, n_out in enumerate(slices):
            A = _f64(A_list[j])
            B = _f64(B_list[j])
            r = A.shape[1]
            z = [0.0] * r
            for q in range(r):
                s = 0.0
                for k in range(d_in):
                    s += X[t][k] * float(A[k, q])
                z[q] = s
            for n in range(n_out):
                s = 0.0
                for q in range(r):
                    s += z[q] * float(B[q, n])
                Y[t][col + n] += float(gamma) * s
            col += n_out
    return np.asarray(Y, dtype=np.float64).reshape(S, d_out)


# --------------------------------------------------------------------------
# unsharded BD-LoRA with explicit block-diagonal factors (Sec. 3, Fig. 3)
# --------------------------------------------------------------------------

def blockdiag(blocks: Sequence[np.ndarray]) -> np.ndarray:
    """Dense block-diagonal matrix with ``blocks`` on the diagonal and zeros
    elsewhere (blocks need not be square, Sec. 3 footnote)."""
    blocks = [_f64(b) for b in blocks]
    R = sum(b.shape[0] for b in blocks)
    C = sum(b.shape[1] for b in blocks)
    out = np.zeros((R, C), dtype=np.float64)
    r = c = 0
    for b in blocks:
        out[r:r + b.shape[0], c:c + b.shape[1]] = b
        r += b.shape[0]
        c += b.shape[1]
    return out


def column_shards(A_full: np.ndarray, B_compact: np.ndarray, N: int):
    """Shard a column-parallel BD-LoRA adapter (App. C.2 storage).

    ``A_full [d_in, r']`` is sharded column-wise; the block-diagonal ``B`` is
    stored compactly as ``[r'/N, d_out]`` with its N blocks side by side.
    Shard i gets ``A_i = A_full[:, i r'/N : (i+1) r'/N]`` and
    ``B_i = B_compact[:, i d_out/N : (i+1) d_out/N]``.
    """
    d_in, r_tot = A_full.shape
    r_s, d_out = B_compact.shape
    if r_tot % N or d_out % N or r_s * N != r_tot:
        raise ValueError("column shards: shapes not divisible by N")
    n_s = d_out // N
    return [(A_full[:, i * r_s:(i + 1) * r_s], B_compact[:, i * n_s:(i + 1) * n_s])
            for i in range(N)]


def row_shards(A_compact: np.ndarray, B_full: np.ndarray, N: int):
    """Shard a row-parallel BD-LoRA adapter (App. C.2 storage).

    The block-diagonal ``A`` is stored compactly as ``[d_in, r'/N]`` with its N
    blocks stacked on top of each other; ``B_full [r', d_out]`` is sharded
    row-wise.  Shard i gets ``A_i = A_compact[i d_in/N : (i+1) d_in/N, :]`` and
    ``B_i = B_full[i r'/N : (i+1) r'/N, :]``.
    """
    d_in, r_s = A_compact.shape
    r_tot, d_out = B_full.shape
    if d_in % N or r_tot % N or r_s * N != r_tot:
        raise ValueError("row shards: shapes not divisible by N")
    k_s = d_in // N
    return [(A_compact[i * k_s:(i + 1) * k_s, :], B_full[i * r_s:(i + 1) * r_s, :])
            for i in range(N)]


def column_full(X, W_full, A_full, B_compact, N: int, gamma: float) -> np.ndarray:
    """Unsharded column layer ``X W + gamma X A blockdiag(B_1..B_N)``."""
    B_blocks = [b for _, b in column_shards(_f64(A_full), _f64(B_compact), N)]
    return _f64(X) @ _f64(W_full) + gamma * (_f64(X) @ _f64(A_full)) @ blockdiag(B_blocks)


def row_full(X, W_full, A_compact, B_full, N: int, gamma: float) -> np.ndarray:
    """Unsharded row layer ``X W + gamma X blockdiag(A_1..A_N) B`` (the value
    the base all-reduce returns once the LoRA partials are added in)."""
    A_blocks = [a for a, _ in row_shards(_f64(A_compact), _f64(B_full), N)]
    return _f64(X) @ _f64(W_full) + gamma * (_f64(X) @ blockdiag(A_blocks)) @ _f64(B_full)


def merged_forward(X, W, A, B, gamma: float) -> np.ndarray:
    """Single adapter merged into the weight: ``X (W + gamma A B)`` (Sec. 1)."""
    return _f64(X) @ (_f64(W) + gamma * (_f64(A) @ _f64(B)))


# --------------------------------------------------------------------------
# comparison rule used by the parity tests
# --------------------------------------------------------------------------

def rel_errors(y: np.ndarray, ref: np.ndarray) -> Dict[str, float]:
    """Errors of ``y`` against ``ref``: the pointwise ratio
    ``|y - ref| / max(|ref|, rms(ref))`` (max over elements), the max
    absolute error over max |ref|, and the Frobenius relative error."""
    y = _f64(y)
    ref = _f64(ref)
    if y.shape != ref.shape:
        raise ValueError(f"shape mismatch {y.shape} vs {ref.shape}")
    if ref.size == 0:
        return {"pointwise": 0.0, "maxabs_over_maxref": 0.0, "frobenius": 0.0}
    rms = float(np.sqrt(np.mean(ref * ref)))
    floor = max(rms, np.finfo(np.float64).tiny)
    d = np.abs(y - ref)
    pw = float(np.max(d / np.maximum(np.abs(ref), floor)))
    mref = float(np.max(np.abs(ref)))
    return {
        "pointwise": pw,
        "maxabs_over_maxref": float(np.max(d)) / max(mref, np.finfo(np.float64).tiny),
        "frobenius": float(np.linalg.norm(y - ref) / max(np.linalg.norm(ref), floor)),
    }


def delta_errors(y: np.ndarray, y_base: np.ndarray, ref: np.ndarray,
                 ref_base: np.ndarray, rounding: float = 2.0 ** -8) -> float:
    """Pointwise error of the LoRA term alone: ``(y - y_base)`` against
    ``(ref - ref_base)``, with the floor taken from the full output's rms.

    ``y`` and ``y_base`` are each rounded once to the output format; the
    difference of two such numbers carries both roundings, so those
    (``rounding`` times ``|y| + |y_base|``, 2^-8 for bfloat16 round to
    nearest) are removed from the discrepancy before it is compared."""
    d = _f64(y) - _f64(y_base)
    dr = _f64(ref) - _f64(ref_base)
    if dr.size == 0:
        return 0.0
    rms = float(np.sqrt(np.mean(_f64(ref) ** 2)))
    floor = max(rms, np.finfo(np.float64).tiny)
    allow = rounding * (np.abs(_f64(y)) + np.abs(_f64(y_base)))
    excess = np.maximum(np.abs(d - dr) - allow, 0.0)
    return float(np.max(excess / np.maximum(np.abs(dr), floor)))
