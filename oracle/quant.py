"""Weight-only INT4 base weight (W4A16) in float64 -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s CPU baseline
may use this package; the GPU path never does.

The paper serves BD-LoRA on top of a base model whose weights are quantized
to INT4 while activations stay 16-bit (Sec. 5.2, results with a quantized base
model; the quantized-backbone table of App. F).  The adapters are unchanged:
the LoRA term is computed exactly as for a 16-bit base.  The paper names the
data type only, so the format here is a reading (recorded with the other
readings of the paper in the design notes):

* symmetric INT4 per group of 128 input channels, one scale per (output
  column, group): ``W[k, n] = scale[n, k // 128] * q[n, k]`` with
  ``q in {-8, ..., 7}``;
* storage: ``q`` as nibbles ``q + 8``, two per byte, row ``n`` of the
  nn.Linear layout ``[d_out, d_in]``; byte ``(n, j)`` holds ``k = 2j`` in its
  low nibble and ``k = 2j + 1`` in its high nibble; scales are bf16 bit
  patterns ``[d_out, d_in / 128]``.

The shard forward with such a base is the forward of :mod:`oracle.bdlora` on
the dequantized weight (dequantization is exact in float64).

Pins (tests/test_oracle_quant.py): hand-built bytes against their nibble
values; a single non-zero nibble lands at the right (k, n) with the right
group's scale (catches a swapped nibble order, a transposed result or an
off-by-one group); Python loops for the dequantized forward on tiny inputs;
the bf16 scale decoding against hand-computed values.
"""
from __future__ import annotations

from typing import Dict, Sequence

import numpy as np

from .bdlora import ProjAdapter, shard_forward

GROUP = 128


def unpack_int4(qbytes: np.ndarray, K: int) -> np.ndarray:
    """``[N, K / 2]`` uint8 -> ``[N, K]`` int64 values in -8..7 (low nibble
    is the even input channel)."""
    qb = np.asarray(qbytes, dtype=np.uint8)
    if qb.ndim != 2 or qb.shape[1] * 2 != K:
        raise ValueError("qbytes must be [N, K/2]")
    lo = (qb & 0x0F).astype(np.int64) - 8
    hi = (qb >> 4).astype(np.int64) - 8
    out = np.empty((qb.shape[0], K), dtype=np.int64)
    out[:, 0::2] = lo
    out[:, 1::2] = hi
    return out


def bf16_bits_value(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> float64 values (the upper half of an fp32)."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def dequantize(qbytes: np.ndarray, scale_bits: np.ndarray, K: int) -> np.ndarray:
    """The base weight in the paper's orientation ``W [K, N]`` (float64):
    ``W[k, n] = scale[n, k // 128] * q[n, k]``."""
    if K % GROUP:
        raise ValueError("K must be a multiple of 128")
    q = unpack_int4(qbytes, K)                               # [N, K]
    s = bf16_bits_value(scale_bits)                          # [N, K / 128]
    if s.shape != (q.shape[0], K // GROUP):
        raise ValueError("scales must be [N, K/128]")
    w = q.astype(np.float64) * np.repeat(s, GROUP, axis=1)    # [N, K]
    return w.T.copy()


def shard_forward_w4(X: np.ndarray, qbytes: np.ndarray, scale_bits: np.ndarray,
                     ids: Sequence[int], adapters: Dict[int, ProjAdapter],
                     slices: Sequence[int]) -> np.ndarray:
    """One projection on one shard with an INT4 base weight: the shard
    forward of Alg. 1 / Alg. 2 on the dequantized weight."""
    K = np.asarray(X).shape[1]
    return shard_forward(X, dequantize(qbytes, scale_bits, K), ids, adapters, slices)


def brute_force_w4(X, qbytes, scale_bits, ids, adapters, slices) -> np.ndarray:
    """:func:`shard_forward_w4` with every step written as Python loops over
    the stored bytes (tiny inputs only)."""
    X = np.asarray(X, dtype=np.float64)
    S, K = X.shape
    qb = np.asarray(qbytes, dtype=np.uint8)
    N = qb.shape[0]
    scl = bf16_bits_value(scale_bits)

    def w(k, n):
        byte = int(qb[n, k // 2])
        nib = (byte & 15) if k % 2 == 0 else (byte >> 4)
        return float(scl[n, k // GROUP]) * (nib - 8)

    out = np.zeros((S, N))
    col0 = np.concatenate([[0], np.cumsum(slices)])
    for t in range(S):
        for n in range(N):
            out[t, n] = sum(X[t, k] * w(k, n) for k in range(K))
        a = int(ids[t])
        if a < 0:
            continue
        gamma, A_l, B_l = adapters[a]
        for j in range(len(slices)):
            A = np.asarray(A_l[j], dtype=np.float64)
            B = np.asarray(B_l[j], dtype=np.float64)
            z = [sum(X[t, k] * A[k, c] for k in range(K)) for c in range(A.shape[1])]
            for n in range(int(slices[j])):
                out[t, col0[j] + n] += gamma * sum(z[c] * B[c, n] for c in range(A.shape[1]))
    return out


def layer_forward_w4(layer, rows=None):
    """All projection calls of a drawn layer whose base weights are INT4
    (``workloads.LayerInputs`` with ``Wq`` / ``Ws_bits`` set), optionally for
    the token rows ``rows`` only."""
    ids = np.asarray(layer.ids)
    outs = []
    for p, pi in enumerate(layer.projs):
        ad = {s: (a.scale, a.A[p], a.B[p]) for s, a in layer.adapters.items()}
        X = pi.X if rows is None else pi.X[np.asarray(rows)]
        ii = ids if rows is None else ids[np.asarray(rows)]
        outs.append(shard_forward_w4(X, pi.Wq, pi.Ws_bits, ii, ad, pi.spec.slices))
    return outs
