"""Parameter, operation and data-movement counts -- TEST INFRASTRUCTURE ONLY.

Follows the cost table of App. A (S-LoRA vs BD-LoRA per LoRA factor, per
device, for one basic MLP) and the trainable-parameter column of the paper's
fine-tuning score table (App. E) and run-time tables (App. F).

Conventions: ``r`` is the S-LoRA (standard LoRA) rank, ``r'`` (``r_total``
here) the total BD-LoRA rank, ``r_s = r'/N`` the per-shard rank (Sec. 3: each
shard carries an independent rank r'/N adapter).

Pins (tests/test_oracle_costs.py): the printed parameter counts of the paper
(golden file with citations), the equal-parameter rank identity of App. A,
and brute-force counting of the elements of drawn adapters.
"""
from __future__ import annotations

from typing import Dict, List, Sequence, Tuple

# (name, kind, d_in_full, d_out_full) of the seven adapted linear layers
_LAYERS = ("q", "k", "v", "o", "gate", "up", "down")


def llama_linears(d_h: int, d_i: int, d_kv: int) -> List[Tuple[str, str, int, int]]:
    """The seven adapted linear layers of a Llama decoder layer: q, k, v
    (column), o (row), gate, up (column), down (row)."""
    return [
        ("q", "column", d_h, d_h), ("k", "column", d_h, d_kv), ("v", "column", d_h, d_kv),
        ("o", "row", d_h, d_h),
        ("gate", "column", d_h, d_i), ("up", "column", d_h, d_i),
        ("down", "row", d_i, d_h),
    ]


def bd_shard_params(kind: str, d_in: int, d_out: int, r_total: int, N: int) -> int:
    """Adapter elements on ONE shard of one BD-LoRA linear layer of full size
    ``d_in x d_out`` (Alg. 1 and Alg. 2 factor shapes).

    column: A_s is d_in x r'/N, B_s (one diagonal block) is r'/N x d_out/N;
    row:    A_s (one diagonal block) is d_in/N x r'/N, B_s is r'/N x d_out.
    """
    if r_total % N:
        raise ValueError("r' must be divisible by N")
    r_s = r_total // N
    if kind == "column":
        return d_in * r_s + r_s * (d_out // N)
    if kind == "row":
        return (d_in // N) * r_s + r_s * d_out
    raise ValueError(kind)


def bd_model_params(d_h: int, d_i: int, d_kv: int, n_layers: int, r_total: int, N: int) -> int:
    """Trainable parameters of a BD-LoRA adapter on all seven linear layers of
    every decoder layer, summed over the N shards."""
    per_layer = sum(N * bd_shard_params(kind, di, do, r_total, N)
                    for _, kind, di, do in llama_linears(d_h, d_i, d_kv))
    return n_layers * per_layer


def lora_model_params(d_h: int, d_i: int, d_kv: int, n_layers: int, r: int) -> int:
    """Trainable parameters of a standard LoRA adapter of rank r on all seven
    linear layers: r (d_in + d_out) per layer (Sec. 1)."""
    return n_layers * sum(r * (di + do) for _, _, di, do in llama_linears(d_h, d_i, d_kv))


def mlp_cost_table(method: str, S: int, d_h: int, d_i: int, rank: int, N: int) -> Dict[str, Dict[str, float]]:
    """Per-device rows of the App. A cost table for one basic MLP
    (W1: d_H x d_I column-parallel, W2: d_I x d_H row-parallel).

    Each row: ``params`` (elements per device), ``ops`` (floating-point
    operations), ``out`` (elements written and read for the output).
    ``rank`` is r for S-LoRA and r' for BD-LoRA.
    """
    r = rank
    if method == "s-lora":
        rows = {
            "A1": (d_h * r / N, S * r / N),
            "B1": (d_i * r / N, S * d_i / N),
            "A2": (d_i * r / N, S * r),
            "B2": (d_h * r / N, S * d_h / N),
        }
    elif method == "bd-lora":
        rows = {
            "A1": (d_h * r / N, S * r / N),
            "B1": ((d_i / N) * (r / N), S * d_i / N),
            "A2": ((d_i / N) * (r / N), S * r / N),
            "B2": (d_h * r / N, S * d_h),
        }
    else:
        raise ValueError(method)
    out = {}
    for k, (p, o) in rows.items():
        out[k] = {"params": p, "ops": 2.0 * S * p, "out": 2.0 * o}
    out["sum"] = {f: sum(out[k][f] for k in rows) for f in ("params", "ops", "out")}
    return out


def equal_param_rank(r: float, d_h: int, d_i: int, N: int) -> float:
    """BD-LoRA total rank with the same per-device parameter count as S-LoRA
    rank r (App. A): r' = r (d_H + d_I) / (d_H + d_I / N)."""
    return r * (d_h + d_i) / (d_h + d_i / N)


# --------------------------------------------------------------------------
# algorithmic work of one batch on one shard (what the method must move)
# --------------------------------------------------------------------------

def batch_bytes(projs, T: int, active_ranks: Sequence[int], elem_bytes: int = 2) -> int:
    """Bytes one shard forward must move for ``T`` tokens: every base weight
    once, every input and output once per projection, and the factors of
    every adapter that some token uses, once each (``active_ranks`` lists the
    true rank of each distinct adapter in the batch).  ``projs`` items carry
    ``d_in`` and ``slices``."""
    total = 0
    for p in projs:
        n = int(sum(p.slices))
        total += p.d_in * n + T * p.d_in + T * n
        for r in active_ranks:
            total += len(p.slices) * p.d_in * r + r * n
    return total * elem_bytes


def batch_flops(projs, token_ranks: Sequence[int]) -> int:
    """Multiply-add work counted as 2 operations each: the base product for
    every token plus, per token, ``X A`` and ``Z B`` of its own adapter
    (matmul cost 2 S #params, App. A); ``token_ranks[t]`` is the rank of
    token t's adapter (0 for none)."""
    T = len(token_ranks)
    total = 0
    for p in projs:
        n = int(sum(p.slices))
        total += 2 * T * p.d_in * n
        for r in token_ranks:
            total += 2 * (len(p.slices) * p.d_in * r + r * n)
    return total
