"""Pins of the BD-LoRA MLP oracle (Alg. 1): loops, sharding, special cases.

Every check compares the oracle against something other than itself: Python
loops, the unsharded block-diagonal MLP assembled from the App. C.2 shard
layout, plain matrix products, scipy's logistic function and hand-computed
bf16 roundings.
"""
import numpy as np
import pytest
from scipy.special import expit

import workloads as wl
from oracle import bdlora, mlp

ACTS = ["none", "silu_mul"]


def _adapter(rng, d_in, r, n_out, gamma):
    return (gamma, [rng.standard_normal((d_in, r))], [rng.standard_normal((r, n_out)) / max(r, 1)])


def _tiny(rng, act, S=6, d_in=7, d_i=5, d_out=4, n_slots=3):
    X = rng.standard_normal((S, d_in))
    n_first = 1 if act == "none" else 2
    first = []
    for _ in range(n_first):
        W = rng.standard_normal((d_in, d_i)) / np.sqrt(d_in)
        ad = {s: _adapter(rng, d_in, 1 + s, d_i, 0.5 + s) for s in range(n_slots)}
        first.append((W, ad))
    W2 = rng.standard_normal((d_i, d_out)) / np.sqrt(d_i)
    ad2 = {s: _adapter(rng, d_i, 2 + s, d_out, 1.5 - 0.25 * s) for s in range(n_slots)}
    ids = rng.integers(-1, n_slots, size=S)
    ids[0] = -1
    return X, first, (W2, ad2), ids


@pytest.mark.parametrize("act", ACTS)
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_mlp_matches_loops(act, seed):
    rng = np.random.default_rng(seed)
    X, first, down, ids = _tiny(rng, act)
    _, y = mlp.mlp_shard_forward(X, first, down, ids, act, round_h=False)
    ref = mlp.mlp_brute_force(X, first, down, ids, act)
    np.testing.assert_allclose(y, ref, rtol=1e-10, atol=1e-12)


def test_silu_is_x_times_logistic():
    x = np.linspace(-30, 30, 1201)
    np.testing.assert_allclose(mlp.silu(x), x * expit(x), rtol=1e-13, atol=1e-300)
    assert mlp.silu(np.array([0.0]))[0] == 0.0


def test_bf16_rounding_by_hand_and_against_the_bit_trick():
    e = 2.0 ** -8
    cases = {1.0: 1.0, 1 + e: 1.0, 1 + 3 * e: 1 + 4 * e, 1 + 5 * e: 1 + 4 * e, 1 + 2.1 * e: 1 + 2 * e,
             -(1 + 3 * e): -(1 + 4 * e), 0.0: 0.0, 3.0: 3.0, 1000.0: 1000.0, 1001.0: 1000.0}
    for x, want in cases.items():
        assert mlp.round_bf16(np.array([x]))[0] == want, x
    # values exactly representable in fp32 round like the integer bit trick
    rng = np.random.default_rng(4)
    f = (rng.standard_normal(20000) * 10.0 ** rng.integers(-6, 6, 20000)).astype(np.float32)
    _, ref = wl.bf16_round(f)
    np.testing.assert_array_equal(mlp.round_bf16(f.astype(np.float64)), ref.astype(np.float64))


@pytest.mark.parametrize("act", ACTS)
def test_rank0_or_no_adapter_reduces_to_plain_products(act):
    rng = np.random.default_rng(7)
    X, first, down, _ = _tiny(rng, act, S=9)
    ids = np.full(9, -1)
    _, y = mlp.mlp_shard_forward(X, first, down, ids, act, round_h=False)
    h = X @ first[0][0] if act == "none" else (X @ first[0][0]) * expit(X @ first[0][0]) * (X @ first[1][0])
    np.testing.assert_allclose(y, h @ down[0], rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("act", ACTS)
@pytest.mark.parametrize("N", [2, 4])
def test_shards_sum_to_the_unsharded_block_diagonal_mlp(act, N):
    """Alg. 1: each device runs a local LoRA-MLP of width d_I/N and rank r/N;
    only the final all-reduce combines them.  The sum of the shards' outputs
    must equal the unsharded MLP whose column factors have a block-diagonal
    B and whose row factor has a block-diagonal A (App. C.2 compact storage)."""
    rng = np.random.default_rng(10 + N)
    S, d_h, d_i, r = 7, 12, 8 * N, 2 * N
    X = rng.standard_normal((S, d_h))
    slots = [0, 1, 2]
    ids = np.array([0, 1, 2, -1, 1, 0, 2])
    n_first = 1 if act == "none" else 2
    Wf = [rng.standard_normal((d_h, d_i)) / np.sqrt(d_h) for _ in range(n_first)]
    W2 = rng.standard_normal((d_i, d_h)) / np.sqrt(d_i)
    # full BD-LoRA factors per slot: column layers A_full [d_h, r], B compact [r/N, d_i];
    # row layer A compact [d_i, r/N], B_full [r, d_h]
    col = {s: [(rng.standard_normal((d_h, r)), rng.standard_normal((r // N, d_i))) for _ in range(n_first)]
           for s in slots}
    row = {s: (rng.standard_normal((d_i, r // N)), rng.standard_normal((r, d_h))) for s in slots}
    gam = {s: 0.5 + 0.5 * s for s in slots}

    # unsharded reference, token group by token group
    ref = np.zeros((S, d_h))
    for t in range(S):
        x = X[t:t + 1]
        a = int(ids[t])
        ys = []
        for j in range(n_first):
            if a < 0:
                ys.append(x @ Wf[j])
            else:
                ys.append(bdlora.column_full(x, Wf[j], col[a][j][0], col[a][j][1], N, gam[a]))
        h = ys[0] if act == "none" else mlp.silu(ys[0]) * ys[1]
        ref[t] = (h @ W2)[0] if a < 0 else bdlora.row_full(h, W2, row[a][0], row[a][1], N, gam[a])[0]

    total = np.zeros((S, d_h))
    n_s = d_i // N
    for i in range(N):
        first = []
        for j in range(n_first):
            ad = {}
            for s in slots:
                A_i, B_i = bdlora.column_shards(col[s][j][0], col[s][j][1], N)[i]
                ad[s] = (gam[s], [A_i], [B_i])
            first.append((Wf[j][:, i * n_s:(i + 1) * n_s], ad))
        ad2 = {}
        for s in slots:
            A_i, B_i = bdlora.row_shards(row[s][0], row[s][1], N)[i]
            ad2[s] = (gam[s], [A_i], [B_i])
        _, y = mlp.mlp_shard_forward(X, first, (W2[i * n_s:(i + 1) * n_s], ad2), ids, act, round_h=False)
        total += y
    np.testing.assert_allclose(total, ref, rtol=1e-10, atol=1e-10)


def test_rounded_intermediate_is_the_bf16_of_the_exact_one():
    rng = np.random.default_rng(3)
    X, first, down, ids = _tiny(rng, "silu_mul", S=8)
    h_exact, _ = mlp.mlp_shard_forward(X, first, down, ids, "silu_mul", round_h=False)
    h, y = mlp.mlp_shard_forward(X, first, down, ids, "silu_mul", round_h=True)
    np.testing.assert_array_equal(h, mlp.round_bf16(h_exact))
    np.testing.assert_allclose(y, bdlora.shard_forward(h, down[0], ids, down[1], [down[0].shape[1]]), rtol=1e-12)


# ---- the pins have teeth: planted mistakes are caught -----------------------

@pytest.mark.parametrize("kind", ["swap_gate_up", "no_down_lora", "act_on_up", "drop_gate_lora"])
def test_planted_mistakes_fail_the_loop_pin(kind):
    rng = np.random.default_rng(11)
    X, first, down, ids = _tiny(rng, "silu_mul", S=6)
    ref = mlp.mlp_brute_force(X, first, down, ids, "silu_mul")
    f, d = list(first), down
    if kind == "swap_gate_up":
        f = [first[1], first[0]]
    elif kind == "no_down_lora":
        d = (down[0], {s: (0.0, a, b) for s, (g, a, b) in down[1].items()})
    elif kind == "drop_gate_lora":
        f = [(first[0][0], {s: (0.0, a, b) for s, (g, a, b) in first[0][1].items()}), first[1]]
    if kind == "act_on_up":
        ys = [bdlora.shard_forward(X, W, ids, ad, [W.shape[1]]) for W, ad in first]
        h = ys[0] * mlp.silu(ys[1])
        y = bdlora.shard_forward(h, down[0], ids, down[1], [down[0].shape[1]])
    else:
        _, y = mlp.mlp_shard_forward(X, f, d, ids, "silu_mul", round_h=False)
    assert not np.allclose(y, ref, rtol=1e-6, atol=1e-8)
