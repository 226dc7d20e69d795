"""Pins for the oracle's shard forward (CPU only).

Each check ties oracle.bdlora to something other than itself: the definition
written out as loops, the block-diagonal identity of Sec. 3, the merged-weight
form of Sec. 1, the "N independent LoRAs" reading of Sec. 3 / App. B, and
plain linear-algebra invariants.  A last test plants mistakes in a copy of the
oracle and checks that the pins catch each of them.
"""
import numpy as np
import pytest

from oracle import bdlora
from workloads import bf16_round


def _bf(rng, shape, scale=1.0):
    return bf16_round(rng.standard_normal(shape).astype(np.float32) * scale)[1]


def _tiny_case(seed=0, T=7, d_in=12, slices=(5, 3, 4), ranks=(0, 1, 2, 4)):
    rng = np.random.default_rng(seed)
    X = _bf(rng, (T, d_in))
    W = _bf(rng, (d_in, sum(slices)), 0.3)
    adapters = {}
    for s, r in enumerate(ranks):
        A = [_bf(rng, (d_in, r), 0.3) for _ in slices]
        B = [_bf(rng, (r, n), 0.5) for n in slices]
        adapters[s] = (0.5 + s, A, B)
    ids = rng.integers(-1, len(ranks), size=T)
    ids[0] = -1
    ids[1] = len(ranks) - 1
    return X, W, ids, adapters, slices


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_matches_brute_force(seed):
    X, W, ids, ad, sl = _tiny_case(seed)
    y = bdlora.shard_forward(X, W, ids, ad, sl)
    yb = bdlora.brute_force(X, W, ids, ad, sl)
    np.testing.assert_allclose(y, yb, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("seed", [0, 1])
def test_float32_evaluation_matches_brute_force_to_single_precision(seed):
    # the single-precision evaluation (the CPU baseline's) computes the same
    # steps: against the float64 brute force it may differ only by float32
    # rounding of sums over at most d_in + r terms
    X, W, ids, ad, sl = _tiny_case(seed, T=9, d_in=40)
    y = bdlora.shard_forward(X, W, ids, ad, sl, dtype=np.float32)
    assert y.dtype == np.float32
    yb = bdlora.brute_force(X, W, ids, ad, sl)
    scale = np.abs(yb).max()
    assert np.max(np.abs(y - yb)) <= 64 * np.finfo(np.float32).eps * scale


def test_empty_batch():
    X, W, ids, ad, sl = _tiny_case(0)
    y = bdlora.shard_forward(X[:0], W, ids[:0], ad, sl)
    assert y.shape == (0, sum(sl))


def test_rank0_and_no_adapter_reduce_to_base():
    X, W, ids, ad, sl = _tiny_case(3)
    base = np.matmul(X.astype(np.float64), W.astype(np.float64))
    for a in (-1, 0):          # slot 0 has rank 0
        y = bdlora.shard_forward(X, W, np.full(len(X), a), ad, sl)
        np.testing.assert_array_equal(y, base)


def test_single_adapter_equals_merged_weight():
    X, W, _, ad, sl = _tiny_case(4, slices=(9,))
    gamma, A, B = ad[3]
    y = bdlora.shard_forward(X, W, np.full(len(X), 3), ad, sl)
    ym = bdlora.merged_forward(X, W, A[0], B[0], gamma)
    np.testing.assert_allclose(y, ym, rtol=1e-12, atol=1e-12)


def test_token_permutation_equivariance():
    X, W, ids, ad, sl = _tiny_case(5, T=11)
    y = bdlora.shard_forward(X, W, ids, ad, sl)
    p = np.random.default_rng(9).permutation(len(X))
    yp = bdlora.shard_forward(X[p], W, ids[p], ad, sl)
    np.testing.assert_allclose(yp, y[p], rtol=0, atol=1e-12)


def test_rows_independent_of_other_tokens():
    X, W, ids, ad, sl = _tiny_case(6, T=9)
    y = bdlora.shard_forward(X, W, ids, ad, sl)
    for t in range(len(X)):
        yt = bdlora.shard_forward(X[t:t + 1], W, ids[t:t + 1], ad, sl)
        np.testing.assert_allclose(yt[0], y[t], rtol=0, atol=1e-12)


def test_linear_in_gamma():
    X, W, ids, ad, sl = _tiny_case(7)
    def with_gamma(g):
        return bdlora.shard_forward(X, W, ids, {s: (g, A, B) for s, (_, A, B) in ad.items()}, sl)
    y0, y1, y3 = with_gamma(0.0), with_gamma(1.0), with_gamma(3.0)
    np.testing.assert_allclose(y3 - y0, 3.0 * (y1 - y0), rtol=1e-12, atol=1e-12)
    np.testing.assert_array_equal(y0, np.matmul(X.astype(np.float64), W.astype(np.float64)))


# ---- block-diagonal identities (Sec. 3, Fig. 3, Alg. 1, App. C.2) ----------

def _bd_column_setup(seed, N=4, d_in=16, d_out=24, r_tot=8, S=5):
    rng = np.random.default_rng(seed)
    X = _bf(rng, (S, d_in))
    Wf = _bf(rng, (d_in, d_out), 0.3)
    Af = _bf(rng, (d_in, r_tot), 0.3)
    Bc = _bf(rng, (r_tot // N, d_out), 0.5)       # compact storage of block-diagonal B
    return X, Wf, Af, Bc


@pytest.mark.parametrize("N", [2, 4])
def test_column_shards_concatenate_to_blockdiag_product(N):
    X, Wf, Af, Bc = _bd_column_setup(10, N=N)
    gamma = 1.7
    n_s = Wf.shape[1] // N
    shards = bdlora.column_shards(Af, Bc, N)
    outs = []
    for i, (A_i, B_i) in enumerate(shards):
        W_i = Wf[:, i * n_s:(i + 1) * n_s]
        outs.append(bdlora.shard_forward(X, W_i, np.zeros(len(X), int),
                                         {0: (gamma, [A_i], [B_i])}, (n_s,)))
    y_cat = np.concatenate(outs, axis=1)
    # the unsharded product with an explicit dense block-diagonal B
    Bd = np.zeros((Af.shape[1], Wf.shape[1]))
    r_s = Af.shape[1] // N
    for i in range(N):
        Bd[i * r_s:(i + 1) * r_s, i * n_s:(i + 1) * n_s] = Bc[:, i * n_s:(i + 1) * n_s]
    y_full = X.astype(np.float64) @ Wf + gamma * (X.astype(np.float64) @ Af) @ Bd
    np.testing.assert_allclose(y_cat, y_full, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(bdlora.column_full(X, Wf, Af, Bc, N, gamma), y_full,
                               rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("N", [2, 4])
def test_row_partials_sum_to_blockdiag_product(N):
    rng = np.random.default_rng(11)
    S, d_in, d_out, r_tot = 5, 16, 20, 8
    X = _bf(rng, (S, d_in))
    Wf = _bf(rng, (d_in, d_out), 0.3)
    Ac = _bf(rng, (d_in, r_tot // N), 0.3)         # compact storage of block-diagonal A
    Bf = _bf(rng, (r_tot, d_out), 0.5)
    gamma = 0.8
    k_s = d_in // N
    total = np.zeros((S, d_out))
    for i, (A_i, B_i) in enumerate(bdlora.row_shards(Ac, Bf, N)):
        X_i = X[:, i * k_s:(i + 1) * k_s]
        W_i = Wf[i * k_s:(i + 1) * k_s, :]
        total += bdlora.shard_forward(X_i, W_i, np.zeros(S, int),
                                      {0: (gamma, [A_i], [B_i])}, (d_out,))
    Ad = np.zeros((d_in, r_tot))
    r_s = r_tot // N
    for i in range(N):
        Ad[i * k_s:(i + 1) * k_s, i * r_s:(i + 1) * r_s] = Ac[i * k_s:(i + 1) * k_s, :]
    y_full = X.astype(np.float64) @ Wf + gamma * (X.astype(np.float64) @ Ad) @ Bf
    np.testing.assert_allclose(total, y_full, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(bdlora.row_full(X, Wf, Ac, Bf, N, gamma), y_full,
                               rtol=1e-12, atol=1e-12)


def test_each_shard_is_an_independent_lora_of_its_weight_shard():
    # Sec. 3 alternative interpretation: shard i == plain LoRA (rank r'/N) merged
    # into its own weight shard
    N = 4
    X, Wf, Af, Bc = _bd_column_setup(12, N=N)
    n_s = Wf.shape[1] // N
    for i, (A_i, B_i) in enumerate(bdlora.column_shards(Af, Bc, N)):
        W_i = Wf[:, i * n_s:(i + 1) * n_s]
        y = bdlora.shard_forward(X, W_i, np.zeros(len(X), int), {0: (2.0, [A_i], [B_i])}, (n_s,))
        np.testing.assert_allclose(y, bdlora.merged_forward(X, W_i, A_i, B_i, 2.0),
                                   rtol=1e-12, atol=1e-12)
        assert A_i.shape == (Af.shape[0], Af.shape[1] // N)
        assert B_i.shape == (Af.shape[1] // N, n_s)


def test_qkv_slices_match_three_separate_layers():
    # the q/k/v call is three column layers, each with its own adapter, outputs
    # side by side
    rng = np.random.default_rng(13)
    S, d_in, sl = 6, 16, (8, 4, 4)
    X = _bf(rng, (S, d_in))
    W = _bf(rng, (d_in, sum(sl)), 0.3)
    A = [_bf(rng, (d_in, 3), 0.3) for _ in sl]
    B = [_bf(rng, (3, n), 0.5) for n in sl]
    ids = np.array([0, -1, 0, 0, -1, 0])
    y = bdlora.shard_forward(X, W, ids, {0: (1.5, A, B)}, sl)
    col = 0
    for j, n in enumerate(sl):
        yj = bdlora.shard_forward(X, W[:, col:col + n], ids, {0: (1.5, [A[j]], [B[j]])}, (n,))
        np.testing.assert_array_equal(y[:, col:col + n], yj)
        col += n


def test_blockdiag_helper():
    a = np.arange(6.0).reshape(2, 3)
    b = np.arange(4.0).reshape(4, 1)
    d = bdlora.blockdiag([a, b])
    assert d.shape == (6, 4)
    np.testing.assert_array_equal(d[:2, :3], a)
    np.testing.assert_array_equal(d[2:, 3:], b)
    assert np.count_nonzero(d[:2, 3:]) == 0 and np.count_nonzero(d[2:, :3]) == 0


def test_error_rule():
    ref = np.array([[1.0, -2.0, 0.0, 1e-9]])
    assert bdlora.rel_errors(ref, ref)["pointwise"] == 0.0
    y = ref + 1e-3
    e = bdlora.rel_errors(y, ref)
    rms = np.sqrt(np.mean(ref ** 2))
    assert abs(e["pointwise"] - 1e-3 / rms) < 1e-12


# ---- the pins have teeth: planted mistakes are caught -----------------------

def _mutant(kind):
    def fwd(X, W, ids, adapters, slices):
        X = np.asarray(X, np.float64)
        W = np.asarray(W, np.float64)
        Y = X @ W if kind != "no_base" else np.zeros((X.shape[0], W.shape[1]))
        for t, a in enumerate(ids):
            if a < 0:
                continue
            g, A_l, B_l = adapters[int(a)]
            col = 0
            for j, n in enumerate(slices):
                A = np.asarray(A_l[j], np.float64)
                B = np.asarray(B_l[j], np.float64)
                src = X[(t + 1) % len(X)] if kind == "wrong_row" else X[t]
                z = src @ A
                gg = 1.0 if kind == "no_gamma" else g
                c0 = col + (1 if kind == "shifted_slice" and j == 1 else 0)
                upd = gg * (z @ B)
                if kind == "sign":
                    upd = -upd
                Y[t, c0:c0 + n] += upd[: max(0, min(n, Y.shape[1] - c0))]
                col += n
        return Y
    return fwd


@pytest.mark.parametrize("kind", ["no_base", "no_gamma", "wrong_row", "shifted_slice", "sign"])
def test_planted_mistakes_fail_the_brute_force_pin(kind):
    X, W, ids, ad, sl = _tiny_case(21)
    yb = bdlora.brute_force(X, W, ids, ad, sl)
    ym = _mutant(kind)(X, W, ids, ad, sl)
    assert not np.allclose(ym, yb, rtol=1e-9, atol=1e-9)


def test_delta_error_rule_allows_only_output_rounding():
    from workloads import bf16_round
    rng = np.random.default_rng(3)
    ref_base = rng.standard_normal(500) * 2
    ref = ref_base + rng.standard_normal(500)
    y = bf16_round(ref)[1].astype(np.float64)
    yb = bf16_round(ref_base)[1].astype(np.float64)
    assert bdlora.delta_errors(y, yb, ref, ref_base) == 0.0      # rounding alone passes
    y_bad = y.copy()
    y_bad[7] += 0.1                                              # a real 0.1 error does not
    assert bdlora.delta_errors(y_bad, yb, ref, ref_base) > 0.01
