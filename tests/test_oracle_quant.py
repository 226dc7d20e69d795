"""Pins of the INT4 base-weight oracle (weight-only quantized base, Sec. 5.2).

Every check compares the oracle against something other than itself: bytes
built by hand, a single planted nibble, Python loops over the stored bytes,
bf16 values computed by hand, and the error bound of round-to-nearest
quantization for the workload generator.
"""
import numpy as np
import pytest

import workloads as wl
from oracle import bdlora, quant


def test_unpack_hand_built_bytes():
    # byte 0x3A: low nibble 0xA -> 10 - 8 = 2 (even k), high nibble 3 -> -5 (odd k)
    qb = np.array([[0x3A, 0x80, 0x0F, 0xF0]], dtype=np.uint8)
    got = quant.unpack_int4(qb, 8)
    np.testing.assert_array_equal(got, [[2, -5, -8, 0, 7, -8, -8, 7]])


def test_bf16_scale_values_by_hand():
    bits = np.array([0x3F80, 0x4000, 0xBF00, 0x3C00, 0x4308], dtype=np.uint16)
    np.testing.assert_array_equal(quant.bf16_bits_value(bits), [1.0, 2.0, -0.5, 2.0 ** -7, 136.0])


@pytest.mark.parametrize("n,k", [(0, 0), (3, 1), (5, 127), (2, 128), (7, 255), (1, 130)])
def test_single_nibble_lands_at_its_place_with_its_groups_scale(n, k):
    N, K = 8, 256
    qb = np.full((N, K // 2), 0x88, dtype=np.uint8)            # every value 0
    byte = qb[n, k // 2]
    qb[n, k // 2] = (byte & 0xF0) | 13 if k % 2 == 0 else (byte & 0x0F) | (2 << 4)
    want_q = 13 - 8 if k % 2 == 0 else 2 - 8
    sb = np.zeros((N, K // 128), dtype=np.uint16)
    sb[:, 0] = 0x3F80                                          # 1.0 for group 0
    sb[:, 1] = 0x4040                                          # 3.0 for group 1
    W = quant.dequantize(qb, sb, K)
    assert W.shape == (K, N)
    want = np.zeros((K, N))
    want[k, n] = want_q * (1.0 if k < 128 else 3.0)
    np.testing.assert_array_equal(W, want)


@pytest.mark.parametrize("seed", [0, 1])
def test_w4_forward_matches_loops_over_the_bytes(seed):
    rng = np.random.default_rng(seed)
    S, K, slices = 5, 256, [16, 8]
    N = sum(slices)
    X = rng.standard_normal((S, K))
    qb = rng.integers(0, 256, size=(N, K // 2), dtype=np.uint8)
    sb, _ = wl.bf16_round(rng.uniform(0.01, 0.1, size=(N, K // 128)).astype(np.float32))
    ad = {s: (0.5 + s, [rng.standard_normal((K, 2 + s)) for _ in slices],
              [rng.standard_normal((2 + s, o)) for o in slices]) for s in range(2)}
    ids = np.array([0, -1, 1, 1, 0])
    got = quant.shard_forward_w4(X, qb, sb, ids, ad, slices)
    ref = quant.brute_force_w4(X, qb, sb, ids, ad, slices)
    np.testing.assert_allclose(got, ref, rtol=1e-10, atol=1e-10)


def test_w4_forward_is_the_forward_on_the_dequantized_weight():
    # the LoRA term does not see the quantization: the difference between the
    # W4 forward and the forward on any other base weight is the difference of
    # the base products alone
    rng = np.random.default_rng(3)
    S, K, N = 6, 128, 32
    X = rng.standard_normal((S, K))
    qb = rng.integers(0, 256, size=(N, K // 2), dtype=np.uint8)
    sb, _ = wl.bf16_round(np.full((N, 1), 0.05, dtype=np.float32))
    ad = {0: (2.0, [rng.standard_normal((K, 4))], [rng.standard_normal((4, N))])}
    ids = np.array([0, 0, -1, 0, -1, 0])
    W0 = rng.standard_normal((K, N))
    d = quant.shard_forward_w4(X, qb, sb, ids, ad, [N]) - bdlora.shard_forward(X, W0, ids, ad, [N])
    np.testing.assert_allclose(d, X @ (quant.dequantize(qb, sb, K) - W0), rtol=1e-10, atol=1e-10)


def test_generator_quantization_error_is_within_half_a_step():
    rng = np.random.default_rng(5)
    _, W = wl.bf16_round((rng.standard_normal((384, 48)) / np.sqrt(384)).astype(np.float32))
    qb, sb = wl.quantize_int4_g128(W)
    Wd = quant.dequantize(qb, sb, 384)
    step = np.repeat(quant.bf16_bits_value(sb), 128, axis=1).T        # [K, N]
    # scale ~ max|W| / 7 rounded to bf16, so |W| / scale stays below 7.03 and
    # rounding to the nearest step is never clipped
    assert np.all(np.abs(W - Wd) <= step / 2 + 1e-12)
    assert np.abs(W).max() > 0 and np.std(Wd) > 0.5 * np.std(W)


@pytest.mark.parametrize("kind", ["swap_nibbles", "transpose_groups", "off_by_one_group"])
def test_planted_mistakes_fail_the_single_nibble_pin(kind):
    N, K = 4, 256
    qb = np.full((N, K // 2), 0x88, dtype=np.uint8)
    qb[1, 64] = 0x8D                                          # k = 128 (even) -> q = 5
    sb = np.zeros((N, K // 128), dtype=np.uint16)
    sb[:, 0], sb[:, 1] = 0x3F80, 0x4040
    want = np.zeros((K, N))
    want[128, 1] = 15.0
    if kind == "swap_nibbles":
        q = quant.unpack_int4(qb, K)
        q[:, 0::2], q[:, 1::2] = q[:, 1::2].copy(), q[:, 0::2].copy()
        W = (q * np.repeat(quant.bf16_bits_value(sb), 128, axis=1)).T
    elif kind == "transpose_groups":
        q = quant.unpack_int4(qb, K)
        W = (q * np.tile(quant.bf16_bits_value(sb), (1, 128))).T
    else:
        q = quant.unpack_int4(qb, K)
        s = np.repeat(quant.bf16_bits_value(sb), 128, axis=1)
        W = (q * np.roll(s, 1, axis=1)).T
    assert not np.array_equal(W, want)
