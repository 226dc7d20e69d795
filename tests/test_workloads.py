"""Input generator checks (CPU only): bfloat16 rounding, determinism, Zipf
law, and the workload shapes."""
import numpy as np
import pytest

import workloads as wl


def _nearest_even_bf16(x: float) -> int:
    # reference by enumeration: the two bf16 neighbours of x and an exact tie rule
    u = int(np.array([x], np.float32).view(np.uint32)[0])
    lo = u >> 16
    cands = [lo, lo + 1]
    vals = [float(wl.bf16_bits_to_float(np.array([c], np.uint16))[0]) for c in cands]
    d = [abs(v - float(np.float32(x))) for v in vals]
    if d[0] < d[1]:
        return cands[0]
    if d[1] < d[0]:
        return cands[1]
    return cands[0] if cands[0] % 2 == 0 else cands[1]


def test_bf16_halfway_cases():
    one = 1.0
    cases = {
        one + 2.0 ** -8: 0x3F80,                  # tie -> even (down)
        one + 3 * 2.0 ** -8: 0x3F82,              # tie -> even (up)
        one + 2.0 ** -8 + 2.0 ** -20: 0x3F81,     # just above the tie -> up
        -(one + 2.0 ** -8): 0xBF80,
        0.0: 0x0000,
    }
    for x, bits in cases.items():
        b, v = wl.bf16_round(np.array([x], np.float32))
        assert int(b[0]) == bits, (x, hex(int(b[0])))


def test_bf16_random_against_enumeration():
    rng = np.random.default_rng(0)
    x = (rng.standard_normal(2000) * 10.0 ** rng.integers(-5, 5, 2000)).astype(np.float32)
    b, v = wl.bf16_round(x)
    for xi, bi in zip(x, b):
        assert int(bi) == _nearest_even_bf16(float(xi))
    assert v.dtype == np.float32
    np.testing.assert_array_equal(wl.bf16_round(v)[0], b)        # idempotent


def test_zipf_law():
    p = wl.finite_zipf_probs(32, 1.0)
    assert abs(p.sum() - 1) < 1e-12
    np.testing.assert_allclose(p[0] / p, np.arange(1, 33), rtol=1e-12)
    ids = wl.draw_ids(wl.workload(1))
    assert ids.min() >= 0 and ids.max() < 32
    big = wl.WorkloadSpec("z", None, 8, [], T=200000, n_slots=32, ranks=[1] * 32,
                          scales=[1.0] * 32, ids_kind="zipf", seed=5)
    freq = np.bincount(wl.draw_ids(big), minlength=32) / 200000
    assert np.max(np.abs(freq - p)) < 0.005


def test_determinism():
    spec = wl.workload(0)
    a, b = wl.draw_layer(spec), wl.draw_layer(spec)
    np.testing.assert_array_equal(a.ids, b.ids)
    np.testing.assert_array_equal(a.projs[0].X_bits, b.projs[0].X_bits)
    np.testing.assert_array_equal(a.adapters[a.ids[0]].A_bits[0][0], b.adapters[a.ids[0]].A_bits[0][0])


def test_workload_shapes():
    p8 = wl.model_projs("llama-3.1-8b", 8)
    assert [(p.name, p.kind, p.d_in, p.slices) for p in p8] == [
        ("qkv", "column", 4096, (512, 128, 128)), ("o", "row", 512, (4096,)),
        ("gate", "column", 4096, (1792,)), ("up", "column", 4096, (1792,)),
        ("down", "row", 1792, (4096,))]
    p70 = wl.model_projs("llama-3.1-70b", 8)
    assert [(p.d_in, p.slices) for p in p70] == [
        (8192, (1024, 128, 128)), (1024, (8192,)), (8192, (3584,)), (8192, (3584,)), (3584, (8192,))]
    s4 = wl.workload(4)
    ids = wl.draw_ids(s4)
    assert ids.size == 4288
    assert len(set(ids[:1024])) == 1 and len(set(int(v) for v in ids) ) <= 64
    assert set(s4.ranks) <= {8, 16, 32, 64}
    s2 = wl.workload(2)
    ids2 = wl.draw_ids(s2)
    assert np.all(np.diff(ids2) >= 0) and np.bincount(ids2).tolist() == [512] * 8


def test_value_distribution():
    lay = wl.draw_layer(wl.workload(0))
    X, W = lay.projs[0].X, lay.projs[0].W
    assert abs(X.std() - 1.0) < 0.05
    assert abs(W.std() * np.sqrt(4096) - 1.0) < 0.05
    a = next(iter(lay.adapters.values()))
    assert abs(a.B[0][0].std() * np.sqrt(8) - 1.0) < 0.1
