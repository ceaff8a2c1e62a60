"""The seeded input generators: determinism, ranges and the N:M rule (CPU only)."""
import numpy as np

from paper_2607_12505_amd import workloads as wl


def test_same_seed_same_bytes():
    g = wl.workload(2).gemms[5]
    a = wl.inputs_for(2, g)
    b = wl.inputs_for(2, g)
    for x, y in zip(a, b):
        assert x.tobytes() == y.tobytes()


def test_value_ranges_and_pattern():
    rng = wl.rng_for(0, 0, 0, 0, wl.ROLE_X)
    X = wl.gen_x(300, 64, rng)
    assert X.min() >= -127 and X.max() <= 127 and X.min() < -120 and X.max() > 120
    for (N, M) in ((1, 4), (2, 4), (1, 8), (2, 8), (4, 8), (8, 8)):
        W, sc = wl.gen_w(64, 128, N, M, wl.rng_for(0, 0, 0, 1, wl.ROLE_W))
        cnt = (W.reshape(64, 128 // M, M) != 0).sum(axis=2)
        assert cnt.max() <= N
        assert np.abs(W).max(axis=1).min() == 127       # the row maximum maps to 127
        assert W.min() >= -127
        assert sc.dtype == np.float32 and (sc > 0).all()


def test_topn_keeps_largest_magnitudes():
    rng = np.random.default_rng(0)
    W, _ = wl.gen_w(8, 16, 2, 4, wl.rng_for(9, 9, 9, 9, 1))
    # recompute the float draw and check that the kept positions are the top-2 per window
    w = wl.rng_for(9, 9, 9, 9, 1).normal(0.0, 0.02, size=(8, 16)).reshape(8, 4, 4)
    kept = W.reshape(8, 4, 4) != 0
    for j in range(8):
        for g in range(4):
            top = set(np.argsort(-np.abs(w[j, g]), kind="stable")[:2])
            assert set(np.flatnonzero(kept[j, g])) <= top


def test_workload_shapes():
    w1 = wl.workload(1)
    assert len(w1.gemms) == 16 and all(g.m == 12608 for g in w1.gemms)
    w2 = wl.workload(2)
    assert {g.m for g in w2.gemms} == {197, 1576, 25216} and len(w2.gemms) == 48
    w3 = wl.workload(3)
    assert len(w3.gemms) == 32
    w4 = wl.workload(4)
    assert len(w4.gemms) == 96 and all(g.m == 18464 for g in w4.gemms)
    assert {(g.N, g.M) for g in w4.gemms} <= set(wl.VIT_L_CHOICES)
