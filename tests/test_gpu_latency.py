"""The latency table and chain timing of the layer-wise search (Sec. 5.1) on
the GPU, at a small ViT-like shape: every (shape, pattern) gets a positive
latency in both timing modes, chains are timed, and Eq. 1 calibrated on them
predicts held-out chains.  (The predictor arithmetic itself is checked against
the oracle on the CPU.)"""
import numpy as np
import pytest

from paper_2607_12505_amd import latency as lt
from paper_2607_12505_amd import nmsearch, nmspmm
import gpu_util as gu

pytestmark = pytest.mark.gpu


def test_lut_chain_and_calibration():
    torch = gu.torch()
    assert torch.cuda.is_available()
    m, C, H = 1024, 256, 1024
    shapes = [(m, C, 3 * C), (m, C, C), (m, C, H), (m, H, C)] * 2
    pats = [(1, 8), (2, 8), (4, 8), (8, 8)]
    cb = lt.ChainBench(torch, shapes, pats, nmspmm.NM_OUT_I32, seed=1)
    print("chain bench prepared", flush=True)
    cold, secs = cb.lut(reps=3, cold=True)
    hot, _ = cb.lut(reps=3, cold=False)
    assert set(cold) == set(hot) == {(s, p) for s in set(shapes) for p in pats}
    assert all(v > 0 and np.isfinite(v) for v in list(cold.values()) + list(hot.values()))
    configs = lt.random_assignments(12, len(shapes), pats, seed=3)
    T = np.array([cb.measure(a, reps=2) for a in configs])
    assert (T > 0).all()
    R = np.array([cb.layer_times(hot, a) for a in configs])
    gamma, b = nmsearch.latency_fit(R[:8], T[:8])
    assert (gamma >= 0).all() and b >= 0
    pred = np.array([nmsearch.latency_predict(r, gamma, b) for r in R[8:]])
    err = np.abs(pred - T[8:]) / T[8:]
    print("held-out chain times (us):", np.round(T[8:], 2).tolist(), "relative errors:", np.round(err, 4).tolist(),
          flush=True)
    # Eq. 1 fitted on 8 chains predicts the held-out ones within 10 % (2-4 % observed)
    assert np.all(err < 0.10)
