"""Packed-weight files and the latency table on disk (CPU only): round trips,
and every corruption the loaders promise to reject."""
import json

import numpy as np
import pytest

from paper_2607_12505_amd import latency, nmspmm
from paper_2607_12505_amd import workloads as wl


@pytest.mark.parametrize("N,M", [(2, 4), (1, 8), (5, 8)])
def test_packed_file_round_trip(tmp_path, N, M):
    rng = np.random.default_rng(3)
    W = wl.random_nm(64, 256, N, M, rng, full=True)
    p = nmspmm.compress(W, N, M)
    f = tmp_path / "w.nmw"
    nmspmm.save_packed(str(f), p)
    q = nmspmm.load_packed(str(f))
    assert np.array_equal(q.vals, p.vals) and np.array_equal(q.meta, p.meta)
    assert (q.desc.n, q.desc.k, q.desc.nm_n, q.desc.nm_m, q.desc.kind) == (64, 256, N, M, p.desc.kind)
    # and it still decodes to W
    assert np.array_equal(nmspmm.decompress(q), W)


def test_packed_file_rejects_corruption(tmp_path):
    rng = np.random.default_rng(4)
    p = nmspmm.compress(wl.random_nm(32, 128, 2, 4, rng, full=True), 2, 4)
    f = tmp_path / "w.nmw"
    nmspmm.save_packed(str(f), p)
    good = f.read_bytes()

    def bad(data):
        f.write_bytes(data)
        with pytest.raises(ValueError):
            nmspmm.load_packed(str(f))

    bad(good[:20])                                        # truncated header
    bad(b"X" + good[1:])                                  # magic
    bad(good[:-1])                                        # truncated payload
    flipped = bytearray(good)
    flipped[-1] ^= 1                                      # a position byte
    bad(bytes(flipped))
    flipped = bytearray(good)
    flipped[nmspmm._PACKED_HEAD.size] ^= 1                # a value byte
    bad(bytes(flipped))
    flipped = bytearray(good)
    flipped[16 + 4 * 4] ^= 1                              # the descriptor's stream count
    bad(bytes(flipped))


def test_lut_round_trip_and_checks(tmp_path):
    table = {((18464, 1024, 3072), (2, 8)): 65.8, ((18464, 1024, 3072), (8, 8)): 86.0,
             ((18464, 4096, 1024), (1, 4)): 60.1}
    f = tmp_path / "lut.json"
    latency.save_lut(str(f), table, gamma=[1.0, 0.9, 1.1], b=3.5, info={"box": "test"})
    t2, g, b, info = latency.load_lut(str(f))
    assert t2 == table and g == [1.0, 0.9, 1.1] and b == 3.5 and info == {"box": "test"}
    latency.save_lut(str(f), table)
    assert latency.load_lut(str(f))[1:3] == (None, None)
    doc = json.loads(f.read_text())
    doc["entries"].append(dict(doc["entries"][0]))
    f.write_text(json.dumps(doc))
    with pytest.raises(ValueError):
        latency.load_lut(str(f))
    doc["entries"].pop()
    doc["entries"][0]["us"] = -1.0
    f.write_text(json.dumps(doc))
    with pytest.raises(ValueError):
        latency.load_lut(str(f))
    doc["format"] = "other"
    f.write_text(json.dumps(doc))
    with pytest.raises(ValueError):
        latency.load_lut(str(f))
