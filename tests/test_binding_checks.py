"""The Python binding validates every tensor before its address reaches the C
ABI (which takes bare pointers): wrong dtype, shape, layout or device raises
ValueError on the host, before any library call.  CPU only."""
import numpy as np
import pytest
import torch

from paper_2607_12505_amd import nmspmm


def _weight(n=64, k=256):
    W = np.zeros((n, k), np.int8)
    W[:, ::4] = 3
    return nmspmm.DeviceWeight.from_packed(nmspmm.compress(W, 2, 4), device="cpu")


def test_spmm_rejects_mismatched_tensors():
    w = _weight()
    X = torch.zeros((32, 256), dtype=torch.int8)
    Y = torch.zeros((32, 64), dtype=torch.int32)
    with pytest.raises(ValueError, match="X: shape"):
        nmspmm.spmm(torch.zeros((32, 128), dtype=torch.int8), w, Y=Y)       # k of X differs from the weight's
    with pytest.raises(ValueError, match="X: dtype"):
        nmspmm.spmm(X.to(torch.int32), w, Y=Y)
    with pytest.raises(ValueError, match="X: 1-D"):
        nmspmm.spmm(X.reshape(-1), w, Y=Y)
    with pytest.raises(ValueError, match="Y: shape"):
        nmspmm.spmm(X, w, Y=torch.zeros((32, 63), dtype=torch.int32))
    with pytest.raises(ValueError, match="Y: dtype"):
        nmspmm.spmm(X, w, Y=torch.zeros((32, 64), dtype=torch.int64))
    with pytest.raises(ValueError, match="Yh: dtype"):
        nmspmm.spmm(X, w, Yh=torch.zeros((32, 64), dtype=torch.float32), scale=torch.ones(64))
    with pytest.raises(ValueError, match="scale: shape"):
        nmspmm.spmm(X, w, Yh=torch.zeros((32, 64), dtype=torch.float16), scale=torch.ones(32))
    with pytest.raises(ValueError, match="Yq: shape"):
        nmspmm.spmm(X, w, Yq=torch.zeros((31, 64), dtype=torch.int8), qscale=torch.ones(64))
    with pytest.raises(ValueError, match="contiguous"):
        nmspmm.spmm(torch.zeros((256, 32), dtype=torch.int8).t(), w, Y=Y)
    short = nmspmm.DeviceWeight(w.vals[:-1], w.meta, w.desc)
    with pytest.raises(ValueError, match="w.vals"):
        nmspmm.spmm(X, short, Y=Y)
    # right types and shapes, but host tensors: refused before the library is called
    with pytest.raises(ValueError, match="device tensor"):
        nmspmm.spmm(X, w, Y=Y)


def test_dense_and_quantiser_reject_mismatched_tensors():
    X = torch.zeros((32, 256), dtype=torch.int8)
    Y = torch.zeros((32, 64), dtype=torch.int32)
    with pytest.raises(ValueError, match="W: shape"):
        nmspmm.gemm_i8_dense(X, torch.zeros((64, 128), dtype=torch.int8), Y=Y)
    with pytest.raises(ValueError, match="Y: shape"):
        nmspmm.gemm_i8_dense(X, torch.zeros((64, 256), dtype=torch.int8), Y=torch.zeros((64, 32), dtype=torch.int32))
    with pytest.raises(ValueError, match="device tensor"):
        nmspmm.gemm_i8_dense(X, torch.zeros((64, 256), dtype=torch.int8), Y=Y)
    with pytest.raises(ValueError, match="x: dtype"):
        nmspmm.quantize_f16(torch.zeros(16, dtype=torch.float32), 1.0)
    with pytest.raises(ValueError, match="xq: shape"):
        nmspmm.quantize_f16(torch.zeros(16, dtype=torch.float16), 1.0, xq=torch.zeros(8, dtype=torch.int8))
    with pytest.raises(ValueError, match="device tensor"):
        nmspmm.quantize_f16(torch.zeros(16, dtype=torch.float16), 1.0)
