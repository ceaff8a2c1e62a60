"""The GEMM entry points under HIP graph capture: a DeiT-Base layer's four
linears at batch 1 (one sparse pattern each, plus the dense baseline and a
split-K plan with its workspace cleared by the library's fill kernel, and a
compact weight expanded once per call into its workspace) are captured once and replayed several times, with eager work and
synchronisations between replays; every replay must reproduce the eager
outputs bit for bit, and the eager outputs match the oracle."""
import numpy as np
import pytest

import oracle
from paper_2607_12505_amd import nmspmm
from paper_2607_12505_amd import workloads as wl

pytestmark = pytest.mark.gpu


def test_captured_layer_replays_bit_exactly():
    import torch
    torch.cuda.set_device(0)
    rng = np.random.default_rng(21)
    m = 197
    shapes = [(768, 2304, 2, 4), (768, 768, 1, 4), (768, 3072, 2, 8), (3072, 768, 1, 8)]   # (k, n, N, M)
    calls, outs, refs = [], [], []
    for k, n, N, M in shapes:
        X = rng.integers(-127, 128, (m, k), dtype=np.int8)
        W = wl.random_nm(n, k, N, M, rng, full=True)
        Xd = torch.from_numpy(X).cuda()
        dw = nmspmm.DeviceWeight.from_packed(nmspmm.compress(W, N, M))
        Y = torch.empty((m, n), dtype=torch.int32, device="cuda")
        calls.append(lambda Xd=Xd, dw=dw, Y=Y: nmspmm.spmm(Xd, dw, Y=Y))
        outs.append(Y)
        refs.append(oracle.matmul_i8(X, W))
    # the dense baseline of the first shape
    k, n = shapes[0][0], shapes[0][1]
    X = rng.integers(-127, 128, (m, k), dtype=np.int8)
    W = wl.random_nm(n, k, 8, 8, rng, full=True)
    Xd, Wd = torch.from_numpy(X).cuda(), torch.from_numpy(W).cuda()
    Yd = torch.empty((m, n), dtype=torch.int32, device="cuda")
    calls.append(lambda: nmspmm.gemm_i8_dense(Xd, Wd, Y=Yd))
    outs.append(Yd)
    refs.append(oracle.matmul_i8(X, W))
    # a split-K plan: its workspace counters are cleared inside the graph by a kernel
    k, n = 3072, 768
    Xs = rng.integers(-127, 128, (m, k), dtype=np.int8)
    Ws = wl.random_nm(n, k, 2, 4, rng, full=True)
    Xsd = torch.from_numpy(Xs).cuda()
    dws = nmspmm.DeviceWeight.from_packed(nmspmm.compress(Ws, 2, 4))
    plan = nmspmm.make_plan(nmspmm.NM_KIND_SP42, 3, 4)
    ws = torch.empty(nmspmm.workspace_size(plan, m, n), dtype=torch.uint8, device="cuda")
    Ys = torch.empty((m, n), dtype=torch.int32, device="cuda")

    def split_call():
        nmspmm.workspace_init(ws)
        nmspmm.spmm(Xsd, dws, Y=Ys, ws=ws, plan=plan)
    calls.append(split_call)
    outs.append(Ys)
    refs.append(oracle.matmul_i8(Xs, Ws))

    # a compact weight expanded once per call into the workspace (the
    # expansion kernel and the 4:2-operand kernel are both captured)
    k, n = 1024, 768
    Xe = rng.integers(-127, 128, (m, k), dtype=np.int8)
    We = wl.random_nm(n, k, 2, 8, rng, full=True)
    Xed = torch.from_numpy(Xe).cuda()
    dwe = nmspmm.DeviceWeight.from_packed(nmspmm.compress(We, 2, 8))
    plan_e = nmspmm.spmm_plan_complete(dwe.desc, m, nmspmm.make_plan(dwe.desc.kind, 0, 1, expand=1))
    ws_e = torch.empty(nmspmm.workspace_size(plan_e, m, n), dtype=torch.uint8, device="cuda")
    nmspmm.workspace_init(ws_e)
    Ye = torch.empty((m, n), dtype=torch.int32, device="cuda")
    calls.append(lambda: nmspmm.spmm(Xed, dwe, Y=Ye, ws=ws_e, plan=plan_e))
    outs.append(Ye)
    refs.append(oracle.matmul_i8(Xe, We))

    for c in calls:                      # eager run
        c()
    torch.cuda.synchronize()
    eager = [o.clone() for o in outs]
    for e, r in zip(eager, refs):
        assert np.array_equal(e.cpu().numpy(), r)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):        # warm-up on the capture stream
        for c in calls:
            c()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for c in calls:
            c()
    for rep in range(4):
        for o in outs:                   # eager work between replays
            o.fill_(-1)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for o, e in zip(outs, eager):
            assert torch.equal(o, e), f"replay {rep} differs"
