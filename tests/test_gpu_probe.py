"""GPU test of the matrix-instruction rate loop (nmprobe.h): it runs through
the C ABI for both instruction kinds, is deterministic, and bench.py turns its
timing into a positive rate."""
import pytest

from paper_2607_12505_amd import nmprobe, nmspmm

pytestmark = pytest.mark.gpu


def test_rate_loop_runs_and_is_deterministic():
    import torch
    g = torch.Generator().manual_seed(5)
    tab = torch.randint(-2 ** 31, 2 ** 31, (nmprobe.NM_PROBE_WORDS,), generator=g, dtype=torch.int64)
    tab = tab.to(torch.int32).cuda()
    for kind in (nmspmm.NM_KIND_SP42, nmspmm.NM_KIND_DENSE):
        out1 = torch.empty(8 * 256, dtype=torch.int32, device="cuda")
        out2 = torch.empty_like(out1)
        nmprobe.probe_mfma_rate(kind, tab, 3, out1)
        nmprobe.probe_mfma_rate(kind, tab, 3, out2)
        torch.cuda.synchronize()
        assert torch.equal(out1, out2)
        # every workgroup runs the same loop on the same table
        assert torch.equal(out1[:256], out1[256:512])
    zero = torch.zeros_like(tab)
    out = torch.empty(256, dtype=torch.int32, device="cuda")
    nmprobe.probe_mfma_rate(nmspmm.NM_KIND_SP42, zero, 2, out)
    torch.cuda.synchronize()
    assert int(out.abs().sum()) == 0


def test_loop_ticks_give_a_plausible_clock():
    import torch
    khz = nmprobe.wall_clock_khz()
    assert khz > 0
    tab = torch.zeros(nmprobe.NM_PROBE_WORDS, dtype=torch.int32, device="cuda")
    out = torch.empty(4 * 256, dtype=torch.int32, device="cuda")
    ticks = torch.zeros(8, dtype=torch.int64, device="cuda")
    nmprobe.probe_mfma_rate(nmspmm.NM_KIND_DENSE, tab, 2000, out, ticks)
    torch.cuda.synchronize()
    t = ticks.cpu().numpy().reshape(-1, 2)
    assert (t > 0).all()
    mhz = t[:, 0] / (t[:, 1] / (khz * 1e3)) / 1e6
    assert ((mhz > 50) & (mhz < 5000)).all()


def test_bench_reports_positive_rates():
    import torch
    import bench
    res = bench.mfma_ceiling(torch, iters=64, reps=1)
    for key in ("smfmac_i32_16x16x128_i8_random", "mfma_i32_16x16x64_i8_random",
                "smfmac_i32_16x16x128_i8_zero", "mfma_i32_16x16x64_i8_zero"):
        assert res[key + "_pops"] > 0 and res[key + "_clock_mhz"] > 0


@pytest.mark.parametrize("m,n", [(1000, 260), (12608, 1152), (33, 4)])
def test_store_only_probe_writes_zeros_exactly_in_the_outputs(m, n):
    # every output-split tile of every kind, on ragged shapes, with and
    # without the multiplier arrays: the probe writes the empty-sum values into
    # [m x n] and nothing past it
    import torch
    bigY = torch.full((m * n + 4096,), 7, dtype=torch.int32, device="cuda")
    bigH = torch.full((m * n + 4096,), 7, dtype=torch.int16, device="cuda")
    bigQ = torch.full((m * n + 4096,), 7, dtype=torch.int8, device="cuda")
    scale = torch.full((n,), 0.5, dtype=torch.float32, device="cuda")
    Y, Yh, Yq = bigY[:m * n].view(m, n), bigH[:m * n].view(m, n), bigQ[:m * n].view(m, n)
    for kind in nmspmm.ALL_KINDS:
        for tile in range(nmspmm.num_tiles()):
            for with_scales in (True, False):
                plan = nmspmm.make_plan(kind, tile, 1)
                outs = dict(Y=Y, scale=scale, Yh=Yh, Yq=Yq, qscale=scale) if with_scales else dict(Y=Y)
                try:
                    nmprobe.probe_store_only(plan, m, n, **outs)
                except nmspmm.NmError as e:
                    assert e.status == nmspmm.NM_ERR_ARG     # not an output-split layout
                    break
                torch.cuda.synchronize()
                assert not Y.any(), (kind, tile)
                if with_scales:
                    assert not Yh.any() and not Yq.any(), (kind, tile)
                assert (bigY[m * n:] == 7).all() and (bigH[m * n:] == 7).all() and (bigQ[m * n:] == 7).all()
                Y.fill_(7)
                Yh.fill_(7)
                Yq.fill_(7)


def test_fence_free_events_time_a_device_sleep_like_torch_events():
    # The timing events of the bench (no system-scope fence) bracket the same
    # work as PyTorch's default events: a device sleep of about 2 ms between
    # them reads the same elapsed time within 5 %, and the interval of two
    # events recorded back to back is short.
    import torch
    from paper_2607_12505_amd import nmprobe
    a, b, c = nmprobe.TimingEvent(), nmprobe.TimingEvent(), nmprobe.TimingEvent()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record()
    a.record()
    torch.cuda._sleep(int(2.0e9 * 2e-3))
    b.record()
    t1.record()
    c.record()
    torch.cuda.synchronize()
    mine, ref = a.elapsed_time(b), t0.elapsed_time(t1)
    assert mine > 0.5 and ref > 0.5
    assert abs(mine - ref) <= 0.05 * ref
    assert 0 <= b.elapsed_time(c) < 0.2
