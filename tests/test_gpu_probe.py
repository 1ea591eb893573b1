"""The measurement aids on the GPU: the probes of libfqprobe.so run (the
XCD-placement probe reports valid XCD numbers), and the instrumented build
libfq_stamps.so records ordered per-wave timestamps while computing what
libfq.so computes."""

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


def test_stream_read_runs(gpu_lib):
    from paper_2608_15531_amd import probe
    buf = torch.ones(1 << 20, dtype=torch.int32, device="cuda")
    sink = torch.zeros(512, dtype=torch.int32, device="cuda")
    probe.fq_probe_stream_read(buf, buf.numel() * 4, 512, 4, 4, sink)
    torch.cuda.synchronize()


@pytest.mark.parametrize("workgroups,threads", [(8, 64), (512, 256), (4096, 1024)])
def test_workgroup_xcd_in_range(gpu_lib, workgroups, threads):
    """Every workgroup writes its XCD number, one of the eight of MI355X."""
    from paper_2608_15531_amd import probe
    out = torch.full((workgroups,), -1, dtype=torch.int32, device="cuda")
    probe.fq_probe_workgroup_xcd(out, workgroups, threads)
    torch.cuda.synchronize()
    ids = out.cpu()
    assert int(ids.min()) >= 0 and int(ids.max()) < 8


@pytest.mark.parametrize("extra", [0, 3, 4, 8, 12, 15, 20, 24])
def test_tile_loads_runs(gpu_lib, extra):
    from paper_2608_15531_amd import probe
    K, N, gpt = 1024, 512, 21
    T = K // 128
    dev = "cuda"
    codes = torch.ones(K * N // 8, dtype=torch.int32, device=dev)
    scales = torch.ones(T * N, dtype=torch.int16, device=dev)
    zeros = torch.ones(T * N // 8, dtype=torch.int32, device=dev)
    x = torch.ones(K, dtype=torch.int16, device=dev)
    groups = torch.ones(T * (N // 64) * gpt * 4, dtype=torch.int32, device=dev)
    sink = torch.zeros(N // 64, dtype=torch.int32, device=dev)
    probe.fq_probe_tile_loads(codes, scales, zeros, x, groups, K, N, gpt, extra, sink)
    torch.cuda.synchronize()


@pytest.mark.parametrize("cols,waves,split", [(16, 8, 1), (16, 4, 2), (32, 8, 1), (32, 4, 2),
                                              (64, 4, 2), (64, 8, 1)])
def test_strip_loads_runs(gpu_lib, cols, waves, split):
    from paper_2608_15531_amd import probe
    K, N, gpt = 1024, 512, 21
    T = K // 128
    dev = "cuda"
    codes = torch.ones(K * N // 8, dtype=torch.int32, device=dev)
    x = torch.ones(K, dtype=torch.int16, device=dev)
    groups = torch.ones(T * (N // 64) * gpt * 4, dtype=torch.int32, device=dev)
    sink = torch.zeros(N // cols * split, dtype=torch.int32, device=dev)
    probe.fq_probe_strip_loads(codes, x, groups, K, N, cols, waves, split, gpt, sink)
    torch.cuda.synchronize()


def test_instrumented_build_stamps_and_results(gpu_lib):
    """The same fused launch through libfq.so and through libfq_stamps.so: the
    results agree to the f32 tolerance, and every wave's four stamps are in
    order (start <= first data <= loop end <= exit)."""
    from synth import make_problem
    import paper_2608_15531_amd as fq
    M, K, N = 4, 4096, 4096
    prob = make_problem(M, K, N, frac=0.01, seed=5)
    X, Wq, s, z = fq.to_device(prob)
    tc = fq.TileCOODevice(fq.fq_pack_tile_coo(K, N, prob.k, prob.n, prob.v))
    ref = fq.fq_w4a16_outlier_matmul(X, Wq, s, z, tc, y_dtype="f32")
    torch.cuda.synchronize()
    saved = fq._lib
    try:
        fq.use_instrumented_build()
        y = fq.fq_w4a16_outlier_matmul(X, Wq, s, z, tc, y_dtype="f32")
        torch.cuda.synchronize()
        c = fq.fq_launch_config(M, K, N)
        nw = c["workgroups"] * (c["dense_waves"] + c["outlier_waves"])
        st = fq.fq_debug_wave_stamps(nw).astype(np.int64)
    finally:
        fq._lib = saved
    a, b = y.cpu().numpy().astype(np.float64), ref.cpu().numpy().astype(np.float64)
    assert np.linalg.norm(a - b) / np.linalg.norm(b) <= 1e-6
    assert (st[:, 0] > 0).all()
    assert (st[:, 1] >= st[:, 0]).all() and (st[:, 2] >= st[:, 1]).all()
    assert (st[:, 3] >= st[:, 2]).all()
    span_us = (st[:, 3].max() - st[:, 0].min()) / 100.0
    assert 0.5 < span_us < 1000.0
