"""The bf16 GEMM comparator (libfqgemm.so, include/fq_gemm_ref.h) on the GPU:
every candidate hipBLASLt offers computes X * W for both weight layouts,
within bf16 rounding of Y plus fp32 accumulation error of an fp64 product of
the same bf16 operands; a HIP graph of it replays to the same result."""

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

WS_BYTES = 64 << 20


def _bf16(shape, seed):
    g = torch.Generator().manual_seed(seed)
    return torch.randn(*shape, generator=g).to(torch.bfloat16)


def _within(y, x, w_kn):
    """y (bf16, device) against the fp64 product of x [M][K] and w_kn [K][N]."""
    xd = x.double().numpy()
    wd = w_kn.double().numpy()
    ref = xd @ wd
    mag = np.abs(xd) @ np.abs(wd)
    yv = y.double().cpu().numpy()
    err = np.abs(yv - ref) - (2.0 ** -8 * np.abs(ref) + 2.0 ** -14 * mag)
    return int((~np.isfinite(yv) | (err > 0)).sum())   # a NaN left in Y counts


@pytest.mark.parametrize("M,K,N", [(1, 512, 384), (4, 1024, 256), (16, 4096, 640),
                                   (5, 1000, 296)])
@pytest.mark.parametrize("layout", ["kn", "nk"])
def test_every_heuristic_candidate(gpu_lib, M, K, N, layout):
    from paper_2608_15531_amd import gemm_ref
    x = _bf16((M, K), 1)
    w_kn = _bf16((K, N), 2)
    w = w_kn if layout == "kn" else w_kn.t().contiguous()
    xd, wd = x.cuda(), w.cuda()
    ws = torch.empty(WS_BYTES, dtype=torch.uint8, device="cuda")
    n = gemm_ref.prepare(M, K, N, layout, gemm_ref.HEURISTIC, 8, WS_BYTES)
    assert 1 <= n <= 8
    for i in range(n):
        need, name = gemm_ref.candidate(M, K, N, layout, i)
        assert need <= WS_BYTES and name
        y = torch.full((M, N), float("nan"), dtype=torch.bfloat16, device="cuda")
        gemm_ref.gemm(xd, wd, y, layout, i, ws)
        torch.cuda.synchronize()
        assert _within(y, x, w_kn) == 0, f"candidate {i} ({name})"


def test_exhaustive_candidates(gpu_lib):
    from paper_2608_15531_amd import gemm_ref
    M, K, N = 4, 1024, 256
    x = _bf16((M, K), 3)
    w = _bf16((K, N), 4)
    xd, wd = x.cuda(), w.cuda()
    ws = torch.empty(WS_BYTES, dtype=torch.uint8, device="cuda")
    n = gemm_ref.prepare(M, K, N, "kn", gemm_ref.EXHAUSTIVE, 8, WS_BYTES)
    assert 1 <= n <= 8
    for i in range(n):
        y = torch.full((M, N), float("nan"), dtype=torch.bfloat16, device="cuda")
        gemm_ref.gemm(xd, wd, y, "kn", i, ws)
        torch.cuda.synchronize()
        assert _within(y, x, w) == 0, f"candidate {i} ({gemm_ref.candidate(M, K, N, 'kn', i)[1]})"


def test_unprepared_and_bad_candidate(gpu_lib):
    from paper_2608_15531_amd import gemm_ref
    lib = gemm_ref.load()
    x = torch.zeros(2, 64, dtype=torch.bfloat16, device="cuda")
    w = torch.zeros(64, 72, dtype=torch.bfloat16, device="cuda")
    y = torch.zeros(2, 72, dtype=torch.bfloat16, device="cuda")
    # never prepared: refused with 2 before hipBLASLt is called
    assert lib.fq_ref_gemm_bf16(x.data_ptr(), w.data_ptr(), y.data_ptr(), 2, 64, 72, 0, 0,
                                None, 0, None) == 2
    n = gemm_ref.prepare(2, 64, 72, "kn")
    assert lib.fq_ref_gemm_bf16(x.data_ptr(), w.data_ptr(), y.data_ptr(), 2, 64, 72, 0, n,
                                None, 0, None) == 2
    assert lib.fq_ref_gemm_bf16_candidate(2, 64, 72, 0, -1, None, None, 0) == 2


def test_graph_replays_match(gpu_lib):
    """A HIP graph of comparator calls, replayed several times with eager
    calls and synchronisations between, gives a correct Y every time."""
    from paper_2608_15531_amd import gemm_ref
    M, K, N = 8, 4096, 1024
    x = _bf16((M, K), 5)
    w = _bf16((K, N), 6)
    x2 = _bf16((M, K), 7)
    xd, wd, x2d = x.cuda(), w.cuda(), x2.cuda()
    ws = torch.empty(WS_BYTES, dtype=torch.uint8, device="cuda")
    gemm_ref.prepare(M, K, N, "kn")
    y = torch.empty(M, N, dtype=torch.bfloat16, device="cuda")
    y2 = torch.empty(M, N, dtype=torch.bfloat16, device="cuda")
    st = torch.cuda.Stream()
    st.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(st):
        gemm_ref.gemm(xd, wd, y, "kn", 0, ws)
    torch.cuda.current_stream().wait_stream(st)
    torch.cuda.synchronize()
    assert _within(y, x, w) == 0
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        gemm_ref.gemm(xd, wd, y, "kn", 0, ws)
    torch.cuda.synchronize()
    for rep in range(3):
        y.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        assert _within(y, x, w) == 0, f"replay {rep}"
        gemm_ref.gemm(x2d, wd, y2, "kn", 0, ws)   # eager work between replays
        torch.cuda.synchronize()
        assert _within(y2, x2, w) == 0
