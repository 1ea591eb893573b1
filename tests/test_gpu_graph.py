"""The fused, unfused and dense-only matmuls captured in a HIP graph.

A graph replays the launches recorded once, with the same kernel arguments:
the split-K and Stream-K counters in the workspace must be back at zero after
every launch, and nothing a launch needs may be recorded as a memset.  Each
graph is replayed several times with the program's own eager work (the same
matmul into another output, sharing the workspace, and a fill of the graph's
output) between the replays; every replay must reproduce the eager result bit
for bit, and on exact-arithmetic inputs both equal the fp64 oracle exactly.
"""

import numpy as np
import pytest
import torch

import oracle
from synth import make_exact_problem

pytestmark = pytest.mark.gpu

REPLAYS = 4
WS_BYTES = 64 << 20

# (M, K, N, split_k, flags by name, sparse mapping)
CASES = [
    (1, 2048, 512, 0, (), "auto"),              # LDS-gather outlier mapping
    (4, 2048, 512, 4, (), "mfma"),              # split-K, one staged X load
    (16, 4096, 1024, 0, (), "auto"),            # four staged X loads
    (8, 14336, 256, 0, (), "auto"),             # long K: the planner splits
    (16, 2048, 512, 0, ("FQ_SCHED_STREAM_K",), "auto"),
    (33, 1024, 256, 2, (), "auto"),             # two 32-row slabs, split-K, eight staged loads
    (20, 2048, 512, 0, (), "auto"),             # two 16-row blocks, six staged loads
    (5, 1024, 384, 2, ("FQ_STRIP_32",), "mfma"),
]


def _flags(fq, names):
    f = 0
    for n in names:
        f |= getattr(fq, n)
    return f


def _call(fq, variant, X, Wq, s, z, tc, Y, ws, split_k, flags, sparse):
    if variant == "dense":
        return fq.fq_w4a16_matmul(X, Wq, s, z, Y=Y, y_dtype="f32", split_k=split_k, ws=ws,
                                  flags=flags)
    fn = fq.fq_w4a16_outlier_matmul if variant == "fused" else \
        fq.fq_w4a16_outlier_matmul_unfused
    return fn(X, Wq, s, z, tc, Y=Y, y_dtype="f32", split_k=split_k, ws=ws, sparse=sparse,
              flags=flags)


@pytest.mark.parametrize("case", CASES, ids=[f"graph{i}" for i in range(len(CASES))])
@pytest.mark.parametrize("variant", ["fused", "unfused", "dense"])
def test_graph_replays_match_eager(gpu_lib, case, variant):
    fq = gpu_lib
    M, K, N, split_k, flag_names, sparse = case
    flags = _flags(fq, flag_names)
    print(f"graph {variant} M={M} K={K} N={N} split_k={split_k} flags={flag_names} {sparse}",
          flush=True)
    prob = make_exact_problem(M, K, N, frac=0.02, seed=3 * M + K + N)
    X, Wq, s, z = fq.to_device(prob)
    tc = fq.TileCOODevice(fq.fq_pack_tile_coo(K, N, prob.k, prob.n, prob.v))
    ws = torch.zeros(WS_BYTES, dtype=torch.uint8, device="cuda")
    if variant == "dense":
        expected = oracle.dense_part(prob.X, prob.Wq, prob.scales, prob.zeros, K, N, prob.group)
    else:
        expected = oracle.matmul(prob.X, prob.Wq, prob.scales, prob.zeros, K, N, prob.group,
                                 prob.k, prob.n, prob.v)
    expected = expected.astype(np.float32)

    Y_eager = torch.empty((M, N), dtype=torch.float32, device="cuda")
    _call(fq, variant, X, Wq, s, z, tc, Y_eager, ws, split_k, flags, sparse)
    torch.cuda.synchronize()
    eager = Y_eager.cpu().numpy()
    assert np.array_equal(eager, expected)

    Y_graph = torch.empty((M, N), dtype=torch.float32, device="cuda")
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):   # warm-up outside the capture
        _call(fq, variant, X, Wq, s, z, tc, Y_graph, ws, split_k, flags, sparse)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        _call(fq, variant, X, Wq, s, z, tc, Y_graph, ws, split_k, flags, sparse)
    torch.cuda.synchronize()

    for r in range(REPLAYS):
        Y_graph.fill_(float("nan"))
        Y_eager.fill_(float("nan"))
        _call(fq, variant, X, Wq, s, z, tc, Y_eager, ws, split_k, flags, sparse)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = Y_graph.cpu().numpy()
        assert np.array_equal(got, eager), f"replay {r} differs from the eager result"
        assert np.array_equal(Y_eager.cpu().numpy(), eager), f"eager call after replay {r}"
