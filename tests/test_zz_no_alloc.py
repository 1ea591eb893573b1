"""The allocation-free entry point against the workspace entry point.

fq_w4a16_outlier_matmul_noalloc runs the same kernels with the same launch
plan as fq_w4a16_outlier_matmul, its workspace being the library's static
device scratch, so the two must agree bit for bit; both are also checked
against the fp64 oracle.  Two calls in a row, the second smaller, both with
cross-workgroup split-K (arrival counters and partial sums in the scratch).
"""

import numpy as np
import pytest
import torch

import oracle
from synth import make_exact_problem, make_problem, seed_for

pytestmark = pytest.mark.gpu


def log(msg):
    print(msg, flush=True)


def _both(fq, prob, y_dtype, split_k=0, params=None):
    X, Wq, s, z = fq.to_device(prob)
    tc = fq.TileCOODevice(fq.fq_pack_tile_coo(prob.K, prob.N, prob.k, prob.n, prob.v, params))
    dt = torch.float32 if y_dtype == "f32" else torch.bfloat16
    y_ws = fq.fq_w4a16_outlier_matmul(X, Wq, s, z, tc, y_dtype=y_dtype, split_k=split_k)
    y_na = torch.empty((prob.M, prob.N), dtype=dt, device=X.device)
    fq.fq_w4a16_outlier_matmul_noalloc(X, Wq, s, z, tc, y_na, y_dtype=y_dtype, split_k=split_k)
    torch.cuda.synchronize()
    if y_dtype == "f32":
        return y_ws.cpu().numpy(), y_na.cpu().numpy()
    return (y_ws.view(torch.int16).cpu().numpy().view(np.uint16),
            y_na.view(torch.int16).cpu().numpy().view(np.uint16))


def test_noalloc_matches_workspace_entry_two_calls(gpu_lib):
    fq = gpu_lib
    # call 1: Llama-3-8B down at 16 rows (64-column strips split 8 ways)
    K, N, M = 14336, 4096, 16
    cfg = fq.fq_launch_config(M, K, N)
    assert cfg["split_k"] > 1, cfg
    log(f"noalloc call 1: M={M} K={K} N={N} {cfg}")
    p1 = make_problem(M, K, N, frac=0.01, seed=seed_for(1, 3, 3))
    for y_dtype in ("bf16", "f32"):
        a, b = _both(fq, p1, y_dtype)
        assert np.array_equal(a, b), y_dtype
    cols = np.unique(np.concatenate([[0, 63, 64, N - 1],
                                     np.random.default_rng(5).choice(N, 96, replace=False)]))
    y_ref = oracle.matmul(p1.X, p1.Wq, p1.scales, p1.zeros, K, N, p1.group, p1.k, p1.n, p1.v,
                          cols)
    rel = np.linalg.norm(b[:, cols] - y_ref) / np.linalg.norm(y_ref)
    assert rel <= 1e-4, rel
    # call 2, smaller: exact arithmetic, explicit split of 3 over fewer strips
    p2 = make_exact_problem(5, 4096, 1024, frac=0.02, seed=11)
    log("noalloc call 2: M=5 K=4096 N=1024 split_k=3")
    a, b = _both(fq, p2, "f32", split_k=3)
    assert np.array_equal(a, b)
    exact = oracle.matmul(p2.X, p2.Wq, p2.scales, p2.zeros, p2.K, p2.N, p2.group, p2.k, p2.n,
                          p2.v).astype(np.float32)
    assert np.array_equal(b, exact)
    a, b = _both(fq, p2, "bf16", split_k=3)
    assert np.array_equal(a, b)
    assert np.array_equal(b, oracle.bf16_rne_bits(exact.astype(np.float64)))


def test_noalloc_rejects_oversize_problem(gpu_lib):
    fq = gpu_lib
    p = make_exact_problem(16, 4096, 28672, frac=0.0, seed=1)
    X, Wq, s, z = fq.to_device(p)
    tc = fq.TileCOODevice(fq.fq_pack_tile_coo(p.K, p.N, p.k, p.n, p.v))
    Y = torch.empty((16, 28672), dtype=torch.bfloat16, device=X.device)
    with pytest.raises(fq.FqError) as e:
        fq.fq_w4a16_outlier_matmul_noalloc(X, Wq, s, z, tc, Y, split_k=8)
    assert e.value.name == "FQ_ERR_SCRATCH_LIMIT"
