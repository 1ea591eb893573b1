"""GPU parity: the HIP path (through the C ABI) against the fp64 CPU oracle.

Bars:
* Tile-COO decode on the device: bit-exact triples.
* Exact-arithmetic inputs (integer X in [-2, 2], scales 2^-4, outliers j/8):
  every fp32 partial sum is exact in any order, so Y must equal the oracle
  bit for bit, in fp32 and after bf16 rounding.
* Random inputs: bf16 Y elementwise |y - y_ref| <= 1e-2 |y_ref| + 1e-2 and
  fp32 Y Frobenius relative error <= 1e-4.
"""

import dataclasses
import os

import numpy as np
import pytest
import torch

import oracle
from synth import make_exact_problem, make_problem, seed_for

pytestmark = pytest.mark.gpu

BF16_RTOL = 1e-2
BF16_ATOL = 1e-2
F32_FROB = 1e-4


def log(msg):
    print(msg, flush=True)


def c_params(**kw):
    d = {"k_tile": 128, "n_tile": 64, "buckets_per_tile": 16, "group_mode": 0, "reorder": 3,
         "elems_per_bank": 2, "n_bank_groups": 4}
    d.update(kw)
    return d


def run(fq, prob, variant="fused", y="bf16", params=None, split_k=0, sparse="auto", flags=0):
    X, Wq, s, z = fq.to_device(prob)
    if variant == "dense":
        Y = fq.fq_w4a16_matmul(X, Wq, s, z, y_dtype=y, split_k=split_k, flags=flags)
    else:
        tc = fq.TileCOODevice(fq.fq_pack_tile_coo(prob.K, prob.N, prob.k, prob.n, prob.v,
                                                  params))
        fn = fq.fq_w4a16_outlier_matmul if variant == "fused" else \
            fq.fq_w4a16_outlier_matmul_unfused
        Y = fn(X, Wq, s, z, tc, y_dtype=y, split_k=split_k, sparse=sparse, flags=flags)
    torch.cuda.synchronize()
    if y == "bf16":
        return Y.view(torch.int16).cpu().numpy().view(np.uint16)
    return Y.cpu().numpy()


def ref(prob, cols=None, dense_only=False):
    if dense_only:
        return oracle.dense_part(prob.X, prob.Wq, prob.scales, prob.zeros, prob.K, prob.N,
                                 prob.group, cols)
    return oracle.matmul(prob.X, prob.Wq, prob.scales, prob.zeros, prob.K, prob.N, prob.group,
                         prob.k, prob.n, prob.v, cols)


def assert_bf16_close(y_bits, y_ref):
    y = oracle.bf16_to_f64(y_bits)
    err = np.abs(y - y_ref)
    bound = BF16_RTOL * np.abs(y_ref) + BF16_ATOL
    bad = np.argwhere(err > bound)
    assert bad.size == 0, f"{bad.shape[0]} elements out of tolerance, first {bad[:5].tolist()}"


def assert_f32_close(y, y_ref):
    rel = np.linalg.norm(y.astype(np.float64) - y_ref) / max(np.linalg.norm(y_ref), 1e-300)
    assert rel <= F32_FROB, f"Frobenius relative error {rel:.3e}"


# ------------------------------------------------------------ device decode --

@pytest.mark.parametrize("params,dist", [
    (c_params(), "uniform"),
    (c_params(buckets_per_tile=8, group_mode=1), "clustered"),
    (c_params(k_tile=64, n_tile=32, buckets_per_tile=3), "uniform"),
])
def test_device_decode_bit_exact(gpu_lib, params, dist):
    fq = gpu_lib
    prob = make_problem(1, 4096, 4096, frac=0.01, seed=seed_for(0, 0, 0), dist=dist)
    log(f"decode {params} {dist}")
    host = fq.fq_pack_tile_coo(4096, 4096, prob.k, prob.n, prob.v, params)
    k, n, v = fq.fq_debug_decode_tile_coo(fq.TileCOODevice(host), 4096, 4096)
    torch.cuda.synchronize()
    k, n = k.cpu().numpy(), n.cpu().numpy()
    v = v.cpu().numpy().view(np.uint16)
    assert k.size == 4 * host.sizes.n_groups
    real = v != 0
    assert (real.sum()) == prob.nnz
    order = np.lexsort((n[real], k[real]))
    gk, gn, gv = k[real][order], n[real][order], v[real][order]
    op = oracle.Params(params["k_tile"], params["n_tile"], params["buckets_per_tile"],
                       params["group_mode"], params["reorder"], params["elems_per_bank"],
                       params["n_bank_groups"])
    ek, en, ev = oracle.unpack_tile_coo(4096, 4096, op, host.tile_indptr, host.bucket_info,
                                        host.packed)
    assert np.array_equal(gk, ek) and np.array_equal(gn, en) and np.array_equal(gv, ev)
    sk, sn, sv = oracle.coo_sorted(prob.k, prob.n, prob.v)
    assert np.array_equal(gk, sk) and np.array_equal(gn, sn) and np.array_equal(gv, sv)
    # padding slots stay inside their tile
    assert k.min() >= 0 and k.max() < 4096 and n.min() >= 0 and n.max() < 4096


# ----------------------------------------------------- exact arithmetic --

EXACT_CASES = [
    # (M, K, N, frac, split_k, params)
    (1, 4096, 4096, 0.01, 0, c_params()),
    (16, 4096, 4096, 0.01, 0, c_params()),
    (5, 896, 320, 0.03, 0, c_params()),
    (13, 896, 320, 0.03, 1, c_params(buckets_per_tile=1)),
    (3, 896, 320, 0.03, 3, c_params(buckets_per_tile=64)),
    (16, 896, 320, 0.03, 7, c_params(buckets_per_tile=256)),
    (17, 1024, 256, 0.02, 0, c_params(group_mode=1, buckets_per_tile=8)),
    (31, 640, 192, 0.05, 2, c_params(reorder=0)),
    (32, 1024, 128, 0.01, 0, c_params()),
    (8, 128, 64, 0.5, 0, c_params()),
    (2, 256, 64, 1.0, 0, c_params(buckets_per_tile=4)),
    (4, 512, 128, 0.0, 0, c_params()),
    # nine rows: the smallest M whose X slice takes four row-wise loads through the LDS stage
    (9, 1152, 448, 0.03, 0, c_params()),
    # one row with by-bucket groups: the default mapping is MFMA here
    (1, 2048, 1024, 0.02, 0, c_params(group_mode=1)),
    # the library default packing: by-bucket groups, one bucket per tile
    (8, 1024, 512, 0.02, 0, c_params(group_mode=1, buckets_per_tile=1)),
    (1, 4096, 4096, 0.01, 0, c_params(group_mode=1, buckets_per_tile=1)),
    (16, 4096, 4096, 0.01, 0, c_params(group_mode=1, buckets_per_tile=1)),
    # more than 32 rows: 32-row slabs in the grid, ragged last slab, split-K
    (33, 1024, 256, 0.02, 0, c_params()),
    (64, 2048, 512, 0.01, 3, c_params()),
    (100, 1024, 192, 0.03, 0, c_params(group_mode=1, buckets_per_tile=8)),
    (128, 4096, 1024, 0.01, 0, c_params()),
    # two 16-row blocks of at most 24 rows: six staged X loads
    (20, 1024, 384, 0.02, 0, c_params()),
    # two 16-row blocks, half the split with eight waves (4096 x 6144-like)
    (24, 8192, 3072, 0.01, 0, c_params()),
    # long K with two 16-row blocks: split-K with eight waves per workgroup
    (32, 14336, 256, 0.01, 0, c_params()),
    (48, 14336, 512, 0.01, 0, c_params(group_mode=1, buckets_per_tile=1)),
]


@pytest.mark.parametrize("case", EXACT_CASES, ids=[f"exact{i}" for i in range(len(EXACT_CASES))])
@pytest.mark.parametrize("variant", ["fused", "unfused"])
@pytest.mark.parametrize("sparse", ["gather", "mfma"])
def test_exact_arithmetic_bit_exact(gpu_lib, case, variant, sparse):
    M, K, N, frac, split_k, params = case
    if sparse == "gather" and M > 4:
        pytest.skip("the gather mapping covers at most four rows")
    log(f"exact {variant} {sparse} M={M} K={K} N={N} frac={frac} split_k={split_k} {params}")
    prob = make_exact_problem(M, K, N, frac=frac, seed=M * 7 + K + N)
    y_ref = ref(prob)
    y32 = run(gpu_lib, prob, variant, "f32", params, split_k, sparse)
    assert np.array_equal(y32, y_ref.astype(np.float32)), \
        f"max diff {np.abs(y32 - y_ref).max()}"
    y16 = run(gpu_lib, prob, variant, "bf16", params, split_k, sparse)
    assert np.array_equal(y16, oracle.bf16_rne_bits(y_ref))


SCHEDULE_FLAGS = {"stream_k": 4, "four_waves": 8, "stream_k+four_waves": 12,
                  "strip32": 16, "strip64": 32, "strip32+four_waves": 24,
                  "strip64+four_waves": 40, "sparse_waves": 64,
                  "strip32+sparse_waves": 80, "strip64+sparse_waves": 96,
                  "four_waves+sparse_waves": 72}


@pytest.mark.parametrize("case", [c for c in EXACT_CASES if c[4] == 0],
                         ids=[f"exact{i}" for i, c in enumerate(EXACT_CASES) if c[4] == 0])
@pytest.mark.parametrize("sched", list(SCHEDULE_FLAGS))
def test_exact_schedules_bit_exact(gpu_lib, case, sched):
    """The ablation schedules (Stream-K ranges, four waves only, outlier
    waves beside the dense waves) and both strip widths (32 and 64 columns) give the same exact
    result as the default one."""
    M, K, N, frac, split_k, params = case
    log(f"exact schedule {sched} M={M} K={K} N={N} frac={frac}")
    fq = gpu_lib
    prob = make_exact_problem(M, K, N, frac=frac, seed=M * 7 + K + N)
    X, Wq, s, z = fq.to_device(prob)
    tc = fq.TileCOODevice(fq.fq_pack_tile_coo(K, N, prob.k, prob.n, prob.v, params))
    f = SCHEDULE_FLAGS[sched]
    y = fq.fq_w4a16_outlier_matmul(X, Wq, s, z, tc, y_dtype="f32", flags=f)
    yu = fq.fq_w4a16_outlier_matmul_unfused(X, Wq, s, z, tc, y_dtype="f32", flags=f)
    torch.cuda.synchronize()
    y_ref = ref(prob).astype(np.float32)
    assert np.array_equal(y.cpu().numpy(), y_ref)
    assert np.array_equal(yu.cpu().numpy(), y_ref)


@pytest.mark.parametrize("case", [c for c in EXACT_CASES if c[4] != 0],
                         ids=[f"exact{i}" for i, c in enumerate(EXACT_CASES) if c[4] != 0])
@pytest.mark.parametrize("strip", [16, 32], ids=["strip32", "strip64"])
def test_exact_split_k_both_strip_widths(gpu_lib, case, strip):
    """Explicit split-K (cross-workgroup partial sums) with 32- and 64-column
    strips, fused, unfused and dense-only."""
    M, K, N, frac, split_k, params = case
    log(f"exact split strip flag={strip} M={M} K={K} N={N} split_k={split_k}")
    prob = make_exact_problem(M, K, N, frac=frac, seed=M * 7 + K + N)
    y_ref = ref(prob).astype(np.float32)
    for variant in ("fused", "unfused"):
        y = run(gpu_lib, prob, variant, "f32", params, split_k, "mfma", flags=strip)
        assert np.array_equal(y, y_ref), variant
    yd = run(gpu_lib, prob, "dense", "f32", split_k=split_k, flags=strip)
    assert np.array_equal(yd, ref(prob, dense_only=True).astype(np.float32))


def _column_pattern_problem(M, counts, seed):
    """Exact-arithmetic problem (K = 256, N = 128) whose first 128 x 64 tile
    holds counts[c] outliers in column c (rows spread over the tile), the other
    tiles a few each; values +-j/8 as in make_exact_problem."""
    prob = make_exact_problem(M, 256, 128, frac=0.0, seed=seed)
    rng = np.random.Generator(np.random.PCG64(seed + 1))
    ks, ns = [], []
    for c, cnt in enumerate(counts):
        rows = rng.choice(128, size=cnt, replace=False)
        ks += list(rows)
        ns += [c] * cnt
    for t_k, t_n in ((1, 0), (0, 1), (1, 1)):   # the other tiles: 3 outliers each
        rows = rng.choice(128, size=3, replace=False)
        ks += list(t_k * 128 + rows)
        ns += list(t_n * 64 + rng.choice(64, size=3, replace=False))
    k = np.array(ks, dtype=np.int32)
    n = np.array(ns, dtype=np.int32)
    mags = rng.integers(1, 33, size=k.size).astype(np.float32) / 8.0
    signs = np.where(rng.integers(0, 2, size=k.size) == 1, -1.0, 1.0).astype(np.float32)
    from synth import bf16_bits_from_f32
    return dataclasses.replace(prob, k=k, n=n, v=bf16_bits_from_f32(mags * signs))


# by-column groups in the first tile: 64 (one load pass), 65 (second pass),
# 128 (both passes full), 129 and 200 (the loop past the preloaded groups)
GROUP_COUNT_CASES = {
    64: [1] * 64,
    65: [5] + [1] * 63,
    128: [5] * 64,
    129: [9] + [5] * 63,
    200: [13] * 8 + [9] * 56,
}


@pytest.mark.parametrize("n_groups", list(GROUP_COUNT_CASES))
@pytest.mark.parametrize("M", [1, 4, 16])
@pytest.mark.parametrize("sparse", ["gather", "mfma"])
def test_exact_group_count_boundaries(gpu_lib, n_groups, M, sparse):
    """Tiles whose group count sits on the boundaries of the per-lane group
    loads (64 and 128 groups) give the exact result with both mappings and
    both strip widths."""
    if sparse == "gather" and M > 4:
        pytest.skip("the gather mapping covers at most four rows")
    counts = GROUP_COUNT_CASES[n_groups]
    assert sum(-(-c // 4) for c in counts) == n_groups
    prob = _column_pattern_problem(M, counts, seed=n_groups * 3 + M)
    log(f"group-count boundary n_groups={n_groups} M={M} {sparse}")
    y_ref = ref(prob).astype(np.float32)
    flags = [0] if sparse == "gather" else [0, 16, 32]
    for f in flags:
        y = run(gpu_lib, prob, "fused", "f32", c_params(), 0, sparse, flags=f)
        assert np.array_equal(y, y_ref), (n_groups, M, sparse, f)


DENSE_VALU = 128   # FQ_DENSE_VALU


@pytest.mark.parametrize("case", [c for c in EXACT_CASES if c[0] == 1],
                         ids=[f"exact{i}" for i, c in enumerate(EXACT_CASES) if c[0] == 1])
@pytest.mark.parametrize("strip", [0, 16, 32], ids=["auto", "strip32", "strip64"])
def test_exact_dense_valu_bit_exact(gpu_lib, case, strip):
    """The dense products on the vector ALUs (bf16 dot products per lane, the
    k-chunks summed across lanes after the last tile) instead of MFMA: one
    row, fused, unfused and dense-only, each strip width, the cases' splits."""
    M, K, N, frac, split_k, params = case
    log(f"exact dense-valu M={M} K={K} N={N} frac={frac} split_k={split_k} strip={strip}")
    prob = make_exact_problem(M, K, N, frac=frac, seed=M * 7 + K + N)
    f = DENSE_VALU | strip
    y_ref = ref(prob)
    for variant in ("fused", "unfused"):
        y32 = run(gpu_lib, prob, variant, "f32", params, split_k, "mfma", flags=f)
        assert np.array_equal(y32, y_ref.astype(np.float32)), (variant, np.abs(y32 - y_ref).max())
    y16 = run(gpu_lib, prob, "fused", "bf16", params, split_k, "mfma", flags=f)
    assert np.array_equal(y16, oracle.bf16_rne_bits(y_ref))
    yd = run(gpu_lib, prob, "dense", "f32", split_k=split_k, flags=f)
    assert np.array_equal(yd, ref(prob, dense_only=True).astype(np.float32))


@pytest.mark.parametrize("shape", [(4096, 6144), (4096, 4096), (4096, 28672), (14336, 4096)],
                         ids=["qkv", "o", "gate_up", "down"])
def test_full_size_dense_valu_sampled_columns(gpu_lib, shape):
    """The dense-path ablation at the Llama-3-8B decode shapes, one row, in the
    launch the benchmark compares with the default: sampled columns against
    the oracle, and the whole output against the default (MFMA) kernel."""
    K, N = shape
    log(f"full dense-valu K={K} N={N}")
    prob = make_problem(1, K, N, frac=0.01, seed=seed_for(1, FULL_SHAPES.index(shape), 0))
    rng = np.random.default_rng(K + N + 5)
    cols = np.unique(np.concatenate([[0, 63, 64, N - 1], rng.choice(N, 192, replace=False)]))
    y_ref = ref(prob, cols)
    y16 = run(gpu_lib, prob, "fused", "bf16", flags=DENSE_VALU)
    assert_bf16_close(y16[:, cols], y_ref)
    y32 = run(gpu_lib, prob, "fused", "f32", flags=DENSE_VALU)
    assert_f32_close(y32[:, cols], y_ref)
    ym = run(gpu_lib, prob, "fused", "f32")
    assert np.linalg.norm(y32 - ym) / np.linalg.norm(ym) <= F32_FROB


def test_exact_dense_only(gpu_lib):
    prob = make_exact_problem(16, 2048, 512, frac=0.02, seed=99)
    y32 = run(gpu_lib, prob, "dense", "f32")
    assert np.array_equal(y32, ref(prob, dense_only=True).astype(np.float32))


# ------------------------------------------------------ random inputs --

@pytest.mark.parametrize("M", [1, 4, 8, 16])
@pytest.mark.parametrize("variant", ["fused", "unfused"])
def test_small_workload_tolerances(gpu_lib, M, variant):
    """4096 x 4096, 1 % uniform outliers, every row count of the decode sweep."""
    log(f"small {variant} M={M}")
    prob = make_problem(M, 4096, 4096, frac=0.01, seed=seed_for(0, 0, [1, 4, 8, 16].index(M)))
    y_ref = ref(prob)
    assert_bf16_close(run(gpu_lib, prob, variant, "bf16"), y_ref)
    assert_f32_close(run(gpu_lib, prob, variant, "f32"), y_ref)


def test_dropping_outliers_fails_the_bar(gpu_lib):
    """The tolerance is tight enough that ignoring W_O cannot pass."""
    prob = make_problem(4, 4096, 4096, frac=0.01, seed=5)
    y = run(gpu_lib, prob, "dense", "f32")
    rel = np.linalg.norm(y - ref(prob)) / np.linalg.norm(ref(prob))
    assert rel > 100 * F32_FROB
    assert_f32_close(y, ref(prob, dense_only=True))


@pytest.mark.parametrize("frac,dist", [(0.0, "uniform"), (0.05, "uniform"),
                                       (0.02, "clustered"), (0.05, "clustered")])
def test_density_sweep_tolerances(gpu_lib, frac, dist):
    log(f"density frac={frac} {dist}")
    prob = make_problem(8, 2048, 2048, frac=frac, seed=int(frac * 1000) + len(dist), dist=dist)
    y_ref = ref(prob)
    assert_bf16_close(run(gpu_lib, prob, "fused", "bf16"), y_ref)
    assert_f32_close(run(gpu_lib, prob, "fused", "f32"), y_ref)


def test_repeat_calls_bit_identical(gpu_lib):
    prob = make_problem(16, 4096, 4096, frac=0.01, seed=77)
    a = run(gpu_lib, prob, "fused", "f32")
    b = run(gpu_lib, prob, "fused", "f32")
    assert np.array_equal(a, b)


def test_repeat_calls_bit_identical_gather_mapping(gpu_lib):
    """The gather mapping adds products with LDS float atomics into per-wave
    buffers; a wave's LDS operations complete in issue order, so repeated
    calls give identical bits.  gate+up at one row, by-column groups (the
    gather mapping's own packing), as the benchmark would launch it."""
    fq = gpu_lib
    K, N = 4096, 28672
    prob = make_problem(1, K, N, frac=0.01, seed=seed_for(1, 2, 0))
    assert fq.fq_launch_config(1, K, N, group_mode=0, buckets_per_tile=16)["mapping"] == "gather"
    X, Wq, s, z = fq.to_device(prob)
    tc = fq.TileCOODevice(fq.fq_pack_tile_coo(K, N, prob.k, prob.n, prob.v, c_params()))
    outs = []
    for _ in range(3):
        y = fq.fq_w4a16_outlier_matmul(X, Wq, s, z, tc, y_dtype="f32", sparse="gather")
        torch.cuda.synchronize()
        outs.append(y.cpu().numpy())
    assert np.array_equal(outs[0], outs[1]) and np.array_equal(outs[0], outs[2])


@pytest.mark.parametrize("flags", [64 | 8, 64 | 32, 64], ids=["sparse_waves+four_waves",
                                                             "sparse_waves+strip64",
                                                             "sparse_waves"])
@pytest.mark.parametrize("M", [4, 32])
def test_exact_outlier_waves_long_k(gpu_lib, flags, M):
    """Outlier waves beside the dense waves with K = 28672 (224 tiles per strip)
    and no split requested: the outlier waves share each K range among half
    as many waves, so the planner must keep them at 63 tiles or fewer each
    (one register of group offsets per wave).  Exact arithmetic, bit for bit."""
    fq = gpu_lib
    K, N = 28672, 128
    cfg = fq.fq_launch_config(M, K, N, split_k=1, flags=flags)
    T = K // 128
    if cfg["outlier_waves"]:
        assert -(-(-(-T // cfg["split_k"])) // cfg["outlier_waves"]) <= 63, cfg
    log(f"exact outlier waves K={K} N={N} M={M} flags={flags} cfg={cfg}")
    prob = make_exact_problem(M, K, N, frac=0.01, seed=M + flags)
    y = run(fq, prob, "fused", "f32", c_params(), split_k=1, sparse="mfma", flags=flags)
    assert np.array_equal(y, ref(prob).astype(np.float32))


def test_workspace_counters_rearmed(gpu_lib):
    fq = gpu_lib
    prob = make_problem(4, 4096, 4096, frac=0.01, seed=8)
    X, Wq, s, z = fq.to_device(prob)
    tc = fq.TileCOODevice(fq.fq_pack_tile_coo(4096, 4096, prob.k, prob.n, prob.v))
    for split_k in (0, 4):
        need = fq.fq_workspace_bytes_unfused(4, 4096, 4096, split_k=split_k)
        ws = torch.zeros(need, dtype=torch.uint8, device="cuda")
        y1 = fq.fq_w4a16_outlier_matmul(X, Wq, s, z, tc, ws=ws, split_k=split_k)
        torch.cuda.synchronize()
        # the counter region (first 256 KiB) is back to zero after the call
        assert int(ws[:256 * 1024].count_nonzero()) == 0, split_k
        y2 = fq.fq_w4a16_outlier_matmul(X, Wq, s, z, tc, ws=ws, split_k=split_k)
        torch.cuda.synchronize()
        assert torch.equal(y1, y2)
        # and after the unfused entry point's two kernels, which share it
        y3 = fq.fq_w4a16_outlier_matmul_unfused(X, Wq, s, z, tc, ws=ws, split_k=split_k)
        torch.cuda.synchronize()
        assert int(ws[:256 * 1024].count_nonzero()) == 0, split_k
        assert_bf16_close(y3.view(torch.int16).cpu().numpy().view(np.uint16), ref(prob))


def test_workspace_shared_across_shapes(gpu_lib):
    """One workspace serving problems of different shapes in turn."""
    fq = gpu_lib
    shapes = [(16, 4096, 4096, 0), (3, 896, 320, 3), (1, 4096, 4096, 0), (5, 896, 192, 2),
              (16, 4096, 4096, 0)]
    ws = torch.zeros(max(fq.fq_workspace_bytes(M, K, N, split_k=sk) for M, K, N, sk in shapes),
                     dtype=torch.uint8, device="cuda")
    for (M, K, N, split_k) in shapes:
        prob = make_exact_problem(M, K, N, frac=0.02, seed=M + K + N)
        X, Wq, s, z = fq.to_device(prob)
        tc = fq.TileCOODevice(fq.fq_pack_tile_coo(K, N, prob.k, prob.n, prob.v))
        need = fq.fq_workspace_bytes(M, K, N, split_k=split_k)
        assert need <= ws.numel()
        Y = fq.fq_w4a16_outlier_matmul(X, Wq, s, z, tc, y_dtype="f32", split_k=split_k, ws=ws)
        torch.cuda.synchronize()
        assert np.array_equal(Y.cpu().numpy(), ref(prob).astype(np.float32)), (M, K, N)


# ------------------------------------------- full-size decode linears --

FULL_SHAPES = [(4096, 6144), (4096, 4096), (4096, 28672), (14336, 4096)]


# (M, strip flag, packing): every row count of the benchmark in the default
# launch configuration with the default packing (what bench.py times), the
# paper's by-column packing (the gather mapping at one row), and each strip
# width forced
PAPER_FORMAT = {"buckets_per_tile": 16, "group_mode": 0}
FULL_CASES = ([(M, 0, None) for M in (1, 4, 8, 16)]
              + [(M, 0, "paper") for M in (1, 4)]
              + [(M, f, None) for M in (1, 16) for f in (16, 32)])


@pytest.mark.parametrize("shape", FULL_SHAPES, ids=["qkv", "o", "gate_up", "down"])
@pytest.mark.parametrize("case", FULL_CASES,
                         ids=[f"M{M}-{ {0: 'auto', 16: 'strip32', 32: 'strip64'}[f]}-"
                              f"{pk or 'default'}" for M, f, pk in FULL_CASES])
def test_full_size_sampled_columns(gpu_lib, shape, case):
    """Llama-3-8B decode linears at full size, in the launch configuration the
    benchmark times (auto, default packing) at every row count, with the
    paper's by-column packing, and with each strip width forced; the oracle
    computes a sample of columns one by one."""
    M, strip, packing = case
    K, N = shape
    params = PAPER_FORMAT if packing == "paper" else None
    log(f"full K={K} N={N} M={M} strip flag={strip} packing={packing or 'default'}")
    prob = make_problem(M, K, N, frac=0.01, seed=seed_for(1, FULL_SHAPES.index(shape),
                                                           [1, 4, 8, 16].index(M)))
    rng = np.random.default_rng(K + N + M)
    cols = np.unique(np.concatenate([[0, 63, 64, N - 1], rng.choice(N, 192, replace=False)]))
    y_ref = ref(prob, cols)
    sparse = "mfma" if strip == 16 else "auto"
    y16 = run(gpu_lib, prob, "fused", "bf16", params=params, sparse=sparse, flags=strip)
    assert_bf16_close(y16[:, cols], y_ref)
    y32 = run(gpu_lib, prob, "fused", "f32", params=params, sparse=sparse, flags=strip)
    assert_f32_close(y32[:, cols], y_ref)
    # property that holds at any size: fused and unfused agree closely everywhere
    yu = run(gpu_lib, prob, "unfused", "f32", params=params, sparse=sparse, flags=strip)
    rel = np.linalg.norm(yu - y32) / np.linalg.norm(y32)
    assert rel <= F32_FROB


@pytest.mark.parametrize("shape", FULL_SHAPES, ids=["qkv", "o", "gate_up", "down"])
@pytest.mark.parametrize("M", [24, 32])
def test_full_size_two_row_blocks_sampled_columns(gpu_lib, shape, M):
    """The Llama-3-8B decode linears at 24 and 32 rows (two 16-row blocks) in
    the default launch configuration (split-K with four or eight waves per
    workgroup, depending on the shape), on sampled columns."""
    K, N = shape
    log(f"full two blocks K={K} N={N} M={M}")
    prob = make_problem(M, K, N, frac=0.01, seed=seed_for(1, FULL_SHAPES.index(shape), 4 + M))
    rng = np.random.default_rng(K + N + M)
    cols = np.unique(np.concatenate([[0, 63, 64, N - 1], rng.choice(N, 128, replace=False)]))
    y_ref = ref(prob, cols)
    assert_bf16_close(run(gpu_lib, prob, "fused", "bf16")[:, cols], y_ref)
    assert_f32_close(run(gpu_lib, prob, "fused", "f32")[:, cols], y_ref)


# --------------------------------------- density sweep at its real shape --

@pytest.mark.parametrize("frac", [0.0, 0.005, 0.01, 0.02, 0.05])
@pytest.mark.parametrize("dist", ["uniform", "clustered"])
def test_density_sweep_full_shape(gpu_lib, frac, dist):
    """M = 8, 4096 x 14336, outlier fraction 0-5 %, uniform or column-clustered
    (2 % of the columns take half of the outliers, capped when they fill up);
    sampled columns against the oracle, every column against the unfused path."""
    K, N, M = 4096, 14336, 8
    log(f"density full frac={frac} {dist}")
    prob = make_problem(M, K, N, frac=frac, dist=dist,
                        seed=seed_for(2, 0, 0) + int(frac * 1000) + (dist == "clustered"))
    rng = np.random.default_rng(K + N + int(frac * 1000))
    heavy = np.unique(prob.n)[:32] if prob.n.size else np.array([], dtype=np.int64)
    cols = np.unique(np.concatenate([[0, N - 1], heavy, rng.choice(N, 96, replace=False)]))
    y_ref = ref(prob, cols)
    assert_bf16_close(run(gpu_lib, prob, "fused", "bf16")[:, cols], y_ref)
    y32 = run(gpu_lib, prob, "fused", "f32")
    assert_f32_close(y32[:, cols], y_ref)
    yu = run(gpu_lib, prob, "unfused", "f32")
    assert np.linalg.norm(yu - y32) <= F32_FROB * max(np.linalg.norm(y32), 1e-30)


# ------------------------------------------ Llama-3-70B decode linears --

SHAPES_70B = [(8192, 10240), (8192, 8192), (8192, 57344), (28672, 8192)]
_PROBLEMS_70B = {}


def _problem_70b(shape, M):
    """One weight set per shape (drawn at M = 32); smaller M use its first rows."""
    if shape not in _PROBLEMS_70B:
        _PROBLEMS_70B.clear()   # keep at most one 70B weight set in host memory
        K, N = shape
        _PROBLEMS_70B[shape] = make_problem(32, K, N, frac=0.01,
                                            seed=seed_for(3, SHAPES_70B.index(shape), 0))
    p = _PROBLEMS_70B[shape]
    return dataclasses.replace(p, M=M, X=np.ascontiguousarray(p.X[:M]))


@pytest.mark.parametrize("shape", SHAPES_70B, ids=["qkv70", "o70", "gate_up70", "down70"])
@pytest.mark.parametrize("M", [1, 8, 16, 32])
def test_70b_full_size_sampled_columns(gpu_lib, shape, M):
    """Llama-3-70B decode linears at full size, every row count of that sweep,
    in the default launch configuration and packing (M = 32: two 16-row MFMA
    blocks); sampled columns against the oracle."""
    K, N = shape
    log(f"70B K={K} N={N} M={M}")
    prob = _problem_70b(shape, M)
    rng = np.random.default_rng(K + N + M)
    cols = np.unique(np.concatenate([[0, 63, 64, N - 1], rng.choice(N, 128, replace=False)]))
    y_ref = ref(prob, cols)
    assert_bf16_close(run(gpu_lib, prob, "fused", "bf16")[:, cols], y_ref)
    assert_f32_close(run(gpu_lib, prob, "fused", "f32")[:, cols], y_ref)


# ------------------------------------------------- up to 128 rows at full size --

SHAPES_LARGE_M = [(4096, 14336), (14336, 4096)]


@pytest.mark.parametrize("shape", SHAPES_LARGE_M, ids=["k4096_n14336", "k14336_n4096"])
@pytest.mark.parametrize("M", [32, 64, 128])
def test_large_m_full_size_sampled_columns(gpu_lib, shape, M):
    """M = 32, 64, 128 on 4096 x 14336 and 14336 x 4096 (32-row slabs); sampled
    columns against the oracle, every element against the unfused path."""
    K, N = shape
    log(f"large M K={K} N={N} M={M}")
    prob = make_problem(M, K, N, frac=0.01,
                        seed=seed_for(4, SHAPES_LARGE_M.index(shape), [32, 64, 128].index(M)))
    rng = np.random.default_rng(K + N + M)
    cols = np.unique(np.concatenate([[0, 63, 64, N - 1], rng.choice(N, 96, replace=False)]))
    y_ref = ref(prob, cols)
    assert_bf16_close(run(gpu_lib, prob, "fused", "bf16")[:, cols], y_ref)
    y32 = run(gpu_lib, prob, "fused", "f32")
    assert_f32_close(y32[:, cols], y_ref)
    yu = run(gpu_lib, prob, "unfused", "f32")
    assert np.linalg.norm(yu - y32) <= F32_FROB * np.linalg.norm(y32)


# ---------------------------------------------- quantiser -> fused kernel --

@pytest.mark.parametrize("fill", [False, True], ids=["outliers", "outliers+padding"])
def test_quantised_weight_through_fused_kernel(gpu_lib, fill):
    """A synthetic dense weight quantised by the library (1 % outliers, padding
    slots optionally filled with original weights) runs through the fused
    kernel; parity against the oracle on the same quantised representation,
    and the result approximates X W of the unquantised weight."""
    from oracle import quant
    from synth import make_activations, make_dense_weight
    fq = gpu_lib
    K, N, M = 4096, 4096, 8
    W = make_dense_weight(K, N, seed=21)
    qw = fq.fq_quantize_outlier_aware(W, 0.01)
    host = fq.fq_pack_tile_coo(K, N, qw.k, qw.n, qw.v)
    if fill:
        assert fq.fq_fill_padding_slots(W, qw, host) > 0
    k, n, v = fq.fq_unpack_tile_coo(K, N, host.params, host.tile_indptr, host.bucket_info,
                                    host.packed)
    X = make_activations(M, K, seed=22)
    Xd, Wq, s, z = fq.to_device(dataclasses.replace(
        make_problem(M, K, N, frac=0.0, seed=0), X=X, Wq=qw.Wq, scales=qw.scales,
        zeros=qw.zeros))
    Y = fq.fq_w4a16_outlier_matmul(Xd, Wq, s, z, fq.TileCOODevice(host), y_dtype="f32")
    torch.cuda.synchronize()
    y = Y.cpu().numpy()
    y_ref = oracle.matmul(X, qw.Wq, qw.scales, qw.zeros, K, N, 128, k, n, v)
    assert_f32_close(y, y_ref)
    exact = oracle.bf16_to_f64(X) @ W.astype(np.float64)
    rel = np.linalg.norm(y - exact) / np.linalg.norm(exact)
    log(f"quantised fill={fill}: relative error of X W_hat against X W = {rel:.4f}")
    assert rel < 0.1
