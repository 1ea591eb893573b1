"""Pins for the CPU oracle (no GPU).

Each test checks the oracle against something other than itself: the bit
layout the format defines, closed forms, library routines in the special
cases that reduce to them, brute force on tiny inputs, exact rational
arithmetic, and hand-derived fixtures.
"""

import itertools
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
from synth import make_exact_problem, make_problem

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------- helpers --

def pack_codes_by_hand(q):
    """Test-side packing of codes [K][N] into words [K/8][N] with Python ints."""
    K, N = q.shape
    out = np.zeros((K // 8, N), dtype=np.uint32)
    for k8 in range(K // 8):
        for n in range(N):
            w = 0
            for j in range(8):
                w |= int(q[8 * k8 + j, n]) << (4 * j)
            out[k8, n] = w
    return out


def pack_zeros_by_hand(z):
    G, N = z.shape
    out = np.zeros((G, N // 8), dtype=np.uint32)
    for g in range(G):
        for n8 in range(N // 8):
            w = 0
            for j in range(8):
                w |= int(z[g, 8 * n8 + j]) << (4 * j)
            out[g, n8] = w
    return out


def f32_to_bf16_bits_torch(x):
    t = torch.tensor(np.asarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def bf16_bits(vals):
    return f32_to_bf16_bits_torch(np.asarray(vals, dtype=np.float32))


# ------------------------------------------------------------ number formats --

def test_codes_nibble_order_is_k_mod_8():
    Wq = np.array([[0x76543210, 0xFEDCBA98]], dtype=np.uint32)
    q = oracle.codes(Wq, 8, 2)
    assert q[:, 0].tolist() == list(range(8))
    assert q[:, 1].tolist() == list(range(8, 16))


def test_zero_points_nibble_order_is_n_mod_8():
    zw = np.array([[0x76543210], [0x89ABCDEF]], dtype=np.uint32)
    z = oracle.zero_points(zw, 2, 8)
    assert z[0].tolist() == list(range(8))
    assert z[1].tolist() == [15, 14, 13, 12, 11, 10, 9, 8]


def test_bf16_rne_known_values():
    one = 1.0
    cases = {
        1.0: 0x3F80, -2.0: 0xC000, 0.0: 0x0000,
        one + 2.0 ** -8: 0x3F80,                 # tie -> even (down)
        one + 3 * 2.0 ** -8: 0x3F82,             # tie -> even (up)
        one + 2.0 ** -8 + 2.0 ** -40: 0x3F81,    # just above the tie
        one + 2.0 ** -8 - 2.0 ** -40: 0x3F80,    # just below the tie
        2.0 ** -133: 0x0001,                     # smallest subnormal
        1e39: 0x7F80,                            # overflow -> inf
    }
    for x, bits in cases.items():
        assert int(oracle.bf16_rne_bits(np.array([x]))[0]) == bits, x


def test_bf16_rne_matches_torch_on_float32_values():
    # For float32 inputs, torch's float32 -> bfloat16 cast (round to nearest
    # even) is an independent implementation of the same rounding.
    rng = np.random.default_rng(5)
    x = np.concatenate([rng.standard_normal(20000) * 10.0 ** rng.integers(-30, 30, 20000),
                        rng.standard_normal(1000) * 1e-39]).astype(np.float32)
    ours = oracle.bf16_rne_bits(x.astype(np.float64))
    assert np.array_equal(ours, f32_to_bf16_bits_torch(x))


def test_bf16_and_f16_decoding():
    assert oracle.bf16_to_f64(np.array([0x3F80, 0xC040, 0x0001], np.uint16)).tolist() == \
        [1.0, -3.0, 2.0 ** -133]
    assert oracle.f16_to_f64(np.array([0x3C00, 0x2C00, 0x0001], np.uint16)).tolist() == \
        [1.0, 0.0625, 2.0 ** -24]


# ------------------------------------------------------------- dense part --

@pytest.mark.parametrize("k0,n0", [(0, 0), (127, 5), (128, 63), (200, 9), (255, 127)])
def test_single_code_closed_form(k0, n0):
    """All codes at their zero-point except one; X = e_k0 picks out s*(q-z)."""
    K, N, G = 256, 128, 128
    rng = np.random.default_rng(k0 * 1000 + n0)
    z = rng.integers(0, 16, size=(K // G, N)).astype(np.uint8)
    q = np.repeat(z, G, axis=0)
    q[k0, n0] = (int(z[k0 // G, n0]) + 5) % 16
    s = rng.uniform(0.005, 0.02, size=(K // G, N)).astype(np.float16)
    X = np.zeros((2, K), dtype=np.uint16)
    X[0, k0] = 0x3F80                                     # 1.0
    X[1, k0] = 0xC000                                     # -2.0
    Y = oracle.dense_part(X, pack_codes_by_hand(q), s.view(np.uint16),
                          pack_zeros_by_hand(z), K, N, G)
    expect = float(s[k0 // G, n0]) * (int(q[k0, n0]) - int(z[k0 // G, n0]))
    assert Y[0, n0] == expect and Y[1, n0] == -2.0 * expect
    Y[:, n0] = 0
    assert not Y.any()


def test_no_outliers_equals_library_matmul():
    """Outlier fraction 0 reduces eq. (1) to X @ W_hat (numpy matmul of a W_hat
    the test builds from the known codes)."""
    M, K, N, G = 3, 512, 96, 128
    rng = np.random.default_rng(7)
    q = rng.integers(0, 16, size=(K, N)).astype(np.uint8)
    z = rng.integers(6, 10, size=(K // G, N)).astype(np.uint8)
    s = rng.uniform(0.005, 0.02, size=(K // G, N)).astype(np.float16)
    Xf = rng.standard_normal((M, K)).astype(np.float32)
    X = f32_to_bf16_bits_torch(Xf)
    W = np.repeat(s.astype(np.float64), G, axis=0) * \
        (q.astype(np.float64) - np.repeat(z.astype(np.float64), G, axis=0))
    X64 = torch.tensor(Xf).to(torch.bfloat16).to(torch.float64).numpy()
    ref = np.matmul(X64, W)
    Y = oracle.matmul(X, pack_codes_by_hand(q), s.view(np.uint16), pack_zeros_by_hand(z),
                      K, N, G, np.zeros(0, np.int32), np.zeros(0, np.int32),
                      np.zeros(0, np.uint16))
    np.testing.assert_allclose(Y, ref, rtol=1e-12, atol=1e-12)


def test_generator_problem_frac0_equals_library_matmul():
    p = make_problem(2, 1024, 256, frac=0.0, seed=11)
    ref_codes = oracle.codes(p.Wq, p.K, p.N)
    # rebuild the words by hand from the decoded codes: the round trip pins
    # the decoder against the hand packer on generator data
    assert np.array_equal(pack_codes_by_hand(ref_codes), p.Wq)
    z = oracle.zero_points(p.zeros, p.K // p.group, p.N)
    assert np.array_equal(pack_zeros_by_hand(z), p.zeros)
    assert z.min() >= 6 and z.max() <= 9
    s = p.scales.view(np.float16).astype(np.float64)
    W = np.repeat(s, 128, axis=0) * (ref_codes - np.repeat(z, 128, axis=0).astype(np.float64))
    X64 = (p.X.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    Y = oracle.matmul(p.X, p.Wq, p.scales, p.zeros, p.K, p.N, p.group, p.k, p.n, p.v)
    np.testing.assert_allclose(Y, np.matmul(X64, W), rtol=1e-12, atol=1e-11)


# ------------------------------------------------------------ outlier part --

def test_all_codes_at_zero_point_equals_spmm():
    """dequant(W_Q) == 0 reduces eq. (1) to X @ W_O (dense scatter of W_O)."""
    M, K, N, G = 4, 384, 64, 128
    rng = np.random.default_rng(3)
    z = rng.integers(0, 16, size=(K // G, N)).astype(np.uint8)
    q = np.repeat(z, G, axis=0)
    s = np.full((K // G, N), 0.01, dtype=np.float16)
    pos = rng.choice(K * N, size=300, replace=False)
    k, n = pos // N, pos % N
    vals = rng.standard_normal(300).astype(np.float32)
    v = f32_to_bf16_bits_torch(vals)
    Wo = np.zeros((K, N))
    Wo[k, n] = torch.tensor(vals).to(torch.bfloat16).double().numpy()
    Xf = rng.standard_normal((M, K)).astype(np.float32)
    X64 = torch.tensor(Xf).to(torch.bfloat16).double().numpy()
    Y = oracle.matmul(f32_to_bf16_bits_torch(Xf), pack_codes_by_hand(q), s.view(np.uint16),
                      pack_zeros_by_hand(z), K, N, G, k, n, v)
    np.testing.assert_allclose(Y, X64 @ Wo, rtol=1e-12, atol=1e-12)


def test_single_outlier_closed_form():
    K, N, G = 256, 64, 128
    z = np.full((K // G, N), 8, np.uint8)
    q = np.repeat(z, G, axis=0)
    X = np.zeros((1, K), np.uint16)
    X[0, 200] = 0x4040                                    # 3.0
    Y = oracle.matmul(X, pack_codes_by_hand(q), np.full((2, N), 0x2C00, np.uint16),
                      pack_zeros_by_hand(z), K, N, G, np.array([200]), np.array([33]),
                      np.array([0xBF00], np.uint16))        # -0.5
    assert Y[0, 33] == -1.5
    Y[0, 33] = 0
    assert not Y.any()


# ---------------------------------------------------------- whole operator --

def test_bruteforce_tiny():
    """eq. (1) by scalar loops over a dense reconstruction W = W_hat + W_O."""
    p = make_problem(3, 256, 32, frac=0.02, seed=21)
    q = oracle.codes(p.Wq, p.K, p.N)
    Y = oracle.matmul(p.X, p.Wq, p.scales, p.zeros, p.K, p.N, p.group, p.k, p.n, p.v)
    xs = torch.tensor(p.X.view(np.int16)).view(torch.bfloat16).double().tolist()
    scales = p.scales.view(np.float16)
    vals = torch.tensor(p.v.view(np.int16)).view(torch.bfloat16).double().tolist()
    outl = {(int(a), int(b)): c for a, b, c in zip(p.k, p.n, vals)}
    for n in range(p.N):
        col = []
        for k in range(p.K):
            g = k // p.group
            zz = (int(p.zeros[g, n // 8]) >> (4 * (n % 8))) & 0xF
            col.append(float(scales[g, n]) * (int(q[k, n]) - zz) + outl.get((k, n), 0.0))
        for m in range(p.M):
            ref = math.fsum(xs[m][k] * col[k] for k in range(p.K))
            assert abs(Y[m, n] - ref) <= 1e-12 * (1 + abs(ref))


def test_exact_case_equals_rational_arithmetic():
    p = make_exact_problem(2, 256, 16, frac=0.05, seed=4)
    Y = oracle.matmul(p.X, p.Wq, p.scales, p.zeros, p.K, p.N, p.group, p.k, p.n, p.v)
    q = oracle.codes(p.Wq, p.K, p.N)
    X64 = oracle.bf16_to_f64(p.X)
    outl = {(int(a), int(b)): Fraction(float(oracle.bf16_to_f64(np.array([c]))[0]))
            for a, b, c in zip(p.k, p.n, p.v)}
    for m, n in itertools.product(range(p.M), range(p.N)):
        acc = Fraction(0)
        for k in range(p.K):
            zz = (int(p.zeros[k // 128, n // 8]) >> (4 * (n % 8))) & 0xF
            w = Fraction(1, 16) * (int(q[k, n]) - zz) + outl.get((k, n), Fraction(0))
            acc += Fraction(float(X64[m, k])) * w
        assert Fraction(Y[m, n]) == acc


def test_linearity_in_X():
    p = make_problem(2, 512, 64, frac=0.01, seed=9)
    rng = np.random.default_rng(1)
    X1 = bf16_bits(rng.integers(-8, 9, size=(2, 512)))
    X2 = bf16_bits(rng.integers(-8, 9, size=(2, 512)))
    Xc = bf16_bits(3.0 * oracle.bf16_to_f64(X1) - 2.0 * oracle.bf16_to_f64(X2))

    def f(X):
        return oracle.matmul(X, p.Wq, p.scales, p.zeros, p.K, p.N, p.group, p.k, p.n, p.v)
    np.testing.assert_allclose(f(Xc), 3 * f(X1) - 2 * f(X2), rtol=1e-12, atol=1e-10)


def test_sampled_columns_equal_full():
    p = make_problem(2, 512, 256, frac=0.02, seed=2)
    full = oracle.matmul(p.X, p.Wq, p.scales, p.zeros, p.K, p.N, p.group, p.k, p.n, p.v)
    cols = np.array([0, 7, 8, 100, 255])
    part = oracle.matmul(p.X, p.Wq, p.scales, p.zeros, p.K, p.N, p.group, p.k, p.n, p.v, cols)
    assert np.array_equal(part, full[:, cols])


def test_generator_outliers_sit_on_zero_points():
    p = make_problem(1, 1024, 128, frac=0.03, seed=5)
    q = oracle.codes(p.Wq, p.K, p.N)
    z = oracle.zero_points(p.zeros, p.K // p.group, p.N)
    assert np.array_equal(q[p.k, p.n], z[p.k // p.group, p.n])
    mags = np.abs(oracle.bf16_to_f64(p.v))
    assert mags.min() >= 0.1
    assert p.nnz == round(0.03 * 1024 * 128)


# ---------------------------------------------------------------- Tile-COO --

def _load_hand():
    with open(os.path.join(GOLDEN, "tilecoo_hand.json")) as f:
        return json.load(f)


def _coo_from_golden(g):
    k = np.array([e[0] for e in g["coo"]])
    n = np.array([e[1] for e in g["coo"]])
    v = np.array([int(e[2], 16) for e in g["coo"]], dtype=np.uint16)
    return k, n, v


def _expected_words(case):
    words = []
    for ks, ns, vs in case["groups"]:
        vb = [int(x, 16) for x in vs]
        words += [ks[0] | ks[1] << 8 | ks[2] << 16 | ks[3] << 24,
                  ns[0] | ns[1] << 8 | ns[2] << 16 | ns[3] << 24,
                  vb[0] | vb[1] << 16, vb[2] | vb[3] << 16]
    return np.array(words, dtype=np.uint32)


@pytest.mark.parametrize("idx", [0, 1, 2])
def test_tilecoo_hand_derived(idx):
    g = _load_hand()
    case = g["cases"][idx]
    k, n, v = _coo_from_golden(g)
    tc = oracle.pack_tile_coo(g["K"], g["N"], k, n, v, oracle.Params(**case["params"]))
    assert tc.tile_indptr.tolist() == case["tile_indptr"]
    assert tc.bucket_info.tolist() == case["bucket_info"]
    assert np.array_equal(tc.packed, _expected_words(case))


def _random_coo(K, N, nnz, rng, clustered=False):
    if clustered:
        cols = rng.choice(N, size=max(1, N // 16), replace=False)
        pos = set()
        while len(pos) < nnz:
            if rng.random() < 0.6:
                pos.add(int(rng.integers(K)) * N + int(rng.choice(cols)))
            else:
                pos.add(int(rng.integers(K * N)))
        pos = np.array(sorted(pos))
    else:
        pos = rng.choice(K * N, size=nnz, replace=False)
    v = rng.integers(1, 0x7F00, size=nnz).astype(np.uint16)
    v[rng.random(nnz) < 0.5] |= 0x8000
    return pos // N, pos % N, v


PARAM_GRID = [
    oracle.Params(),
    oracle.Params(buckets=8),
    oracle.Params(buckets=4, group_mode=oracle.BY_BUCKET),
    oracle.Params(buckets=64, reorder=0),
    oracle.Params(buckets=16, reorder=1),
    oracle.Params(buckets=16, reorder=2, group_mode=oracle.BY_BUCKET),
    oracle.Params(k_tile=64, n_tile=32, buckets=3, elems_per_bank=1, n_bank_groups=8),
    oracle.Params(k_tile=256, n_tile=256, buckets=32),
]


@pytest.mark.parametrize("p", PARAM_GRID)
@pytest.mark.parametrize("clustered", [False, True])
def test_tilecoo_round_trip_and_invariants(p, clustered):
    K, N = 512, 512
    rng = np.random.default_rng(hash((p, clustered)) % 2 ** 32)
    nnz = int(0.03 * K * N)
    k, n, v = _random_coo(K, N, nnz, rng, clustered)
    tc = oracle.pack_tile_coo(K, N, k, n, v, p)
    kk, nn, vv = oracle.unpack_tile_coo(K, N, p, tc.tile_indptr, tc.bucket_info, tc.packed)
    ek, en, ev = oracle.coo_sorted(k, n, v)
    assert np.array_equal(kk, ek) and np.array_equal(nn, en) and np.array_equal(vv, ev)
    check_invariants(tc, K, N, k, n)


def check_invariants(tc, K, N, k, n):
    p = tc.params
    kt_count = K // p.k_tile
    n_tiles = kt_count * (N // p.n_tile)
    assert tc.tile_indptr.shape == (n_tiles + 1,)
    assert tc.tile_indptr[0] == 0 and tc.tile_indptr[-1] == tc.n_groups
    assert np.all(np.diff(tc.tile_indptr.astype(np.int64)) >= 0)
    assert tc.bytes == 4 * (n_tiles + 1) + 4 * n_tiles * p.buckets + 16 * tc.n_groups
    g = tc.packed.reshape(-1, 4)
    tile_of = (np.asarray(n) // p.n_tile) * kt_count + np.asarray(k) // p.k_tile
    info = tc.bucket_info.reshape(n_tiles, p.buckets, 2).astype(np.int64)
    for t in range(n_tiles):
        t0, t1 = int(tc.tile_indptr[t]), int(tc.tile_indptr[t + 1])
        offs, cnts = info[t, :, 0], info[t, :, 1]
        # buckets contiguous, in bucket order, covering the tile exactly
        assert offs[0] == 0 and np.array_equal(offs[1:], np.cumsum(cnts)[:-1])
        assert cnts.sum() == t1 - t0
        owner = {}
        loads = np.zeros(p.buckets, np.int64)
        for b in range(p.buckets):
            gg = g[t0 + offs[b]: t0 + offs[b] + cnts[b]]
            for w in gg:
                ks = [(int(w[0]) >> (8 * j)) & 0xFF for j in range(4)]
                ns = [(int(w[1]) >> (8 * j)) & 0xFF for j in range(4)]
                vs = [(int(w[2 + j // 2]) >> (16 * (j % 2))) & 0xFFFF for j in range(4)]
                assert max(ks) < p.k_tile and max(ns) < p.n_tile
                if p.group_mode == oracle.BY_COLUMN:
                    assert len(set(ns)) == 1
                for kk_, nn_, vv_ in zip(ks, ns, vs):
                    if vv_:
                        loads[b] += 1
                        # column ownership: one bucket per column per tile
                        assert owner.setdefault(nn_, b) == b
        c_per_col = np.bincount(np.asarray(n)[tile_of == t] % p.n_tile, minlength=p.n_tile)
        if p.reorder & oracle.REORDER_COLUMNS and c_per_col.sum():
            # greedy list scheduling bound
            bound = math.ceil(c_per_col.sum() / p.buckets) + c_per_col.max()
            assert loads.max() <= bound
        if p.group_mode == oracle.BY_COLUMN:
            assert t1 - t0 == sum((c + 3) // 4 for c in c_per_col)


def test_tilecoo_independent_of_input_order():
    K, N = 256, 256
    rng = np.random.default_rng(8)
    k, n, v = _random_coo(K, N, 2000, rng)
    p = oracle.Params(buckets=8)
    a = oracle.pack_tile_coo(K, N, k, n, v, p)
    perm = rng.permutation(k.size)
    b = oracle.pack_tile_coo(K, N, k[perm], n[perm], v[perm], p)
    assert np.array_equal(a.packed, b.packed)
    assert np.array_equal(a.bucket_info, b.bucket_info)
    assert np.array_equal(a.tile_indptr, b.tile_indptr)


def test_tilecoo_rejects_bad_input():
    p = oracle.Params(k_tile=8, n_tile=8, buckets=2)
    with pytest.raises(oracle.FormatError):
        oracle.pack_tile_coo(16, 16, [0, 0], [1, 1], np.array([1, 2], np.uint16), p)
    with pytest.raises(oracle.FormatError):
        oracle.pack_tile_coo(16, 16, [16], [1], np.array([1], np.uint16), p)
    with pytest.raises(oracle.FormatError):
        oracle.pack_tile_coo(16, 16, [1], [1], np.array([0x8000], np.uint16), p)
    with pytest.raises(oracle.FormatError):
        oracle.pack_tile_coo(20, 16, [1], [1], np.array([1], np.uint16), p)


def test_storage_formula_worked_example():
    """Storage Analysis (Sec. 3.2.1), worked by hand for a 4096 x 4096 matrix,
    128 x 64 tiles, 16 buckets per tile and 167,772 outliers (1 %)."""
    with open(os.path.join(GOLDEN, "storage_formula.json")) as f:
        g = json.load(f)
    assert oracle.storage_bytes(g["n_tiles"], g["n_buckets"], g["nnz"]) == g["tile_coo_bytes"]
    assert oracle.csr_bytes(g["K"], g["nnz"]) == g["csr_bytes"]


def test_element_reordering_reduces_bank_group_collisions():
    """Metric, not an invariant: over many random tiles the reordered encoding
    makes lockstep buckets collide on bank groups no more often."""
    K, N = 1024, 512
    rng = np.random.default_rng(12)
    k, n, v = _random_coo(K, N, int(0.03 * K * N), rng)
    base = oracle.Params(buckets=4, group_mode=oracle.BY_BUCKET, reorder=1)
    reo = oracle.Params(buckets=4, group_mode=oracle.BY_BUCKET, reorder=3)
    a = oracle.pack_tile_coo(K, N, k, n, v, base)
    b = oracle.pack_tile_coo(K, N, k, n, v, reo)
    ca = sum(oracle.oracle.bank_group_collisions(a, t) for t in range(a.n_tiles))
    cb = sum(oracle.oracle.bank_group_collisions(b, t) for t in range(b.n_tiles))
    assert cb < ca


def test_bank_group_collisions_hand_counted():
    """The collision metric of Sec. 3.2.2 on a hand-written tile whose counts
    were worked out by hand (tests/golden/bank_collisions_hand.json), for two
    bank geometries and three lockstep widths."""
    with open(os.path.join(GOLDEN, "bank_collisions_hand.json")) as f:
        g = json.load(f)
    words = []
    for rows, cols in g["groups"]:
        words += [sum(r << (8 * j) for j, r in enumerate(rows)),
                  sum(c << (8 * j) for j, c in enumerate(cols)), 0x3F803F80, 0x3F803F80]
    for e in g["expected"]:
        params = oracle.Params(k_tile=128, n_tile=64, buckets=g["buckets"],
                               group_mode=oracle.BY_BUCKET, reorder=0,
                               elems_per_bank=e["elems_per_bank"],
                               n_bank_groups=e["n_bank_groups"])
        tc = oracle.TileCOO(params, np.array(g["tile_indptr"], np.uint32),
                            np.array(g["bucket_info"], np.uint16),
                            np.array(words, np.uint32), nnz=4 * len(g["groups"]))
        got = oracle.oracle.bank_group_collisions(tc, 0, e["lanes_per_step"])
        assert got == e["collisions"], e


@pytest.mark.parametrize("params", [oracle.Params(),
                                    oracle.Params(buckets=1, group_mode=oracle.BY_BUCKET),
                                    oracle.Params(buckets=8, group_mode=oracle.BY_BUCKET,
                                                  reorder=0)])
def test_matmul_through_tile_coo_equals_bruteforce(params):
    """eq. (1) with W_O read back through the oracle's own Tile-COO (pack then
    unpack) against scalar sums over the dense reconstruction W_hat + W_O,
    and bit for bit against the exact rational result on exact-arithmetic
    inputs: a dropped, duplicated or misplaced outlier in the round trip
    changes the sum."""
    p = make_problem(2, 256, 128, frac=0.03, seed=31)
    tc = oracle.pack_tile_coo(p.K, p.N, p.k, p.n, p.v, params)
    Y = oracle.matmul_tile_coo(p.X, p.Wq, p.scales, p.zeros, p.K, p.N, p.group, tc)
    q = oracle.codes(p.Wq, p.K, p.N)
    xs = oracle.bf16_to_f64(p.X)
    scales = oracle.f16_to_f64(p.scales)
    vals = oracle.bf16_to_f64(p.v)
    W = np.zeros((p.K, p.N))
    for k in range(p.K):
        for n in range(p.N):
            zz = (int(p.zeros[k // p.group, n // 8]) >> (4 * (n % 8))) & 0xF
            W[k, n] = scales[k // p.group, n] * (int(q[k, n]) - zz)
    for a, b, c in zip(p.k, p.n, vals):
        W[a, b] += c
    for m in range(p.M):
        for n in range(p.N):
            ref = math.fsum(xs[m, k] * W[k, n] for k in range(p.K))
            assert abs(Y[m, n] - ref) <= 1e-12 * (1 + abs(ref))
    e = make_exact_problem(2, 256, 64, frac=0.05, seed=32)
    te = oracle.pack_tile_coo(e.K, e.N, e.k, e.n, e.v, params)
    Ye = oracle.matmul_tile_coo(e.X, e.Wq, e.scales, e.zeros, e.K, e.N, e.group, te)
    assert np.array_equal(Ye, oracle.matmul(e.X, e.Wq, e.scales, e.zeros, e.K, e.N, e.group,
                                            e.k, e.n, e.v))
    # and a copy with one outlier dropped from the packed groups does not match
    bad = oracle.TileCOO(te.params, te.tile_indptr, te.bucket_info, te.packed.copy(), te.nnz)
    g = bad.packed.reshape(-1, 4)
    real = np.argwhere((g[:, 2] & 0xFFFF) != 0)[0, 0]
    g[real, 2] &= np.uint32(0xFFFF0000)
    Yb = oracle.matmul_tile_coo(e.X, e.Wq, e.scales, e.zeros, e.K, e.N, e.group, bad)
    assert not np.array_equal(Yb, Ye)
