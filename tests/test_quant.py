"""Offline outlier-aware quantiser: the oracle against its pins, and the
library's host implementation against the oracle (bit-exact)."""

import json
import os

import numpy as np
import pytest

import oracle
from oracle import quant
from synth import make_dense_weight

HERE = os.path.dirname(os.path.abspath(__file__))


def _fq():
    import paper_2608_15531_amd as fq
    try:
        fq.load()
    except ImportError:
        pytest.skip("libfq.so is not built")
    return fq


def _hand_matrix(fx):
    W = np.zeros((fx["K"], fx["N"]), np.float32)
    for c in fx["columns"]:
        for k, v in c["values"].items():
            W[int(k), c["col"]] = v
    return W


# ------------------------------------------------------------------ pins --

def test_hand_derived_groups():
    """eq. (2) worked by hand on four groups (tests/golden/quant_hand.json)."""
    fx = json.load(open(os.path.join(HERE, "golden", "quant_hand.json")))
    W = _hand_matrix(fx)
    Wq, scales, zeros, k, n, v = quant.quantize(W, 0.0, fx["group"])
    q = oracle.codes(Wq, fx["K"], fx["N"])
    z = oracle.zero_points(zeros, 1, fx["N"])
    assert k.size == 0
    for c in fx["columns"]:
        assert int(scales[0, c["col"]]) == c["scale_bits"], c["note"]
        assert int(z[0, c["col"]]) == c["zero"], c["note"]
        for kk, code in c["codes"].items():
            assert int(q[int(kk), c["col"]]) == code, (c["note"], kk)


def test_fp16_not_below_examples():
    """Smallest fp16 >= s: exact fp16 values map to themselves, others to the
    next fp16 up (0.1 -> 0x2E67 = 0.1000976..., 1/3 -> 0x3556)."""
    assert quant.fp16_not_below(0.5) == 0x3800
    assert quant.fp16_not_below(1.0) == 0x3C00
    assert quant.fp16_not_below(0.1) == 0x2E67
    assert quant.fp16_not_below(1.0 / 3.0) == 0x3556
    assert quant.fp16_not_below(2.0 ** -24) == 0x0001
    assert quant.fp16_not_below(1.5 * 2.0 ** -24) == 0x0002


def test_weights_on_an_affine_grid_are_reproduced():
    """Closed form: w = s (q - z) with s a power of two, each group holding codes
    0 and 15, is quantised back to the same codes and reconstructed exactly."""
    rng = np.random.default_rng(3)
    K, N, G = 256, 16, 128
    s = 2.0 ** -6
    qt = rng.integers(0, 16, (K, N))
    qt[0::G] = 0
    qt[1::G] = 15
    zt = rng.integers(0, 16, (K // G, N))
    W = (s * (qt - np.repeat(zt, G, axis=0))).astype(np.float32)
    Wq, scales, zeros, k, n, v = quant.quantize(W, 0.0, G)
    assert np.array_equal(oracle.codes(Wq, K, N), qt)
    assert np.array_equal(oracle.zero_points(zeros, K // G, N), zt)
    assert np.all(oracle.f16_to_f64(scales) == s)
    Wh = quant.reconstruct(Wq, scales, zeros, K, N, G, k, n, v)
    assert np.array_equal(Wh, W.astype(np.float64))


def test_rounding_error_bound():
    """Every non-outlier weight is within s16 of its reconstruction, and within
    s16 / 2 unless its code was clamped; outliers are exact in bf16."""
    W = make_dense_weight(512, 64, seed=11)
    Wq, scales, zeros, k, n, v = quant.quantize(W, 0.01)
    Wh = quant.reconstruct(Wq, scales, zeros, 512, 64, 128, k, n, v)
    s16 = np.repeat(oracle.f16_to_f64(scales), 128, axis=0)
    err = np.abs(Wh - W.astype(np.float64))
    out = np.zeros_like(err, bool)
    out[k, n] = True
    assert np.all(err[~out] <= s16[~out] * (1 + 1e-12))
    assert np.mean(err[~out] <= 0.5 * s16[~out] * (1 + 1e-12)) > 0.999
    assert np.array_equal(Wh[k, n], oracle.bf16_to_f64(oracle.bf16_rne_bits(W[k, n].astype(np.float64))))


def test_outlier_selection_brute_force():
    """The outliers are the round(frac K N) largest |w|, ties to the lower
    row-major index (checked with a plain sort on a matrix full of ties)."""
    rng = np.random.default_rng(5)
    W = (rng.integers(-6, 7, (128, 16)) * 0.25).astype(np.float32)
    for frac in (0.0, 0.01, 0.1, 0.5):
        sel = quant.select_outliers(W, frac)
        flat = W.ravel()
        order = sorted((i for i in range(flat.size) if flat[i] != 0),
                       key=lambda i: (-abs(float(flat[i])), i))
        want = min(int(np.round(frac * flat.size)), len(order))
        assert sel.tolist() == sorted(order[:want]), frac


def test_error_falls_with_outlier_fraction():
    W = make_dense_weight(1024, 128, seed=2)
    errs = []
    for frac in (0.0, 0.005, 0.01, 0.02):
        Wq, scales, zeros, k, n, v = quant.quantize(W, frac)
        Wh = quant.reconstruct(Wq, scales, zeros, 1024, 128, 128, k, n, v)
        errs.append(np.linalg.norm(Wh - W) / np.linalg.norm(W))
    assert all(a > b for a, b in zip(errs, errs[1:])), errs


def test_padding_reuse_lowers_error_and_stays_valid():
    K, N = 512, 128
    W = make_dense_weight(K, N, seed=4)
    Wq, scales, zeros, k, n, v = quant.quantize(W, 0.01)
    before = np.linalg.norm(quant.reconstruct(Wq, scales, zeros, K, N, 128, k, n, v) - W)
    tc = oracle.pack_tile_coo(K, N, k, n, v)
    filled = quant.fill_padding(W, 128, tc, Wq, zeros)
    assert filled > 0
    k2, n2, v2 = oracle.unpack_tile_coo(K, N, tc.params, tc.tile_indptr, tc.bucket_info,
                                         tc.packed)
    assert k2.size == k.size + filled
    Wh = quant.reconstruct(Wq, scales, zeros, K, N, 128, k2, n2, v2)
    assert np.linalg.norm(Wh - W) < before
    assert np.array_equal(Wh[k2, n2],
                          oracle.bf16_to_f64(oracle.bf16_rne_bits(W[k2, n2].astype(np.float64))))


# ---------------------------------------------- library against the oracle --

@pytest.mark.parametrize("seed,frac", [(0, 0.0), (1, 0.01), (2, 0.05), (3, 0.3)])
def test_library_quantiser_matches_oracle(seed, frac):
    fq = _fq()
    W = make_dense_weight(384, 96, seed=seed)
    W[:128, 0] = 0.0           # all-zero group
    W[128:256, 1] = 0.125      # constant positive group
    W[256:, 2] = -0.5          # constant negative group
    W[7, 9] = W[8, 9] = W.max() * 2   # a tie at the top
    got = fq.fq_quantize_outlier_aware(W, frac)
    ref = quant.quantize(W, frac)
    for name, a, b in zip(("Wq", "scales", "zeros", "k", "n", "v"),
                          (got.Wq, got.scales, got.zeros, got.k, got.n, got.v), ref):
        assert np.array_equal(a, b), name


@pytest.mark.parametrize("buckets,group_mode", [(16, 0), (1, 1)],
                         ids=["by_column_16", "by_bucket_1"])
def test_library_padding_fill_matches_oracle(buckets, group_mode):
    fq = _fq()
    K, N = 512, 192
    W = make_dense_weight(K, N, seed=9)
    got = fq.fq_quantize_outlier_aware(W, 0.02)
    Wq, scales, zeros, k, n, v = quant.quantize(W, 0.02)
    host = fq.fq_pack_tile_coo(K, N, got.k, got.n, got.v,
                               {"buckets_per_tile": buckets, "group_mode": group_mode})
    tc = oracle.pack_tile_coo(K, N, k, n, v, oracle.Params(buckets=buckets, group_mode=group_mode))
    assert fq.fq_fill_padding_slots(W, got, host) == quant.fill_padding(W, 128, tc, Wq, zeros)
    assert np.array_equal(host.packed, np.asarray(tc.packed, np.uint32))
    assert np.array_equal(got.Wq, Wq)
    fq.fq_validate_tile_coo(K, N, host.params, host.tile_indptr, host.bucket_info, host.packed)


def test_library_quantiser_errors():
    fq = _fq()
    W = make_dense_weight(256, 64, seed=1)
    bad = W.copy()
    bad[3, 3] = np.nan
    with pytest.raises(fq.FqError, match="FQ_ERR_RANGE|range"):
        fq.fq_quantize_outlier_aware(bad, 0.01)
    with pytest.raises(fq.FqError):
        fq.fq_quantize_outlier_aware(W, 1.5)
    with pytest.raises(fq.FqError):
        fq.fq_quantize_outlier_aware(W[:200], 0.01)
