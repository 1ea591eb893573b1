"""Host-side tests of libfq (no GPU): exports, Tile-COO packer against the
oracle's independent packer, validation, and the C ABI's argument checks."""

import ctypes as C
import os
import re

import numpy as np
import pytest

import oracle
import paper_2608_15531_amd as fq
from synth import make_problem

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(fq.LIB_PATH):
        from paper_2608_15531_amd.build import build
        build()
    return fq.load()


def to_c_params(p: oracle.Params):
    return {"k_tile": p.k_tile, "n_tile": p.n_tile, "buckets_per_tile": p.buckets,
            "group_mode": p.group_mode, "reorder": p.reorder,
            "elems_per_bank": p.elems_per_bank, "n_bank_groups": p.n_bank_groups}


def test_exports_every_declared_symbol(lib):
    with open(os.path.join(ROOT, "include", "fq.h")) as f:
        header = f.read()
    declared = set(re.findall(r"^\s*(?:fq_status|fq_tilecoo_params|const char\*)\s+(fq_\w+)\(",
                              header, re.M))
    assert declared, "no declarations parsed"
    assert declared == set(fq.EXPORTS)
    for name in declared:
        assert getattr(lib, name) is not None


def test_probe_library_exports_its_header(lib):
    """libfqprobe.so (the streaming-read probe) exports what include/fq_probe.h
    declares, and rejects bad arguments on the host without launching."""
    from paper_2608_15531_amd import probe
    with open(os.path.join(ROOT, "include", "fq_probe.h")) as f:
        header = f.read()
    declared = set(re.findall(r"^\s*int\s+(fq_\w+)\(", header, re.M))
    assert declared == set(probe.EXPORTS)
    plib = probe.load()
    for name in declared:
        assert getattr(plib, name) is not None
    buf = (C.c_uint32 * 128)()
    addr = (C.addressof(buf) + 15) & ~15   # 16-byte aligned: only the named argument is bad
    f = plib.fq_probe_stream_read
    assert f(None, 256, 1, 1, 1, addr, None) == 1                # null source
    assert f(addr, 0, 1, 1, 1, addr, None) == 1                  # no bytes
    assert f(addr, 100, 1, 1, 1, addr, None) == 1                # not a multiple of 16
    assert f(addr, 256, 0, 1, 1, addr, None) == 1                # no workgroups
    assert f(addr, 256, 1, 3, 1, addr, None) == 1                # bad wave count
    assert f(addr, 256, 1, 1, 3, addr, None) == 1                # bad loads in flight
    t = plib.fq_probe_tile_loads
    assert t(addr, addr, addr, addr, None, 128, 64, 21, 0, addr, None) == 1      # null groups
    assert t(addr, addr, addr, addr, addr, 100, 64, 21, 0, addr, None) == 1      # K % 128
    assert t(addr, addr, addr, addr, addr, 128, 96, 21, 0, addr, None) == 1      # N % 64
    assert t(addr, addr, addr, addr, addr, 128, 64, 65, 0, addr, None) == 1      # > 64 groups
    assert t(addr, addr, addr, addr, addr, 128, 64, 21, 32, addr, None) == 1     # no such load
    assert t(addr, addr, addr, addr, addr, 128, 64, 21, 1, addr, None) == 1      # scales alone
    assert t(addr + 8, addr, addr, addr, addr, 128, 64, 21, 0, addr, None) == 1  # codes misaligned
    sl = plib.fq_probe_strip_loads
    assert sl(None, addr, addr, 1024, 512, 32, 8, 1, 21, addr, None) == 1      # null codes
    assert sl(addr, addr, addr, 1000, 512, 32, 8, 1, 21, addr, None) == 1      # K % 128
    assert sl(addr, addr, addr, 1024, 96, 32, 8, 1, 21, addr, None) == 1       # N % 64
    assert sl(addr, addr, addr, 1024, 512, 48, 8, 1, 21, addr, None) == 1      # strip width
    assert sl(addr, addr, addr, 1024, 512, 32, 2, 1, 21, addr, None) == 1      # wave count
    assert sl(addr, addr, addr, 1024, 512, 32, 8, 0, 21, addr, None) == 1      # no split
    assert sl(addr, addr, addr, 1024, 512, 32, 8, 2, 21, addr, None) == 1      # 4 tiles < 8 waves
    assert sl(addr, addr, addr, 1024, 512, 32, 4, 1, 65, addr, None) == 1      # > 64 groups
    assert sl(addr + 8, addr, addr, 1024, 512, 32, 4, 1, 21, addr, None) == 1  # codes misaligned
    assert sl(addr, addr, addr, 1024, 512, 32, 4, 1, 21, addr + 2, None) == 1  # sink misaligned
    x = plib.fq_probe_workgroup_xcd
    assert x(None, 8, 64, None) == 1                             # null output
    assert x(addr + 2, 8, 64, None) == 1                         # misaligned output
    assert x(addr, 0, 64, None) == 1                             # no workgroups
    assert x(addr, 8, 96, None) == 1                             # bad thread count


def test_gemm_ref_library_exports_its_header(lib):
    """libfqgemm.so (the hipBLASLt bf16 GEMM comparator) exports what
    include/fq_gemm_ref.h declares, and rejects bad arguments on the host
    before any HIP or hipBLASLt call."""
    from paper_2608_15531_amd import gemm_ref
    with open(os.path.join(ROOT, "include", "fq_gemm_ref.h")) as f:
        header = f.read()
    declared = set(re.findall(r"^\s*(?:int|const char\*)\s+(fq_\w+)\(", header, re.M))
    assert declared == set(gemm_ref.EXPORTS)
    for name, value in (("FQ_REF_W_KN", gemm_ref.W_KN), ("FQ_REF_W_NK", gemm_ref.W_NK),
                        ("FQ_REF_HEURISTIC", gemm_ref.HEURISTIC),
                        ("FQ_REF_EXHAUSTIVE", gemm_ref.EXHAUSTIVE)):
        assert re.search(rf"#define {name} {value}\b", header)
    glib = gemm_ref.load()
    for name in declared:
        assert getattr(glib, name) is not None
    n = C.c_int32(-1)
    prep = glib.fq_ref_gemm_bf16_prepare
    assert prep(0, 64, 64, 0, 0, 4, 0, C.byref(n)) == 1              # M = 0
    assert prep(1, 64, 64, 2, 0, 4, 0, C.byref(n)) == 1              # unknown layout
    assert prep(1, 64, 64, 0, 2, 4, 0, C.byref(n)) == 1              # unknown source
    assert prep(1, 64, 64, 0, 0, 0, 0, C.byref(n)) == 1              # no candidates asked
    assert prep(1, 64, 64, 0, 0, 4097, 0, C.byref(n)) == 1           # too many asked
    assert prep(1, 64, 1 << 21, 0, 0, 4, 0, C.byref(n)) == 1         # N beyond 2^20
    assert prep(1, 64, 64, 0, 0, 4, 0, None) == 1                    # no output
    assert glib.fq_ref_gemm_last_error() == b"n_candidates is NULL"
    assert n.value == -1
    assert glib.fq_ref_gemm_bf16_candidate(1, 64, 64, 3, 0, None, None, 0) == 1
    assert glib.fq_ref_gemm_bf16(None, None, None, 1, 64, 64, 0, 0, None, 0, None) == 1
    assert b"device pointers" in glib.fq_ref_gemm_last_error()


def test_instrumented_build_exports(lib):
    """libfq_stamps.so, the build with per-wave timestamps, exports every entry
    point of include/fq.h and what include/fq_debug.h declares, and rejects
    bad arguments of the stamp reader on the host."""
    path = fq.STAMPS_LIB_PATH
    assert os.path.exists(path)
    slib = C.CDLL(path)
    for name in fq.EXPORTS:
        assert getattr(slib, name) is not None
    with open(os.path.join(ROOT, "include", "fq_debug.h")) as f:
        declared = set(re.findall(r"^\s*int\s+(fq_\w+)\(", f.read(), re.M))
    assert declared == {"fq_debug_wave_stamps"}
    f = slib.fq_debug_wave_stamps
    f.argtypes = [C.c_void_p, C.c_int64]
    buf = (C.c_uint64 * 4)()
    assert f(None, 1) == 1
    assert f(C.addressof(buf), 0) == 1
    assert f(C.addressof(buf), 8193) == 1


def test_default_params(lib):
    p = fq.fq_default_tilecoo_params().as_dict()
    assert p == {"k_tile": 128, "n_tile": 64, "buckets_per_tile": 1, "group_mode": 1,
                 "reorder": 3, "elems_per_bank": 2, "n_bank_groups": 4}


def test_status_strings(lib):
    for s in range(12):
        assert fq.fq_status_string(s) and fq.fq_status_string(s) != "unknown status"
    assert fq.fq_status_string(0) == "ok"


PACK_CASES = [
    (oracle.Params(), 1024, 512, 0.01, "uniform"),
    (oracle.Params(), 512, 256, 0.05, "clustered"),
    (oracle.Params(buckets=8), 512, 512, 0.02, "uniform"),
    (oracle.Params(buckets=1), 256, 128, 0.03, "uniform"),
    (oracle.Params(buckets=64, reorder=0), 512, 256, 0.02, "clustered"),
    (oracle.Params(buckets=16, reorder=1), 512, 256, 0.02, "uniform"),
    (oracle.Params(buckets=16, reorder=2), 512, 256, 0.02, "uniform"),
    (oracle.Params(buckets=4, group_mode=1), 512, 256, 0.03, "clustered"),
    (oracle.Params(buckets=5, group_mode=1, reorder=2), 512, 256, 0.03, "uniform"),
    (oracle.Params(k_tile=64, n_tile=32, buckets=3, elems_per_bank=1, n_bank_groups=8),
     512, 256, 0.02, "uniform"),
    (oracle.Params(k_tile=256, n_tile=256, buckets=256), 512, 512, 0.01, "clustered"),
    (oracle.Params(), 256, 128, 0.0, "uniform"),
    (oracle.Params(), 128, 64, 1.0, "uniform"),
]


@pytest.mark.parametrize("case", PACK_CASES, ids=[f"case{i}" for i in range(len(PACK_CASES))])
def test_pack_matches_oracle_bytes(lib, case):
    p, K, N, frac, dist = case
    prob = make_problem(1, K, N, frac=frac, seed=K + N + int(frac * 1000),
                        dist=dist if frac < 0.5 else "uniform")
    ref = oracle.pack_tile_coo(K, N, prob.k, prob.n, prob.v, p)
    got = fq.fq_pack_tile_coo(K, N, prob.k, prob.n, prob.v, to_c_params(p))
    assert np.array_equal(got.tile_indptr, ref.tile_indptr)
    assert np.array_equal(got.bucket_info, ref.bucket_info)
    assert np.array_equal(got.packed, ref.packed)
    s = got.sizes
    assert s.n_tiles == ref.n_tiles and s.n_buckets == ref.n_buckets
    assert s.n_groups == ref.n_groups and s.nnz == prob.nnz
    assert s.n_pad == 4 * s.n_groups - s.nnz and s.bytes == ref.bytes
    per_tile = np.diff(ref.tile_indptr.astype(np.int64))
    assert s.max_tile_groups == (per_tile.max() if per_tile.size else 0)
    # host decode round trip, and the oracle's decode of the library's bytes
    k, n, v = fq.fq_unpack_tile_coo(K, N, to_c_params(p), got.tile_indptr, got.bucket_info,
                                    got.packed)
    ek, en, ev = oracle.coo_sorted(prob.k, prob.n, prob.v)
    assert np.array_equal(k, ek) and np.array_equal(n, en) and np.array_equal(v, ev)
    fq.fq_validate_tile_coo(K, N, to_c_params(p), got.tile_indptr, got.bucket_info, got.packed)


def test_pack_order_independent(lib):
    prob = make_problem(1, 512, 256, frac=0.02, seed=3)
    a = fq.fq_pack_tile_coo(512, 256, prob.k, prob.n, prob.v)
    perm = np.random.default_rng(0).permutation(prob.nnz)
    b = fq.fq_pack_tile_coo(512, 256, prob.k[perm], prob.n[perm], prob.v[perm])
    assert np.array_equal(a.packed, b.packed) and np.array_equal(a.bucket_info, b.bucket_info)


def test_pack_hand_fixture(lib):
    import json
    with open(os.path.join(ROOT, "tests", "golden", "tilecoo_hand.json")) as f:
        g = json.load(f)
    k = np.array([e[0] for e in g["coo"]])
    n = np.array([e[1] for e in g["coo"]])
    v = np.array([int(e[2], 16) for e in g["coo"]], dtype=np.uint16)
    for case in g["cases"]:
        pr = dict(case["params"])
        pr["buckets_per_tile"] = pr.pop("buckets")
        got = fq.fq_pack_tile_coo(g["K"], g["N"], k, n, v, pr)
        assert got.tile_indptr.tolist() == case["tile_indptr"]
        assert got.bucket_info.tolist() == case["bucket_info"]
        words = []
        for ks, ns, vs in case["groups"]:
            vb = [int(x, 16) for x in vs]
            words += [ks[0] | ks[1] << 8 | ks[2] << 16 | ks[3] << 24,
                      ns[0] | ns[1] << 8 | ns[2] << 16 | ns[3] << 24,
                      vb[0] | vb[1] << 16, vb[2] | vb[3] << 16]
        assert got.packed.tolist() == words


@pytest.mark.parametrize("bad,status", [
    (dict(k=[0, 0], n=[1, 1], v=[1, 2]), "FQ_ERR_DUPLICATE"),
    (dict(k=[256], n=[1], v=[1]), "FQ_ERR_RANGE"),
    (dict(k=[-1], n=[1], v=[1]), "FQ_ERR_RANGE"),
    (dict(k=[1], n=[128], v=[1]), "FQ_ERR_RANGE"),
    (dict(k=[1], n=[1], v=[0x8000]), "FQ_ERR_ZERO_VALUE"),
    (dict(k=[1], n=[1], v=[0]), "FQ_ERR_ZERO_VALUE"),
])
def test_pack_rejects_bad_coo(lib, bad, status):
    with pytest.raises(fq.FqError) as e:
        fq.fq_pack_tile_coo(256, 128, np.array(bad["k"]), np.array(bad["n"]),
                            np.array(bad["v"], dtype=np.uint16))
    assert e.value.name == status


@pytest.mark.parametrize("params,K,N,status", [
    ({"k_tile": 300}, 600, 128, "FQ_ERR_FORMAT"),
    ({"n_tile": 0}, 256, 128, "FQ_ERR_FORMAT"),
    ({}, 250, 128, "FQ_ERR_SHAPE"),
    ({}, 256, 100, "FQ_ERR_SHAPE"),
    ({"buckets_per_tile": 0}, 256, 128, "FQ_ERR_FORMAT"),
    ({"group_mode": 2}, 256, 128, "FQ_ERR_FORMAT"),
    ({"reorder": 4}, 256, 128, "FQ_ERR_FORMAT"),
    ({"elems_per_bank": 64, "n_bank_groups": 4}, 256, 128, "FQ_ERR_FORMAT"),
])
def test_pack_rejects_bad_params(lib, params, K, N, status):
    with pytest.raises(fq.FqError) as e:
        fq.fq_pack_tile_coo(K, N, np.array([1]), np.array([1]), np.array([1], np.uint16), params)
    assert e.value.name == status


def test_pack_null_arguments(lib):
    sizes = fq.fq_tilecoo_sizes()
    p = fq.fq_default_tilecoo_params()
    k = np.array([1], np.int32)
    v = np.array([1], np.uint16)
    assert lib.fq_pack_tile_coo(256, 128, 1, None, k.ctypes.data, v.ctypes.data, C.byref(p),
                                C.byref(sizes), None, None, None) == 1
    assert lib.fq_pack_tile_coo(256, 128, 1, k.ctypes.data, k.ctypes.data, v.ctypes.data,
                                C.byref(p), None, None, None, None) == 1
    ti = np.zeros(16, np.uint32)
    assert lib.fq_pack_tile_coo(256, 128, 1, k.ctypes.data, k.ctypes.data, v.ctypes.data,
                                C.byref(p), C.byref(sizes), ti.ctypes.data, None, None) == 1
    # NULL params -> defaults
    assert lib.fq_pack_tile_coo(256, 128, 1, k.ctypes.data, k.ctypes.data, v.ctypes.data,
                                None, C.byref(sizes), None, None, None) == 0
    assert sizes.n_tiles == 4 and sizes.n_groups == 1 and sizes.n_pad == 3


def _corrupt_cases(tc):
    ti, bi, pk = tc.tile_indptr.copy(), tc.bucket_info.copy(), tc.packed.copy()
    yield "indptr_start", (ti + np.uint32(1)), bi, pk
    t2 = ti.copy(); t2[1], t2[2] = t2[2], t2[1]
    if t2[1] != ti[1]:
        yield "indptr_order", t2, bi, pk
    b2 = bi.copy(); b2[1] += 1
    yield "bucket_count", ti, b2, pk
    b3 = bi.copy(); b3[2] += 1
    yield "bucket_offset", ti, b3, pk
    p2 = pk.copy(); p2[0] |= 0x80   # row 128+ in a 128-row tile
    yield "row_range", ti, bi, p2
    p3 = pk.copy(); p3[1] = (p3[1] & 0xFFFFFF00) | 0x40   # column 64 in a 64-column tile
    yield "col_range", ti, bi, p3
    p4 = pk.copy(); p4[1] = (p4[1] & 0xFFFFFF00) | ((p4[1] + 1) & 0x3F)   # split one group
    yield "group_column", ti, bi, p4
    # duplicate position: copy slot 0 of group 0 onto slot 0 of group 1 (same tile)
    p5 = pk.copy().reshape(-1, 4)
    p5[1] = p5[0]
    yield "duplicate", ti, bi, p5.ravel()


# the format of the paper's decoding kernel: by-column groups, 16 buckets per tile
PAPER_FORMAT = {"buckets_per_tile": 16, "group_mode": 0}


def test_validate_rejects_corruption(lib):
    prob = make_problem(1, 512, 256, frac=0.03, seed=17)
    tc = fq.fq_pack_tile_coo(512, 256, prob.k, prob.n, prob.v, PAPER_FORMAT)
    fq.fq_validate_tile_coo(512, 256, tc.params, tc.tile_indptr, tc.bucket_info, tc.packed)
    names = []
    for name, ti, bi, pk in _corrupt_cases(tc):
        with pytest.raises(fq.FqError) as e:
            fq.fq_validate_tile_coo(512, 256, tc.params, ti, bi, pk)
        assert e.value.name == "FQ_ERR_FORMAT", name
        names.append(name)
    assert len(names) >= 7


def test_validate_rejects_shared_column(lib):
    # two buckets of one tile claiming the same column
    p = {"k_tile": 8, "n_tile": 4, "buckets_per_tile": 2, "elems_per_bank": 2,
         "n_bank_groups": 4}
    tc = fq.fq_pack_tile_coo(8, 4, np.array([0, 1]), np.array([0, 1]),
                             np.array([0x3F80, 0x4000], np.uint16), p)
    pk = tc.packed.copy().reshape(-1, 4)
    assert pk.shape[0] == 2
    pk[1, 1] = pk[0, 1]    # second bucket's group now names the first bucket's column
    pk[1, 0] = 0x07070707 & pk[1, 0] | 0x05050505   # keep rows distinct from group 0
    with pytest.raises(fq.FqError):
        fq.fq_validate_tile_coo(8, 4, p, tc.tile_indptr, tc.bucket_info, pk.ravel())


def test_storage_formula_on_library_output(lib):
    prob = make_problem(1, 4096, 4096, frac=0.01, seed=0)
    for params, buckets in ((PAPER_FORMAT, 16), (None, 1)):
        tc = fq.fq_pack_tile_coo(4096, 4096, prob.k, prob.n, prob.v, params)
        s = tc.sizes
        assert s.n_tiles == 2048 and s.n_buckets == 2048 * buckets and s.nnz == 167772
        assert s.bytes == oracle.storage_bytes(s.n_tiles, s.n_buckets, 4 * s.n_groups)
        # padded Tile-COO still beats the paper's CSR count at 1 %
        assert s.bytes < oracle.csr_bytes(4096, s.nnz)
    # the default (by-bucket, one bucket per tile) pads only each tile's tail:
    # fewer than 4 padding slots per tile
    assert s.n_pad < 4 * s.n_tiles


# ---------------------------------------------------- device entry points --
# Only argument checks that fail before any launch are exercised here.

def _problem(**kw):
    d = dict(M=4, K=1024, N=512, group_size=128, y_dtype=0, split_k=0, flags=0)
    d.update(kw)
    return fq.fq_problem(**d)


FAKE = 1 << 20   # 16-byte aligned, never dereferenced: validation fails first


def _tc(**kw):
    p = fq.fq_default_tilecoo_params()
    for k, v in kw.pop("params", {}).items():
        setattr(p, k, v)
    d = dict(tile_indptr=FAKE, bucket_info=FAKE, packed=FAKE, params=p, n_groups=10,
             max_tile_groups=2)
    d.update(kw)
    return fq.fq_tilecoo_dev(**d)


def _call(lib, pr, X=FAKE, Wq=FAKE, s=FAKE, z=FAKE, tc=None, Y=FAKE, ws=FAKE, wsb=1 << 30):
    tc = tc if tc is not None else _tc()
    return fq.STATUS_NAMES[lib.fq_w4a16_outlier_matmul(C.byref(pr), X, Wq, s, z, C.byref(tc),
                                                       Y, ws, wsb, None)]


@pytest.mark.parametrize("kw,status", [
    (dict(M=0), "FQ_ERR_SHAPE"),
    (dict(M=129), "FQ_ERR_UNSUPPORTED"),
    (dict(K=1000), "FQ_ERR_SHAPE"),
    (dict(N=96), "FQ_ERR_SHAPE"),
    (dict(group_size=64), "FQ_ERR_UNSUPPORTED"),
    (dict(y_dtype=5), "FQ_ERR_UNSUPPORTED"),
    (dict(split_k=-1), "FQ_ERR_SHAPE"),
    (dict(flags=3), "FQ_ERR_UNSUPPORTED"),
    (dict(flags=1, M=5), "FQ_ERR_UNSUPPORTED"),
    (dict(flags=256), "FQ_ERR_UNSUPPORTED"),       # no such switch
    (dict(flags=128, M=2), "FQ_ERR_UNSUPPORTED"),  # dense products on the VALUs: one row only
    (dict(flags=128 | 1, M=1), "FQ_ERR_UNSUPPORTED"),    # ... with the MFMA outlier mapping
    (dict(flags=128 | 4, M=1), "FQ_ERR_UNSUPPORTED"),    # ... uniform split-K
    (dict(flags=128 | 64, M=1), "FQ_ERR_UNSUPPORTED"),   # ... no outlier waves
    (dict(flags=16 | 32), "FQ_ERR_UNSUPPORTED"),   # both strip widths
    (dict(flags=16 | 4), "FQ_ERR_UNSUPPORTED"),    # 32-column strips with Stream-K
    (dict(flags=16 | 1), "FQ_ERR_UNSUPPORTED"),    # 32-column strips with the gather mapping
    (dict(flags=4 | 8 | 3), "FQ_ERR_UNSUPPORTED"),
    # 32-bit byte offsets: packed weights of 2^31 bytes, partial sums of 2^31 bytes
    (dict(K=131072, N=32768), "FQ_ERR_UNSUPPORTED"),
    (dict(M=128, K=32768, N=65536, split_k=64), "FQ_ERR_UNSUPPORTED"),
])
def test_matmul_rejects_bad_problem(lib, kw, status):
    assert _call(lib, _problem(**kw)) == status


def test_matmul_rejects_bad_pointers(lib):
    pr = _problem()
    assert _call(lib, pr, X=None) == "FQ_ERR_NULL"
    assert _call(lib, pr, Y=None) == "FQ_ERR_NULL"
    assert _call(lib, pr, X=FAKE + 2) == "FQ_ERR_ALIGN"
    assert _call(lib, pr, Wq=FAKE + 4) == "FQ_ERR_ALIGN"
    assert _call(lib, pr, s=FAKE + 2) == "FQ_ERR_ALIGN"
    assert _call(lib, pr, Y=FAKE + 8) == "FQ_ERR_ALIGN"
    assert lib.fq_w4a16_outlier_matmul(C.byref(pr), FAKE, FAKE, FAKE, FAKE, None, FAKE, FAKE,
                                       1 << 30, None) == 1


def _call_noalloc(lib, pr, X=FAKE, Wq=FAKE, s=FAKE, z=FAKE, tc=None, Y=FAKE):
    tc = tc if tc is not None else _tc()
    return fq.STATUS_NAMES[lib.fq_w4a16_outlier_matmul_noalloc(C.byref(pr), X, Wq, s, z,
                                                               C.byref(tc), Y, None)]


def test_noalloc_rejects_before_touching_the_device(lib):
    """The allocation-free entry point checks its arguments like the fused one
    and rejects a problem whose launch plan needs more workspace than its
    static scratch, all before any device call (this container has no GPU)."""
    assert fq.NOALLOC_SCRATCH_BYTES == 256 * 1024 + (8 << 20)
    with open(os.path.join(ROOT, "include", "fq.h")) as f:
        assert "#define FQ_NOALLOC_SCRATCH_BYTES ((size_t)(256 * 1024 + (8 << 20)))" in f.read()
    assert _call_noalloc(lib, _problem(M=0)) == "FQ_ERR_SHAPE"
    assert _call_noalloc(lib, _problem(), X=None) == "FQ_ERR_NULL"
    assert _call_noalloc(lib, _problem(), Y=FAKE + 8) == "FQ_ERR_ALIGN"
    assert _call_noalloc(lib, _problem(), tc=_tc(params={"k_tile": 64})) == "FQ_ERR_UNSUPPORTED"
    # explicit split-K over many strips: 448 strips x 8 splits x 32 rows x 64 x 4 B of partials
    big = _problem(M=16, K=4096, N=28672, split_k=8)
    need = C.c_size_t(0)
    assert lib.fq_workspace_bytes(C.byref(big), C.byref(need)) == 0
    assert need.value > fq.NOALLOC_SCRATCH_BYTES
    assert _call_noalloc(lib, big) == "FQ_ERR_SCRATCH_LIMIT"
    # every decode workload's default plan fits the static scratch
    for M, K, N in [(16, 14336, 4096), (16, 28672, 8192), (32, 28672, 8192), (1, 4096, 6144),
                    (128, 14336, 4096), (128, 4096, 14336), (16, 8192, 57344)]:
        pr = _problem(M=M, K=K, N=N)
        assert lib.fq_workspace_bytes(C.byref(pr), C.byref(need)) == 0
        assert need.value <= fq.NOALLOC_SCRATCH_BYTES, (M, K, N, need.value)


def test_matmul_rejects_bad_tilecoo(lib):
    pr = _problem()
    assert _call(lib, pr, tc=_tc(params={"k_tile": 64})) == "FQ_ERR_UNSUPPORTED"
    assert _call(lib, pr, tc=_tc(params={"n_tile": 128})) == "FQ_ERR_UNSUPPORTED"
    assert _call(lib, pr, tc=_tc(params={"buckets_per_tile": 512})) == "FQ_ERR_UNSUPPORTED"
    assert _call(lib, pr, tc=_tc(packed=None)) == "FQ_ERR_NULL"
    assert _call(lib, pr, tc=_tc(packed=FAKE + 8)) == "FQ_ERR_ALIGN"
    assert _call(lib, pr, tc=_tc(n_groups=-1)) == "FQ_ERR_FORMAT"
    assert _call(lib, pr, tc=_tc(n_groups=1 << 27)) == "FQ_ERR_UNSUPPORTED"


def test_matmul_rejects_small_workspace(lib):
    pr = _problem(N=4096, K=4096)
    need = C.c_size_t(0)
    assert lib.fq_workspace_bytes(C.byref(pr), C.byref(need)) == 0
    assert need.value > 0
    assert _call(lib, pr, wsb=1024) == "FQ_ERR_WORKSPACE"
    assert _call(lib, pr, ws=None) == "FQ_ERR_WORKSPACE"
    assert _call(lib, pr, ws=FAKE + 16) == "FQ_ERR_WORKSPACE"
    un = C.c_size_t(0)
    assert lib.fq_workspace_bytes_unfused(C.byref(pr), C.byref(un)) == 0
    assert un.value >= need.value + 4 * 4 * 4096


def test_debug_decode_rejects(lib):
    tc = _tc()
    assert lib.fq_debug_decode_tile_coo(None, 256, 128, FAKE, FAKE, FAKE, None) == 1
    assert lib.fq_debug_decode_tile_coo(C.byref(tc), 250, 128, FAKE, FAKE, FAKE, None) == 2
    assert lib.fq_debug_decode_tile_coo(C.byref(tc), 256, 128, None, FAKE, FAKE, None) == 1


# ----------------------------------------------------- launch configuration --

@pytest.mark.parametrize("M,K,N,expect", [
    # wide matrices: 64-column strips, no split; the gather mapping at M = 1 with
    # by-column groups, the MFMA mapping with the default by-bucket groups
    (1, 4096, 28672, dict(strip_cols=64, split_k=1, mapping="gather", group_mode=0)),
    (1, 4096, 28672, dict(strip_cols=64, split_k=1, mapping="mfma")),
    (16, 4096, 28672, dict(strip_cols=64, split_k=1, mapping="mfma", x_stage_loads=4)),
    # narrow, K <= 8192: 32-column strips without split-K
    (1, 4096, 4096, dict(strip_cols=32, split_k=1, dense_waves=8, mapping="mfma", x_stage_loads=1)),
    (8, 4096, 6144, dict(strip_cols=32, split_k=1, dense_waves=8, x_stage_loads=2)),
    # few strips, up to 16 rows: 32-column strips, no split
    (16, 4096, 4096, dict(strip_cols=32, split_k=1, dense_waves=8, workgroups=128)),
    # few strips and two 16-row blocks: 64-column strips split to 256 workgroups, eight waves
    (32, 4096, 4096, dict(strip_cols=64, split_k=4, dense_waves=8, workgroups=256)),
    (24, 8192, 8192, dict(strip_cols=64, split_k=2, dense_waves=8, workgroups=256)),
    # 32-column strips already give 192 workgroups of 32 tiles: no split
    (16, 4096, 6144, dict(strip_cols=32, split_k=1, dense_waves=8, x_stage_loads=4)),
    # X slices through the LDS stage with ceil(M/4) row-wise loads, one 16-row block
    (4, 4096, 6144, dict(x_stage_loads=1)),
    (5, 4096, 6144, dict(x_stage_loads=2)),
    (9, 4096, 6144, dict(x_stage_loads=4)),
    # two 16-row blocks: six or eight row-wise loads (the stage lives in the outlier image)
    (17, 4096, 6144, dict(x_staged=True, x_stage_loads=6)),
    (25, 4096, 6144, dict(x_staged=True, x_stage_loads=8)),
    (128, 4096, 14336, dict(x_stage_loads=8)),
    # 160+ 64-column strips: 64-column strips, no split, eight waves
    (8, 4096, 14336, dict(strip_cols=64, split_k=1, dense_waves=8)),
    (1, 8192, 10240, dict(strip_cols=64, mapping="gather", x_staged=False, group_mode=0)),
    # the gather mapping (by-column groups at one row) stages its own X slice
    (1, 4096, 28672, dict(mapping="gather", x_stage_loads=0, group_mode=0)),
    # the default packing (by-bucket groups) takes the MFMA mapping at one row too
    (1, 4096, 28672, dict(mapping="mfma", x_stage_loads=1)),
    # long K: 64-column strips split to about 512 workgroups
    (4, 14336, 4096, dict(strip_cols=64, split_k=8, dense_waves=4, workgroups=512)),
    # two 16-row blocks where four-wave workgroups would overflow one round:
    # half that split, eight waves
    (32, 4096, 6144, dict(strip_cols=64, split_k=2, dense_waves=8, workgroups=192)),
    (24, 8192, 3072, dict(strip_cols=64, split_k=4, dense_waves=8, workgroups=192)),
    # long K with two 16-row blocks: about 256 workgroups of eight waves
    (32, 14336, 4096, dict(strip_cols=64, split_k=4, dense_waves=8, workgroups=256)),
    (64, 14336, 4096, dict(strip_cols=64, split_k=2, dense_waves=8, workgroups=256)),
    (32, 28672, 8192, dict(strip_cols=64, split_k=2, dense_waves=8, workgroups=256)),
])
def test_launch_config_defaults(lib, M, K, N, expect):
    expect = dict(expect)
    gm = expect.pop("group_mode", None)
    cfg = fq.fq_launch_config(M, K, N, group_mode=gm, buckets_per_tile=None if gm is None else 16)
    for k, v in expect.items():
        assert cfg[k] == v, (k, cfg)
    assert cfg["outlier_waves"] == 0 and not cfg["stream_k"]
    assert cfg["lds_bytes"] <= 160 * 1024


def test_launch_config_switches(lib):
    assert fq.fq_launch_config(4, 4096, 4096, flags=fq.FQ_STRIP_64)["strip_cols"] == 64
    assert fq.fq_launch_config(4, 4096, 28672, flags=fq.FQ_STRIP_32)["strip_cols"] == 32
    ew = fq.fq_launch_config(4, 4096, 28672, flags=fq.FQ_SPARSE_WAVES)
    assert ew["outlier_waves"] == ew["dense_waves"] // 2
    assert fq.fq_launch_config(4, 4096, 28672, flags=fq.FQ_SCHED_STREAM_K)["stream_k"]
    assert fq.fq_launch_config(4, 4096, 4096, split_k=3)["split_k"] == 3
    # groups spanning columns (by-bucket) take the MFMA mapping at M = 1 too
    assert fq.fq_launch_config(1, 4096, 28672, group_mode=fq.FQ_GROUP_BY_COLUMN)["mapping"] == "gather"
    assert fq.fq_launch_config(1, 4096, 28672, group_mode=fq.FQ_GROUP_BY_BUCKET)["mapping"] == "mfma"
    assert fq.fq_launch_config(1, 4096, 28672)["mapping"] == "mfma"   # default: by-bucket
    assert fq.fq_launch_config(1, 4096, 28672, sparse="gather",
                               group_mode=fq.FQ_GROUP_BY_BUCKET)["mapping"] == "gather"
    with pytest.raises(fq.FqError):
        fq.fq_launch_config(1, 4096, 4096, group_mode=2)
    with pytest.raises(fq.FqError):
        fq.fq_launch_config(5, 4096, 4096, sparse="gather")
    # the dense-path ablation (VALU dot products) runs the MFMA outlier mapping
    # in the default shape, at one row only
    dv = fq.fq_launch_config(1, 4096, 28672, flags=fq.FQ_DENSE_VALU, group_mode=fq.FQ_GROUP_BY_COLUMN)
    assert dv["mapping"] == "mfma" and dv["x_stage_loads"] == 1
    base = fq.fq_launch_config(1, 4096, 28672)
    assert {k: dv[k] for k in ("strip_cols", "split_k", "dense_waves", "workgroups")} == \
        {k: base[k] for k in ("strip_cols", "split_k", "dense_waves", "workgroups")}
    with pytest.raises(fq.FqError):
        fq.fq_launch_config(4, 4096, 4096, flags=fq.FQ_DENSE_VALU)


def test_launch_plans_stay_within_kernel_limits(lib):
    """Every launch the planner accepts, over a sweep of shapes, splits and
    switches, fits the kernel's limits: at most 160 KB of LDS, at most 63
    tiles per wave (one register of group offsets), a grid of strips x
    splits x 32-row slabs, the gather mapping only at up to four rows on
    64-column strips, and X staging exactly when the MFMA mapping is used
    (one 16-row block, or two without outlier waves and
    Stream-K).  The default (no split, no switch) is accepted for every
    shape."""
    Ms = [1, 2, 3, 4, 5, 8, 9, 16, 17, 24, 32, 33, 48, 64, 100, 128]
    Ks = [128, 256, 1024, 4096, 8192, 14336, 28672, 57344]
    Ns = [64, 128, 192, 512, 4096, 6144, 14336, 28672, 57344]
    switches = [0, fq.FQ_STRIP_32, fq.FQ_STRIP_64, fq.FQ_FOUR_WAVES, fq.FQ_SCHED_STREAM_K,
                fq.FQ_SPARSE_WAVES, fq.FQ_STRIP_32 | fq.FQ_FOUR_WAVES,
                fq.FQ_SPARSE_WAVES | fq.FQ_FOUR_WAVES, fq.FQ_SPARSE_WAVES | fq.FQ_STRIP_64,
                fq.FQ_SPARSE_WAVES | fq.FQ_STRIP_32,
                fq.FQ_SCHED_STREAM_K | fq.FQ_FOUR_WAVES]
    accepted = 0
    for M in Ms:
        for K in Ks:
            for N in Ns:
                if K * N // 2 >= 1 << 31:
                    continue
                T = K // 128
                for split_k in (0, 1, 2, 3, 7):
                    for flags in switches:
                        try:
                            c = fq.fq_launch_config(M, K, N, split_k=split_k, flags=flags)
                        except Exception:
                            assert (split_k, flags) != (0, 0), (M, K, N)
                            continue
                        accepted += 1
                        where = (M, K, N, split_k, flags, c)
                        assert c["lds_bytes"] <= 160 * 1024, where
                        assert c["dense_waves"] in (4, 8), where
                        assert c["outlier_waves"] in (0, c["dense_waves"] // 2), where
                        assert c["strip_cols"] in (32, 64), where
                        if c["mapping"] == "gather":
                            assert M <= 4 and c["strip_cols"] == 64, where
                        stage = {1: 1, 2: 1, 3: 1, 4: 1, 5: 2, 8: 2, 17: 6, 24: 6}.get(
                            M, 4 if M <= 16 else 8)
                        if M > 16 and (c["outlier_waves"] or c["stream_k"]):
                            stage = 0   # two blocks stage only without outlier waves and Stream-K
                        assert c["x_stage_loads"] == (stage if c["mapping"] == "mfma" else 0), where
                        if not c["stream_k"]:
                            S = c["split_k"]
                            assert 1 <= S <= T, where
                            slabs = -(-M // 32)
                            assert c["workgroups"] == N // c["strip_cols"] * S * slabs, where
                            assert -(-(-(-T // S)) // c["dense_waves"]) <= 63, where
                            if c["outlier_waves"]:
                                # the outlier waves share the same K range among half as
                                # many waves: the same one-register bound applies to them
                                assert -(-(-(-T // S)) // c["outlier_waves"]) <= 63, where
                        else:
                            # Stream-K: a workgroup's segment lies in one strip and holds
                            # at most its even share of the units
                            U = N // c["strip_cols"] * T
                            share = min(T, -(-U // c["workgroups"]))
                            assert -(-share // c["dense_waves"]) <= 63, where
    assert accepted > 10000
