"""Python binding of libfq (fused outlier-aware W4A16 decode matmul, MI355X).

Argument marshalling only: every step of the computation runs in the HIP
kernels of libfq.so, behind the C ABI declared in include/fq.h.  PyTorch
provides device memory and streams.  Function names follow the C names.

There is no CPU fallback: if libfq.so has not been built, every call raises.
"""

from __future__ import annotations

import ctypes as C
import os
import threading
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libfq.so")

FQ_OK = 0
STATUS_NAMES = {0: "FQ_OK", 1: "FQ_ERR_NULL", 2: "FQ_ERR_SHAPE", 3: "FQ_ERR_RANGE",
                4: "FQ_ERR_DUPLICATE", 5: "FQ_ERR_ZERO_VALUE", 6: "FQ_ERR_FORMAT",
                7: "FQ_ERR_UNSUPPORTED", 8: "FQ_ERR_WORKSPACE", 9: "FQ_ERR_HIP",
                10: "FQ_ERR_ALIGN", 11: "FQ_ERR_SCRATCH_LIMIT"}
# static device scratch of fq_w4a16_outlier_matmul_noalloc (FQ_NOALLOC_SCRATCH_BYTES)
NOALLOC_SCRATCH_BYTES = 256 * 1024 + (8 << 20)
FQ_GROUP_BY_COLUMN = 0
FQ_GROUP_BY_BUCKET = 1
FQ_REORDER_COLUMNS = 1
FQ_REORDER_ELEMENTS = 2
FQ_Y_BF16 = 0
FQ_Y_F32 = 1
FQ_SPARSE_AUTO = 0
FQ_SPARSE_GATHER = 1
FQ_SPARSE_MFMA = 2
_SPARSE_MODES = {"auto": FQ_SPARSE_AUTO, "gather": FQ_SPARSE_GATHER, "mfma": FQ_SPARSE_MFMA}
FQ_SCHED_STREAM_K = 4
FQ_FOUR_WAVES = 8
FQ_STRIP_32 = 16
FQ_STRIP_64 = 32
FQ_SPARSE_WAVES = 64
FQ_DENSE_VALU = 128


class FqError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        self.name = STATUS_NAMES.get(status, f"status {status}")
        super().__init__(f"{where}: {self.name}")


class fq_tilecoo_params(C.Structure):
    _fields_ = [("k_tile", C.c_int32), ("n_tile", C.c_int32), ("buckets_per_tile", C.c_int32),
                ("group_mode", C.c_int32), ("reorder", C.c_int32),
                ("elems_per_bank", C.c_int32), ("n_bank_groups", C.c_int32)]

    def as_dict(self):
        return {f: getattr(self, f) for f, _ in self._fields_}


class fq_tilecoo_sizes(C.Structure):
    _fields_ = [("n_tiles", C.c_int64), ("n_buckets", C.c_int64), ("n_groups", C.c_int64),
                ("nnz", C.c_int64), ("n_pad", C.c_int64), ("bytes", C.c_int64),
                ("max_tile_groups", C.c_int64)]

    def as_dict(self):
        return {f: getattr(self, f) for f, _ in self._fields_}


class fq_tilecoo_dev(C.Structure):
    _fields_ = [("tile_indptr", C.c_void_p), ("bucket_info", C.c_void_p),
                ("packed", C.c_void_p), ("params", fq_tilecoo_params),
                ("n_groups", C.c_int64), ("max_tile_groups", C.c_int64)]


class fq_problem(C.Structure):
    _fields_ = [("M", C.c_int32), ("K", C.c_int32), ("N", C.c_int32),
                ("group_size", C.c_int32), ("y_dtype", C.c_int32), ("split_k", C.c_int32),
                ("flags", C.c_int32)]


_lib = None
_lock = threading.Lock()

_P = C.c_void_p
_SIGS = {
    "fq_default_tilecoo_params": ([], fq_tilecoo_params),
    "fq_pack_tile_coo": ([C.c_int32, C.c_int32, C.c_int64, _P, _P, _P,
                          C.POINTER(fq_tilecoo_params), C.POINTER(fq_tilecoo_sizes), _P, _P, _P],
                         C.c_int),
    "fq_unpack_tile_coo": ([C.c_int32, C.c_int32, C.POINTER(fq_tilecoo_params), C.c_int64,
                            _P, _P, _P, C.POINTER(C.c_int64), _P, _P, _P], C.c_int),
    "fq_validate_tile_coo": ([C.c_int32, C.c_int32, C.POINTER(fq_tilecoo_params), C.c_int64,
                              _P, _P, _P], C.c_int),
    "fq_workspace_bytes": ([C.POINTER(fq_problem), C.POINTER(C.c_size_t)], C.c_int),
    "fq_workspace_bytes_unfused": ([C.POINTER(fq_problem), C.POINTER(C.c_size_t)], C.c_int),
    "fq_w4a16_outlier_matmul": ([C.POINTER(fq_problem), _P, _P, _P, _P,
                                 C.POINTER(fq_tilecoo_dev), _P, _P, C.c_size_t, _P], C.c_int),
    "fq_w4a16_outlier_matmul_unfused": ([C.POINTER(fq_problem), _P, _P, _P, _P,
                                         C.POINTER(fq_tilecoo_dev), _P, _P, C.c_size_t, _P],
                                        C.c_int),
    "fq_w4a16_outlier_matmul_noalloc": ([C.POINTER(fq_problem), _P, _P, _P, _P,
                                         C.POINTER(fq_tilecoo_dev), _P, _P], C.c_int),
    "fq_w4a16_matmul": ([C.POINTER(fq_problem), _P, _P, _P, _P, _P, _P, C.c_size_t, _P],
                        C.c_int),
    "fq_debug_decode_tile_coo": ([C.POINTER(fq_tilecoo_dev), C.c_int32, C.c_int32, _P, _P, _P,
                                  _P], C.c_int),
    "fq_status_string": ([C.c_int], C.c_char_p),
    "fq_launch_config": ([C.POINTER(fq_problem), C.c_int32, C.c_int32, C.POINTER(C.c_int32)],
                         C.c_int),
    "fq_quantize_outlier_aware": ([C.c_int32, C.c_int32, _P, C.c_int32, C.c_double,
                                   C.POINTER(C.c_int64), _P, _P, _P, _P, _P, _P], C.c_int),
    "fq_fill_padding_slots": ([C.c_int32, C.c_int32, _P, C.c_int32,
                               C.POINTER(fq_tilecoo_params), C.c_int64, _P, _P, _P, _P, _P,
                               C.POINTER(C.c_int64)], C.c_int),
}
EXPORTS = tuple(_SIGS)


def load() -> C.CDLL:
    """Load libfq.so (built in-tree by build.py); raise if it is missing."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise ImportError(f"libfq.so is not built ({LIB_PATH}); run "
                                  "paper_2608_15531_amd.build.build() first")
            lib = C.CDLL(LIB_PATH)
            for name, (args, res) in _SIGS.items():
                fn = getattr(lib, name)
                fn.argtypes = args
                fn.restype = res
            _lib = lib
    return _lib


STAMPS_LIB_PATH = os.path.join(os.path.dirname(LIB_PATH), "libfq_stamps.so")


def use_instrumented_build() -> C.CDLL:
    """Switch this process to libfq_stamps.so, the build of the same sources
    in which every wave of a matmul launch records timestamps
    (include/fq_debug.h), for measurement only.  Call it before anything else
    uses the library; raises if that build is missing."""
    global _lib
    with _lock:
        if not os.path.exists(STAMPS_LIB_PATH):
            raise ImportError(f"libfq_stamps.so is not built ({STAMPS_LIB_PATH})")
        lib = C.CDLL(STAMPS_LIB_PATH)
        for name, (args, res) in _SIGS.items():
            fn = getattr(lib, name)
            fn.argtypes = args
            fn.restype = res
        lib.fq_debug_wave_stamps.argtypes = [C.c_void_p, C.c_int64]
        lib.fq_debug_wave_stamps.restype = C.c_int
        _lib = lib
    return _lib


def fq_debug_wave_stamps(n_waves: int) -> np.ndarray:
    """The per-wave timestamps of the last matmul launch (instrumented build
    only): uint64 [n_waves][4] = start, first tile's data, end of the tile
    loop, exit, in ticks of the 100 MHz s_memrealtime counter."""
    lib = load()
    if not hasattr(lib, "fq_debug_wave_stamps") or lib.fq_debug_wave_stamps.argtypes is None:
        raise RuntimeError("fq_debug_wave_stamps: call use_instrumented_build() first")
    out = np.zeros((n_waves, 4), np.uint64)
    if lib.fq_debug_wave_stamps(out.ctypes.data, n_waves) != 0:
        raise RuntimeError("fq_debug_wave_stamps failed")
    return out


def _check(status: int, where: str) -> None:
    if status != FQ_OK:
        raise FqError(status, where)


def _ptr(a: np.ndarray) -> int | None:
    return a.ctypes.data if a.size else None


def _params(p) -> fq_tilecoo_params:
    if p is None:
        return load().fq_default_tilecoo_params()
    if isinstance(p, fq_tilecoo_params):
        return p
    d = load().fq_default_tilecoo_params().as_dict()
    d.update(p if isinstance(p, dict) else vars(p))
    return fq_tilecoo_params(**{k: int(d[k]) for k, _ in fq_tilecoo_params._fields_})


def fq_default_tilecoo_params() -> fq_tilecoo_params:
    return load().fq_default_tilecoo_params()


def fq_status_string(status: int) -> str:
    return load().fq_status_string(status).decode()


# ------------------------------------------------------------------ host --

@dataclass
class TileCOOHost:
    params: fq_tilecoo_params
    sizes: fq_tilecoo_sizes
    tile_indptr: np.ndarray   # uint32
    bucket_info: np.ndarray   # uint16
    packed: np.ndarray        # uint32


def fq_pack_tile_coo(K: int, N: int, k, n, v, params=None) -> TileCOOHost:
    """Encode COO outliers (k, n int32; v bf16 bits uint16) into Tile-COO."""
    lib = load()
    k = np.ascontiguousarray(k, dtype=np.int32)
    n = np.ascontiguousarray(n, dtype=np.int32)
    v = np.ascontiguousarray(v, dtype=np.uint16)
    if not (k.shape == n.shape == v.shape):
        raise ValueError("k, n, v must have the same length")
    p = _params(params)
    sizes = fq_tilecoo_sizes()
    _check(lib.fq_pack_tile_coo(K, N, k.size, _ptr(k), _ptr(n), _ptr(v), C.byref(p),
                                C.byref(sizes), None, None, None), "fq_pack_tile_coo")
    tile_indptr = np.empty(sizes.n_tiles + 1, dtype=np.uint32)
    bucket_info = np.empty(2 * sizes.n_buckets, dtype=np.uint16)
    packed = np.empty(max(4 * sizes.n_groups, 4), dtype=np.uint32)
    _check(lib.fq_pack_tile_coo(K, N, k.size, _ptr(k), _ptr(n), _ptr(v), C.byref(p),
                                C.byref(sizes), tile_indptr.ctypes.data,
                                bucket_info.ctypes.data, packed.ctypes.data), "fq_pack_tile_coo")
    return TileCOOHost(p, sizes, tile_indptr, bucket_info, packed[:4 * sizes.n_groups])


def fq_validate_tile_coo(K: int, N: int, params, tile_indptr, bucket_info, packed) -> None:
    lib = load()
    p = _params(params)
    ti = np.ascontiguousarray(tile_indptr, dtype=np.uint32)
    bi = np.ascontiguousarray(bucket_info, dtype=np.uint16)
    pk = np.ascontiguousarray(packed, dtype=np.uint32)
    _check(lib.fq_validate_tile_coo(K, N, C.byref(p), pk.size // 4, _ptr(ti), _ptr(bi),
                                    _ptr(pk)), "fq_validate_tile_coo")


def fq_unpack_tile_coo(K: int, N: int, params, tile_indptr, bucket_info, packed):
    """Decode Tile-COO on the host; returns (k, n, v) sorted by (k, n)."""
    lib = load()
    p = _params(params)
    ti = np.ascontiguousarray(tile_indptr, dtype=np.uint32)
    bi = np.ascontiguousarray(bucket_info, dtype=np.uint16)
    pk = np.ascontiguousarray(packed, dtype=np.uint32)
    nnz = C.c_int64(0)
    _check(lib.fq_unpack_tile_coo(K, N, C.byref(p), pk.size // 4, _ptr(ti), _ptr(bi), _ptr(pk),
                                  C.byref(nnz), None, None, None), "fq_unpack_tile_coo")
    k = np.empty(max(nnz.value, 1), np.int32)
    n = np.empty(max(nnz.value, 1), np.int32)
    v = np.empty(max(nnz.value, 1), np.uint16)
    _check(lib.fq_unpack_tile_coo(K, N, C.byref(p), pk.size // 4, _ptr(ti), _ptr(bi), _ptr(pk),
                                  C.byref(nnz), k.ctypes.data, n.ctypes.data, v.ctypes.data),
           "fq_unpack_tile_coo")
    return k[:nnz.value], n[:nnz.value], v[:nnz.value]


@dataclass
class QuantizedWeight:
    K: int
    N: int
    group: int
    Wq: np.ndarray       # uint32 [K/8][N]
    scales: np.ndarray   # uint16 [K/G][N] fp16 bits
    zeros: np.ndarray    # uint32 [K/G][N/8]
    k: np.ndarray        # int32 [nnz] outlier rows
    n: np.ndarray        # int32 [nnz] outlier columns
    v: np.ndarray        # uint16 [nnz] bf16 bits


def fq_quantize_outlier_aware(W, outlier_frac: float, group: int = 128) -> QuantizedWeight:
    """Split fp32 W [K][N] into INT4 W_Q (per-group affine) and bf16 outliers."""
    lib = load()
    W = np.ascontiguousarray(W, dtype=np.float32)
    K, N = W.shape
    nnz = C.c_int64(0)
    _check(lib.fq_quantize_outlier_aware(K, N, W.ctypes.data, group, float(outlier_frac),
                                         C.byref(nnz), None, None, None, None, None, None),
           "fq_quantize_outlier_aware")
    Wq = np.empty((K // 8, N), np.uint32)
    scales = np.empty((K // group, N), np.uint16)
    zeros = np.empty((K // group, N // 8), np.uint32)
    m = max(nnz.value, 1)
    k, n, v = np.empty(m, np.int32), np.empty(m, np.int32), np.empty(m, np.uint16)
    _check(lib.fq_quantize_outlier_aware(K, N, W.ctypes.data, group, float(outlier_frac),
                                         C.byref(nnz), Wq.ctypes.data, scales.ctypes.data,
                                         zeros.ctypes.data, k.ctypes.data, n.ctypes.data,
                                         v.ctypes.data), "fq_quantize_outlier_aware")
    c = nnz.value
    return QuantizedWeight(K, N, group, Wq, scales, zeros, k[:c], n[:c], v[:c])


def fq_fill_padding_slots(W, qw: QuantizedWeight, host: TileCOOHost) -> int:
    """Store original weights in the padding slots of `host` (in place) and set
    the matching codes of qw.Wq to their zero-points; returns the slots filled."""
    lib = load()
    W = np.ascontiguousarray(W, dtype=np.float32)
    K, N = W.shape
    filled = C.c_int64(0)
    pk = host.packed if host.packed.size else np.zeros(4, np.uint32)
    _check(lib.fq_fill_padding_slots(K, N, W.ctypes.data, qw.group, C.byref(host.params),
                                     int(host.sizes.n_groups), host.tile_indptr.ctypes.data,
                                     host.bucket_info.ctypes.data, pk.ctypes.data,
                                     qw.Wq.ctypes.data, qw.zeros.ctypes.data, C.byref(filled)),
           "fq_fill_padding_slots")
    return int(filled.value)


# ---------------------------------------------------------------- device --

def _torch():
    import torch
    return torch


class TileCOODevice:
    """Tile-COO arrays resident in device memory (torch tensors)."""

    def __init__(self, host: TileCOOHost, device="cuda"):
        torch = _torch()
        self.params = host.params
        self.sizes = host.sizes
        self.tile_indptr = torch.from_numpy(host.tile_indptr.view(np.int32).copy()).to(device)
        self.bucket_info = torch.from_numpy(host.bucket_info.view(np.int16).copy()).to(device)
        pk = host.packed if host.packed.size else np.zeros(4, np.uint32)
        self.packed = torch.from_numpy(pk.view(np.int32).copy()).to(device)
        self.n_groups = int(host.sizes.n_groups)
        self.max_tile_groups = int(host.sizes.max_tile_groups)

    def struct(self) -> fq_tilecoo_dev:
        return fq_tilecoo_dev(self.tile_indptr.data_ptr(), self.bucket_info.data_ptr(),
                              self.packed.data_ptr(), self.params, self.n_groups,
                              self.max_tile_groups)

    @property
    def nbytes(self) -> int:
        return int(self.sizes.bytes)


_workspaces: dict = {}


def _stream_handle(stream, device) -> int:
    torch = _torch()
    if stream is None:
        stream = torch.cuda.current_stream(device)
    return int(stream.cuda_stream)


def workspace(nbytes: int, device, stream_handle: int):
    """Zero-filled workspace kept per (device, stream); the kernels leave it zeroed.
    Call it with the kernel's stream current (see _on_stream): the allocation
    and its zero fill are then ordered before the kernel on that stream."""
    torch = _torch()
    key = (torch.device(device).index, stream_handle)
    buf = _workspaces.get(key)
    if buf is None or buf.numel() < nbytes:
        buf = torch.zeros(max(nbytes, 256), dtype=torch.uint8, device=device)
        _workspaces[key] = buf
    return buf


def _on_stream(stream):
    """Makes `stream` current while Y and the workspace are allocated, so the
    caching allocator ties them to the stream the kernel runs on and the
    workspace's zero fill precedes the kernel there."""
    import contextlib
    if stream is None:
        return contextlib.nullcontext()
    return _torch().cuda.stream(stream)


def _problem(M, K, N, y_dtype, split_k, group=128, sparse="auto", flags=0) -> fq_problem:
    return fq_problem(M, K, N, group, y_dtype, split_k, _SPARSE_MODES[sparse] | flags)


def _check_tensor(t, dtype, shape, name):
    torch = _torch()
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype != dtype or tuple(t.shape) != tuple(shape) or not t.is_contiguous():
        raise ValueError(f"{name}: expected contiguous {dtype} {tuple(shape)}, got "
                         f"{t.dtype} {tuple(t.shape)}")


def _matmul_args(X, Wq, scales, zeros, Y, y_dtype, group):
    torch = _torch()
    M, K = X.shape
    N = Wq.shape[1]
    _check_tensor(X, torch.bfloat16, (M, K), "X")
    _check_tensor(Wq, torch.int32, (K // 8, N), "Wq")
    _check_tensor(scales, torch.float16, (K // group, N), "scales")
    _check_tensor(zeros, torch.int32, (K // group, N // 8), "zeros")
    ydt = FQ_Y_F32 if y_dtype in ("f32", "fp32", torch.float32) else FQ_Y_BF16
    if Y is None:
        Y = torch.empty((M, N), dtype=torch.float32 if ydt == FQ_Y_F32 else torch.bfloat16,
                        device=X.device)
    else:
        _check_tensor(Y, torch.float32 if ydt == FQ_Y_F32 else torch.bfloat16, (M, N), "Y")
    return M, K, N, ydt, Y


def fq_w4a16_outlier_matmul(X, Wq, scales, zeros, tc: TileCOODevice, Y=None, y_dtype="bf16",
                            split_k: int = 0, stream=None, ws=None, group: int = 128,
                            sparse: str = "auto", flags: int = 0):
    """Fused Y = X dequant(W_Q) + X W_O on the GPU; returns Y.  flags: any of
    FQ_SCHED_STREAM_K, FQ_FOUR_WAVES."""
    lib = load()
    with _on_stream(stream):
        M, K, N, ydt, Y = _matmul_args(X, Wq, scales, zeros, Y, y_dtype, group)
        pr = _problem(M, K, N, ydt, split_k, group, sparse, flags)
        need = C.c_size_t(0)
        _check(lib.fq_workspace_bytes(C.byref(pr), C.byref(need)), "fq_workspace_bytes")
        sh = _stream_handle(stream, X.device)
        if ws is None:
            ws = workspace(need.value, X.device, sh)
    tcs = tc.struct()
    _check(lib.fq_w4a16_outlier_matmul(C.byref(pr), X.data_ptr(), Wq.data_ptr(),
                                       scales.data_ptr(), zeros.data_ptr(), C.byref(tcs),
                                       Y.data_ptr(), ws.data_ptr(), ws.numel(), sh),
           "fq_w4a16_outlier_matmul")
    return Y


def fq_w4a16_outlier_matmul_noalloc(X, Wq, scales, zeros, tc: TileCOODevice, Y,
                                    y_dtype="bf16", split_k: int = 0, stream=None,
                                    group: int = 128, sparse: str = "auto", flags: int = 0):
    """Fused Y = X dequant(W_Q) + X W_O without a workspace: the library's
    static device scratch serves as one.  Y is the caller's output tensor
    (nothing is allocated here either); returns Y."""
    lib = load()
    if Y is None:
        raise ValueError("fq_w4a16_outlier_matmul_noalloc: pass the output tensor Y")
    M, K, N, ydt, Y = _matmul_args(X, Wq, scales, zeros, Y, y_dtype, group)
    pr = _problem(M, K, N, ydt, split_k, group, sparse, flags)
    tcs = tc.struct()
    _check(lib.fq_w4a16_outlier_matmul_noalloc(C.byref(pr), X.data_ptr(), Wq.data_ptr(),
                                               scales.data_ptr(), zeros.data_ptr(),
                                               C.byref(tcs), Y.data_ptr(),
                                               _stream_handle(stream, X.device)),
           "fq_w4a16_outlier_matmul_noalloc")
    return Y


def fq_w4a16_outlier_matmul_unfused(X, Wq, scales, zeros, tc: TileCOODevice, Y=None,
                                    y_dtype="bf16", split_k: int = 0, stream=None, ws=None,
                                    group: int = 128, sparse: str = "auto", flags: int = 0):
    """Two-kernel baseline (dense W4A16 then Tile-COO SpMM); returns Y."""
    lib = load()
    with _on_stream(stream):
        M, K, N, ydt, Y = _matmul_args(X, Wq, scales, zeros, Y, y_dtype, group)
        pr = _problem(M, K, N, ydt, split_k, group, sparse, flags)
        need = C.c_size_t(0)
        _check(lib.fq_workspace_bytes_unfused(C.byref(pr), C.byref(need)),
               "fq_workspace_bytes_unfused")
        sh = _stream_handle(stream, X.device)
        if ws is None:
            ws = workspace(need.value, X.device, sh)
    tcs = tc.struct()
    _check(lib.fq_w4a16_outlier_matmul_unfused(C.byref(pr), X.data_ptr(), Wq.data_ptr(),
                                               scales.data_ptr(), zeros.data_ptr(),
                                               C.byref(tcs), Y.data_ptr(), ws.data_ptr(),
                                               ws.numel(), sh),
           "fq_w4a16_outlier_matmul_unfused")
    return Y


def fq_w4a16_matmul(X, Wq, scales, zeros, Y=None, y_dtype="bf16", split_k: int = 0,
                    stream=None, ws=None, group: int = 128, flags: int = 0):
    """Dense-only Y = X dequant(W_Q) (outliers ignored); returns Y."""
    lib = load()
    with _on_stream(stream):
        M, K, N, ydt, Y = _matmul_args(X, Wq, scales, zeros, Y, y_dtype, group)
        pr = _problem(M, K, N, ydt, split_k, group, flags=flags)
        need = C.c_size_t(0)
        _check(lib.fq_workspace_bytes(C.byref(pr), C.byref(need)), "fq_workspace_bytes")
        sh = _stream_handle(stream, X.device)
        if ws is None:
            ws = workspace(need.value, X.device, sh)
    _check(lib.fq_w4a16_matmul(C.byref(pr), X.data_ptr(), Wq.data_ptr(), scales.data_ptr(),
                               zeros.data_ptr(), Y.data_ptr(), ws.data_ptr(), ws.numel(), sh),
           "fq_w4a16_matmul")
    return Y


def fq_debug_decode_tile_coo(tc: TileCOODevice, K: int, N: int, stream=None):
    """Device decode of every group; returns (k, n, v) torch tensors of 4*n_groups."""
    torch = _torch()
    lib = load()
    dev = tc.packed.device
    G = tc.n_groups
    with _on_stream(stream):
        k = torch.empty(max(4 * G, 1), dtype=torch.int32, device=dev)
        n = torch.empty(max(4 * G, 1), dtype=torch.int32, device=dev)
        v = torch.empty(max(4 * G, 1), dtype=torch.int16, device=dev)
    tcs = tc.struct()
    _check(lib.fq_debug_decode_tile_coo(C.byref(tcs), K, N, k.data_ptr(), n.data_ptr(),
                                        v.data_ptr(), _stream_handle(stream, dev)),
           "fq_debug_decode_tile_coo")
    return k[:4 * G], n[:4 * G], v[:4 * G]


def fq_launch_config(M: int, K: int, N: int, split_k: int = 0, sparse: str = "auto",
                     flags: int = 0, buckets_per_tile: int | None = None,
                     group_mode: int | None = None) -> dict:
    """The launch the fused entry point would make (nothing is launched) for a
    Tile-COO packed with the given bucket count and grouping (default: the
    library's default packing)."""
    lib = load()
    if buckets_per_tile is None or group_mode is None:
        d = lib.fq_default_tilecoo_params()
        buckets_per_tile = d.buckets_per_tile if buckets_per_tile is None else buckets_per_tile
        group_mode = d.group_mode if group_mode is None else group_mode
    pr = _problem(M, K, N, FQ_Y_BF16, split_k, 128, sparse, flags)
    cfg = (C.c_int32 * 10)()
    _check(lib.fq_launch_config(C.byref(pr), buckets_per_tile, group_mode, cfg),
           "fq_launch_config")
    return {"strip_cols": cfg[0], "split_k": cfg[1], "dense_waves": cfg[2],
            "outlier_waves": cfg[3], "mapping": "gather" if cfg[4] == FQ_SPARSE_GATHER else "mfma",
            "workgroups": cfg[5], "stream_k": bool(cfg[6]), "lds_bytes": cfg[7],
            "x_staged": bool(cfg[8]), "x_stage_loads": cfg[8], "bulk_scales": bool(cfg[9])}


def fq_workspace_bytes(M: int, K: int, N: int, y_dtype=FQ_Y_BF16, split_k: int = 0,
                       group: int = 128, flags: int = 0) -> int:
    lib = load()
    pr = _problem(M, K, N, y_dtype, split_k, group, flags=flags)
    need = C.c_size_t(0)
    _check(lib.fq_workspace_bytes(C.byref(pr), C.byref(need)), "fq_workspace_bytes")
    return need.value


def fq_workspace_bytes_unfused(M: int, K: int, N: int, y_dtype=FQ_Y_BF16, split_k: int = 0,
                               group: int = 128, flags: int = 0) -> int:
    lib = load()
    pr = _problem(M, K, N, y_dtype, split_k, group, flags=flags)
    need = C.c_size_t(0)
    _check(lib.fq_workspace_bytes_unfused(C.byref(pr), C.byref(need)),
           "fq_workspace_bytes_unfused")
    return need.value


# ---------------------------------------------------- numpy -> device --

def to_device(problem, device="cuda"):
    """Upload a synth.Problem's dense arrays as torch tensors in the library layout."""
    torch = _torch()
    X = torch.from_numpy(problem.X.view(np.int16).copy()).view(torch.bfloat16).to(device)
    Wq = torch.from_numpy(problem.Wq.view(np.int32).copy()).to(device)
    scales = torch.from_numpy(problem.scales.view(np.int16).copy()).view(torch.float16).to(device)
    zeros = torch.from_numpy(problem.zeros.view(np.int32).copy()).to(device)
    return X, Wq, scales, zeros
