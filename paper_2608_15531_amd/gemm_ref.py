"""Binding of libfqgemm.so, the bf16 GEMM comparator on hipBLASLt declared in
include/fq_gemm_ref.h (a measurement reference for the matmul kernels;
argument marshalling only).  Raises if the library has not been built."""

from __future__ import annotations

import ctypes as C
import os
import threading

_HERE = os.path.dirname(os.path.abspath(__file__))
GEMM_LIB_PATH = os.path.join(_HERE, "libfqgemm.so")
EXPORTS = ("fq_ref_gemm_bf16_prepare", "fq_ref_gemm_bf16_candidate", "fq_ref_gemm_bf16",
           "fq_ref_gemm_last_error")
W_KN, W_NK = 0, 1
HEURISTIC, EXHAUSTIVE = 0, 1
_LAYOUTS = {"kn": W_KN, "nk": W_NK}

_lib = None
_lock = threading.Lock()


def load() -> C.CDLL:
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(GEMM_LIB_PATH):
                raise ImportError(f"libfqgemm.so is not built ({GEMM_LIB_PATH}); run "
                                  "paper_2608_15531_amd.build.build() first")
            lib = C.CDLL(GEMM_LIB_PATH)
            i32, u64 = C.c_int32, C.c_uint64
            lib.fq_ref_gemm_bf16_prepare.argtypes = [i32, i32, i32, i32, i32, i32, u64,
                                                     C.POINTER(i32)]
            lib.fq_ref_gemm_bf16_prepare.restype = C.c_int
            lib.fq_ref_gemm_bf16_candidate.argtypes = [i32, i32, i32, i32, i32, C.POINTER(u64),
                                                       C.c_char_p, C.c_size_t]
            lib.fq_ref_gemm_bf16_candidate.restype = C.c_int
            lib.fq_ref_gemm_bf16.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p, i32, i32, i32, i32,
                                             i32, C.c_void_p, u64, C.c_void_p]
            lib.fq_ref_gemm_bf16.restype = C.c_int
            lib.fq_ref_gemm_last_error.argtypes = []
            lib.fq_ref_gemm_last_error.restype = C.c_char_p
            _lib = lib
    return _lib


def _check(rc: int, what: str) -> None:
    if rc != 0:
        msg = load().fq_ref_gemm_last_error().decode(errors="replace")
        raise RuntimeError(f"{what} failed ({rc}): {msg}")


def prepare(M: int, K: int, N: int, layout: str = "kn", source: int = HEURISTIC,
            max_candidates: int = 16, max_workspace: int = 64 << 20) -> int:
    """Collect candidate algorithms for Y[M][N] = X[M][K] * W on the current
    device; returns how many there are."""
    n = C.c_int32(0)
    _check(load().fq_ref_gemm_bf16_prepare(M, K, N, _LAYOUTS[layout], source, max_candidates,
                                            max_workspace, C.byref(n)), "fq_ref_gemm_bf16_prepare")
    return n.value


def candidate(M: int, K: int, N: int, layout: str, index: int) -> tuple[int, str]:
    """(workspace bytes, kernel name) of a prepared candidate."""
    ws = C.c_uint64(0)
    buf = C.create_string_buffer(512)
    _check(load().fq_ref_gemm_bf16_candidate(M, K, N, _LAYOUTS[layout], index, C.byref(ws), buf,
                                              len(buf)), "fq_ref_gemm_bf16_candidate")
    return ws.value, buf.value.decode(errors="replace")


def gemm(X, W, Y, layout: str, index: int, workspace=None, stream=None) -> None:
    """Enqueue Y = X * W (bf16 device tensors: X [M][K], W [K][N] for layout
    "kn" or [N][K] for "nk", Y [M][N]) with candidate `index` on `stream`
    (torch stream, default: current)."""
    import torch
    M, K = X.shape
    N = Y.shape[1]
    w_shape = (K, N) if layout == "kn" else (N, K)
    for t, shape in ((X, (M, K)), (W, w_shape), (Y, (M, N))):
        if t.dtype != torch.bfloat16 or tuple(t.shape) != shape or not t.is_contiguous():
            raise ValueError(f"gemm: expected a contiguous bf16 tensor of shape {shape}")
    if stream is None:
        stream = torch.cuda.current_stream(X.device)
    ws_ptr, ws_bytes = (None, 0) if workspace is None else (
        workspace.data_ptr(), workspace.numel() * workspace.element_size())
    _check(load().fq_ref_gemm_bf16(X.data_ptr(), W.data_ptr(), Y.data_ptr(), M, K, N,
                                   _LAYOUTS[layout], index, ws_ptr, ws_bytes,
                                   int(stream.cuda_stream)), "fq_ref_gemm_bf16")
