"""Binding of libfqprobe.so, the streaming-read probe declared in
include/fq_probe.h (a measurement reference for the matmul kernels; argument
marshalling only).  Raises if the library has not been built."""

from __future__ import annotations

import ctypes as C
import os
import threading

_HERE = os.path.dirname(os.path.abspath(__file__))
PROBE_LIB_PATH = os.path.join(_HERE, "libfqprobe.so")
EXPORTS = ("fq_probe_stream_read", "fq_probe_workgroup_xcd", "fq_probe_tile_loads",
           "fq_probe_strip_loads")
FQ_PROBE_SCALES, FQ_PROBE_ZEROS, FQ_PROBE_X, FQ_PROBE_GROUPS, FQ_PROBE_MASKED = 1, 2, 4, 8, 16

_lib = None
_lock = threading.Lock()


def load() -> C.CDLL:
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(PROBE_LIB_PATH):
                raise ImportError(f"libfqprobe.so is not built ({PROBE_LIB_PATH}); run "
                                  "paper_2608_15531_amd.build.build() first")
            lib = C.CDLL(PROBE_LIB_PATH)
            lib.fq_probe_stream_read.argtypes = [C.c_void_p, C.c_size_t, C.c_int32, C.c_int32,
                                                 C.c_int32, C.c_void_p, C.c_void_p]
            lib.fq_probe_stream_read.restype = C.c_int
            lib.fq_probe_workgroup_xcd.argtypes = [C.c_void_p, C.c_int32, C.c_int32, C.c_void_p]
            lib.fq_probe_workgroup_xcd.restype = C.c_int
            lib.fq_probe_tile_loads.argtypes = [C.c_void_p] * 5 + [C.c_int32, C.c_int32, C.c_int32,
                                                                   C.c_uint32, C.c_void_p, C.c_void_p]
            lib.fq_probe_tile_loads.restype = C.c_int
            lib.fq_probe_strip_loads.argtypes = [C.c_void_p] * 3 + [C.c_int32] * 6 + [
                C.c_void_p, C.c_void_p]
            lib.fq_probe_strip_loads.restype = C.c_int
            _lib = lib
    return _lib


def fq_probe_stream_read(src, nbytes: int, workgroups: int, waves: int, loads_in_flight: int,
                         sink, stream=None) -> None:
    """Enqueue one streaming read of nbytes of the device tensor src on
    `stream` (torch stream, default: current).  sink: device tensor of at
    least `workgroups` int32 words."""
    import torch
    if nbytes > src.numel() * src.element_size() or sink.numel() * sink.element_size() < 4 * workgroups:
        raise ValueError("fq_probe_stream_read: buffer too small")
    if stream is None:
        stream = torch.cuda.current_stream(src.device)
    rc = load().fq_probe_stream_read(src.data_ptr(), nbytes, workgroups, waves,
                                     loads_in_flight, sink.data_ptr(), int(stream.cuda_stream))
    if rc != 0:
        raise RuntimeError(f"fq_probe_stream_read failed ({rc})")


def fq_probe_workgroup_xcd(out, workgroups: int, threads: int, stream=None) -> None:
    """Enqueue the XCD-placement probe: out (device int32 tensor of at least
    `workgroups` words) receives the XCD each workgroup ran on."""
    import torch
    if out.numel() * out.element_size() < 4 * workgroups:
        raise ValueError("fq_probe_workgroup_xcd: buffer too small")
    if stream is None:
        stream = torch.cuda.current_stream(out.device)
    rc = load().fq_probe_workgroup_xcd(out.data_ptr(), workgroups, threads, int(stream.cuda_stream))
    if rc != 0:
        raise RuntimeError(f"fq_probe_workgroup_xcd failed ({rc})")


def fq_probe_tile_loads(codes, scales, zeros, x, groups, K: int, N: int, groups_per_tile: int,
                        extra: int, sink, stream=None) -> None:
    """Enqueue the per-tile load probe (see include/fq_probe.h) on device
    tensors; sink: device tensor of at least N / 64 int32 words."""
    import torch
    if (codes.numel() * codes.element_size() < K * N // 2
            or sink.numel() * sink.element_size() < 4 * (N // 64)
            or groups.numel() * groups.element_size() < 16 * groups_per_tile * (K // 128) * (N // 64)
            or x.numel() * x.element_size() < 2 * K):
        raise ValueError("fq_probe_tile_loads: buffer too small")
    if stream is None:
        stream = torch.cuda.current_stream(codes.device)
    rc = load().fq_probe_tile_loads(codes.data_ptr(), scales.data_ptr(), zeros.data_ptr(),
                                    x.data_ptr(), groups.data_ptr(), K, N, groups_per_tile,
                                    extra, sink.data_ptr(), int(stream.cuda_stream))
    if rc != 0:
        raise RuntimeError(f"fq_probe_tile_loads failed ({rc})")


def fq_probe_strip_loads(codes, x, groups, K: int, N: int, strip_cols: int, waves: int,
                         split: int, groups_per_tile: int, sink, stream=None) -> None:
    """Enqueue the strip-width load probe (see include/fq_probe.h) on device
    tensors; sink: device tensor of at least (N / strip_cols) * split int32
    words."""
    import torch
    T = K // 128
    if (codes.numel() * codes.element_size() < K * N // 2
            or x.numel() * x.element_size() < 2 * K
            or groups.numel() * groups.element_size() < 16 * groups_per_tile * T * (N // 64)
            or sink.numel() * sink.element_size() < 4 * (N // max(1, strip_cols)) * split):
        raise ValueError("fq_probe_strip_loads: buffer too small")
    if stream is None:
        stream = torch.cuda.current_stream(codes.device)
    rc = load().fq_probe_strip_loads(codes.data_ptr(), x.data_ptr(), groups.data_ptr(), K, N,
                                     strip_cols, waves, split, groups_per_tile, sink.data_ptr(),
                                     int(stream.cuda_stream))
    if rc != 0:
        raise RuntimeError(f"fq_probe_strip_loads failed ({rc})")
