"""Binding of libasymspec_probe.so: the read-ceiling probe.

A plain read-reduce kernel that streams one device buffer with the same
16-byte non-temporal loads as the decision kernel; its rate over a buffer far
larger than the caches is the practical HBM read ceiling, reported beside the
decision kernel's achieved bandwidth.  Not part of the decision step.
"""

from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
PROBE_PATH = os.path.join(HERE, "libasymspec_probe.so")
E_ARG = -1
E_DEVICE = -2
MAX_BLOCKS = 1 << 20

_lib = None


def load_library():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(PROBE_PATH):
        raise ImportError(f"{PROBE_PATH} is missing: build it with `python -m paper_2608_26004_amd.build`")
    lib = ctypes.CDLL(PROBE_PATH)
    lib.asymspec_probe_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p,
                                        ctypes.c_int, ctypes.c_void_p]
    lib.asymspec_probe_read.restype = ctypes.c_int
    lib.asymspec_probe_clock.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_uint32, ctypes.c_void_p]
    lib.asymspec_probe_clock.restype = ctypes.c_int
    _lib = lib
    return lib


def read_xor(buf, out, nblocks: int, stream=None) -> None:
    """Enqueue one read of every byte of the contiguous device tensor `buf`
    into per-workgroup XORs out[0:nblocks] (an int32 device tensor); on
    torch's current stream unless `stream` (a torch stream) is given."""
    import torch
    if not (buf.is_cuda and out.is_cuda and buf.is_contiguous() and out.is_contiguous()):
        raise ValueError("buf and out must be contiguous device tensors")
    if out.dtype != torch.int32 or out.numel() < nblocks:
        raise ValueError("out must be int32 with at least nblocks elements")
    s = stream if stream is not None else torch.cuda.current_stream(buf.device)
    st = load_library().asymspec_probe_read(
        ctypes.c_void_p(buf.data_ptr()), buf.numel() * buf.element_size(),
        ctypes.c_void_p(out.data_ptr()), int(nblocks), ctypes.c_void_p(s.cuda_stream))
    if st != 0:
        raise RuntimeError(f"asymspec_probe_read failed with status {st}")


def read_ceiling(nbytes: int = 1 << 31, grids=(2048, 4096, 8192, 16384), reps: int = 10,
                 device=None) -> dict:
    """Median read rate of the probe over an nbytes buffer for each grid size
    (HIP events on the launching stream); the best grid is the ceiling."""
    import numpy as np
    import torch
    dev = device or torch.device("cuda")
    buf = torch.empty(nbytes // 2, dtype=torch.int16, device=dev)
    out = torch.empty(max(grids), dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream(dev)
    best = None
    per_grid = {}
    for nb in grids:
        for _ in range(3):
            read_xor(buf, out, nb, stream)
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(reps)]
        for a, b in ev:
            a.record(stream)
            read_xor(buf, out, nb, stream)
            b.record(stream)
        torch.cuda.synchronize(dev)
        ms = float(np.median([a.elapsed_time(b) for a, b in ev]))
        gbs = nbytes / (ms * 1e-3) / 1e9
        per_grid[nb] = gbs
        if best is None or gbs > best[1]:
            best = (nb, gbs, ms)
    del buf, out
    return {"GBps": best[1], "bytes": nbytes, "nblocks": best[0], "ms": best[2],
            "per_grid_GBps": per_grid}


def clock_mhz(device=None, nblocks: int = 256, ticks: int = 2000) -> dict:
    """Core clock in MHz, sampled by nblocks single-wave workgroups that each
    wait `ticks` ticks (10 ns each) of the real-time counter: mean, min and
    max over the workgroups.  Synchronises the device."""
    import numpy as np
    import torch
    dev = device or torch.device("cuda")
    out = torch.zeros(2 * nblocks, dtype=torch.int32, device=dev)
    s = torch.cuda.current_stream(dev)
    st = load_library().asymspec_probe_clock(ctypes.c_void_p(out.data_ptr()), int(nblocks),
                                             int(ticks), ctypes.c_void_p(s.cuda_stream))
    if st != 0:
        raise RuntimeError(f"asymspec_probe_clock failed with status {st}")
    w = out.cpu().numpy().view(np.uint32).astype(np.float64).reshape(nblocks, 2)
    mhz = 100.0 * w[:, 0] / np.maximum(w[:, 1], 1.0)
    return {"mean": float(mhz.mean()), "min": float(mhz.min()), "max": float(mhz.max())}
