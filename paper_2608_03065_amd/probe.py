"""Binding of libpsc_probe.so (a measurement aid, not part of the mask path):
the latency of the classifier walk's dependent loads against the table's
size, in a given launch shape.  Argument marshalling only; the chain runs in
psc_probe_chase."""
from __future__ import annotations

import ctypes as C
import os

HERE = os.path.dirname(os.path.abspath(__file__))
PROBE_LIB_PATH = os.path.join(HERE, "libpsc_probe.so")
WAVE_LOAD, SCALAR_LOAD = 0, 1
ROW_INTS = 256

_lib = None


def lib() -> C.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(PROBE_LIB_PATH):
            raise ImportError(f"{PROBE_LIB_PATH} is missing: run __graft_entry__.build() first")
        L = C.CDLL(PROBE_LIB_PATH)
        L.psc_probe_chase.argtypes = [C.c_int32, C.c_void_p, C.c_void_p, C.c_int32, C.c_int32, C.c_int32,
                                      C.c_int32, C.c_int32, C.c_uint32, C.c_void_p]
        L.psc_probe_chase.restype = C.c_int
        _lib = L
    return _lib


def chase(mode, out, table, n_rows, k, fill, grid, seed, stream) -> None:
    """One launch of psc_probe_chase; raises on a nonzero hipError_t."""
    rc = lib().psc_probe_chase(int(mode), out.data_ptr() if out is not None else None, table.data_ptr(),
                               int(n_rows), int(k), int(fill), int(grid[0]), int(grid[1]), int(seed) & 0xFFFFFFFF,
                               C.c_void_p(stream.cuda_stream))
    if rc != 0:
        raise RuntimeError(f"psc_probe_chase: hipError_t {rc}")


def _device_delay(stream):
    """A function that queues a device-side delay of about n launches on
    `stream`, so that a timed loop is queued whole before its first event
    fires and the host's launch rate stays out of it."""
    import torch
    a, z = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(stream):
        torch.cuda._sleep(1000)
        a.record(stream)
        torch.cuda._sleep(1 << 20)
        z.record(stream)
    torch.cuda.synchronize()
    cycles_per_us = (1 << 20) / max(a.elapsed_time(z) * 1e3, 1.0)

    def delay(n):
        with torch.cuda.stream(stream):
            torch.cuda._sleep(int(min(100.0 + 20.0 * n, 60000.0) * cycles_per_us))
    return delay


def chase_latency(device, stream, grid, sizes_mb=(1, 16, 128, 256, 512, 1024), k=8, launches=500) -> dict:
    """ns per dependent load, (t(k) - t(0)) / k over `launches` back-to-back
    launches, each starting its chains at other rows (a new seed per launch),
    for each table size and load path, with and without the store stream."""
    import torch
    gx, gy = grid
    prequeue = _device_delay(stream)
    out = torch.empty(gx * gy * 16384, dtype=torch.uint8, device=device)
    gen = torch.Generator(device=device).manual_seed(0x9E37)
    res = {}
    for mb in sizes_mb:
        n_rows = mb * 1024
        tab = torch.randint(-2**31, 2**31 - 1, (n_rows * ROW_INTS,), generator=gen, dtype=torch.int32, device=device)

        def timed(mode, kk, fill):
            with torch.cuda.stream(stream):
                for j in range(10):
                    chase(mode, out, tab, n_rows, kk, fill, grid, 1_000_000 + j, stream)
                torch.cuda.synchronize()
                prequeue(launches)
                a, z = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record(stream)
                for j in range(launches):
                    chase(mode, out, tab, n_rows, kk, fill, grid, j + 1, stream)
                z.record(stream)
                torch.cuda.synchronize()
            return a.elapsed_time(z) / launches * 1e3

        for mode, name in ((WAVE_LOAD, "wave_1KiB"), (SCALAR_LOAD, "scalar_8B")):
            row = {}
            for fill in (1, 0):
                t0, tk = timed(mode, 0, fill), timed(mode, k, fill)
                tag = "with_stores" if fill else "no_stores"
                row[tag] = {"launch_us_k0": round(t0, 3), f"launch_us_k{k}": round(tk, 3),
                            "ns_per_load": round((tk - t0) / k * 1e3, 1)}
            res[f"{mb}MiB_{name}"] = row
        del tab
        torch.cuda.empty_cache()
    return res
