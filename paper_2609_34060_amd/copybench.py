"""Copy ceilings beside the apply (measurement only): plain copies with the apply's 16-byte accesses, timed with HIP
events on the stream they run on.  The kernels are in csrc/kvc_copybench.hip (libkvc_copybench.so)."""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional

import numpy as np
import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libkvc_copybench.so")
_lib = None


def load() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with paper_2609_34060_amd/build.py")
        lib = ctypes.CDLL(LIB_PATH)
        vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
        for name, args in (("kvcb_copy", [vp, vp, i64, i32, i32, vp]),
                           ("kvcb_read", [vp, i64, i32, i32, ctypes.c_uint32, vp, vp]),
                           ("kvcb_write", [vp, i64, i32, i32, ctypes.c_uint32, vp]),
                           ("kvcb_paged_blocks", [vp, vp, vp, vp, vp, i32, i32, i32, vp]),
                           ("kvcb_paged_heads", [vp, vp, vp, vp, i32, i32, i32, i32, i32, i32, i32, vp])):
            getattr(lib, name).restype = ctypes.c_int
            getattr(lib, name).argtypes = args
        _lib = lib
    return _lib


def _time(launch, reps: int, warmup: int = 2) -> float:
    """Mean milliseconds of `launch` over `reps` launches (HIP events on the current stream)."""
    for _ in range(warmup):
        launch()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(reps):
        launch()
    end.record()
    end.synchronize()
    return start.elapsed_time(end) / reps


def _check(rc: int, what: str) -> None:
    if rc != 0:
        raise RuntimeError(f"{what}: hipError {rc}")


def xcd_blocked(n: int, per_wg: int = 1) -> np.ndarray:
    """A work order in which the workgroups of each XCD (workgroup i runs on XCD i mod 8) take one contiguous eighth
    of the slots 0 .. n - 1, per_wg slots per workgroup."""
    wgs = -(-n // per_wg)
    out = np.empty(wgs * per_wg, dtype=np.int64)
    per_xcd = -(-wgs // 8)
    for w in range(wgs):
        src = (w % 8) * per_xcd + w // 8
        out[w * per_wg:(w + 1) * per_wg] = np.arange(src * per_wg, (src + 1) * per_wg)
    out = out[out < n]
    if len(out) != n or len(np.unique(out)) != n:   # an uneven split: fall back to the identity
        return np.arange(n)
    return out


def ceilings(device: str = "cuda", gib: float = 4.0, reps: int = 10, seed: int = 5) -> Dict[str, dict]:
    """GB/s of each copy pattern moving `gib` GiB read + `gib` GiB written (read-only / write-only: `gib` GiB).

    Paged patterns use one pool of 32 KiB blocks (16 tokens x 8 KV heads x 128 bf16 features, the benchmark's block)
    with the source and destination sequences on disjoint, seeded random block sets."""
    lib = load()
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    n16 = int(gib * 2 ** 30) // 16
    out: Dict[str, dict] = {}

    def record(name, ms, moved):
        out[name] = {"ms": round(ms, 4), "gbps": round(moved / ms / 1e6, 1), "frac": round(moved / ms / 1e6 / 8000, 4)}

    a = torch.empty(n16 * 16, dtype=torch.uint8, device=device)
    b = torch.empty_like(a)
    a.random_(0, 255)
    sink = torch.zeros(1, dtype=torch.int32, device=device)
    wgs = 256 * 8
    for name, mode in (("contiguous_gridstride", 0), ("contiguous_chunked", 1), ("contiguous_xcd", 2)):
        ms = _time(lambda: _check(lib.kvcb_copy(a.data_ptr(), b.data_ptr(), n16, wgs, mode, stream), name), reps)
        record(name, ms, 2 * n16 * 16)
    ms = _time(lambda: _check(lib.kvcb_read(a.data_ptr(), n16, wgs, 1, 0xDEADBEEF, sink.data_ptr(), stream),
                              "read"), reps)
    record("read_only_xcd", ms, n16 * 16)
    ms = _time(lambda: _check(lib.kvcb_write(b.data_ptr(), n16, wgs, 1, 7, stream), "write"), reps)
    record("write_only_xcd", ms, n16 * 16)
    del a, b

    block_bytes = 16 * 8 * 256
    nblk = int(gib * 2 ** 30) // block_bytes
    pool = torch.empty(2 * nblk * block_bytes, dtype=torch.uint8, device=device)
    rng = np.random.Generator(np.random.PCG64(seed))
    perm = rng.permutation(2 * nblk).astype(np.int32)
    st_np, dt_np = perm[:nblk], perm[nblk:]
    st = torch.from_numpy(st_np).to(device)
    dt = torch.from_numpy(dt_np).to(device)
    orders = {"logical": np.arange(nblk), "logical_xcd": xcd_blocked(nblk),
              "src_sorted": np.argsort(st_np, kind="stable"), "dst_sorted": np.argsort(dt_np, kind="stable")}
    orders["src_sorted_xcd"] = orders["src_sorted"][xcd_blocked(nblk)]
    orders["dst_sorted_xcd"] = orders["dst_sorted"][xcd_blocked(nblk)]
    for oname, order in orders.items():
        od = torch.from_numpy(np.ascontiguousarray(order, dtype=np.int32)).to(device)
        for per in (1, 4):
            name = f"paged_blocks_{oname}_x{per}"
            ms = _time(lambda: _check(lib.kvcb_paged_blocks(pool.data_ptr(), pool.data_ptr(), st.data_ptr(),
                                                            dt.data_ptr(), od.data_ptr(), nblk, per,
                                                            block_bytes // 16, stream), name), reps)
            record(name, ms, 2 * nblk * block_bytes)
    ms = _time(lambda: _check(lib.kvcb_paged_heads(pool.data_ptr(), pool.data_ptr(), st.data_ptr(), dt.data_ptr(),
                                                   nblk * 16, 8, 1024, 16, block_bytes // 16, 8 * 16, 16, stream),
                              "paged_heads"), reps)
    record("paged_heads_1024", ms, 2 * nblk * block_bytes)
    torch.cuda.synchronize()
    return out
