"""Loaders for the C host and HIP device twins of the generator.

``build()`` compiles both into this directory; the loaders only open what is
already built and raise if it is missing.
"""

from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

from . import gen

HERE = os.path.dirname(os.path.abspath(__file__))
HOST_LIB = os.path.join(HERE, "libsynth_host.so")
DEV_LIB = os.path.join(HERE, "libsynth_dev.so")

HIP_FLAGS = ["-O3", "--offload-arch=gfx950", "-ffp-contract=off", "-fPIC", "-shared",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def build(verbose: bool = False) -> None:
    src_host = os.path.join(HERE, "csrc", "synth_host.c")
    src_dev = os.path.join(HERE, "csrc", "synth_dev.hip")
    cmds = [
        ["gcc", "-O2", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared", src_host, "-o", HOST_LIB],
        ["hipcc", *HIP_FLAGS, src_dev, "-o", DEV_LIB],
    ]
    for cmd in cmds:
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)


_host = None
_dev = None


def _load_host():
    global _host
    if _host is None:
        if not os.path.exists(HOST_LIB):
            raise RuntimeError(f"{HOST_LIB} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(HOST_LIB)
        lib.synth_logits_host.restype = None
        lib.synth_logits_host.argtypes = [
            ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64,
            ctypes.c_int64, ctypes.c_uint64, ctypes.c_double, ctypes.c_void_p, ctypes.c_void_p,
            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int]
        _host = lib
    return _host


def default_threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(n, 16))


def logits_rows_host(wl: gen.Workload, rows, out: np.ndarray | None = None, nthreads: int | None = None):
    """Same values as ``gen.logits_rows_numpy`` (bit-exact), via the C twin."""
    lib = _load_host()
    rows = np.ascontiguousarray(np.asarray(rows, dtype=np.int64).reshape(-1))
    dt = np.float32 if wl.dtype == "f32" else np.uint16
    if out is None:
        out = np.empty((rows.size, wl.V), dtype=dt)
    assert out.dtype == dt and out.shape == (rows.size, wl.V) and out.flags.c_contiguous
    assert rows.size == 0 or (rows.min() >= 0 and rows.max() < wl.T)
    q = gen.normal_table()
    lib.synth_logits_host(
        out.ctypes.data, 0 if wl.dtype == "f32" else 1, rows.size, rows.ctypes.data, wl.V, wl.V,
        gen.base_key(wl.seed), wl.sigma, wl.kind.ctypes.data, wl.src_row.ctypes.data,
        wl.spike_col.ctypes.data, wl.spike_val.ctypes.data, q.ctypes.data,
        nthreads or default_threads())
    return out


def gaussian_bits_host(seed: int, stream_id: int, rows: int, cols: int, sigma: float,
                       nthreads: int | None = None) -> np.ndarray:
    """gen.gaussian_bits (bit-exact) via the C twin, for matrices too large for
    numpy's temporaries (the 152064 x 3584 LM-head weight)."""
    lib = _load_host()
    out = np.empty((rows, cols), dtype=np.uint16)
    idx = np.arange(rows, dtype=np.int64)
    kind = np.zeros(rows, np.int32)
    src_row = np.arange(rows, dtype=np.int32)
    spike_col = np.full(rows, -1, np.int32)
    spike_val = np.zeros(rows, np.float64)
    q = gen.normal_table()
    lib.synth_logits_host(out.ctypes.data, 1, rows, idx.ctypes.data, cols, cols,
                          gen.stream_key(seed, stream_id), float(sigma), kind.ctypes.data,
                          src_row.ctypes.data, spike_col.ctypes.data, spike_val.ctypes.data,
                          q.ctypes.data, nthreads or default_threads())
    return out


def _load_dev():
    global _dev
    if _dev is None:
        if not os.path.exists(DEV_LIB):
            raise RuntimeError(f"{DEV_LIB} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(DEV_LIB)
        lib.synth_logits_device.restype = ctypes.c_int
        lib.synth_logits_device.argtypes = [
            ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64,
            ctypes.c_uint64, ctypes.c_double, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
        _dev = lib
    return _dev


class DeviceRecipe:
    """The per-row recipe arrays of a workload, resident on the GPU (torch tensors)."""

    def __init__(self, wl: gen.Workload, device="cuda"):
        import torch

        self.wl = wl
        self.kind = torch.from_numpy(wl.kind).to(device)
        self.src_row = torch.from_numpy(wl.src_row).to(device)
        self.spike_col = torch.from_numpy(wl.spike_col).to(device)
        self.spike_val = torch.from_numpy(wl.spike_val).to(device)
        self.Q = torch.from_numpy(np.array(gen.normal_table())).to(device)


def fill_gaussian_device(out, seed: int, stream_id: int, sigma: float, stream=None) -> None:
    """Fill the bf16 device tensor ``out`` [rows, cols] with gen.gaussian_bits
    (seed, stream_id, rows, cols, sigma), bit for bit, with the logits kernel:
    every row Gaussian, no spike, the stream folded into the key."""
    import torch

    if out.dtype != torch.bfloat16 or out.dim() != 2 or out.stride(1) != 1:
        raise ValueError("out must be a 2-D bfloat16 tensor with contiguous rows")
    rows, cols = out.shape
    dev = out.device
    kind = torch.zeros(rows, dtype=torch.int32, device=dev)
    src_row = torch.arange(rows, dtype=torch.int32, device=dev)
    spike_col = torch.full((rows,), -1, dtype=torch.int32, device=dev)
    spike_val = torch.zeros(rows, dtype=torch.float64, device=dev)
    Q = torch.from_numpy(np.array(gen.normal_table())).to(dev)
    if stream is None:
        stream = torch.cuda.current_stream().cuda_stream
    rc = _load_dev().synth_logits_device(
        out.data_ptr(), 1, rows, cols, out.stride(0), gen.stream_key(seed, stream_id), float(sigma),
        kind.data_ptr(), src_row.data_ptr(), spike_col.data_ptr(), spike_val.data_ptr(),
        Q.data_ptr(), stream)
    if rc != 0:
        raise RuntimeError(f"synth_logits_device failed with code {rc}")


def fill_logits_device(recipe: DeviceRecipe, out, stream=None) -> None:
    """Fill the torch device tensor ``out`` ([T, ld], float32 or bfloat16) with
    the workload's logits on ``stream`` (default: torch's current stream)."""
    import torch

    wl = recipe.wl
    lib = _load_dev()
    want = torch.float32 if wl.dtype == "f32" else torch.bfloat16
    if out.dtype != want or out.dim() != 2 or out.shape[0] != wl.T or out.shape[1] < wl.V:
        raise ValueError("output tensor does not match the workload")
    if out.stride(1) != 1:
        raise ValueError("output rows must be contiguous")
    if stream is None:
        stream = torch.cuda.current_stream().cuda_stream
    rc = lib.synth_logits_device(
        out.data_ptr(), 0 if wl.dtype == "f32" else 1, wl.T, wl.V, out.stride(0),
        gen.base_key(wl.seed), wl.sigma, recipe.kind.data_ptr(), recipe.src_row.data_ptr(),
        recipe.spike_col.data_ptr(), recipe.spike_val.data_ptr(), recipe.Q.data_ptr(), stream)
    if rc != 0:
        raise RuntimeError(f"synth_logits_device failed with code {rc}")
