"""The benchmark's measurement helpers: a register-only bf16 MFMA loop that
gives the sustained matrix-core rate of the part, the practical ceiling the
attention kernel is compared with beside the data-sheet peak, and unit probes
of the exponential, FMA and 16-byte LDS read issue rates.

It is not a step of the method: it lives in its own library,
libmfma_probe.so (built from mfma_probe.hip next to this file by the
package's build step), outside libsparsp and its C ABI.
"""

from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(_HERE, "libmfma_probe.so")
_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            raise RuntimeError(f"{LIB} is not built; run python -m paper_2609_32197_amd.build")
        _lib = ctypes.CDLL(LIB)
        _lib.mfma_probe_run.argtypes = [ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p,
                                        ctypes.c_void_p]
        _lib.mfma_probe_run.restype = ctypes.c_int
        _lib.unit_probe_run.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.c_int32,
                                        ctypes.c_void_p, ctypes.c_void_p]
        _lib.unit_probe_run.restype = ctypes.c_int
    return _lib


def run(iters: int, workgroups: int, sink, stream=None) -> None:
    """Enqueue workgroups * iters * 524,288 FLOP of register-only bf16 MFMA work;
    sink: float32 cuda tensor of at least workgroups * 256 elements."""
    import torch
    if sink.numel() < int(workgroups) * 256 or sink.dtype != torch.float32 or not sink.is_cuda:
        raise ValueError("sink must be a float32 cuda tensor of workgroups * 256 elements")
    st = stream if stream is not None else torch.cuda.current_stream(sink.device)
    rc = _load().mfma_probe_run(int(iters), int(workgroups), sink.data_ptr(), st.cuda_stream)
    if rc != 0:
        raise RuntimeError(f"mfma probe failed with status {rc}")


def status(iters: int, workgroups: int, sink_ptr) -> int:
    """The raw return code for the given arguments (argument checks only: the
    rejected cases launch nothing)."""
    return int(_load().mfma_probe_run(int(iters), int(workgroups), sink_ptr, None))


UNIT_KINDS = {"exp": 0, "fma": 1, "lds": 2}


def run_unit(kind: str, iters: int, workgroups: int, sink, stream=None) -> None:
    """Enqueue one unit probe ("exp", "fma": 16 instructions per wave and
    iteration; "lds": 32 ds_read_b128 per wave and iteration)."""
    import torch
    if sink.numel() < int(workgroups) * 256 or sink.dtype != torch.float32 or not sink.is_cuda:
        raise ValueError("sink must be a float32 cuda tensor of workgroups * 256 elements")
    st = stream if stream is not None else torch.cuda.current_stream(sink.device)
    rc = _load().unit_probe_run(UNIT_KINDS[kind], int(iters), int(workgroups), sink.data_ptr(),
                                st.cuda_stream)
    if rc != 0:
        raise RuntimeError(f"unit probe {kind} failed with status {rc}")
