"""Pinned, device-mapped host buffers for the offloaded KV pools (HIP runtime through ctypes).

torch's pinned allocator rounds large requests up (a 34 GB pool would take 64 GB), so the pools
of the offloaded decode path are allocated with hipHostMalloc directly.  The memory is mapped
into the GPU address space, which is what the gather kernel reads over PCIe.
"""
from __future__ import annotations

import ctypes

import numpy as np
import torch

_hip = None
HIP_HOST_MALLOC_MAPPED = 0x2
HIP_MEMCPY_HOST_TO_DEVICE = 1
HIP_MEMCPY_DEVICE_TO_HOST = 2


def _rt():
    global _hip
    if _hip is None:
        lib = ctypes.CDLL("libamdhip64.so")
        lib.hipHostMalloc.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_size_t, ctypes.c_uint]
        lib.hipHostMalloc.restype = ctypes.c_int
        lib.hipHostFree.argtypes = [ctypes.c_void_p]
        lib.hipHostFree.restype = ctypes.c_int
        lib.hipMemcpyAsync.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int, ctypes.c_void_p]
        lib.hipMemcpyAsync.restype = ctypes.c_int
        lib.hipHostGetDevicePointer.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_void_p, ctypes.c_uint]
        lib.hipHostGetDevicePointer.restype = ctypes.c_int
        _hip = lib
    return _hip


def device_pointer(host_ptr: int) -> int:
    """The device address of pinned host memory mapped for the device (hipHostMalloc'd, including
    torch's pinned tensors)."""
    d = ctypes.c_void_p()
    rc = _rt().hipHostGetDevicePointer(ctypes.byref(d), ctypes.c_void_p(host_ptr), 0)
    if rc != 0 or not d.value:
        raise RuntimeError(f"hipHostGetDevicePointer failed with {rc}")
    return int(d.value)


class PinnedBuffer:
    """`nbytes` of pinned host memory mapped into the device address space."""

    def __init__(self, nbytes: int):
        self.nbytes = int(nbytes)
        p = ctypes.c_void_p()
        rc = _rt().hipHostMalloc(ctypes.byref(p), self.nbytes, HIP_HOST_MALLOC_MAPPED)
        if rc != 0 or not p.value:
            raise MemoryError(f"hipHostMalloc({self.nbytes}) failed with {rc}")
        self.ptr = int(p.value)

    def as_tensor(self, dtype=torch.uint8) -> torch.Tensor:
        """A CPU tensor viewing the buffer (no copy)."""
        arr = np.ctypeslib.as_array(ctypes.cast(self.ptr, ctypes.POINTER(ctypes.c_uint8)), shape=(self.nbytes,))
        return torch.from_numpy(arr).view(dtype)

    def copy_from_device(self, offset: int, src: torch.Tensor, stream=None):
        """Asynchronous device -> pinned copy of `src` to byte `offset` on `stream`."""
        n = src.numel() * src.element_size()
        assert 0 <= offset and offset + n <= self.nbytes
        s = (stream or torch.cuda.current_stream()).cuda_stream
        rc = _rt().hipMemcpyAsync(self.ptr + offset, src.data_ptr(), n, HIP_MEMCPY_DEVICE_TO_HOST, s)
        if rc != 0:
            raise RuntimeError(f"hipMemcpyAsync D2H failed with {rc}")

    def copy_to_device(self, offset: int, dst: torch.Tensor, stream=None):
        """Asynchronous pinned -> device copy into `dst` from byte `offset` on `stream`."""
        n = dst.numel() * dst.element_size()
        assert 0 <= offset and offset + n <= self.nbytes
        s = (stream or torch.cuda.current_stream()).cuda_stream
        rc = _rt().hipMemcpyAsync(dst.data_ptr(), self.ptr + offset, n, HIP_MEMCPY_HOST_TO_DEVICE, s)
        if rc != 0:
            raise RuntimeError(f"hipMemcpyAsync H2D failed with {rc}")

    def free(self):
        if self.ptr:
            _rt().hipHostFree(self.ptr)
            self.ptr = 0

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass
