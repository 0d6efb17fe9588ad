"""Seeded synthetic inputs shared by the oracle side and the HIP side.

Holds no part of the KV transfer method: it fills flat byte ranges of named
streams (see synth_host.c for the definition: a counter-based splitmix64 stream
mapped to bf16 N(0,1) through a quantile table, or raw bytes). A KV-cache
tensor for layer l, K or V, is the stream ``cache_stream(role, l, kv)``; the
content of block b is that stream's bytes at offset ``b * slab_bytes``, so a
host mirror of any subset of blocks can be regenerated without a full copy.

Host fills run in C (``libkvsynth_host.so``); device fills run a small HIP
kernel (``libkvsynth_dev.so``) that implements the same definition.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

MODE_NORMAL_BF16 = 0
MODE_RAW = 1

_HERE = os.path.dirname(os.path.abspath(__file__))
HOST_LIB = os.path.join(_HERE, "libkvsynth_host.so")
DEV_LIB = os.path.join(_HERE, "libkvsynth_dev.so")

_host = None
_dev = None
_dev_tables = {}


def _host_lib():
    global _host
    if _host is None:
        if not os.path.exists(HOST_LIB):
            raise RuntimeError(f"{HOST_LIB} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(HOST_LIB)
        lib.kvs_stream_key.restype = ctypes.c_uint64
        lib.kvs_stream_key.argtypes = [ctypes.c_uint64, ctypes.c_uint64]
        lib.kvs_word.restype = ctypes.c_uint64
        lib.kvs_word.argtypes = [ctypes.c_uint64, ctypes.c_uint64]
        lib.kvs_normal_table.restype = ctypes.POINTER(ctypes.c_uint16)
        lib.kvs_normal_table.argtypes = []
        lib.kvs_fill_ranges.restype = ctypes.c_int
        lib.kvs_fill_ranges.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint64,
                                        ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64,
                                        ctypes.c_int, ctypes.c_int]
        lib.kvs_fill_host.restype = ctypes.c_int
        lib.kvs_fill_host.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint64,
                                      ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int, ctypes.c_int]
        _host = lib
    return _host


def _dev_lib():
    global _dev
    if _dev is None:
        if not os.path.exists(DEV_LIB):
            raise RuntimeError(f"{DEV_LIB} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(DEV_LIB)
        lib.kvs_fill_device.restype = ctypes.c_int
        lib.kvs_fill_device.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint64,
                                        ctypes.c_uint64, ctypes.c_int, ctypes.c_void_p,
                                        ctypes.c_void_p]
        _dev = lib
    return _dev


# ---- stream naming ---------------------------------------------------------

ROLE_SRC = 1      # cache blocks that hold prefix KV before a gather
ROLE_DST = 2      # background content of the cache (free / untouched blocks)
ROLE_IMAGE = 3    # a packed transfer image (restore input)
ROLE_NEW = 4      # newly computed blocks (batched offload)


def cache_stream(role: int, layer: int, kv: int, tag: int = 0) -> int:
    """Stream id of the cache tensor (layer, K=0 / V=1) under a role."""
    return (0x4B56 << 48) | ((tag & 0xFFFF) << 32) | ((role & 0xFF) << 24) | (layer << 1) | kv


def image_stream(tag: int = 0) -> int:
    return (0x494D << 48) | ((tag & 0xFFFF) << 32) | (ROLE_IMAGE << 24)


def stream_key(seed: int, stream: int) -> int:
    return int(_host_lib().kvs_stream_key(seed & (2**64 - 1), stream & (2**64 - 1)))


def word(key: int, w: int) -> int:
    return int(_host_lib().kvs_word(key, w))


def normal_table() -> np.ndarray:
    p = _host_lib().kvs_normal_table()
    return np.ctypeslib.as_array(p, shape=(65536,)).copy()


def fill_host(buf: np.ndarray, seed: int, stream: int, byte_offset: int = 0,
              mode: int = MODE_NORMAL_BF16, threads: int = 8) -> None:
    """Fill a C-contiguous host array with stream bytes [byte_offset, +nbytes)."""
    if not buf.flags["C_CONTIGUOUS"]:
        raise ValueError("fill_host needs a C-contiguous array")
    rc = _host_lib().kvs_fill_host(buf.ctypes.data, buf.nbytes, seed & (2**64 - 1),
                                   stream & (2**64 - 1), byte_offset, mode, threads)
    if rc != 0:
        raise ValueError(f"kvs_fill_host rejected nbytes={buf.nbytes} offset={byte_offset}")


def fill_ranges(buf: np.ndarray, offsets, length: int, seed: int, stream: int,
                mode: int = MODE_NORMAL_BF16, threads: int = 8) -> None:
    """For each offset o: buf[o:o+length] = stream bytes [o, o+length)."""
    offs = np.ascontiguousarray(np.asarray(offsets, dtype=np.uint64))
    if offs.size and int(offs.max()) + length > buf.nbytes:
        raise ValueError("range past the end of the buffer")
    if not buf.flags["C_CONTIGUOUS"]:
        raise ValueError("fill_ranges needs a C-contiguous array")
    rc = _host_lib().kvs_fill_ranges(buf.ctypes.data, offs.ctypes.data, offs.size, length,
                                     seed & (2**64 - 1), stream & (2**64 - 1), mode, threads)
    if rc != 0:
        raise ValueError("kvs_fill_ranges rejected its arguments")


def host_bytes(nbytes: int, seed: int, stream: int, byte_offset: int = 0,
               mode: int = MODE_NORMAL_BF16, threads: int = 8) -> np.ndarray:
    out = np.empty(nbytes, dtype=np.uint8)
    fill_host(out, seed, stream, byte_offset, mode, threads)
    return out


def fill_device(t, seed: int, stream: int, byte_offset: int = 0,
                mode: int = MODE_NORMAL_BF16, hip_stream: int | None = None) -> None:
    """Fill a contiguous device tensor (torch, on a GPU) with stream bytes."""
    import torch

    if not t.is_contiguous() or not t.is_cuda:
        raise ValueError("fill_device needs a contiguous GPU tensor")
    dev = t.device.index if t.device.index is not None else torch.cuda.current_device()
    tab = _dev_tables.get(dev)
    if tab is None:
        tab = torch.from_numpy(normal_table().view(np.int16)).to(f"cuda:{dev}")
        _dev_tables[dev] = tab
    if hip_stream is None:
        hip_stream = torch.cuda.current_stream(dev).cuda_stream
    nbytes = t.numel() * t.element_size()
    rc = _dev_lib().kvs_fill_device(t.data_ptr(), nbytes, stream_key(seed, stream), byte_offset,
                                    mode, tab.data_ptr(), hip_stream)
    if rc != 0:
        raise RuntimeError(f"kvs_fill_device failed with hip error {rc}")
