"""CPU oracle for the paged-KV gather / scatter / staged-restore path.

TEST INFRASTRUCTURE ONLY: only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package. The product path
(``paper_2609_11744_amd``) never imports it, and it imports nothing from there.

Two independent implementations of the same definitions:
  * O2, ``gather`` / ``scatter``: plain C slab memcpy (kvx_oracle.c), the one
    timed as the CPU baseline;
  * O1, ``gather_elementwise`` / ``scatter_elementwise``: Python loops over
    every element (elementwise.py), for tiny shapes.

``restore`` is defined as the scatter of the whole packed image: splitting the
transfer into bounded staging pieces (Sec. 6.4) must not change the result.

Host mirrors: a cache is two lists (K, V) of per-layer 1-D uint8 numpy arrays
of num_blocks * slab_bytes bytes each.

Parity: pinned by the paper's printed size figures (Sec. 2.1, Sec. 6.4), by
the reduction of special cases to plain memcpy / numpy indexing, by the
round-trip, relabelling, untouched-bytes, chunk-size and layer-split
invariants, and by O1 == O2 brute force on tiny shapes (tests/test_oracle_pins.py).
"""
from __future__ import annotations

import ctypes
import dataclasses
import os

import numpy as np

from .elementwise import gather_elementwise, scatter_elementwise  # noqa: F401

_HERE = os.path.dirname(os.path.abspath(__file__))
# KVX_ORACLE_LIB lets the mutation tests load a deliberately broken build of
# kvx_oracle.c in a child process; nothing else sets it.
LIB_PATH = os.environ.get("KVX_ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")

OK, EINVAL, EBADBLOCK = 0, -1, -4


LAYOUT_NHD, LAYOUT_HND, LAYOUT_PAGED_ATTN = 0, 1, 2


class _Shape(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in
                ("num_layers", "num_blocks", "block_size", "kv_heads", "head_dim", "elem_bytes",
                 "layout")]


@dataclasses.dataclass(frozen=True)
class Shape:
    num_layers: int
    num_blocks: int
    block_size: int
    kv_heads: int
    head_dim: int
    elem_bytes: int = 2
    layout: int = LAYOUT_NHD

    @property
    def row_bytes(self) -> int:
        return self.kv_heads * self.head_dim * self.elem_bytes

    @property
    def slab_bytes(self) -> int:
        return self.block_size * self.row_bytes

    def _c(self) -> _Shape:
        return _Shape(self.num_layers, self.num_blocks, self.block_size, self.kv_heads,
                      self.head_dim, self.elem_bytes, self.layout)


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(LIB_PATH)
        i64, vp = ctypes.c_int64, ctypes.c_void_p
        lib.kvo_bytes_per_token.restype = i64
        lib.kvo_bytes_per_token.argtypes = [i64, i64, i64, i64]
        lib.kvo_packed_bytes.restype = i64
        lib.kvo_packed_bytes.argtypes = [ctypes.POINTER(_Shape), i64, i64, i64]
        for name in ("kvo_gather", "kvo_scatter"):
            f = getattr(lib, name)
            f.restype = ctypes.c_int
            f.argtypes = [ctypes.POINTER(_Shape), ctypes.POINTER(vp), ctypes.POINTER(vp), i64, i64,
                          vp, i64, i64, vp]
        _lib = lib
    return _lib


def bytes_per_token(layers: int, kv_heads: int, head_dim: int, elem_bytes: int) -> int:
    """Size model of Sec. 2.1."""
    return int(_load().kvo_bytes_per_token(layers, kv_heads, head_dim, elem_bytes))


def packed_bytes(shape: Shape, l0: int, l1: int, n_blocks: int) -> int:
    s = shape._c()
    return int(_load().kvo_packed_bytes(ctypes.byref(s), l0, l1, n_blocks))


def _ptrs(bufs):
    arr = (ctypes.c_void_p * len(bufs))()
    for i, b in enumerate(bufs):
        if not b.flags["C_CONTIGUOUS"]:
            raise ValueError("mirror arrays must be C-contiguous")
        arr[i] = b.ctypes.data
    return arr


def _bt(block_table):
    bt = np.ascontiguousarray(np.asarray(block_table, dtype=np.int32))
    return bt, (bt.ctypes.data if bt.size else None)


def gather(shape: Shape, k, v, l0: int, l1: int, block_table, chunk_tokens: int,
           out: np.ndarray | None = None) -> np.ndarray:
    """O2 gather into a new (or given) uint8 array of packed_bytes bytes."""
    bt, btp = _bt(block_table)
    nbytes = packed_bytes(shape, l0, l1, bt.size) if l1 >= l0 else 0
    if out is None:
        out = np.empty(max(nbytes, 0), dtype=np.uint8)
    if out.nbytes < nbytes:
        raise ValueError("output too small")
    s = shape._c()
    rc = _load().kvo_gather(ctypes.byref(s), _ptrs(k), _ptrs(v), l0, l1, btp, bt.size,
                            chunk_tokens, out.ctypes.data if out.size else None)
    if rc != OK:
        raise _error(rc)
    return out


def scatter(shape: Shape, k, v, l0: int, l1: int, block_table, chunk_tokens: int,
            packed: np.ndarray) -> None:
    """O2 scatter of a packed uint8 image into the mirror, in place."""
    bt, btp = _bt(block_table)
    nbytes = packed_bytes(shape, l0, l1, bt.size) if l1 >= l0 else 0
    if packed.nbytes < nbytes:
        raise ValueError("packed image too small")
    s = shape._c()
    rc = _load().kvo_scatter(ctypes.byref(s), _ptrs(k), _ptrs(v), l0, l1, btp, bt.size,
                             chunk_tokens, packed.ctypes.data if packed.size else None)
    if rc != OK:
        raise _error(rc)


def restore(shape: Shape, k, v, l0: int, l1: int, block_table, chunk_tokens: int,
            image: np.ndarray) -> None:
    """Restore = scatter of the whole packed image (piece split is invisible)."""
    scatter(shape, k, v, l0, l1, block_table, chunk_tokens, image)


def _error(rc: int) -> Exception:
    if rc == EBADBLOCK:
        return IndexError("block id out of range")
    return ValueError(f"invalid argument (status {rc})")


def new_mirror(shape: Shape):
    """Zeroed host mirror (lists of per-layer K and V byte arrays)."""
    nbytes = shape.num_blocks * shape.slab_bytes
    k = [np.zeros(nbytes, dtype=np.uint8) for _ in range(shape.num_layers)]
    v = [np.zeros(nbytes, dtype=np.uint8) for _ in range(shape.num_layers)]
    return k, v


def element_view(buf: np.ndarray, shape: Shape) -> np.ndarray:
    """View a per-layer byte array of the default layout as
    [num_blocks, block_size, kv_heads, head_dim] words."""
    dt = {1: np.uint8, 2: np.uint16, 4: np.uint32, 8: np.uint64}[shape.elem_bytes]
    return buf.view(dt).reshape(shape.num_blocks, shape.block_size, shape.kv_heads,
                                shape.head_dim)


def canonical_view(buf: np.ndarray, shape: Shape, kv: int) -> np.ndarray:
    """A per-layer K (kv=0) or V (kv=1) byte array of any layout, seen as
    [num_blocks, block_size, kv_heads, head_dim] words (a numpy view built by
    reshaping and transposing the layout's own axes)."""
    dt = {1: np.uint8, 2: np.uint16, 4: np.uint32, 8: np.uint64}[shape.elem_bytes]
    w = buf.view(dt)
    NB, BS, H, D = shape.num_blocks, shape.block_size, shape.kv_heads, shape.head_dim
    if shape.layout == LAYOUT_NHD:
        return w.reshape(NB, BS, H, D)
    if shape.layout == LAYOUT_HND:
        return w.reshape(NB, H, BS, D).transpose(0, 2, 1, 3)
    if kv == 1:  # [NB][H][D][BS]
        return w.reshape(NB, H, D, BS).transpose(0, 3, 1, 2)
    x = 16 // shape.elem_bytes  # [NB][H][D/x][BS][x]
    return w.reshape(NB, H, D // x, BS, x).transpose(0, 3, 1, 2, 4).reshape(NB, BS, H, D)
