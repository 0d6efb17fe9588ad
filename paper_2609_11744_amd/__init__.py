"""Paged-KV gather / scatter / staged restore on MI355X (gfx950).

Thin Python binding over the C ABI of ``libkvx.so`` (include/kvx.h): the
functions below marshal arguments and call the library; every byte of the
path is moved by the library's HIP kernels, DMA-engine copies and file I/O. PyTorch provides
device memory and streams only. There is no CPU fallback: importing works
without a GPU, but any call that moves data needs the built library and a GPU.

Operations (sections of the paper they follow):
  * kvx_gather_blocks  -- pack paged KV blocks into contiguous transfer chunks
    (offload side of the batched block copy, Secs. 6.2 and 6.4);
  * kvx_scatter_blocks -- unpack chunks into paged blocks (load side);
  * kvx_restore_from_staging -- feed scatters through a bounded pinned
    staging ring, the host-to-device copies on a DMA engine (Sec. 6.4);
  * kvx_offload_to_staging -- the reverse pipeline for stores.
"""
from __future__ import annotations

import ctypes
import os

from . import _native
from ._native import KvxCache, KvxChunkRef, KvxHostChunk, KvxPiece, KvxRingStats

KVX_OK, KVX_EINVAL, KVX_ENOMEM, KVX_EHIP, KVX_EBADBLOCK, KVX_ECLOSED, KVX_EINTERNAL, KVX_EIO = (
    0, -1, -2, -3, -4, -5, -6, -7)
KVX_EBUSY = -8
KVX_MAX_LAYERS = 128
KVX_LAYOUT_NHD, KVX_LAYOUT_HND, KVX_LAYOUT_PAGED_ATTN = 0, 1, 2


class KvxError(RuntimeError):
    def __init__(self, status: int, where: str):
        msg = _native.lib().kvx_strerror(status).decode()
        super().__init__(f"{where}: {msg} (status {status})")
        self.status = status


def _ok(status: int, where: str) -> None:
    if status != KVX_OK:
        raise KvxError(status, where)


def _stream_handle(stream):
    import torch

    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


_ELEM = None


def _elem_bytes(dtype) -> int:
    import torch

    return torch.empty((), dtype=dtype).element_size()


def layer_shapes(num_blocks, block_size, num_kv_heads, head_dim, elem_bytes,
                 layout=KVX_LAYOUT_NHD):
    """Per-layer (K shape, V shape) of a cache layout."""
    if layout == KVX_LAYOUT_NHD:
        s = (num_blocks, block_size, num_kv_heads, head_dim)
        return s, s
    if layout == KVX_LAYOUT_HND:
        s = (num_blocks, num_kv_heads, block_size, head_dim)
        return s, s
    if layout == KVX_LAYOUT_PAGED_ATTN:
        x = 16 // elem_bytes
        if head_dim % x:
            raise ValueError(f"head_dim must be a multiple of {x} for this layout")
        return ((num_blocks, num_kv_heads, head_dim // x, block_size, x),
                (num_blocks, num_kv_heads, head_dim, block_size))
    raise ValueError(f"unknown layout {layout}")


class PagedKVCache:
    """A paged KV cache: per layer, K and V device tensors in one of the
    layouts of kvx.h (default [num_blocks, block_size, num_kv_heads, head_dim])."""

    def __init__(self, k, v, layout=KVX_LAYOUT_NHD):
        if len(k) != len(v) or not k:
            raise ValueError("need the same positive number of K and V layers")
        ks = tuple(k[0].shape)
        if layout == KVX_LAYOUT_NHD and len(ks) == 4:
            nb, bs, h, d = ks
        elif layout == KVX_LAYOUT_HND and len(ks) == 4:
            nb, h, bs, d = ks
        elif layout == KVX_LAYOUT_PAGED_ATTN and len(ks) == 5:
            nb, h, dx, bs, x = ks
            d = dx * x
        else:
            raise ValueError("cache tensor shape does not match the layout")
        elem = k[0].element_size()
        kshape, vshape = layer_shapes(nb, bs, h, d, elem, layout)
        for t in k:
            if tuple(t.shape) != kshape:
                raise ValueError("all K tensors must share the layout's shape")
        for t in v:
            if tuple(t.shape) != vshape:
                raise ValueError("all V tensors must share the layout's shape")
        for t in list(k) + list(v):
            if t.dtype != k[0].dtype or not t.is_contiguous() or t.device != k[0].device:
                raise ValueError("all cache tensors must share dtype and device and be contiguous")
        self.k, self.v = list(k), list(v)
        self.num_blocks, self.block_size, self.num_kv_heads, self.head_dim = nb, bs, h, d
        self.num_layers = len(k)
        self.layout = layout
        self.dtype = k[0].dtype
        self.device = k[0].device
        self.elem_bytes = elem
        self._kp = (ctypes.c_void_p * self.num_layers)(*[t.data_ptr() for t in self.k])
        self._vp = (ctypes.c_void_p * self.num_layers)(*[t.data_ptr() for t in self.v])
        self._c = KvxCache(self._kp, self._vp, self.num_layers, self.num_blocks, self.block_size,
                           self.num_kv_heads, self.head_dim, self.elem_bytes, layout)

    @property
    def slab_bytes(self) -> int:
        return self.block_size * self.num_kv_heads * self.head_dim * self.elem_bytes

    @classmethod
    def allocate(cls, num_layers, num_blocks, block_size, num_kv_heads, head_dim, dtype, device,
                 layout=KVX_LAYOUT_NHD):
        import torch

        e = torch.empty((), dtype=dtype).element_size()
        ks, vs = layer_shapes(num_blocks, block_size, num_kv_heads, head_dim, e, layout)
        return cls([torch.empty(ks, dtype=dtype, device=device) for _ in range(num_layers)],
                   [torch.empty(vs, dtype=dtype, device=device) for _ in range(num_layers)],
                   layout)

    @classmethod
    def from_host(cls, k_bytes, v_bytes, num_blocks, block_size, num_kv_heads, head_dim, dtype,
                  device, layout=KVX_LAYOUT_NHD):
        """Upload per-layer host byte arrays (numpy uint8) into a new cache."""
        import torch

        e = torch.empty((), dtype=dtype).element_size()
        ks, vs = layer_shapes(num_blocks, block_size, num_kv_heads, head_dim, e, layout)
        up = lambda b, shp: torch.from_numpy(b).to(device).view(dtype).view(shp)  # noqa: E731
        return cls([up(b, ks) for b in k_bytes], [up(b, vs) for b in v_bytes], layout)

    def c_struct(self) -> KvxCache:
        return self._c


def shape_only_cache(num_layers, num_blocks, block_size, num_kv_heads, head_dim, elem_bytes,
                     layout=KVX_LAYOUT_NHD):
    """A kvx_cache description with no tensors (for planning on the host)."""
    return KvxCache(None, None, num_layers, num_blocks, block_size, num_kv_heads, head_dim,
                    elem_bytes, layout)


def _cstruct(cache):
    return cache.c_struct() if isinstance(cache, PagedKVCache) else cache


def kvx_bytes_per_token(layers, kv_heads, head_dim, elem_bytes) -> int:
    return int(_native.lib().kvx_bytes_per_token(layers, kv_heads, head_dim, elem_bytes))


def kvx_packed_bytes(cache, l0, l1, n_blocks) -> int:
    c = _cstruct(cache)
    return int(_native.lib().kvx_packed_bytes(ctypes.byref(c), l0, l1, n_blocks))


def _table_ptr(cache, block_table, n_blocks):
    import torch

    if n_blocks == 0:
        return block_table.data_ptr() if block_table is not None else None
    if block_table.dtype != torch.int32 or not block_table.is_contiguous():
        raise ValueError("block_table must be a contiguous int32 tensor")
    if block_table.device != cache.device:
        raise ValueError("block_table must be on the cache's device")
    if block_table.numel() < n_blocks:
        raise ValueError("block_table shorter than n_blocks")
    return block_table.data_ptr()


def _buffer_ptr(cache, buf, need):
    if need <= 0:
        return buf.data_ptr() if buf is not None else None
    if buf.device != cache.device or not buf.is_contiguous():
        raise ValueError("packed buffer must be contiguous on the cache's device")
    if buf.numel() * buf.element_size() < need:
        raise ValueError(f"packed buffer holds {buf.numel() * buf.element_size()} bytes, "
                         f"needs {need}")
    return buf.data_ptr()


def kvx_chunk_stride(cache, l0, l1, chunk_tokens) -> int:
    """Bytes from one chunk of a packed image to the next (-1 if invalid)."""
    c = _cstruct(cache)
    return int(_native.lib().kvx_chunk_stride(ctypes.byref(c), l0, l1, chunk_tokens))


def kvx_gather_blocks(cache: PagedKVCache, l0, l1, block_table, n_blocks, chunk_tokens, dst,
                      stream=None) -> None:
    need = max(kvx_packed_bytes(cache, l0, l1, n_blocks), 0)
    st = _native.lib().kvx_gather_blocks(
        ctypes.byref(cache.c_struct()), l0, l1, _table_ptr(cache, block_table, n_blocks),
        n_blocks, chunk_tokens, _buffer_ptr(cache, dst, need), _stream_handle(stream))
    _ok(st, "kvx_gather_blocks")


def kvx_scatter_blocks(cache: PagedKVCache, l0, l1, block_table, n_blocks, chunk_tokens, src,
                       stream=None) -> None:
    need = max(kvx_packed_bytes(cache, l0, l1, n_blocks), 0)
    st = _native.lib().kvx_scatter_blocks(
        ctypes.byref(cache.c_struct()), l0, l1, _table_ptr(cache, block_table, n_blocks),
        n_blocks, chunk_tokens, _buffer_ptr(cache, src, need), _stream_handle(stream))
    _ok(st, "kvx_scatter_blocks")


KVX_NOALLOC_MAX_BLOCKS = 65536


def kvx_scatter_blocks_noalloc(cache: PagedKVCache, l0, l1, block_table, n_blocks, chunk_tokens,
                               src, stream=None) -> None:
    """kvx_scatter_blocks that allocates nothing (its ordering scratch is a
    fixed device array of the library's; calls on one GPU must not overlap)."""
    need = max(kvx_packed_bytes(cache, l0, l1, n_blocks), 0)
    st = _native.lib().kvx_scatter_blocks_noalloc(
        ctypes.byref(cache.c_struct()), l0, l1, _table_ptr(cache, block_table, n_blocks),
        n_blocks, chunk_tokens, _buffer_ptr(cache, src, need), _stream_handle(stream))
    _ok(st, "kvx_scatter_blocks_noalloc")


CHUNK_REF_DTYPE = [("packed_offset", "<i8"), ("bt_offset", "<i4"), ("n_blocks", "<i4")]


def chunk_refs(refs, device):
    """Device array of kvx_chunk_ref from (packed_offset, bt_offset, n_blocks) rows."""
    import numpy as np
    import torch

    a = np.zeros(len(refs), dtype=CHUNK_REF_DTYPE)
    for i, (off, bt0, nb) in enumerate(refs):
        a[i] = (off, bt0, nb)
    return torch.from_numpy(a.view(np.uint8).copy()).to(device)


def _chunks_call(fn, cache, l0, l1, block_table, table_len, refs_dev, n_chunks, chunk_tokens,
                 packed, stream, where):
    import torch

    if n_chunks > 0:
        if refs_dev.device != cache.device or refs_dev.numel() * refs_dev.element_size() < 16 * n_chunks:
            raise ValueError("chunk refs must be a device buffer of n_chunks kvx_chunk_ref")
        if block_table.dtype != torch.int32 or block_table.numel() < table_len:
            raise ValueError("block_table must be int32 with at least table_len entries")
        if packed.device != cache.device or not packed.is_contiguous():
            raise ValueError("packed buffer must be contiguous on the cache's device")
    nbytes = packed.numel() * packed.element_size() if packed is not None else 0
    st = fn(ctypes.byref(cache.c_struct()), l0, l1,
            block_table.data_ptr() if block_table is not None else None, table_len,
            refs_dev.data_ptr() if refs_dev is not None else None, n_chunks, chunk_tokens,
            packed.data_ptr() if packed is not None else None, nbytes, _stream_handle(stream))
    _ok(st, where)


def kvx_gather_chunks(cache, l0, l1, block_table, table_len, refs_dev, n_chunks, chunk_tokens,
                      packed, stream=None) -> None:
    """Fused batched gather of a chunk list (refs_dev from chunk_refs())."""
    _chunks_call(_native.lib().kvx_gather_chunks, cache, l0, l1, block_table, table_len,
                 refs_dev, n_chunks, chunk_tokens, packed, stream, "kvx_gather_chunks")


def kvx_scatter_chunks(cache, l0, l1, block_table, table_len, refs_dev, n_chunks, chunk_tokens,
                       packed, stream=None) -> None:
    _chunks_call(_native.lib().kvx_scatter_chunks, cache, l0, l1, block_table, table_len,
                 refs_dev, n_chunks, chunk_tokens, packed, stream, "kvx_scatter_chunks")


def kvx_check(stream=None) -> None:
    _ok(_native.lib().kvx_check(_stream_handle(stream)), "kvx_check")


KVX_RAMP_NONE, KVX_RAMP_FIRST, KVX_RAMP_LAST = 0, 1, 2

# kvx_trace_event kinds (include/kvx.h)
TRACE_KINDS = {1: "fill", 2: "drain", 3: "wait", 4: "h2d", 5: "d2h", 6: "scatter", 7: "gather"}


def trace_chrome(events, name="ring") -> dict:
    """A ring timeline (StagingRing.trace) as Chrome trace-event JSON: one
    complete event per interval, one track per fill or drain thread and one
    each for the enqueuing thread's waits, the host-link copies and the
    launches; times in microseconds from the first interval."""
    t0 = min((e["t0_ns"] for e in events), default=0)
    tracks = {"wait": (1, "enqueue thread: waits for fill / drain"),
              "h2d": (2, "host-to-device copies"), "d2h": (2, "device-to-host copies"),
              "scatter": (3, "scatter launches"), "gather": (3, "gather launches")}
    out, named = [], set()
    for e in events:
        if e["kind"] in ("fill", "drain"):
            tid, label = 10 + e["lane"], f'{e["kind"]} thread {e["lane"]}'
        else:
            tid, label = tracks.get(e["kind"], (0, e["kind"]))
        if tid not in named:
            named.add(tid)
            out.append({"ph": "M", "name": "thread_name", "pid": 1, "tid": tid,
                        "args": {"name": label}})
        out.append({"ph": "X", "name": f'{e["kind"]} piece {e["piece"]}', "pid": 1, "tid": tid,
                    "ts": (e["t0_ns"] - t0) / 1e3, "dur": (e["t1_ns"] - e["t0_ns"]) / 1e3,
                    "args": {"piece": e["piece"], "slot": e["slot"], "bytes": e["bytes"]}})
    out.append({"ph": "M", "name": "process_name", "pid": 1, "args": {"name": name}})
    return {"traceEvents": out, "displayTimeUnit": "ms"}


def kvx_copy_walk(cache, l0, l1, n_blocks, chunk_tokens, to_packed: bool) -> dict:
    """The walk a gather (to_packed) or scatter of these arguments takes (pure
    host computation, kvx_copy_walk)."""
    c = _cstruct(cache)
    w = _native.KvxWalk()
    _ok(_native.lib().kvx_copy_walk(ctypes.byref(c), l0, l1, n_blocks, chunk_tokens,
                                    1 if to_packed else 0, ctypes.byref(w)), "kvx_copy_walk")
    return {f: getattr(w, f) for f, _ in _native.KvxWalk._fields_ if f != "reserved"}


def kvx_plan_pieces(cache, l0, l1, n_blocks, chunk_tokens, slot_bytes, ramp=KVX_RAMP_NONE):
    """Staging pieces as a list of dicts (pure host computation)."""
    c = _cstruct(cache)
    n = ctypes.c_int32(0)
    _ok(_native.lib().kvx_plan_pieces(ctypes.byref(c), l0, l1, n_blocks, chunk_tokens,
                                      slot_bytes, ramp, None, 0, ctypes.byref(n)),
        "kvx_plan_pieces")
    arr = (KvxPiece * max(n.value, 1))()
    _ok(_native.lib().kvx_plan_pieces(ctypes.byref(c), l0, l1, n_blocks, chunk_tokens,
                                      slot_bytes, ramp, arr, n.value, ctypes.byref(n)),
        "kvx_plan_pieces")
    return [{f: getattr(arr[i], f) for f, _ in KvxPiece._fields_} for i in range(n.value)]


class PinnedBuffer:
    """Exactly-sized pinned host memory (kvx_pinned_alloc), with a numpy view."""

    def __init__(self, nbytes: int):
        import numpy as np

        p = ctypes.c_void_p()
        _ok(_native.lib().kvx_pinned_alloc(nbytes, ctypes.byref(p)), "kvx_pinned_alloc")
        self.ptr = p.value
        self.nbytes = nbytes
        self.array = np.ctypeslib.as_array((ctypes.c_uint8 * nbytes).from_address(self.ptr))

    def free(self):
        if self.ptr:
            self.array = None
            _native.lib().kvx_pinned_free(self.ptr)
            self.ptr = None

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


class StagingRing:
    """A bounded pinned staging ring (kvx_ring_*)."""

    def __init__(self, device, n_slots: int, slot_bytes: int, landing=None):
        import torch

        dev = torch.device(device)
        idx = dev.index if dev.index is not None else torch.cuda.current_device()
        if landing is not None:
            if landing.numel() * landing.element_size() < n_slots * slot_bytes:
                raise ValueError("landing buffer too small")
            lp = landing.data_ptr()
        else:
            lp = None
        self._landing = landing
        h = ctypes.c_void_p()
        _ok(_native.lib().kvx_ring_create(idx, n_slots, slot_bytes, lp, ctypes.byref(h)),
            "kvx_ring_create")
        self.handle = h.value
        self.n_slots, self.slot_bytes = n_slots, slot_bytes
        self._source = None
        self._cache = None
        self.n_blocks = 0

    def bind(self, cache: PagedKVCache, l0, l1, n_blocks, chunk_tokens, host_source,
             fill_threads=4):
        """host_source: numpy uint8 array, PinnedBuffer or pinned CPU tensor."""
        need = max(kvx_packed_bytes(cache, l0, l1, n_blocks), 0)
        if isinstance(host_source, PinnedBuffer):
            ptr, size = host_source.ptr, host_source.nbytes
        elif hasattr(host_source, "ctypes"):
            if not host_source.flags["C_CONTIGUOUS"]:
                raise ValueError("host image must be contiguous")
            ptr, size = host_source.ctypes.data, host_source.nbytes
        else:
            ptr, size = host_source.data_ptr(), host_source.numel() * host_source.element_size()
        if size < need:
            raise ValueError(f"host image holds {size} bytes, needs {need}")
        _ok(_native.lib().kvx_ring_bind(self.handle, ctypes.byref(cache.c_struct()), l0, l1,
                                        n_blocks, chunk_tokens, ptr, fill_threads),
            "kvx_ring_bind")
        self._source = host_source  # keep alive while bound
        self._cache = cache
        self.n_blocks = n_blocks

    def _host_chunks(self, chunks):
        arr = (KvxHostChunk * max(len(chunks), 1))()
        keep = []
        for i, (buf, bt0, nb) in enumerate(chunks):
            if isinstance(buf, int):
                ptr = buf
            elif isinstance(buf, PinnedBuffer):
                ptr = buf.ptr
            else:
                if not buf.flags["C_CONTIGUOUS"]:
                    raise ValueError("host chunk buffers must be contiguous")
                ptr = buf.ctypes.data
            keep.append(buf)
            arr[i] = KvxHostChunk(ptr, bt0, nb)
        return arr, keep

    def bind_chunks(self, cache, l0, l1, chunk_tokens, chunks, fill_threads=4):
        """Restore binding over a chunk list [(host image, bt_offset, n_blocks)];
        a host image is a numpy uint8 array, a PinnedBuffer or a raw address."""
        arr, keep = self._host_chunks(chunks)
        _ok(_native.lib().kvx_ring_bind_chunks(self.handle, ctypes.byref(cache.c_struct()), l0, l1,
                                               chunk_tokens, arr, len(chunks), fill_threads),
            "kvx_ring_bind_chunks")
        self._source, self._cache = keep, cache
        self.n_blocks = max((bt0 + nb for _, bt0, nb in chunks), default=0)

    def bind_offload(self, cache, l0, l1, chunk_tokens, chunks, drain_threads=4):
        """Offload binding over a chunk list [(host destination, bt_offset, n_blocks)]."""
        arr, keep = self._host_chunks(chunks)
        _ok(_native.lib().kvx_ring_bind_offload(self.handle, ctypes.byref(cache.c_struct()), l0,
                                                l1, chunk_tokens, arr, len(chunks), drain_threads),
            "kvx_ring_bind_offload")
        self._source, self._cache = keep, cache
        self.n_blocks = max((bt0 + nb for _, bt0, nb in chunks), default=0)

    def _file_chunks(self, chunks):
        arr = (_native.KvxFileChunk * max(len(chunks), 1))()
        keep = []
        for i, (path, bt0, nb) in enumerate(chunks):
            b = os.fsencode(path)
            keep.append(b)
            arr[i] = _native.KvxFileChunk(b, bt0, nb)
        return arr, keep

    def bind_files(self, cache, l0, l1, chunk_tokens, chunks, io_depth=8):
        """Restore binding over chunk files [(path, bt_offset, n_blocks)] (storage tier)."""
        arr, keep = self._file_chunks(chunks)
        _ok(_native.lib().kvx_ring_bind_files(self.handle, ctypes.byref(cache.c_struct()), l0, l1,
                                              chunk_tokens, arr, len(chunks), io_depth),
            "kvx_ring_bind_files")
        self._source, self._cache = keep, cache
        self.n_blocks = max((bt0 + nb for _, bt0, nb in chunks), default=0)

    def bind_offload_files(self, cache, l0, l1, chunk_tokens, chunks, io_depth=8):
        """Offload binding to chunk files [(path, bt_offset, n_blocks)], published on completion."""
        arr, keep = self._file_chunks(chunks)
        _ok(_native.lib().kvx_ring_bind_offload_files(self.handle, ctypes.byref(cache.c_struct()),
                                                      l0, l1, chunk_tokens, arr, len(chunks),
                                                      io_depth),
            "kvx_ring_bind_offload_files")
        self._source, self._cache = keep, cache
        self.n_blocks = max((bt0 + nb for _, bt0, nb in chunks), default=0)

    def bind_preloaded(self, cache, l0, l1, chunk_tokens, preloader, chunks):
        """Restore binding over chunk files [(path, bt_offset, n_blocks)] held in a
        preloader's pool: each restore holds the files and copies every piece as
        soon as its files are staged."""
        arr, keep = self._file_chunks(chunks)
        _ok(_native.lib().kvx_ring_bind_preloaded(self.handle, ctypes.byref(cache.c_struct()), l0,
                                                  l1, chunk_tokens, preloader.handle, arr,
                                                  len(chunks)),
            "kvx_ring_bind_preloaded")
        self._source, self._cache = (keep, preloader), cache
        self.n_blocks = max((bt0 + nb for _, bt0, nb in chunks), default=0)

    def stats(self) -> dict:
        s = KvxRingStats()
        _ok(_native.lib().kvx_ring_stats_get(self.handle, ctypes.byref(s)), "kvx_ring_stats_get")
        return {f: getattr(s, f) for f, _ in KvxRingStats._fields_}

    def set_trace(self, enable=True):
        """Record the next transfers' timeline (kvx_ring_set_trace)."""
        _ok(_native.lib().kvx_ring_set_trace(self.handle, 1 if enable else 0),
            "kvx_ring_set_trace")

    def trace(self) -> list:
        """The last traced transfer's intervals (kvx_ring_trace_get), ordered by
        start: dicts with kind (a TRACE_KINDS name), piece, lane, slot, bytes,
        t0_ns, t1_ns (host monotonic clock, as time.monotonic_ns)."""
        n = ctypes.c_int32()
        _ok(_native.lib().kvx_ring_trace_get(self.handle, None, 0, ctypes.byref(n)),
            "kvx_ring_trace_get")
        arr = (_native.KvxTraceEvent * max(n.value, 1))()
        _ok(_native.lib().kvx_ring_trace_get(self.handle, arr, n.value, ctypes.byref(n)),
            "kvx_ring_trace_get")
        return [{"kind": TRACE_KINDS.get(e.kind, str(e.kind)), "piece": e.piece, "lane": e.lane,
                 "slot": e.slot, "bytes": e.bytes, "t0_ns": e.t0_ns, "t1_ns": e.t1_ns}
                for e in arr[:n.value]]

    def abort(self):
        _ok(_native.lib().kvx_ring_abort(self.handle), "kvx_ring_abort")

    def set_test_hooks(self, max_delay_us=0, poison=False, hip_copies=False):
        """Fault injection: random fill/drain pauses, poisoning of released slots;
        hip_copies routes the host-link copies (both directions) through the HIP
        runtime instead of the DMA engines."""
        flags = (1 if poison else 0) | (2 if hip_copies else 0)
        _ok(_native.lib().kvx_ring_set_test_hooks(self.handle, max_delay_us, flags),
            "kvx_ring_set_test_hooks")

    def close(self):
        if self.handle:
            _native.lib().kvx_ring_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def kvx_restore_from_staging(ring: StagingRing, block_table, stream=None) -> None:
    ptr = _table_ptr(ring._cache, block_table, ring.n_blocks) if ring._cache is not None else None
    st = _native.lib().kvx_restore_from_staging(ring.handle, ptr, _stream_handle(stream))
    _ok(st, "kvx_restore_from_staging")


def kvx_block_hashes(tokens, block_size, parent_hash=0):
    """Prefix-hash chain over the full blocks of `tokens` (numpy int32 array)."""
    import numpy as np

    t = np.ascontiguousarray(tokens, dtype=np.int32)
    out = np.empty(max(t.size // block_size, 1), dtype=np.uint64)
    n = _native.lib().kvx_block_hashes(t.ctypes.data if t.size else None, t.size, block_size,
                                       parent_hash & (2**64 - 1), out.ctypes.data)
    if n < 0:
        raise KvxError(KVX_EINVAL, "kvx_block_hashes")
    return out[:n]


def kvx_dedupe_keys(keys):
    """first_of[i] = index of the first occurrence of keys[i]."""
    import numpy as np

    k = np.ascontiguousarray(keys, dtype=np.uint64)
    first = np.empty(max(k.size, 1), dtype=np.int32)
    _ok(_native.lib().kvx_dedupe_keys(k.ctypes.data if k.size else None, k.size, first.ctypes.data),
        "kvx_dedupe_keys")
    return first[:k.size]


def kvx_probe_stream(src, dst, nbytes: int, mode: int, stream=None) -> None:
    """HBM probe (roofline context): mode 0 read src, 1 write dst, 2 copy src -> dst."""
    for t in (src, dst):
        if t is not None and (not t.is_cuda or t.numel() * t.element_size() < nbytes):
            raise ValueError("probe buffers must be device tensors of at least nbytes")
    st = _native.lib().kvx_probe_stream(src.data_ptr() if src is not None else None,
                                        dst.data_ptr() if dst is not None else None, nbytes, mode,
                                        _stream_handle(stream))
    _ok(st, "kvx_probe_stream")


def kvx_chunk_path(root: str, tag: str, key: int) -> str:
    """Hash-addressed chunk file path: <root>/<tag>/<k0>/<k1>/<key>.kvc."""
    out = ctypes.create_string_buffer(4096)
    n = _native.lib().kvx_chunk_path(os.fsencode(root), os.fsencode(tag), key & (2**64 - 1), out,
                                     len(out))
    if n < 0:
        raise KvxError(KVX_EINVAL, "kvx_chunk_path")
    return os.fsdecode(out.value)


def _file_ios(ops):
    import numpy as np

    arr = (_native.KvxFileIo * max(len(ops), 1))()
    keep = []
    for i, (path, buf, offset) in enumerate(ops):
        if isinstance(buf, PinnedBuffer):
            ptr, size = buf.ptr, buf.nbytes
        else:
            a = np.asarray(buf)
            if a.dtype != np.uint8 or not a.flags.c_contiguous:
                raise ValueError("file buffers must be contiguous uint8 arrays")
            ptr, size = a.ctypes.data, a.nbytes
            keep.append(a)
        b = os.fsencode(path)
        keep.append(b)
        arr[i] = _native.KvxFileIo(b, ptr, offset, size)
    return arr, keep


def kvx_read_files(ops, io_depth: int = 8) -> None:
    """Read [(path, buffer, file offset)]: each buffer is filled from its file."""
    arr, keep = _file_ios(ops)
    _ok(_native.lib().kvx_read_files(arr, len(ops), io_depth), "kvx_read_files")


def kvx_write_files(ops, io_depth: int = 8) -> None:
    """Write and publish files from [(path, buffer, file offset)]; a file's ops
    must tile it exactly."""
    arr, keep = _file_ios(ops)
    _ok(_native.lib().kvx_write_files(arr, len(ops), io_depth), "kvx_write_files")


def _paths(paths):
    enc = [os.fsencode(p) for p in paths]
    arr = (ctypes.c_char_p * max(len(enc), 1))(*enc)
    return arr, enc


class Preloader:
    """Bounded pool of host slots that chunk files are read into ahead of their
    requests (kvx_preloader_*): hint() queues speculative reads, fetch() claims
    staged images (reading the rest first, before any speculative work) and
    returns numpy views of them, release() drops the holds."""

    def __init__(self, n_slots: int, slot_bytes: int, io_depth: int = 8, reserve: int = 0,
                 pinned: bool = True):
        h = ctypes.c_void_p()
        _ok(_native.lib().kvx_preloader_create(n_slots, slot_bytes, io_depth, reserve,
                                               1 if pinned else 0, ctypes.byref(h)),
            "kvx_preloader_create")
        self.handle = h.value

    def hint(self, paths) -> None:
        arr, keep = _paths(paths)
        _ok(_native.lib().kvx_preload_hint(self.handle, arr, len(paths)), "kvx_preload_hint")

    def fetch(self, paths):
        """Hold the named files' images; returns one uint8 array view per path
        (valid until release)."""
        import numpy as np

        arr, keep = _paths(paths)
        n = len(paths)
        imgs = (ctypes.c_void_p * max(n, 1))()
        sizes = (ctypes.c_int64 * max(n, 1))()
        _ok(_native.lib().kvx_preload_fetch(self.handle, arr, n, imgs, sizes), "kvx_preload_fetch")
        return [np.ctypeslib.as_array((ctypes.c_uint8 * sizes[i]).from_address(imgs[i]))
                for i in range(n)]

    def release(self, paths) -> None:
        arr, keep = _paths(paths)
        _ok(_native.lib().kvx_preload_release(self.handle, arr, len(paths)),
            "kvx_preload_release")

    def wait_idle(self) -> None:
        _ok(_native.lib().kvx_preload_wait_idle(self.handle), "kvx_preload_wait_idle")

    def set_test_hooks(self, delay_us: int = 0) -> None:
        """Pause the reactor delay_us after each batch of completed pieces."""
        _ok(_native.lib().kvx_preload_set_test_hooks(self.handle, delay_us),
            "kvx_preload_set_test_hooks")

    def stats(self) -> dict:
        s = _native.KvxPreloadStats()
        _ok(_native.lib().kvx_preload_stats_get(self.handle, ctypes.byref(s)),
            "kvx_preload_stats_get")
        return {f: getattr(s, f) for f, _ in _native.KvxPreloadStats._fields_}

    def close(self) -> None:
        if self.handle:
            _native.lib().kvx_preloader_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def kvx_offload_to_staging(ring: StagingRing, block_table, stream=None) -> None:
    ptr = _table_ptr(ring._cache, block_table, ring.n_blocks) if ring._cache is not None else None
    st = _native.lib().kvx_offload_to_staging(ring.handle, ptr, _stream_handle(stream))
    _ok(st, "kvx_offload_to_staging")


def kvx_offload_begin(ring: StagingRing, block_table, stream=None) -> None:
    """Start the bound offload in the background (the deferred store); finish
    it with kvx_offload_wait. The block table is kept alive until then."""
    ptr = _table_ptr(ring._cache, block_table, ring.n_blocks) if ring._cache is not None else None
    st = _native.lib().kvx_offload_begin(ring.handle, ptr, _stream_handle(stream))
    _ok(st, "kvx_offload_begin")
    ring._pending = block_table


def kvx_offload_wait(ring: StagingRing) -> None:
    st = _native.lib().kvx_offload_wait(ring.handle)
    ring._pending = None
    _ok(st, "kvx_offload_wait")


def kvx_restore_begin(ring: StagingRing, block_table, stream=None) -> None:
    """Start the bound restore in the background; kvx_restore_wait orders a
    stream after its scatters. The block table is kept alive until then."""
    ptr = _table_ptr(ring._cache, block_table, ring.n_blocks) if ring._cache is not None else None
    st = _native.lib().kvx_restore_begin(ring.handle, ptr, _stream_handle(stream))
    _ok(st, "kvx_restore_begin")
    ring._pending = block_table


def kvx_restore_wait(ring: StagingRing, stream=None) -> None:
    st = _native.lib().kvx_restore_wait(ring.handle, _stream_handle(stream))
    ring._pending = None
    _ok(st, "kvx_restore_wait")


__all__ = [
    "KvxError", "PagedKVCache", "PinnedBuffer", "StagingRing", "kvx_bytes_per_token",
    "kvx_packed_bytes", "kvx_gather_blocks", "kvx_scatter_blocks", "kvx_check",
    "kvx_plan_pieces", "kvx_restore_from_staging", "shape_only_cache", "KVX_MAX_LAYERS",
    "kvx_gather_chunks", "kvx_scatter_chunks", "chunk_refs", "kvx_offload_to_staging",
    "kvx_block_hashes", "kvx_dedupe_keys", "KVX_LAYOUT_NHD", "KVX_LAYOUT_HND",
    "KVX_LAYOUT_PAGED_ATTN", "layer_shapes", "kvx_probe_stream", "kvx_chunk_path", "Preloader",
    "kvx_read_files", "kvx_write_files", "KVX_EIO", "KVX_EBUSY", "kvx_offload_begin",
    "kvx_offload_wait", "kvx_restore_begin", "kvx_restore_wait", "kvx_chunk_stride",
    "KVX_RAMP_NONE", "KVX_RAMP_FIRST", "KVX_RAMP_LAST", "kvx_scatter_blocks_noalloc",
    "KVX_NOALLOC_MAX_BLOCKS", "TRACE_KINDS", "trace_chrome", "kvx_copy_walk",
]
