"""ctypes binding of ``libpaged_attn.so`` (argument marshalling only).

Every function here has the name and argument order of the C function it
calls; see ``include/paged_attn.h`` for meanings, layouts and ownership.
Device buffers may be given as torch tensors (their ``data_ptr()`` is
passed) or as raw integer addresses; ``stream`` is a HIP stream handle as an
integer (for example ``torch.cuda.current_stream().cuda_stream``) or None
for the default stream.  A negative status raises ``PagedAttnError`` with
the library's message.  If the library has not been built, importing this
module raises ImportError: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libpaged_attn.so")

PA_OK, PA_EINVAL, PA_ENOMEM, PA_EUNSUPPORTED, PA_EHIP, PA_ESTATE = 0, -1, -2, -3, -4, -5
BLOCK_SIZE = 16

# Every symbol the header declares, with (restype, argtypes).
_c_int, _i32, _i64, _f32, _vp, _sz = (ctypes.c_int, ctypes.c_int32, ctypes.c_int64,
                                      ctypes.c_float, ctypes.c_void_p, ctypes.c_size_t)
_pi32 = ctypes.POINTER(ctypes.c_int32)
_pi64 = ctypes.POINTER(ctypes.c_int64)
SIGNATURES = {
    "pa_last_error": (ctypes.c_char_p, []),
    "pa_version": (_i32, []),
    "kv_pool_create": (_c_int, [_i32, _i32, _i32, _i32, _vp, _vp, ctypes.POINTER(_vp)]),
    "kv_pool_destroy": (_c_int, [_vp]),
    "kv_pool_alloc": (_c_int, [_vp, _i32, _pi32]),
    "kv_pool_claim": (_c_int, [_vp, _i32, _pi32]),
    "kv_pool_retain": (_c_int, [_vp, _i32, _pi32]),
    "kv_pool_release": (_c_int, [_vp, _i32, _pi32]),
    "kv_pool_num_free": (_c_int, [_vp, _pi32]),
    "kv_pool_refcount": (_c_int, [_vp, _i32, _pi32]),
    "kv_pool_num_shared": (_c_int, [_vp, _pi64]),
    "kv_pool_layout": (_c_int, [_vp, _pi64, _pi64]),
    "paged_attn_num_partitions": (_c_int, [_i32, _i32, _pi32]),
    "paged_attn_workspace_size": (_c_int, [_i32, _i32, _i32, _i32, _i32,
                                           ctypes.POINTER(_sz), ctypes.POINTER(_sz)]),
    "paged_attn_decode": (_c_int, [_vp, _vp, _vp, _i32, _vp, _i32, _i32, _f32, _i32, _i32,
                                   _vp, _vp, _vp, _vp]),
    "paged_attn_reduce": (_c_int, [_vp, _vp, _vp, _i32, _i32, _i32, _i32, _i32, _vp, _vp]),
    "paged_attn_decode_trace": (_c_int, [_vp, _vp, _vp, _i32, _vp, _i32, _i32, _f32, _i32,
                                         _i32, _vp, _vp, _vp, _vp, _i64, _vp]),
    "pa_stream_copy": (_c_int, [_vp, _vp, _sz, _vp]),
    "pa_gather_tiles": (_c_int, [_vp, _vp, _i32, _i32, _vp, _i32, _i32, _vp, _vp]),
    "paged_attn_append_kv": (_c_int, [_vp, _vp, _vp, _vp, _i32, _vp, _i32, _vp]),
    "paged_attn_schedule": (_c_int, [_pi32, _i32, _i32, _i32, _i32, _pi32, _i32, _pi32]),
    "paged_attn_cascade_groups_workspace_size": (_c_int, [_i32, _i32, _i32, _i32, _i32, _i32, _i32,
                                                         _i32, ctypes.POINTER(_sz),
                                                         ctypes.POINTER(_sz), _pi32]),
    "paged_attn_decode_cascade_groups": (_c_int, [_vp, _vp, _vp, _i32, _vp, _i32, _i32, _f32, _i32,
                                                  _i32, _i32, _i32, _vp, _i32, _i32, _i32, _vp, _i32,
                                                  _vp, _vp, _vp]),
    "paged_attn_reduce_cascade_groups": (_c_int, [_vp, _vp, _vp, _i32, _i32, _i32, _i32, _i32, _i32,
                                                  _i32, _i32, _vp, _vp]),
    "paged_attn_decode_append": (_c_int, [_vp, _vp, _vp, _vp, _vp, _i32, _vp, _i32, _i32, _f32, _i32,
                                          _i32, _vp, _i32, _vp, _vp, _vp, _vp]),
    "paged_attn_decode_cascade_append": (_c_int, [_vp, _vp, _vp, _vp, _vp, _i32, _vp, _i32, _i32, _f32,
                                                  _i32, _i32, _i32, _i32, _vp, _i32, _i32, _i32, _vp,
                                                  _i32, _vp, _vp, _vp]),
    "paged_attn_decode_scheduled": (_c_int, [_vp, _vp, _vp, _i32, _vp, _i32, _i32, _f32, _i32, _i32,
                                             _vp, _i32, _vp, _vp, _vp, _vp]),
    "paged_attn_decode_cascade_scheduled": (_c_int, [_vp, _vp, _vp, _i32, _vp, _i32, _i32, _f32, _i32,
                                                     _i32, _i32, _i32, _vp, _i32, _vp, _vp, _vp]),
    "paged_attn_extend": (_c_int, [_vp, _vp, _vp, _i32, _vp, _i32, _vp, _i32, _i32, _f32, _i32, _i32,
                                   _vp, _vp]),
    "paged_attn_decode_scheduled_trace": (_c_int, [_vp, _vp, _vp, _i32, _vp, _i32, _i32, _f32, _i32,
                                                   _i32, _vp, _i32, _vp, _vp, _vp, _vp, _i64, _vp]),
    "paged_attn_cascade_trace_layout": (_c_int, [_vp, _i32, _i32, _i32, _i32, _i32, _i32, _i32, _i32,
                                                 _pi64]),
    "paged_attn_decode_cascade_trace": (_c_int, [_vp, _vp, _vp, _i32, _vp, _i32, _i32, _f32, _i32,
                                                 _i32, _i32, _i32, _vp, _i32, _i32, _i32, _vp, _i32,
                                                 _vp, _vp, _vp, _i64, _vp]),
    "paged_attn_decode_noalloc": (_c_int, [_vp, _vp, _vp, _i32, _vp, _i32, _i32, _f32, _i32, _i32,
                                           _vp, _vp]),
    "paged_attn_check_tables": (_c_int, [_vp, _pi32, _i32, _pi32, _i32, _i32, _pi32, _i32, _i32,
                                         _pi32]),
    "paged_attn_cascade_workspace_size": (_c_int, [_i32, _i32, _i32, _i32, _i32, _i32, _i32,
                                                   ctypes.POINTER(_sz), ctypes.POINTER(_sz),
                                                   _pi32]),
    "paged_attn_decode_cascade": (_c_int, [_vp, _vp, _vp, _i32, _vp, _i32, _i32, _f32, _i32,
                                           _i32, _i32, _i32, _vp, _vp, _vp]),
    "paged_attn_reduce_cascade": (_c_int, [_vp, _vp, _vp, _i32, _i32, _i32, _i32, _i32, _i32,
                                           _i32, _vp, _vp]),
}


class PagedAttnError(RuntimeError):
    def __init__(self, code: int, message: str):
        super().__init__(f"[{code}] {message}")
        self.code = code


def _load(path: str = LIB_PATH) -> ctypes.CDLL:
    # torch owns the device memory and streams handed to the library, so the
    # library must resolve libamdhip64 to the HIP runtime torch already
    # loaded (same SONAME); loaded first, it would bring in a second runtime
    # whose device context and streams are unrelated to torch's.
    import torch  # noqa: F401
    if not os.path.exists(path):
        raise ImportError(
            f"{path} is missing: build the HIP library first "
            "(python -c 'import __graft_entry__ as g; g.build()')")
    lib = ctypes.CDLL(path)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


_lib = _load()


def library() -> ctypes.CDLL:
    return _lib


def _check(rc: int) -> None:
    if rc != PA_OK:
        raise PagedAttnError(rc, _lib.pa_last_error().decode())


def _ptr(x):
    if x is None:
        return None
    if hasattr(x, "data_ptr"):
        return x.data_ptr() or None
    return int(x) or None


def _ids(ids):
    arr = (ctypes.c_int32 * len(ids))(*[int(i) for i in ids])
    return len(ids), arr


def pa_last_error() -> str:
    return _lib.pa_last_error().decode()


def pa_version() -> int:
    return int(_lib.pa_version())


class KVPool:
    """Handle of a KV block pool (host metadata over caller-owned device pools)."""

    def __init__(self, handle: int, num_blocks: int, num_kv_heads: int, head_dim: int,
                 k_pool=None, v_pool=None):
        self.handle = handle
        self.num_blocks = num_blocks
        self.num_kv_heads = num_kv_heads
        self.head_dim = head_dim
        self._keep = (k_pool, v_pool)   # keeps tensors alive while the handle lives

    def close(self) -> None:
        if self.handle:
            _lib.kv_pool_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def _handle(self):
        if not self.handle:
            raise PagedAttnError(PA_EINVAL, "pool handle is closed")
        return self.handle


def kv_pool_create(num_blocks, block_size, num_kv_heads, head_dim, k_pool, v_pool) -> KVPool:
    h = ctypes.c_void_p()
    _check(_lib.kv_pool_create(num_blocks, block_size, num_kv_heads, head_dim, _ptr(k_pool),
                               _ptr(v_pool), ctypes.byref(h)))
    return KVPool(h.value, num_blocks, num_kv_heads, head_dim, k_pool, v_pool)


def kv_pool_destroy(pool: KVPool) -> None:
    pool.close()


def kv_pool_alloc(pool: KVPool, n: int) -> list:
    arr = (ctypes.c_int32 * max(n, 1))()
    _check(_lib.kv_pool_alloc(pool._handle(), n, arr))
    return [arr[i] for i in range(n)]


def kv_pool_claim(pool: KVPool, ids) -> None:
    n, arr = _ids(ids)
    _check(_lib.kv_pool_claim(pool._handle(), n, arr))


def kv_pool_retain(pool: KVPool, ids) -> None:
    n, arr = _ids(ids)
    _check(_lib.kv_pool_retain(pool._handle(), n, arr))


def kv_pool_release(pool: KVPool, ids) -> None:
    n, arr = _ids(ids)
    _check(_lib.kv_pool_release(pool._handle(), n, arr))


def kv_pool_num_free(pool: KVPool) -> int:
    n = ctypes.c_int32()
    _check(_lib.kv_pool_num_free(pool._handle(), ctypes.byref(n)))
    return n.value


def kv_pool_refcount(pool: KVPool, block_id: int) -> int:
    n = ctypes.c_int32()
    _check(_lib.kv_pool_refcount(pool._handle(), block_id, ctypes.byref(n)))
    return n.value


def kv_pool_num_shared(pool: KVPool) -> int:
    n = ctypes.c_int64()
    _check(_lib.kv_pool_num_shared(pool._handle(), ctypes.byref(n)))
    return n.value


def kv_pool_layout(pool: KVPool):
    """Returns (element strides [block, head, token, dim], bytes of one pool)."""
    strides = (ctypes.c_int64 * 4)()
    nbytes = ctypes.c_int64()
    _check(_lib.kv_pool_layout(pool._handle(), strides, ctypes.byref(nbytes)))
    return list(strides), nbytes.value


def paged_attn_num_partitions(max_context_len: int, partition_size: int) -> int:
    p = ctypes.c_int32()
    _check(_lib.paged_attn_num_partitions(max_context_len, partition_size, ctypes.byref(p)))
    return p.value


def paged_attn_workspace_size(batch, num_q_heads, head_dim, max_context_len, partition_size):
    a, b = ctypes.c_size_t(), ctypes.c_size_t()
    _check(_lib.paged_attn_workspace_size(batch, num_q_heads, head_dim, max_context_len,
                                          partition_size, ctypes.byref(a), ctypes.byref(b)))
    return a.value, b.value


def paged_attn_decode(pool: KVPool, q, block_tables, bt_stride, context_lens, batch, num_q_heads,
                      scale, max_context_len, partition_size, out, partial_out=None,
                      partial_lse=None, stream=None) -> None:
    _check(_lib.paged_attn_decode(pool._handle(), _ptr(q), _ptr(block_tables), bt_stride,
                                  _ptr(context_lens), batch, num_q_heads, scale, max_context_len,
                                  partition_size, _ptr(out), _ptr(partial_out), _ptr(partial_lse),
                                  _ptr(stream)))


def paged_attn_reduce(partial_out, partial_lse, context_lens, batch, num_q_heads, head_dim,
                      partition_size, max_partitions, out, stream=None) -> None:
    _check(_lib.paged_attn_reduce(_ptr(partial_out), _ptr(partial_lse), _ptr(context_lens), batch,
                                  num_q_heads, head_dim, partition_size, max_partitions, _ptr(out),
                                  _ptr(stream)))


def paged_attn_decode_trace(pool: KVPool, q, block_tables, bt_stride, context_lens, batch,
                            num_q_heads, scale, max_context_len, partition_size, out,
                            partial_out, partial_lse, trace, trace_capacity, stream=None) -> None:
    _check(_lib.paged_attn_decode_trace(pool._handle(), _ptr(q), _ptr(block_tables), bt_stride,
                                        _ptr(context_lens), batch, num_q_heads, scale,
                                        max_context_len, partition_size, _ptr(out),
                                        _ptr(partial_out), _ptr(partial_lse), _ptr(trace),
                                        trace_capacity, _ptr(stream)))


def pa_stream_copy(src, dst, nbytes, stream=None) -> None:
    _check(_lib.pa_stream_copy(_ptr(src), _ptr(dst), nbytes, _ptr(stream)))


def pa_gather_tiles(pool: KVPool, block_tables, bt_stride, batch, spans, num_spans, sink,
                    stream=None, tiles_in_flight: int = 2) -> None:
    handle = pool._handle() if pool is not None else None
    _check(_lib.pa_gather_tiles(handle, _ptr(block_tables), bt_stride, batch, _ptr(spans),
                                num_spans, tiles_in_flight, _ptr(sink), _ptr(stream)))


def paged_attn_append_kv(pool: KVPool, k_new, v_new, block_tables, bt_stride, context_lens, batch,
                         stream=None) -> None:
    _check(_lib.paged_attn_append_kv(pool._handle(), _ptr(k_new), _ptr(v_new), _ptr(block_tables),
                                     bt_stride, _ptr(context_lens), batch, _ptr(stream)))


def paged_attn_decode_append(pool: KVPool, q, k_new, v_new, block_tables, bt_stride, context_lens,
                             batch, num_q_heads, scale, max_context_len, partition_size, items,
                             num_items, out, partial_out=None, partial_lse=None, stream=None) -> None:
    _check(_lib.paged_attn_decode_append(
        pool._handle(), _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(block_tables), bt_stride,
        _ptr(context_lens), batch, num_q_heads, scale, max_context_len, partition_size, _ptr(items),
        num_items, _ptr(out), _ptr(partial_out), _ptr(partial_lse), _ptr(stream)))


def paged_attn_decode_cascade_append(pool: KVPool, q, k_new, v_new, block_tables, bt_stride,
                                     context_lens, batch, num_q_heads, scale, max_context_len,
                                     partition_size, prefix_len, prefix_partition_size, group_start,
                                     num_groups, max_group_size, group_len, items, num_items,
                                     partial_out, partial_lse, stream=None) -> None:
    _check(_lib.paged_attn_decode_cascade_append(
        pool._handle(), _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(block_tables), bt_stride,
        _ptr(context_lens), batch, num_q_heads, scale, max_context_len, partition_size, prefix_len,
        prefix_partition_size, _ptr(group_start), num_groups, max_group_size, group_len, _ptr(items),
        num_items, _ptr(partial_out), _ptr(partial_lse), _ptr(stream)))


def paged_attn_cascade_workspace_size(batch, num_q_heads, head_dim, max_context_len,
                                      partition_size, prefix_len, prefix_partition_size):
    """Returns (partial_out bytes, partial_lse bytes, max_partitions)."""
    a, b, m = ctypes.c_size_t(), ctypes.c_size_t(), ctypes.c_int32()
    _check(_lib.paged_attn_cascade_workspace_size(batch, num_q_heads, head_dim, max_context_len,
                                                  partition_size, prefix_len,
                                                  prefix_partition_size, ctypes.byref(a),
                                                  ctypes.byref(b), ctypes.byref(m)))
    return a.value, b.value, m.value


def paged_attn_decode_cascade(pool: KVPool, q, block_tables, bt_stride, context_lens, batch,
                              num_q_heads, scale, max_context_len, partition_size, prefix_len,
                              prefix_partition_size, partial_out, partial_lse, stream=None) -> None:
    _check(_lib.paged_attn_decode_cascade(pool._handle(), _ptr(q), _ptr(block_tables), bt_stride,
                                          _ptr(context_lens), batch, num_q_heads, scale,
                                          max_context_len, partition_size, prefix_len,
                                          prefix_partition_size, _ptr(partial_out),
                                          _ptr(partial_lse), _ptr(stream)))


def paged_attn_cascade_groups_workspace_size(batch, num_q_heads, head_dim, max_context_len,
                                             partition_size, prefix_len, prefix_partition_size,
                                             group_len):
    """Returns (partial_out bytes, partial_lse bytes, max_partitions)."""
    a, b, m = ctypes.c_size_t(), ctypes.c_size_t(), ctypes.c_int32()
    _check(_lib.paged_attn_cascade_groups_workspace_size(
        batch, num_q_heads, head_dim, max_context_len, partition_size, prefix_len,
        prefix_partition_size, group_len, ctypes.byref(a), ctypes.byref(b), ctypes.byref(m)))
    return a.value, b.value, m.value


def paged_attn_decode_cascade_groups(pool: KVPool, q, block_tables, bt_stride, context_lens, batch,
                                     num_q_heads, scale, max_context_len, partition_size,
                                     prefix_len, prefix_partition_size, group_start, num_groups,
                                     max_group_size, group_len, items, num_items, partial_out,
                                     partial_lse, stream=None) -> None:
    _check(_lib.paged_attn_decode_cascade_groups(
        pool._handle(), _ptr(q), _ptr(block_tables), bt_stride, _ptr(context_lens), batch,
        num_q_heads, scale, max_context_len, partition_size, prefix_len, prefix_partition_size,
        _ptr(group_start), num_groups, max_group_size, group_len, _ptr(items), num_items,
        _ptr(partial_out), _ptr(partial_lse), _ptr(stream)))


def paged_attn_reduce_cascade_groups(partial_out, partial_lse, context_lens, batch, num_q_heads,
                                     head_dim, partition_size, prefix_len, prefix_partition_size,
                                     group_len, max_partitions, out, stream=None) -> None:
    _check(_lib.paged_attn_reduce_cascade_groups(
        _ptr(partial_out), _ptr(partial_lse), _ptr(context_lens), batch, num_q_heads, head_dim,
        partition_size, prefix_len, prefix_partition_size, group_len, max_partitions, _ptr(out),
        _ptr(stream)))


def paged_attn_reduce_cascade(partial_out, partial_lse, context_lens, batch, num_q_heads,
                              head_dim, partition_size, prefix_len, prefix_partition_size,
                              max_partitions, out, stream=None) -> None:
    _check(_lib.paged_attn_reduce_cascade(_ptr(partial_out), _ptr(partial_lse),
                                          _ptr(context_lens), batch, num_q_heads, head_dim,
                                          partition_size, prefix_len, prefix_partition_size,
                                          max_partitions, _ptr(out), _ptr(stream)))


def paged_attn_extend(pool: KVPool, q, q_start, total_q, block_tables, bt_stride, context_lens, batch,
                      num_q_heads, scale, max_context_len, max_chunk, out, stream=None) -> None:
    _check(_lib.paged_attn_extend(pool._handle(), _ptr(q), _ptr(q_start), total_q, _ptr(block_tables),
                                  bt_stride, _ptr(context_lens), batch, num_q_heads, scale,
                                  max_context_len, max_chunk, _ptr(out), _ptr(stream)))


def paged_attn_schedule(context_lens, max_context_len, partition_size, prefix_len=0):
    """Work list (numpy int32, item = part * batch + b) from host context lengths."""
    import numpy as np
    ctx = np.ascontiguousarray(np.asarray(context_lens, dtype=np.int32))
    batch = int(ctx.size)
    n = ctypes.c_int32()
    cap = max(1, batch * max(1, -(-max(max_context_len - prefix_len, 1) // partition_size)
                             if partition_size else 1))
    items = np.zeros(cap, dtype=np.int32)
    _check(_lib.paged_attn_schedule(ctx.ctypes.data_as(_pi32), batch, max_context_len, partition_size,
                                    prefix_len, items.ctypes.data_as(_pi32), cap, ctypes.byref(n)))
    return items[: n.value].copy()


def paged_attn_decode_scheduled(pool: KVPool, q, block_tables, bt_stride, context_lens, batch,
                                num_q_heads, scale, max_context_len, partition_size, items, num_items,
                                out, partial_out=None, partial_lse=None, stream=None) -> None:
    _check(_lib.paged_attn_decode_scheduled(pool._handle(), _ptr(q), _ptr(block_tables), bt_stride,
                                            _ptr(context_lens), batch, num_q_heads, scale,
                                            max_context_len, partition_size, _ptr(items), num_items,
                                            _ptr(out), _ptr(partial_out), _ptr(partial_lse),
                                            _ptr(stream)))


def paged_attn_decode_cascade_scheduled(pool: KVPool, q, block_tables, bt_stride, context_lens, batch,
                                        num_q_heads, scale, max_context_len, partition_size,
                                        prefix_len, prefix_partition_size, items, num_items,
                                        partial_out, partial_lse, stream=None) -> None:
    _check(_lib.paged_attn_decode_cascade_scheduled(
        pool._handle(), _ptr(q), _ptr(block_tables), bt_stride, _ptr(context_lens), batch,
        num_q_heads, scale, max_context_len, partition_size, prefix_len, prefix_partition_size,
        _ptr(items), num_items, _ptr(partial_out), _ptr(partial_lse), _ptr(stream)))


def paged_attn_decode_scheduled_trace(pool: KVPool, q, block_tables, bt_stride, context_lens, batch,
                                      num_q_heads, scale, max_context_len, partition_size, items,
                                      num_items, out, partial_out, partial_lse, trace,
                                      trace_capacity, stream=None) -> None:
    _check(_lib.paged_attn_decode_scheduled_trace(
        pool._handle(), _ptr(q), _ptr(block_tables), bt_stride, _ptr(context_lens), batch,
        num_q_heads, scale, max_context_len, partition_size, _ptr(items), num_items, _ptr(out),
        _ptr(partial_out), _ptr(partial_lse), _ptr(trace), trace_capacity, _ptr(stream)))


def paged_attn_cascade_trace_layout(pool: KVPool, batch, num_q_heads, max_context_len,
                                    partition_size, prefix_len, prefix_partition_size,
                                    num_groups=0, group_len=0) -> dict:
    """Offsets (int32 values) and tiles per item of the trace sections."""
    lay = (ctypes.c_int64 * 7)()
    _check(_lib.paged_attn_cascade_trace_layout(pool._handle(), batch, num_q_heads, max_context_len,
                                                partition_size, prefix_len, prefix_partition_size,
                                                num_groups, group_len, lay))
    keys = ("prefix_offset", "prefix_tiles", "group_offset", "group_tiles", "decode_offset",
            "decode_tiles", "total")
    return dict(zip(keys, [int(x) for x in lay]))


def paged_attn_decode_cascade_trace(pool: KVPool, q, block_tables, bt_stride, context_lens, batch,
                                    num_q_heads, scale, max_context_len, partition_size, prefix_len,
                                    prefix_partition_size, group_start, num_groups, max_group_size,
                                    group_len, items, num_items, partial_out, partial_lse, trace,
                                    trace_capacity, stream=None) -> None:
    _check(_lib.paged_attn_decode_cascade_trace(
        pool._handle(), _ptr(q), _ptr(block_tables), bt_stride, _ptr(context_lens), batch,
        num_q_heads, scale, max_context_len, partition_size, prefix_len, prefix_partition_size,
        _ptr(group_start), num_groups, max_group_size, group_len, _ptr(items), num_items,
        _ptr(partial_out), _ptr(partial_lse), _ptr(trace), trace_capacity, _ptr(stream)))


def paged_attn_check_tables(pool: KVPool, block_tables, context_lens, prefix_len=0,
                            group_start=None, group_len=0) -> None:
    """Host-side check of numpy block tables and lengths (raises PagedAttnError
    with the failing sequence in ``.bad_seq``)."""
    import numpy as np
    bt = np.ascontiguousarray(np.asarray(block_tables, dtype=np.int32))
    ctx = np.ascontiguousarray(np.asarray(context_lens, dtype=np.int32))
    gs = None if group_start is None else np.ascontiguousarray(np.asarray(group_start, dtype=np.int32))
    bad = ctypes.c_int32(-1)
    rc = _lib.paged_attn_check_tables(
        pool._handle(), bt.ctypes.data_as(_pi32), int(bt.shape[1]) if bt.ndim == 2 else 1,
        ctx.ctypes.data_as(_pi32), int(ctx.size), prefix_len,
        gs.ctypes.data_as(_pi32) if gs is not None else None,
        int(gs.size - 1) if gs is not None else 0, group_len, ctypes.byref(bad))
    if rc != PA_OK:
        err = PagedAttnError(rc, _lib.pa_last_error().decode())
        err.bad_seq = bad.value
        raise err


NOALLOC_SCRATCH_BYTES = 64 << 20


def paged_attn_decode_noalloc(pool: KVPool, q, block_tables, bt_stride, context_lens, batch,
                              num_q_heads, scale, max_context_len, partition_size, out,
                              stream=None) -> None:
    _check(_lib.paged_attn_decode_noalloc(pool._handle(), _ptr(q), _ptr(block_tables), bt_stride,
                                          _ptr(context_lens), batch, num_q_heads, scale,
                                          max_context_len, partition_size, _ptr(out), _ptr(stream)))
