"""MI355X (gfx950) paged decode attention.

The compute lives in the HIP library ``libpaged_attn.so`` behind the C ABI in
``include/paged_attn.h``; ``binding`` is its ctypes binding and ``device``
moves one decode step's inputs into device memory with torch.  Importing the
package fails if the library has not been built.
"""
from . import binding  # noqa: F401  (raises ImportError when the library is missing)
from .binding import (  # noqa: F401
    KVPool, PagedAttnError, kv_pool_alloc, kv_pool_claim, kv_pool_create, kv_pool_destroy,
    kv_pool_layout, kv_pool_num_free, kv_pool_num_shared, kv_pool_refcount, kv_pool_release, kv_pool_retain,
    pa_last_error, pa_stream_copy, pa_version, paged_attn_decode, paged_attn_decode_trace,
    paged_attn_num_partitions, paged_attn_reduce, paged_attn_workspace_size,
    paged_attn_cascade_workspace_size, paged_attn_decode_cascade, paged_attn_reduce_cascade,
)
