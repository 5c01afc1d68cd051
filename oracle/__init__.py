"""CPU oracle for paged decode attention -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, the package smoke check and the benchmark's CPU-baseline leg
may import this package.  It shares no code with the HIP path.

Modules: ``attention`` (fp64 numpy oracle, split partials and their merge),
``brute`` (pure-Python fsum brute force), ``gate`` (parity tolerance),
``kvcache`` (appending a decode step's K/V to the paged cache), ``extend``
(causal attention of a chunk of new tokens over the paged cache).
Every function is pinned by the CPU tests against closed forms, invariants,
brute force and hand-derived golden values; no function is parity-unpinned.
"""
from .attention import (  # noqa: F401
    bf16_to_f64, decode_workload, gather_sequence, merge_partials, paged_decode,
    softmax_attention, split_partials,
)
from .gate import GateReport, compare  # noqa: F401
from .extend import extend_attention  # noqa: F401
from .kvcache import append_kv  # noqa: F401
