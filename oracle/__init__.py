"""Plain, slow fp64 CPU oracles: paged chunked-prefill attention, the KV append, and chunked
prefill of a KDA (gated delta-rule) layer with state snapshot and resume.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the bench's CPU-baseline leg
may import this package.  It shares no code with the HIP path: no kernels, helpers, tables or
pre/post-processing, and it never imports the product package.

Every function states the passage of the paper it follows.  All functions are pinned by the
``-m "not gpu"`` tests (library cross-check, closed forms, invariants, brute force), so none is
"parity unpinned".
"""
from .attention import (  # noqa: F401
    bf16_bits_to_f64,
    num_blocks,
    gather_positions,
    append_kv,
    attention_rows,
    chunked_prefill,
    chunked_prefill_rows,
    probabilities,
    merge_partials,
)
from . import kda  # noqa: F401,E402
