"""Span-query prefill attention over a paged KV cache, for AMD MI355X (gfx950).

Thin Python binding of ``libspanq.so`` (C-ABI declared in ``include/spanq.h``).
This module only marshals arguments: hashing, planning, page writes and every
attention step run in the native library and its HIP kernels.  PyTorch is used
by callers for device memory and streams; it is imported first so that the
library binds to the same HIP runtime as torch.
"""
from ._lib import (  # noqa: F401
    SPAN_BF16,
    SPAN_F32,
    SPAN_HASH_FRAG_TAG,
    SPAN_HASH_ROOT,
    Model,
    Plan,
    Pool,
    SpanError,
    hash_mix,
    hash_pages,
    library_path,
    load,
    probe_mfma_peak,
    probe_read_peak,
)
