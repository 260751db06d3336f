"""MI355X (gfx950) paged decode attention with beLLMan's length controller,
and the prompt (prefill) path that fills the cache before decoding.

The numerical work runs in ``libbellman.so`` (HIP kernels behind a C ABI,
declared in ``include/bellman.h``); this package marshals torch tensors into
that ABI and nothing more.  There is no fallback: every call raises if the
library is not built.
"""
from ._binding import (  # noqa: F401
    FIXED_SCRATCH_BYTES,
    BellmanError,
    Controller,
    calibrate_thresholds,
    decode_attention,
    decode_attention_noalloc,
    decode_step,
    device_errors,
    kv_append,
    kv_write,
    last_error,
    length_cap,
    library,
    library_path,
    prefill_attention,
    probe_gather,
    reserve_workspace,
    shutdown,
    version,
)
