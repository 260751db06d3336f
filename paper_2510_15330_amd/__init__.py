"""MI355X (gfx950) paged decode attention with beLLMan's length controller.

The numerical work runs in ``libbellman.so`` (HIP kernels behind a C ABI,
declared in ``include/bellman.h``); this package marshals torch tensors into
that ABI and nothing more.  There is no fallback: every call raises if the
library is not built.
"""
from ._binding import (  # noqa: F401
    BellmanError,
    Controller,
    IMPL_AUTO,
    IMPL_MFMA,
    IMPL_VALU,
    calibrate_thresholds,
    decode_attention,
    device_errors,
    kv_append,
    last_error,
    length_cap,
    library,
    library_path,
    reserve_workspace,
    shutdown,
    version,
)
