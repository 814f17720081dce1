"""MI355X-native Fibonacci-offset sparse attention (fibattn).

The compute path is libfibattn.so (hand-written HIP for gfx950 behind the C ABI in
include/fibattn.h); `fibattn` is its thin Python binding.  Importing this package
does not load the library; the first call does, and raises if it is not built.
"""
from .fibattn import (FibattnError, fibattn_backward, fibattn_backward_workspace_bytes,  # noqa: F401
                      fibattn_forward, fibattn_rope, fibattn_rope_qk, fibattn_rung_table, fibattn_timing_begin,
                      fibattn_timing_end)
