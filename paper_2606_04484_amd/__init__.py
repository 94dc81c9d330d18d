"""MI355X-native merged actor update for multi-turn agentic RL.

Timeline merging (Section 4.4.2, Algorithm 1), a packed variable-length
decoder block and the fused LM-head / clipped policy-gradient loss, as
hand-written HIP kernels for gfx950 behind the C ABI in include/aj.h.
This package is the thin binding (capi) plus the host-side step driver
(actor); importing it does not load the library until a call needs it.
"""
from .capi import AjError  # noqa: F401
