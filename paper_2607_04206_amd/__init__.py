"""MI355X (gfx950) attention for cached diffusion-LLM serving: one call over a
mixed batch of block decodes and whole non-causal prefills on a paged KV cache.

The C ABI lives in include/sangam_attn.h and libsangam_attn.so; this package is
its thin Python binding (``plan`` and ``forward``)."""
from .attn import Plan, forward, plan  # noqa: F401
from ._lib import SangamError  # noqa: F401
