"""PASK decode hot path on MI355X (gfx950): structure-conditioned KV
persistence and decode attention over the mixed bf16 / int4 cache.

`pask` is the binding of the C ABI (libpask.so); `session` allocates a cache
and its workspace with torch and drives the ABI for a batch of sequences.
"""

__all__ = ["pask", "session"]
