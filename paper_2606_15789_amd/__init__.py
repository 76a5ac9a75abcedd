"""MI355X-native chunked rANS decoder for lossless LLM weight compression.

``wc``     -- ctypes binding of libwc (include/wc.h): analyze, encode, decode.
``synth``  -- seeded synthetic weight tensors (inputs only, no codec arithmetic).
``build``  -- compiles libwc.so for gfx950.
"""

__all__ = ["wc", "synth", "build"]
