"""MI355X-native forward/backward of one skip-collocated Pulse pipeline stage.

The compute lives in ``libpulse_stage.so`` (hand-written HIP for gfx950 behind
a C ABI declared in ``include/pulse_stage.h``); :mod:`.stage` is a thin ctypes
binding over it that marshals torch device pointers and streams.  Importing
this package does not load the library; ``paper_2606_19163_amd.stage`` does,
and fails loudly when it has not been built.
"""

__all__ = ["configs", "synth"]
