"""MI355X-native prefill / decode hot path of a dense GQA decoder layer.

The compute lives in ``libps.so`` (hand-written HIP for gfx950 behind a C
ABI, declared in ``include/ps.h``); ``binding`` marshals arguments to it and
fails loudly when the library is missing. ``accounting`` holds the
algorithmic FLOP/byte counts used to express timings as roofline fractions.
Importing the package does not load the library.
"""
__version__ = "0.2.0"
