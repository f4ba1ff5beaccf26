"""metro: an MI355X-native batched agent-LLM forward pass (chunked prefill + decode).

The compute lives in ``libmetro.so`` (hand-written HIP for gfx950 behind a C ABI,
declared in ``include/metro.h``).  ``paper_2411_03519_amd.metro`` is the thin
ctypes binding; importing it fails loudly when the library has not been built.
``paper_2411_03519_amd.synth`` draws the seeded synthetic inputs.
"""

__version__ = "0.1.0"
