"""SpeechKV hot path for AMD Instinct MI355X (gfx950).

SpeechKV (arXiv 2607.06827) pools the speech keys and values of deep LLM layers
window by window with a learned gate and lets full-resolution queries attend
over the shorter cache.  The work is done by HIP kernels in libspeechkv.so;
`paper_2607_06827_amd.speechkv` is the ctypes binding (it raises on import if
the library is not built), `paper_2607_06827_amd.inputs` the seeded synthetic
inputs.
"""

__version__ = "0.1.0"
