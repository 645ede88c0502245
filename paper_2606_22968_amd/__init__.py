"""libmocap_attn: chunked causal prefill attention for AMD Instinct MI355X.

The HIP kernels and the C ABI live in ``csrc/`` and ``include/mocap_attn.h``;
``binding`` wraps the C entry points with ctypes, ``prefill`` drives a whole
chunk sequence, ``synth`` builds seeded synthetic inputs and ``build``
compiles the library for gfx950.  Importing the package loads nothing; the
shared library is loaded on first use and its absence is an error.
"""
__all__ = ["binding", "prefill", "synth", "build"]
