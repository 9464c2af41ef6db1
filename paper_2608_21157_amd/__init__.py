"""MI355X-native structured-grid stencil library: HIP kernels for gfx950 behind a C ABI.

``binding`` wraps ``libstencil.so`` (built by ``build``); ``inputs`` generates the seeded
synthetic workloads.  Importing the package loads nothing: the library is loaded on the
first binding call and a missing build raises ImportError there.
"""
