"""MI355X-native structured-grid stencil library (HIP for gfx950 behind a C ABI)."""
