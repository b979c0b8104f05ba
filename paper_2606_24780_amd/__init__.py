"""MI355X (gfx950) FP32 GPT-2 training step: HIP kernels behind a C ABI
(libbt.so, include/bt.h) with a thin ctypes binding (``bt``) and seeded
synthetic inputs (``synth``).  The library is loaded on first use."""
__version__ = "0.1.0"
