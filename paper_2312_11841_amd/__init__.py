"""MI355X (gfx950) implementation of MixRT's per-pixel rendering path.

- `mixrt`: ctypes binding of libmixrt.so (the C ABI of include/mixrt.h).
- `synth`: seeded synthetic inputs shaped like the paper's workloads.
- `build`: hipcc build of libmixrt.so.
"""
__all__ = ["mixrt", "synth", "build"]
