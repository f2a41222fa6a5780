"""MI355X (gfx950) implementation of MixRT's per-pixel rendering path.

- `mixrt`: ctypes binding of libmixrt.so (the C ABI of include/mixrt.h).
- `synth`: seeded synthetic inputs shaped like the paper's workloads.
- `build`: hipcc build of libmixrt.so and libmixrt_microbench.so.
- `microbench`: binding of the roofline microbenchmarks (gather, copy, MFMA,
  device properties) the measurements are quoted against.
"""
__all__ = ["mixrt", "synth", "build", "microbench"]
