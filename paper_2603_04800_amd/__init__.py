"""MI355X (gfx950) implementation of MASQuant's modality-aware quantized linear.

The inference rule of MASQuant (Sec. 4.3): token rows are smoothed by their
modality's factors S_m^-1, quantized per token to int8, multiplied by one
shared int8 weight Q(S_t W) with int32 accumulation, dequantized, and rows of
non-text modalities receive the low-rank Cross-Modal Compensation
(x S_m^-1) L1^m L2^m.

Submodules
  ops        ctypes binding of the HIP library libmasq.so (the C ABI of
             include/masq.h); importing it requires the built library.
  calibrate  offline host-side calibration producing the layer's artifacts.
  build      compiles libmasq.so for gfx950.
"""

__all__ = ["ops", "calibrate", "build"]
