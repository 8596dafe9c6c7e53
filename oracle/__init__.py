"""CPU oracle for the modality-aware W8A8 + low-rank linear (MASQuant).

TEST INFRASTRUCTURE ONLY.  This package is the slow, plain reference that the
GPU library is checked against.  Only the test suite, the smoke check and the
CPU-baseline leg of the benchmark may import it; the product path never does,
and it shares no code with the HIP kernels or their Python binding.

Modules
-------
``inference``   the inference rule of Sec. 4.3 (final case equation) with every
                rounding point fixed: smoothing, per-token int8 quantization
                (eq. PTQ), exact int32 GEMM, dequantization, low-rank
                compensation, output cast.
``calibration`` the offline factors the inference consumes: MAS initial
                smoothing factors (Sec. 4.2), the shared weight Q(S_t W)
                (eq. PTQ per output channel), and the Cross-Modal Compensation
                factors L1, L2 from SVD whitening (Sec. 4.3, eq. l1l2).
``bf16``        bit-level bfloat16 conversions used by both.

Pins (checked by the CPU test suite, not by retyping formulas):
  * codes / scales: brute force with numpy.float32 scalars on tiny shapes,
    amax -> +-127, |q| <= 127, idempotent re-quantization, the rounding-error
    bound |xs - q*delta| <= delta/2 of eq. PTQ, zero rows;
  * int32 GEMM: int64 einsum vs fp64 BLAS, known answers (q = 1, Wq = 127 I);
  * computational invariance (Sec. 3.1): activations unquantized and full-rank
    factors give X W to fp64 rounding for every modality;
  * s_m = s_t with the float difference base makes the compensation vanish,
    leaving plain SmoothQuant W8A8 bit-for-bit;
  * full-rank truncation reproduces diag(s_m) W exactly (eq. l1l2);
  * Theorem 2 (optimal low-rank compensation) against an independent SVD of
    X_m S_m^-1 dW (Eckart-Young), and no worse than other rank-r choices;
  * Theorem 1 (Sec. 4.2), qualitatively: per-modality factors recover the
    activation SQNR that a unified factor set by another modality loses;
  * bf16 helpers exhaustively against torch's CPU casts;
  * the whole layer element by element against its definition in Python
    scalars and exact rationals on tiny inputs (brute force).
The paper prints no worked numerical example for the layer, so no pin uses
printed values.
"""
