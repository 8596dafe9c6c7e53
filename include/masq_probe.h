/*
 * masq_probe.h -- peak probes for the benchmark (libmasq_probe.so).  They
 * measure what the MI355X sustains, to report the layer's kernels against a
 * measured peak beside the spec-sheet one.  Not part of the layer's ABI.
 *
 * All pointers are device pointers owned by the caller; stream is a
 * hipStream_t as void* (NULL = default stream).  The calls only enqueue work.
 * Return 0 on success, -1 for invalid arguments (nothing enqueued), -2 if the
 * launch was rejected.
 */
#ifndef MASQ_PROBE_H
#define MASQ_PROBE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* int8 MFMA issue with no memory traffic in the loop: `blocks` workgroups of
 * four wave64s, each wave running `iters` rounds of 8 independent
 * v_mfma_i32_32x32x32_i8 chains on register operands.  out: int32
 * [blocks * 256], one value per thread (keeps the chains live).  The number
 * of int8 operations it performs is masq_probe_mfma_i8_ops(blocks, iters). */
int masq_probe_mfma_i8(int32_t blocks, int32_t iters, int32_t* out, void* stream);
int64_t masq_probe_mfma_i8_ops(int32_t blocks, int32_t iters);

/* Linear read of `bytes` bytes of buf (16-byte aligned, bytes % 16 == 0) with
 * coalesced 16-byte loads by `blocks` workgroups of 256 threads.  out: int32
 * [blocks * 256], an xor of what each thread read. */
int masq_probe_read(const void* buf, int64_t bytes, int32_t blocks, int32_t* out, void* stream);

/* L2 -> LDS transfer through LDS DMA (global_load_lds_dwordx4), the path
 * that feeds the GEMM's K stages: `blocks` workgroups of 8 waves, each wave
 * moving `iters` rounds of four 1 KB instructions (16 rows x 64 bytes, the
 * GEMM's stage-row pattern) into LDS, from rows spread over the first
 * `region` bytes of buf (4 KB pitch; region >= 256 KB, buf 16-byte
 * aligned).  Bytes moved: masq_probe_lds_dma_bytes(blocks, iters).  out:
 * int32 [blocks]. */
int masq_probe_lds_dma(const void* buf, int64_t region, int32_t blocks, int32_t iters,
                       int32_t* out, void* stream);
int64_t masq_probe_lds_dma_bytes(int32_t blocks, int32_t iters);

#ifdef __cplusplus
}
#endif

#endif /* MASQ_PROBE_H */
