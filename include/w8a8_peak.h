/*
 * w8a8_peak.h -- measured ceilings of the device for the benchmark's roofline
 * columns (libw8a8_peak.so; not part of the W8A8 path).
 *
 * The benchmark reports each kernel against the published peaks (dense INT8
 * matrix rate, HBM bandwidth) and against what these probes reach on the
 * device it runs on.  All launch asynchronously on `stream` (a hipStream_t);
 * the caller times them.  Return 0, 1 for a bad argument, 3 for a launch error.
 */
#ifndef W8A8_PEAK_H
#define W8A8_PEAK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* `blocks` workgroups of 4 waves, each wave running 8 independent chains of
   `iters` v_mfma_i32_16x16x64_i8 on register operands.  sink: device int[blocks]
   (written only in a case the operands cannot produce). */
int w8a8_peak_mfma_i8(int blocks, int iters, int* sink, void* stream);
/* Integer operations (2 per multiply-add) one such launch performs. */
double w8a8_peak_mfma_i8_ops(int blocks, int iters);

/* Reads `bytes` (a multiple of 16, 16-byte aligned device buffer) once with
   16-byte non-temporal loads, `blocks` workgroups of 256 threads.
   sink: device unsigned[1] (written only in a case the data make unlikely). */
int w8a8_peak_read(const void* buf, size_t bytes, int blocks, unsigned* sink, void* stream);

/* The traffic of a wide INT8 GEMM with one pass over its weights and no
   arithmetic: w holds n rows of k bytes (n and k multiples of 64, k at most
   1536, 16-byte aligned), read once with 16-byte non-temporal loads in runs
   of 64 rows; after each run its 64 columns of `rows` bf16 output rows are
   written to out (rows x n bf16, row-major, 16-byte aligned) as 128-byte row
   segments.  `blocks` workgroups of 256 threads take the runs grid-stride.
   sink as above. */
int w8a8_peak_read_write(const void* w, int64_t n, int k, void* out, int rows, int blocks,
                         unsigned* sink, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* W8A8_PEAK_H */
