/* Measurement helper library (libsa_bench.so), separate from the attention
 * path: a sustained bf16 MFMA throughput probe, used to quote the attention
 * kernel's MFMA utilisation against the matrix-core rate the chip actually
 * sustains, next to the published peak.
 */
#ifndef SA_BENCH_H
#define SA_BENCH_H

#ifdef __cplusplus
extern "C" {
#endif

/* Runs v_mfma_f32_32x32x16_bf16 back to back (four independent accumulation
 * chains per wave, 1024 workgroups of 4 waves) for `iters` iterations of 16
 * MFMAs each, `reps` times, on the current device and the null stream.
 * Operands are bf16 values in [-2, -1] U [1, 2] whose mantissa bits change
 * every iteration (random_operands = 1), or all zero (random_operands = 0);
 * MFMA power, and with it the sustained clock, depends on the operand bits.
 * Writes the best of the `reps` runs: *tflops (TFLOP/s over the whole launch)
 * and *ghz (shader clock from s_memtime against s_memrealtime).
 * Allocates and frees a small device buffer.  Returns 0, or -1 on a HIP
 * error or iters < 1 or reps < 1 or a NULL output pointer.
 */
int sa_bench_mfma_peak(int random_operands, int iters, int reps, float* tflops, float* ghz);

#ifdef __cplusplus
}
#endif

#endif
