/*
 * libsteel measurement helpers (not part of the attention path): the
 * achievable rate of the bf16 matrix-core instruction the attention kernels
 * use (v_mfma_f32_32x32x16_bf16), as the context for their roofline
 * fraction, and the issue rates of the softmax's exponential and fma
 * (v_exp_f32, v_fma_f32), the basis of the plain-ALU estimate.  The paper measures against its device's
 * peak (Section V-A); here the published peak (256 CU x 2.4 GHz x 4096 bf16
 * flop/clk/CU) is the denominator, and the matrix-core rate shows what the
 * chip sustains under the matrix cores' power draw for given operand data.
 */
#ifndef STEEL_BENCH_H
#define STEEL_BENCH_H

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Enqueue grid workgroups of waves_per_wg waves; every wave runs iters
 * iterations of 16 v_mfma_f32_32x32x16_bf16 (2 * 32 * 32 * 16 flop each).
 *
 *   operands  device, 8 x 64 x 8 bf16 (512 x 16 bytes), 16-byte aligned:
 *             four A then four B fragments, 16 bytes per lane each; the
 *             caller chooses the values (constant, N(0,1), ...)
 *   sink      device float [grid * 64 * waves_per_wg]: one sum per lane, so
 *             the products are not optimised away
 *   clocks    device uint64 [2 * grid]: per workgroup, shader-clock cycles
 *             (s_memtime) and 100 MHz reference ticks (s_memrealtime) over
 *             its loop; their ratio is the average clock of that workgroup
 *   stream    hipStream_t as void*, or NULL
 *
 * Returns 0 when enqueued, 1 on an invalid argument (nothing enqueued), 3 on
 * a launch error.  Timing is the caller's (events around the call).
 */
int steel_mfma_peak(const void* operands, int iters, int grid, int waves_per_wg, float* sink,
                    unsigned long long* clocks, void* stream);

/*
 * Enqueue grid workgroups of waves_per_wg waves; every lane runs iters
 * iterations over eight independent floats of one VALU instruction of the
 * online softmax (Algorithm 1, second stage): op 0 x <- 2^(-x) (eight
 * v_exp_f32 per iteration, the negation folded into the instruction), op 1
 * x <- x * 0.999 + 0.0001 (eight v_fma_f32).
 *
 *   seed    device float [8]: the starting values (any finite values)
 *   sink    device float [grid * 64 * waves_per_wg], as for steel_mfma_peak
 *   clocks  device uint64 [2 * grid], as for steel_mfma_peak: shader-clock
 *           cycles over the loop give the cycles per 64-lane instruction
 *   stream  hipStream_t as void*, or NULL
 *
 * Returns 0 when enqueued, 1 on an invalid argument (nothing enqueued), 3 on
 * a launch error.
 */
int steel_valu_rate(int op, const float* seed, int iters, int grid, int waves_per_wg, float* sink,
                    unsigned long long* clocks, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* STEEL_BENCH_H */
