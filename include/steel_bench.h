/*
 * libsteel measurement helpers (not part of the attention path): the
 * achievable rate of the bf16 matrix-core instruction the attention kernels
 * use (v_mfma_f32_32x32x16_bf16), as the context for their roofline
 * fraction, the issue rates of the softmax's exponential and fma
 * (v_exp_f32, v_fma_f32), the basis of the plain-ALU estimate, and the LDS
 * and global -> LDS copy rates that the tiles of Algorithm 1 move through.
 * The paper measures against its device's peak (Section V-A); here the published peak (256 CU x 2.4 GHz x 4096 bf16
 * flop/clk/CU) is the denominator, and the matrix-core rate shows what the
 * chip sustains under the matrix cores' power draw for given operand data.
 */
#ifndef STEEL_BENCH_H
#define STEEL_BENCH_H

#include <stddef.h>

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

/*
 * Enqueue grid workgroups of waves_per_wg waves; every lane moves 16 bytes
 * between its VGPRs and a 32 KiB LDS buffer eight times per iteration, each
 * time in another 1 KiB block of lane-contiguous slots (no bank conflicts):
 * op 0 ds_read_b128, op 1 two ds_read_b64_tr_b16 (the transposed reads the
 * P V product takes its V fragments with), op 2 ds_write_b128.  Bytes moved
 * per CU over the loop's shader-clock cycles give the LDS rate of that
 * instruction at that number of resident waves.
 *
 *   sink    device uint32 [grid * 64 * waves_per_wg]: one value per lane
 *   clocks  device uint64 [2 * grid], as for steel_mfma_peak
 *   stream  hipStream_t as void*, or NULL
 *
 * Returns 0 when enqueued, 1 on an invalid argument (nothing enqueued), 3 on
 * a launch error.
 */
int steel_lds_rate(int op, int iters, int grid, int waves_per_wg, unsigned* sink,
                   unsigned long long* clocks, void* stream);

/*
 * Enqueue grid workgroups of waves_per_wg waves (1, 2, 4, 8 or 16); each
 * fills a 32 KiB LDS buffer from src with global_load_lds_dwordx4 (the tile
 * copy of the attention kernels), waits for its copies, and refills, iters
 * times.  Workgroup b reads within the (b % 8)-th eighth of src, at offsets
 * that move by 32 KiB per fill, so a source of a few MiB stays in the L2s.
 *
 *   src        device, 16-byte aligned, src_bytes >= 512 KiB
 *   sink, clocks, stream  as for steel_lds_rate
 *
 * Returns 0 when enqueued, 1 on an invalid argument (nothing enqueued), 3 on
 * a launch error.
 */
int steel_copy_rate(const void* src, size_t src_bytes, int iters, int grid, int waves_per_wg,
                    unsigned* sink, unsigned long long* clocks, void* stream);

/*
 * Enqueue grid workgroups of eight waves (one per CU for grid = 256); waves
 * w and w + 4 share SIMD w % 4.  Waves 0-3 run mfma_iters iterations of four
 * v_mfma_f32_32x32x16_bf16 when bit 0 of mode is set; waves 4-7 run
 * valu_iters iterations of eight independent VALU chains (vop 0 v_exp_f32,
 * vop 1 v_fma_f32, as steel_valu_rate) when bit 1 is set (mode 1, 2 or 3).
 * Comparing each role's cycles with both on against each alone measures how
 * far one wave's matrix-core work and another wave's VALU work on the same
 * SIMD overlap.
 *
 *   operands  device, as for steel_mfma_peak (fragments 0, 1, 4 and 5 used);
 *             may be NULL when bit 0 of mode is clear
 *   seed      device float [8], as for steel_valu_rate; may be NULL when bit
 *             1 of mode is clear
 *   sink      device float [grid * 512]: one value per lane
 *   clocks    device uint64 [2 * 8 * grid]: per wave (workgroup-major),
 *             shader-clock cycles and 100 MHz reference ticks of its own loop
 *   stream    hipStream_t as void*, or NULL
 *
 * Returns 0 when enqueued, 1 on an invalid argument (nothing enqueued), 3 on
 * a launch error.
 */
int steel_mix_rate(int mode, int vop, const void* operands, int mfma_iters, const float* seed,
                   int valu_iters, int grid, float* sink, unsigned long long* clocks, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* STEEL_BENCH_H */
