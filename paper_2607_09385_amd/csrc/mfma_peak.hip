// Achievable bf16 matrix-core rate on this chip, and the issue rates of the
// softmax's VALU instructions (measurement only; not part of the attention
// path).  Every wave streams v_mfma_f32_32x32x16_bf16 (the
// instruction of the score and output products) over operands loaded once
// from memory: four A and four B fragments per lane, combined in a rotating
// pattern so consecutive instructions see different data, into four
// independent accumulators.  The operand values decide how much power the
// matrix cores draw and therefore the clock the chip holds: constant operands
// against N(0,1) operands bound what the attention kernels can reach.
//
// Each workgroup's first lane also records the elapsed shader-clock cycles
// (s_memtime) and the elapsed 100 MHz reference ticks (s_memrealtime) of its
// loop, from which the average clock during the run follows.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/steel_bench.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__global__ __launch_bounds__(1024) void k_mfma_peak(const bf16x8* __restrict__ ops, int iters,
                                                    float* __restrict__ sink,
                                                    unsigned long long* __restrict__ clocks) {
  const int lane = threadIdx.x & 63;
  bf16x8 a0 = ops[0 * 64 + lane], a1 = ops[1 * 64 + lane], a2 = ops[2 * 64 + lane],
         a3 = ops[3 * 64 + lane];
  bf16x8 b0 = ops[4 * 64 + lane], b1 = ops[5 * 64 + lane], b2 = ops[6 * 64 + lane],
         b3 = ops[7 * 64 + lane];
  f32x16 c0 = {}, c1 = {}, c2 = {}, c3 = {};
  const unsigned long long t0 = __builtin_amdgcn_s_memtime();
  const unsigned long long r0 = __builtin_amdgcn_s_memrealtime();
  for (int it = 0; it < iters; ++it) {
    c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b0, c0, 0, 0, 0);
    c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b1, c1, 0, 0, 0);
    c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a2, b2, c2, 0, 0, 0);
    c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a3, b3, c3, 0, 0, 0);
    c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b2, c0, 0, 0, 0);
    c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a2, b3, c1, 0, 0, 0);
    c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a3, b0, c2, 0, 0, 0);
    c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b1, c3, 0, 0, 0);
    c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a2, b0, c0, 0, 0, 0);
    c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a3, b1, c1, 0, 0, 0);
    c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b2, c2, 0, 0, 0);
    c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b3, c3, 0, 0, 0);
    c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a3, b2, c0, 0, 0, 0);
    c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b3, c1, 0, 0, 0);
    c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b0, c2, 0, 0, 0);
    c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a2, b1, c3, 0, 0, 0);
  }
  const unsigned long long t1 = __builtin_amdgcn_s_memtime();
  const unsigned long long r1 = __builtin_amdgcn_s_memrealtime();
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < 16; ++i) s += c0[i] + c1[i] + c2[i] + c3[i];
  sink[(size_t)blockIdx.x * blockDim.x + threadIdx.x] = s;
  if (threadIdx.x == 0) {
    clocks[2 * (size_t)blockIdx.x] = t1 - t0;
    clocks[2 * (size_t)blockIdx.x + 1] = r1 - r0;
  }
}

// Issue rates of the softmax's VALU instructions: every lane iterates eight
// independent chains, x <- 2^(-x) (op 0: eight v_exp_f32 per iteration, the
// negation an operand modifier; the values settle near 0.64) or
// x <- x * 0.999 + 1e-4 (op 1: eight v_fma_f32).  The shader-clock cycles of
// the loop give the cycles per 64-lane instruction whatever the clock; with
// one wave per SIMD that is the issue interval of a single wave, with several
// the SIMD's throughput.
template <int OP>
__global__ __launch_bounds__(1024) void k_valu_rate(const float* __restrict__ seed, int iters,
                                                    float* __restrict__ sink,
                                                    unsigned long long* __restrict__ clocks) {
  const int lane = threadIdx.x & 63;
  float x[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) x[i] = seed[i] + 0.001f * lane;
  const unsigned long long t0 = __builtin_amdgcn_s_memtime();
  const unsigned long long r0 = __builtin_amdgcn_s_memrealtime();
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      if constexpr (OP == 0) x[i] = __builtin_amdgcn_exp2f(-x[i]);
      else x[i] = __builtin_fmaf(x[i], 0.999f, 1e-4f);
    }
  }
  const unsigned long long t1 = __builtin_amdgcn_s_memtime();
  const unsigned long long r1 = __builtin_amdgcn_s_memrealtime();
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i) s += x[i];
  sink[(size_t)blockIdx.x * blockDim.x + threadIdx.x] = s;
  if (threadIdx.x == 0) {
    clocks[2 * (size_t)blockIdx.x] = t1 - t0;
    clocks[2 * (size_t)blockIdx.x + 1] = r1 - r0;
  }
}

}  // namespace

extern "C" int steel_valu_rate(int op, const float* seed, int iters, int grid, int waves_per_wg,
                               float* sink, unsigned long long* clocks, void* stream) {
  if ((op != 0 && op != 1) || !seed || !sink || !clocks || iters < 1 || grid < 1 ||
      waves_per_wg < 1 || waves_per_wg > 16)
    return 1;
  if (op == 0)
    hipLaunchKernelGGL(k_valu_rate<0>, dim3(grid), dim3(64 * waves_per_wg), 0,
                       static_cast<hipStream_t>(stream), seed, iters, sink, clocks);
  else
    hipLaunchKernelGGL(k_valu_rate<1>, dim3(grid), dim3(64 * waves_per_wg), 0,
                       static_cast<hipStream_t>(stream), seed, iters, sink, clocks);
  return hipGetLastError() == hipSuccess ? 0 : 3;
}

extern "C" int steel_mfma_peak(const void* operands, int iters, int grid, int waves_per_wg,
                               float* sink, unsigned long long* clocks, void* stream) {
  if (!operands || !sink || !clocks || iters < 1 || grid < 1 || waves_per_wg < 1 ||
      waves_per_wg > 16)
    return 1;
  hipLaunchKernelGGL(k_mfma_peak, dim3(grid), dim3(64 * waves_per_wg), 0,
                     static_cast<hipStream_t>(stream), static_cast<const bf16x8*>(operands), iters,
                     sink, clocks);
  return hipGetLastError() == hipSuccess ? 0 : 3;
}
