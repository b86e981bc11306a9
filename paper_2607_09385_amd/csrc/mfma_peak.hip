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
// loop, from which the average clock during the run follows.  The same file
// measures the LDS and global -> LDS copy rates the attention kernels lean
// on (steel_lds_rate, steel_copy_rate).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/steel_bench.h"
#include "attn_common.h"

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
  __syncthreads();  // the loop is timed from the first wave's start to the last wave's end
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
  __syncthreads();
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
  __syncthreads();  // the loop is timed from the first wave's start to the last wave's end
  const unsigned long long t0 = __builtin_amdgcn_s_memtime();
  const unsigned long long r0 = __builtin_amdgcn_s_memrealtime();
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      if constexpr (OP == 0) x[i] = __builtin_amdgcn_exp2f(-x[i]);
      else x[i] = __builtin_fmaf(x[i], 0.999f, 1e-4f);
    }
  }
  __syncthreads();
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

// LDS throughput: every wave of a workgroup moves 16 bytes per lane eight
// times per iteration between VGPRs and a 32 KiB LDS buffer, each time in a
// different 1 KiB block (lane-contiguous slots, no bank conflicts): op 0
// ds_read_b128, op 1 two ds_read_b64_tr_b16 (the transposed reads of the V
// fragments), op 2 ds_write_b128.  Bytes per CU over the shader-clock cycles
// of the loop give the rate whatever the clock.
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) u32x4 lds_u32x4;

template <int OP>
__global__ __launch_bounds__(1024) void k_lds_rate(int iters, unsigned* __restrict__ sink,
                                                   unsigned long long* __restrict__ clocks) {
  __shared__ __attribute__((aligned(1024))) char buf[32768];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  for (int i = t; i < 32768 / 16; i += blockDim.x) ((u32x4*)buf)[i] = u32x4{(unsigned)i, 1u, 2u, 3u};
  __syncthreads();
  u32x4 acc = {0u, 0u, 0u, 0u};
  s16x4 acc2 = {0, 0, 0, 0};
  __syncthreads();  // the loop is timed from the first wave's start to the last wave's end
  const unsigned long long t0 = __builtin_amdgcn_s_memtime();
  const unsigned long long r0 = __builtin_amdgcn_s_memrealtime();
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const uint32_t off = (uint32_t)((((wave * 8 + j + it) & 31) * 64 + lane) * 16);
      // volatile: every access is made, none is merged, hoisted or dropped
      if constexpr (OP == 0) {
        acc += *(const volatile lds_u32x4*)(buf + off);
      } else if constexpr (OP == 1) {
        const s16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(buf + off));
        const s16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(buf + off + 8));
        acc2 += a + b;
      } else {
        *(volatile lds_u32x4*)(buf + off) = u32x4{(unsigned)it, (unsigned)j, 0u, 0u};
      }
    }
  }
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): the last LDS operations are done
  __syncthreads();
  const unsigned long long t1 = __builtin_amdgcn_s_memtime();
  const unsigned long long r1 = __builtin_amdgcn_s_memrealtime();
  sink[(size_t)blockIdx.x * blockDim.x + t] = acc[0] + acc[1] + (unsigned)(acc2[0] + acc2[1]);
  if (t == 0) {
    clocks[2 * (size_t)blockIdx.x] = t1 - t0;
    clocks[2 * (size_t)blockIdx.x + 1] = r1 - r0;
  }
}

// Global -> LDS copy throughput with the attention kernels' copy instruction
// (global_load_lds_dwordx4): each workgroup fills a 32 KiB LDS buffer from
// its XCD's eighth of the source (L2-resident when the source is a few MiB),
// waits for the copies, and starts the next fill at another offset.
__global__ __launch_bounds__(1024) void k_copy_rate(const char* __restrict__ src, long long region,
                                                    int iters, unsigned* __restrict__ sink,
                                                    unsigned long long* __restrict__ clocks) {
  __shared__ __attribute__((aligned(1024))) char buf[32768];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6, nw = (int)blockDim.x >> 6;
  const int per = 32 / nw;  // 1 KiB copies per wave per fill
  const char* base = src + (size_t)(blockIdx.x & 7) * region;
  const uint32_t lds0 = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)buf;
  unsigned acc = 0;
  __syncthreads();  // the loop is timed from the first wave's start to the last wave's end
  const unsigned long long t0 = __builtin_amdgcn_s_memtime();
  const unsigned long long r0 = __builtin_amdgcn_s_memrealtime();
  for (int it = 0; it < iters; ++it) {
    const long long off = (((long long)(blockIdx.x >> 3) * 7919 * 64 + (long long)it * 32768) %
                           (region - 32768 + 1)) & ~1023ll;
    for (int j = 0; j < per; ++j)
      steel::copy16_to_lds(base + off, (uint32_t)(((wave * per + j) * 64 + lane) * 16),
                           lds0 + (uint32_t)(wave * per + j) * 1024u);
    steel::wait_vm<0>();
    __syncthreads();
    acc += *(const unsigned*)(buf + ((t * 16 + it * 64) & 32767));
    __syncthreads();
  }
  __syncthreads();
  const unsigned long long t1 = __builtin_amdgcn_s_memtime();
  const unsigned long long r1 = __builtin_amdgcn_s_memrealtime();
  sink[(size_t)blockIdx.x * blockDim.x + t] = acc;
  if (t == 0) {
    clocks[2 * (size_t)blockIdx.x] = t1 - t0;
    clocks[2 * (size_t)blockIdx.x + 1] = r1 - r0;
  }
}

// Overlap of matrix-core and VALU work of two waves on one SIMD: a workgroup
// of eight waves per CU, waves w and w + 4 on SIMD w % 4.  Waves 0-3 stream
// v_mfma_f32_32x32x16_bf16 (as k_mfma_peak, four accumulators) when bit 0 of
// MODE is set; waves 4-7 run the eight-chain loop of k_valu_rate (VOP 0
// v_exp_f32, 1 v_fma_f32) when bit 1 is set.  Every wave records the
// shader-clock cycles and reference ticks of its own loop: with both roles
// on, each role's cycles against its cycles alone show whether the two kinds
// of work share the SIMD or run side by side (the split the wave-specialised
// attention kernel is built on).
template <int MODE, int VOP>
__global__ __launch_bounds__(512) void k_mix_rate(const bf16x8* __restrict__ ops, int mfma_iters,
                                                  const float* __restrict__ seed, int valu_iters,
                                                  float* __restrict__ sink,
                                                  unsigned long long* __restrict__ clocks) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  float s = 0.f;
  __syncthreads();
  const unsigned long long t0 = __builtin_amdgcn_s_memtime();
  const unsigned long long r0 = __builtin_amdgcn_s_memrealtime();
  if (wave < 4) {
    if constexpr ((MODE & 1) != 0) {
      const bf16x8 a0 = ops[0 * 64 + lane], a1 = ops[1 * 64 + lane], b0 = ops[4 * 64 + lane],
                   b1 = ops[5 * 64 + lane];
      f32x16 c0 = {}, c1 = {}, c2 = {}, c3 = {};
      for (int it = 0; it < mfma_iters; ++it) {
        c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b0, c0, 0, 0, 0);
        c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b1, c1, 0, 0, 0);
        c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b1, c2, 0, 0, 0);
        c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b0, c3, 0, 0, 0);
      }
#pragma unroll
      for (int i = 0; i < 16; ++i) s += c0[i] + c1[i] + c2[i] + c3[i];
    }
  } else {
    if constexpr ((MODE & 2) != 0) {
      float x[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) x[i] = seed[i] + 0.001f * lane;
      for (int it = 0; it < valu_iters; ++it) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          if constexpr (VOP == 0) x[i] = __builtin_amdgcn_exp2f(-x[i]);
          else x[i] = __builtin_fmaf(x[i], 0.999f, 1e-4f);
        }
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) s += x[i];
    }
  }
  const unsigned long long t1 = __builtin_amdgcn_s_memtime();
  const unsigned long long r1 = __builtin_amdgcn_s_memrealtime();
  sink[(size_t)blockIdx.x * blockDim.x + threadIdx.x] = s;
  if (lane == 0) {
    clocks[2 * ((size_t)blockIdx.x * 8 + wave)] = t1 - t0;
    clocks[2 * ((size_t)blockIdx.x * 8 + wave) + 1] = r1 - r0;
  }
}

}  // namespace

extern "C" int steel_lds_rate(int op, int iters, int grid, int waves_per_wg, unsigned* sink,
                              unsigned long long* clocks, void* stream) {
  if (op < 0 || op > 2 || !sink || !clocks || iters < 1 || grid < 1 || waves_per_wg < 1 ||
      waves_per_wg > 16)
    return 1;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const dim3 g(grid), b(64 * waves_per_wg);
  if (op == 0) hipLaunchKernelGGL(k_lds_rate<0>, g, b, 0, s, iters, sink, clocks);
  else if (op == 1) hipLaunchKernelGGL(k_lds_rate<1>, g, b, 0, s, iters, sink, clocks);
  else hipLaunchKernelGGL(k_lds_rate<2>, g, b, 0, s, iters, sink, clocks);
  return hipGetLastError() == hipSuccess ? 0 : 3;
}

extern "C" int steel_copy_rate(const void* src, size_t src_bytes, int iters, int grid,
                               int waves_per_wg, unsigned* sink, unsigned long long* clocks,
                               void* stream) {
  const bool pow2 = waves_per_wg > 0 && (waves_per_wg & (waves_per_wg - 1)) == 0;
  if (!src || ((uintptr_t)src & 15u) || !sink || !clocks || iters < 1 || grid < 1 || !pow2 ||
      waves_per_wg > 16 || src_bytes < (size_t)8 * 65536)
    return 1;
  const long long region = (long long)(src_bytes / 8) & ~1023ll;  // each XCD's eighth, >= 64 KiB
  hipLaunchKernelGGL(k_copy_rate, dim3(grid), dim3(64 * waves_per_wg), 0,
                     static_cast<hipStream_t>(stream), static_cast<const char*>(src), region,
                     iters, sink, clocks);
  return hipGetLastError() == hipSuccess ? 0 : 3;
}

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

extern "C" int steel_mix_rate(int mode, int vop, const void* operands, int mfma_iters,
                              const float* seed, int valu_iters, int grid, float* sink,
                              unsigned long long* clocks, void* stream) {
  if (mode < 1 || mode > 3 || (vop != 0 && vop != 1) || grid < 1 || !sink || !clocks ||
      ((mode & 1) && (!operands || mfma_iters < 1)) || ((mode & 2) && (!seed || valu_iters < 1)))
    return 1;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const bf16x8* ops = static_cast<const bf16x8*>(operands);
  const dim3 g(grid), b(512);
#define STEEL_MIX(M, V) hipLaunchKernelGGL((k_mix_rate<M, V>), g, b, 0, s, ops, mfma_iters, seed, valu_iters, sink, clocks)
  if (mode == 1) STEEL_MIX(1, 0);
  else if (mode == 2 && vop == 0) STEEL_MIX(2, 0);
  else if (mode == 2) STEEL_MIX(2, 1);
  else if (vop == 0) STEEL_MIX(3, 0);
  else STEEL_MIX(3, 1);
#undef STEEL_MIX
  return hipGetLastError() == hipSuccess ? 0 : 3;
}
