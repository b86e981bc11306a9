// Pre-pass of the fp8 form: the E4M3 operands of K and V.
//
// The paper's datapath multiplies bf16 operands into fp32 (Section II-C).  The
// fp8 form feeds the two products of Algorithm 1 with E4M3 operands instead:
// K and V get one power-of-two scale per (batch, key/value head), Q one per
// query row (taken inside the attention kernel), and P is rounded there.
// Here, in two launches (K is skipped when only P V takes E4M3 operands):
//   k_fp8_amax   largest |K| and |V| over each of kFp8Chunks row chunks of
//                every (b, g) (no atomics: each chunk writes its own pair);
//   k_fp8_tiles  per (b, g, key block) the scales from those maxima and the
//                tile of each tensor in the layout the attention kernels
//                keep in LDS (Fp8Buffers): K row-major, V transposed with its
//                keys in the P operand's order, both swizzled, keys past S_k
//                zero.  The tile of key block 0 also stores the inverse scales.
#include "internal.h"

namespace steel {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float wave_max(float x) {
  for (int off = 32; off > 0; off >>= 1) x = fmaxf(x, __shfl_xor(x, off));
  return x;
}

// Four consecutive values scaled and rounded to E4M3 (nearest even), packed
// into one dword in memory order.
__device__ __forceinline__ uint32_t pack4(float a, float b, float c, float d) {
  int w = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0, false);
  w = __builtin_amdgcn_cvt_pk_fp8_f32(c, d, w, true);
  return (uint32_t)w;
}

}  // namespace

__global__ __launch_bounds__(256) void k_fp8_amax(Problem p, const __bf16* __restrict__ k,
                                                  const __bf16* __restrict__ v,
                                                  float* __restrict__ part, int with_k) {
  const int bh = (int)blockIdx.x / kFp8Chunks, ch = (int)blockIdx.x % kFp8Chunks;
  const int per = (p.S_k + kFp8Chunks - 1) / kFp8Chunks;
  const int r0 = min(ch * per, p.S_k), r1 = min(r0 + per, p.S_k);
  const size_t base = ((size_t)bh * p.S_k + r0) * p.D;
  const int n8 = (r1 - r0) * p.D / 8;  // 16-byte groups
  float ak = 0.f, av = 0.f;
  // four 16-byte loads in flight per thread and tensor
  auto amax8 = [](float m, const bf16x8& x) {
#pragma unroll
    for (int e = 0; e < 8; ++e) m = fmaxf(m, fabsf((float)x[e]));
    return m;
  };
  int i = threadIdx.x;
  for (; i + 3 * 256 < n8; i += 4 * 256) {
    bf16x8 xv[4], xk[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) xv[u] = *(const bf16x8*)(v + base + 8 * (size_t)(i + u * 256));
    if (with_k) {
#pragma unroll
      for (int u = 0; u < 4; ++u) xk[u] = *(const bf16x8*)(k + base + 8 * (size_t)(i + u * 256));
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      av = amax8(av, xv[u]);
      if (with_k) ak = amax8(ak, xk[u]);
    }
  }
  for (; i < n8; i += 256) {
    av = amax8(av, *(const bf16x8*)(v + base + 8 * (size_t)i));
    if (with_k) ak = amax8(ak, *(const bf16x8*)(k + base + 8 * (size_t)i));
  }
  __shared__ float sh[2][4];
  ak = wave_max(ak);
  av = wave_max(av);
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    sh[0][wave] = ak;
    sh[1][wave] = av;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    part[2 * blockIdx.x] = fmaxf(fmaxf(sh[0][0], sh[0][1]), fmaxf(sh[0][2], sh[0][3]));
    part[2 * blockIdx.x + 1] = fmaxf(fmaxf(sh[1][0], sh[1][1]), fmaxf(sh[1][2], sh[1][3]));
  }
}

template <int D>
__global__ __launch_bounds__(256) void k_fp8_tiles(Problem p, const __bf16* __restrict__ k,
                                                   const __bf16* __restrict__ v,
                                                   const float* __restrict__ part, Fp8Buffers f) {
  constexpr int C = D / 16;  // 16-byte chunks per K8 row
  const int bh = (int)blockIdx.x / p.nKB, kb = (int)blockIdx.x % p.nKB;
  // the head's maxima from its chunk partials (one per thread, then waves)
  __shared__ float red[2][4];
  float ak = 0.f, av = 0.f;
  for (int c = threadIdx.x; c < kFp8Chunks; c += 256) {
    ak = fmaxf(ak, part[2 * (bh * kFp8Chunks + c)]);
    av = fmaxf(av, part[2 * (bh * kFp8Chunks + c) + 1]);
  }
  ak = wave_max(ak);
  av = wave_max(av);
  if ((threadIdx.x & 63) == 0) {
    red[0][threadIdx.x >> 6] = ak;
    red[1][threadIdx.x >> 6] = av;
  }
  __syncthreads();
  ak = fmaxf(fmaxf(red[0][0], red[0][1]), fmaxf(red[0][2], red[0][3]));
  av = fmaxf(fmaxf(red[1][0], red[1][1]), fmaxf(red[1][2], red[1][3]));
  const float sk = e4m3_scale(ak), sv = e4m3_scale(av);
  if (kb == 0 && threadIdx.x == 0) {
    f.scale[2 * bh] = 1.f / sk;
    f.scale[2 * bh + 1] = 1.f / sv;
  }
  const int key0 = kb * kBlk;
  const size_t src = ((size_t)bh * p.S_k + key0) * D;     // element offset of the block
  const size_t dst = ((size_t)bh * p.nKB + kb) * kBlk * D;  // byte offset of the tile

  // V block into LDS, row-major [key][D] (rows past S_k zero)
  __shared__ __bf16 vs[kBlk * D];
  for (int i = threadIdx.x; i < kBlk * D / 8; i += 256) {
    const int key = (8 * i) / D;
    bf16x8 x = {};
    if (key0 + key < p.S_k) x = *(const bf16x8*)(v + src + 8 * (size_t)i);
    *(bf16x8*)(vs + 8 * i) = x;
  }

  // K8: output chunk (row r, slot s) holds dims 16 (s ^ kswz(r)) .. +15
  for (int oc = threadIdx.x; f.k8 != nullptr && oc < kBlk * C; oc += 256) {
    const int r = oc / C, slot = oc % C;
    const int c = slot ^ kswz8<D>(r);
    u32x4 w = {0u, 0u, 0u, 0u};
    if (key0 + r < p.S_k) {
      const bf16x8 x0 = *(const bf16x8*)(k + src + (size_t)r * D + 16 * c);
      const bf16x8 x1 = *(const bf16x8*)(k + src + (size_t)r * D + 16 * c + 8);
      w[0] = pack4((float)x0[0] * sk, (float)x0[1] * sk, (float)x0[2] * sk, (float)x0[3] * sk);
      w[1] = pack4((float)x0[4] * sk, (float)x0[5] * sk, (float)x0[6] * sk, (float)x0[7] * sk);
      w[2] = pack4((float)x1[0] * sk, (float)x1[1] * sk, (float)x1[2] * sk, (float)x1[3] * sk);
      w[3] = pack4((float)x1[4] * sk, (float)x1[5] * sk, (float)x1[6] * sk, (float)x1[7] * sk);
    }
    *(u32x4*)(f.k8 + dst + (size_t)r * D + 16 * slot) = w;
  }
  __syncthreads();

  // V8: output chunk (row d, slot s) holds logical chunk c = s ^ ((d >> 2) & 3):
  // byte i of it is key 32 (c % 2) + 8 (i / 4) + 4 (c / 2) + i % 4
  for (int oc = threadIdx.x; oc < D * 4; oc += 256) {
    const int d = oc / 4, slot = oc % 4;
    const int c = slot ^ ((d >> 2) & 3);
    const int kbase = 32 * (c & 1) + 4 * (c >> 1);
    float x[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) x[i] = (float)vs[(kbase + 8 * (i >> 2) + (i & 3)) * D + d] * sv;
    const u32x4 w = {pack4(x[0], x[1], x[2], x[3]), pack4(x[4], x[5], x[6], x[7]),
                     pack4(x[8], x[9], x[10], x[11]), pack4(x[12], x[13], x[14], x[15])};
    *(u32x4*)(f.v8 + dst + (size_t)d * kBlk + 16 * slot) = w;
  }
}

hipError_t launch_fp8_prepass(const Problem& p, const void* k, const void* v, const Fp8Buffers& f,
                              hipStream_t s) {
  const int heads = p.B * p.Hkv;
  hipLaunchKernelGGL(k_fp8_amax, dim3(heads * kFp8Chunks), dim3(256), 0, s, p, (const __bf16*)k,
                     (const __bf16*)v, f.part, f.k8 != nullptr ? 1 : 0);
  if (p.D == 64)
    hipLaunchKernelGGL(k_fp8_tiles<64>, dim3(heads * p.nKB), dim3(256), 0, s, p, (const __bf16*)k,
                       (const __bf16*)v, (const float*)f.part, f);
  else
    hipLaunchKernelGGL(k_fp8_tiles<128>, dim3(heads * p.nKB), dim3(256), 0, s, p,
                       (const __bf16*)k, (const __bf16*)v, (const float*)f.part, f);
  return hipGetLastError();
}

}  // namespace steel
