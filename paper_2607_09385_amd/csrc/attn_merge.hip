// Merge of partial attention results computed over disjoint key sets (key
// chunks of one long sequence, or keys held on different devices).
//
// With the row log-sum-exp lse_c of each part (the m and l statistics of
// Algorithm 1, lse = (m + log2 l) ln 2), the attention over the union of the
// key sets is sum_c w_c O_c with w_c = exp(lse_c - lse), lse = log sum_c
// exp(lse_c); rows that see no key in any part stay 0 with lse = -inf.
// Memory bound: each part's O and lse are read once, O and lse written once.
#include "internal.h"

namespace steel {

typedef float f32x4_t __attribute__((ext_vector_type(4)));

// One thread per (row, 4 columns).
__global__ __launch_bounds__(256) void k_attn_merge(const float* __restrict__ o_parts,
                                                    const float* __restrict__ lse_parts,
                                                    int n_parts, long long rows, int D,
                                                    float* __restrict__ out,
                                                    float* __restrict__ lse_out) {
  const int c4n = D / 4;
  const long long idx = (long long)blockIdx.x * 256 + threadIdx.x;
  const long long row = idx / c4n;
  if (row >= rows) return;
  const int c4 = (int)(idx - row * c4n);
  float top = -INFINITY;
  for (int c = 0; c < n_parts; ++c) top = fmaxf(top, lse_parts[(size_t)c * rows + row]);
  f32x4_t* dst = reinterpret_cast<f32x4_t*>(out + (size_t)row * D) + c4;
  if (top == -INFINITY) {
    *dst = f32x4_t{0.f, 0.f, 0.f, 0.f};
    if (lse_out != nullptr && c4 == 0) lse_out[row] = -INFINITY;
    return;
  }
  float den = 0.f;
  f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
  for (int c = 0; c < n_parts; ++c) {
    const float w = expf(lse_parts[(size_t)c * rows + row] - top);  // 0 for lse = -inf
    den += w;
    const f32x4_t o = reinterpret_cast<const f32x4_t*>(o_parts + ((size_t)c * rows + row) * D)[c4];
    acc += w * o;
  }
  *dst = acc * (1.f / den);
  if (lse_out != nullptr && c4 == 0) lse_out[row] = top + logf(den);
}

hipError_t launch_merge(const float* o_parts, const float* lse_parts, int n_parts, long long rows,
                        int D, float* out, float* lse_out, hipStream_t s) {
  const long long threads = rows * (D / 4);
  hipLaunchKernelGGL(k_attn_merge, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, s,
                     o_parts, lse_parts, n_parts, rows, D, out, lse_out);
  return hipGetLastError();
}

}  // namespace steel
