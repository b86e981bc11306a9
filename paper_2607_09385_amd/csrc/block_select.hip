// Block-mask producer on gfx950: for every query block, the key blocks whose
// mean-pooled keys score highest against the mean-pooled queries (top-k of
// the causal candidates, ties to the smaller block), plus the diagonal block.
//
// The paper builds its masks on the compute core instead of fetching them
// (Section III-B) and runs any block mask through the three tile classes of
// Section IV-A; this is the selection rule the sparse workload is defined
// with, moved onto the GPU ahead of the index build.
//
// Floating point decides which blocks are kept, so the arithmetic is fixed:
// float64 throughout, each block sum adds its rows in increasing order, the
// mean divides that sum by the row count (correctly rounded), and each score
// adds the D products in increasing d with every product and sum rounded on
// its own (no fused multiply-add).  Three launches:
//   block_means   one workgroup per (head, block) of Q and of K: the rows
//                 staged in LDS, one thread per column
//   block_scores  64 x 64 score tiles per workgroup from LDS-staged means
//                 (tiles above the diagonal skipped when causal)
//   topk_select   one wave per (head, query block): a radix select over
//                 order-preserving integer keys of the scores (rows of up to
//                 512 key blocks), or a bitonic sort of the candidates in
//                 LDS (longer rows), then the mask row
#include <algorithm>
#include <climits>

#include "internal.h"

namespace steel {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));

// One workgroup per (head, block): the block's rows (contiguous in memory)
// are staged into LDS with 16-byte loads, then thread d sums column d over the
// rows in increasing order.
__global__ __launch_bounds__(128) void k_block_means(const __bf16* __restrict__ x, int S, int nb,
                                                     int D, double* __restrict__ out) {
  __shared__ __attribute__((aligned(16))) __bf16 tile[kBlk * 128];
  const int g = blockIdx.x;  // (head, block)
  const int bh = g / nb, bi = g - bh * nb;
  const int r0 = bi * kBlk;
  const int cnt = min(kBlk, S - r0);
  const __bf16* p = x + ((size_t)bh * S + r0) * D;
  const int nvec = cnt * D / 8;
  for (int v = threadIdx.x; v < nvec; v += 128)
    *(bf16x8_t*)(tile + 8 * v) = *(const bf16x8_t*)(p + 8 * v);
  __syncthreads();
  const int d = threadIdx.x;
  if (d >= D) return;
  double acc = 0.0;
  for (int r = 0; r < cnt; ++r) acc = acc + (double)(float)tile[r * D + d];
  out[(size_t)g * D + d] = acc / (double)cnt;
}

// scores[bh][qb][kb] = dot(qm[bh][qb], km[bh / G][kb]) for one 64 x 64 tile.
// Thread t owns rows 4*(t/16) .. +3 and columns 4*(t%16) .. +3 of the tile.
__global__ __launch_bounds__(256) void k_block_scores(const double* __restrict__ qm,
                                                      const double* __restrict__ km, int nQB,
                                                      int nKB, int D, int G, int Hq, int Hkv,
                                                      int causal, int ntq, int ntk,
                                                      double* __restrict__ scores) {
#pragma clang fp contract(off)
  constexpr int DC = 32;  // d chunk staged in LDS
  static_assert(kBlk * DC % 256 == 0, "whole staging rounds");
  // rows padded by 2 doubles: the staging writes step over banks and every row
  // stays 16-byte aligned for the paired operand reads
  __shared__ __attribute__((aligned(16))) double qs[DC][kBlk + 2];
  __shared__ __attribute__((aligned(16))) double ks[DC][kBlk + 2];
  const int t = threadIdx.x;
  int g = blockIdx.x;
  const int tk = g % ntk;
  g /= ntk;
  const int tq = g % ntq;
  const int bh = g / ntq;  // b * Hq + h
  if (causal && tk > tq) return;  // every kb of the tile lies past every qb
  const int b = bh / Hq, h = bh - b * Hq;
  const double* qrow = qm + (size_t)bh * nQB * D;
  const double* krow = km + ((size_t)b * Hkv + h / G) * nKB * D;
  const int i0 = 4 * (t >> 4), j0 = 4 * (t & 15);
  double acc[4][4];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[a][c] = 0.0;
  for (int d0 = 0; d0 < D; d0 += DC) {
    // stage qm / km rows of the tile, d-major: every load is issued before
    // the first LDS write, so their latencies overlap
    constexpr int PER = kBlk * DC / 256;
    double qv[PER], kv[PER];
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int e = t + 256 * u;
      const int r = e / DC, dd = e - r * DC;
      const int qb = tq * kBlk + r, kb = tk * kBlk + r;
      qv[u] = qb < nQB ? qrow[(size_t)qb * D + d0 + dd] : 0.0;
      kv[u] = kb < nKB ? krow[(size_t)kb * D + d0 + dd] : 0.0;
    }
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int e = t + 256 * u;
      const int r = e / DC, dd = e - r * DC;
      qs[dd][r] = qv[u];
      ks[dd][r] = kv[u];
    }
    __syncthreads();
    // operands of step dd + 1 are read while step dd computes
    double a[2][4], c[2][4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      a[0][u] = qs[0][i0 + u];
      c[0][u] = ks[0][j0 + u];
    }
#pragma unroll
    for (int dd = 0; dd < DC; ++dd) {
      const int cur = dd & 1;
      if (dd + 1 < DC) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          a[cur ^ 1][u] = qs[dd + 1][i0 + u];
          c[cur ^ 1][u] = ks[dd + 1][j0 + u];
        }
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int w = 0; w < 4; ++w) acc[u][w] = acc[u][w] + a[cur][u] * c[cur][w];
    }
    __syncthreads();
  }
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int qb = tq * kBlk + i0 + u;
    if (qb >= nQB) continue;
    double* out = scores + ((size_t)bh * nQB + qb) * nKB;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const int kb = tk * kBlk + j0 + w;
      if (kb < nKB) out[kb] = acc[u][w];
    }
  }
}

// Does candidate a come before candidate b (larger score, then smaller kb)?
__device__ __forceinline__ bool before(double sa, int ia, double sb, int ib) {
  return sa > sb || (sa == sb && ia < ib);
}

// One wave per (head, query block) row, blockDim/64 rows per workgroup.  Each wave
// has its own LDS segment (n2max scores, n2max indices, nKB flags); the
// steps of the sort are separated by a wave-level wait, not a barrier.
__device__ __forceinline__ void wave_lds_sync() {
  // this wave's LDS accesses are done, and the compiler moves none across
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
}

__global__ __launch_bounds__(256) void k_topk_select(const double* __restrict__ scores, int nQB,
                                                     int nKB, int n2max, size_t seg, int causal,
                                                     long long keep_num, long long keep_den,
                                                     long long n_rows,
                                                     uint8_t* __restrict__ mask) {
  extern __shared__ __attribute__((aligned(16))) char sel_lds[];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const long long row = (long long)blockIdx.x * (blockDim.x >> 6) + w;  // (b*Hq + h)*nQB + qb
  if (row >= n_rows) return;  // the whole wave; no workgroup barrier follows
  char* base = sel_lds + (size_t)w * seg;
  double* s = reinterpret_cast<double*>(base);
  int* id = reinterpret_cast<int*>(base + 8 * (size_t)n2max);
  uint8_t* flag = reinterpret_cast<uint8_t*>(base + 12 * (size_t)n2max);
  const int qb = (int)(row % nQB);
  const int ncand = causal ? min(qb + 1, nKB) : nKB;
  const int keep = (int)((keep_num * ncand + keep_den - 1) / keep_den);
  int n2 = 1;
  while (n2 < ncand) n2 <<= 1;
  const double* src = scores + (size_t)row * nKB;
  for (int j = lane; j < n2; j += 64) {
    s[j] = j < ncand ? src[j] : -INFINITY;
    id[j] = j;
  }
  for (int j = lane; j < nKB; j += 64) flag[j] = 0;
  wave_lds_sync();
  // bitonic sort of n2 entries into "before" order; in each step every lane
  // takes whole compare-exchange pairs (i, i + j), i with bit j clear
  for (int k = 2; k <= n2; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int pr = lane; pr < (n2 >> 1); pr += 64) {
        const int i = ((pr & ~(j - 1)) << 1) | (pr & (j - 1));
        const int l = i + j;
        const bool up = (i & k) == 0;
        const double si = s[i], sl = s[l];
        const int ii = id[i], il = id[l];
        const bool swap = up ? before(sl, il, si, ii) : before(si, ii, sl, il);
        if (swap) {
          s[i] = sl;
          s[l] = si;
          id[i] = il;
          id[l] = ii;
        }
      }
      wave_lds_sync();
    }
  }
  for (int j = lane; j < keep; j += 64) flag[id[j]] = 1;
  if (lane == 0 && qb < nKB) flag[qb] = 1;
  wave_lds_sync();
  uint8_t* dst = mask + (size_t)row * nKB;
  for (int kb = lane; kb < nKB; kb += 64) dst[kb] = flag[kb];
}

// Rows of at most 64 * kSelPerLane key blocks: a radix select in registers.
// Each score becomes an unsigned key in the order of the doubles (both zeros
// give the key of +0, so equal scores give equal keys).  Eight passes, one
// byte each from the top, narrow down the key of the keep-th largest score
// with a 256-bin histogram per wave in LDS; every candidate with a larger
// key is kept, and of those with that key the ones with the smallest key
// block indices, as many as are still missing.  The result is the same set
// as a full sort by (score descending, kb ascending).
constexpr int kSelPerLane = 8;

__device__ __forceinline__ uint64_t order_key(double x) {
  if (x == 0.0) x = 0.0;  // -0 and +0 compare equal
  const uint64_t u = (uint64_t)__double_as_longlong(x);
  return (u >> 63) ? ~u : (u | 0x8000000000000000ull);
}

__global__ __launch_bounds__(256) void k_topk_select_radix(const double* __restrict__ scores,
                                                           int nQB, int nKB, int causal,
                                                           long long keep_num, long long keep_den,
                                                           long long n_rows,
                                                           uint8_t* __restrict__ mask) {
  __shared__ unsigned hist_all[4][256];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const long long row = (long long)blockIdx.x * 4 + w;  // (b*Hq + h)*nQB + qb
  if (row >= n_rows) return;  // the whole wave; no workgroup barrier follows
  unsigned* hist = hist_all[w];
  const int qb = (int)(row % nQB);
  const int ncand = causal ? min(qb + 1, nKB) : nKB;
  int need = (int)((keep_num * ncand + keep_den - 1) / keep_den);
  const double* src = scores + (size_t)row * nKB;
  uint64_t key[kSelPerLane];  // 0: not a candidate (below every score's key)
#pragma unroll
  for (int c = 0; c < kSelPerLane; ++c) {
    const int j = lane + 64 * c;
    key[c] = j < ncand ? order_key(src[j]) : 0ull;
  }
  uint64_t prefix = 0;  // the bytes of the boundary key found so far
#pragma unroll 1
  for (int pass = 0; pass < 8; ++pass) {
    const int shift = 56 - 8 * pass;
#pragma unroll
    for (int i = 0; i < 4; ++i) hist[4 * lane + i] = 0u;
    wave_lds_sync();
#pragma unroll
    for (int c = 0; c < kSelPerLane; ++c)
      if (key[c] != 0ull && ((key[c] >> shift) >> 8) == prefix)  // higher bytes match
        atomicAdd(&hist[(unsigned)(key[c] >> shift) & 255u], 1u);
    wave_lds_sync();
    // bins 4*lane .. 4*lane+3; counts of the higher bins come from the
    // lanes above (a suffix sum over the wave)
    unsigned h[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) h[i] = hist[4 * lane + i];
    const unsigned tot = h[0] + h[1] + h[2] + h[3];
    unsigned suf = tot;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const unsigned t = __shfl_down(suf, o);
      if (lane + o < 64) suf += t;
    }
    unsigned above = suf - tot;
    int found = -1;
    unsigned found_above = 0;
#pragma unroll
    for (int i = 3; i >= 0; --i) {
      if (found < 0 && above < (unsigned)need && above + h[i] >= (unsigned)need) {
        found = 4 * lane + i;
        found_above = above;
      }
      above += h[i];
    }
    // exactly one bin holds the need-th largest remaining key
    const int src_lane = __builtin_ctzll(__ballot(found >= 0));
    const int v = __shfl(found, src_lane);
    need -= (int)__shfl(found_above, src_lane);
    prefix = (prefix << 8) | (uint64_t)v;
  }
  uint8_t* dst = mask + (size_t)row * nKB;
  int eq_before = 0;  // candidates with the boundary key in earlier lane groups
#pragma unroll
  for (int c = 0; c < kSelPerLane; ++c) {
    const int j = lane + 64 * c;
    const bool eq = key[c] == prefix;
    const uint64_t m = __ballot(eq);
    const int rank = eq_before + __popcll(m & ((1ull << lane) - 1ull));
    const bool keep = key[c] > prefix || (eq && rank < need) || j == qb;
    eq_before += __popcll(m);
    if (j < nKB) dst[j] = keep ? 1 : 0;
  }
}

hipError_t launch_topk_mask(const Problem& p, const __bf16* q, const __bf16* k, int keep_num,
                            int keep_den, uint8_t* mask, double* qm, double* km, double* scores,
                            hipStream_t s) {
  const int ntq = (p.nQB + kBlk - 1) / kBlk, ntk = (p.nKB + kBlk - 1) / kBlk;
  hipLaunchKernelGGL(k_block_means, dim3(p.B * p.Hq * p.nQB), dim3(128), 0, s, q, p.S_q, p.nQB,
                     p.D, qm);
  hipLaunchKernelGGL(k_block_means, dim3(p.B * p.Hkv * p.nKB), dim3(128), 0, s, k, p.S_k, p.nKB,
                     p.D, km);
  hipLaunchKernelGGL(k_block_scores, dim3(p.B * p.Hq * ntq * ntk), dim3(256), 0, s, qm, km, p.nQB,
                     p.nKB, p.D, p.G, p.Hq, p.Hkv, p.causal, ntq, ntk, scores);
  const long long rows = (long long)p.B * p.Hq * p.nQB;
  if (p.nKB <= 64 * kSelPerLane) {
    hipLaunchKernelGGL(k_topk_select_radix, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, s,
                       scores, p.nQB, p.nKB, p.causal, (long long)keep_num, (long long)keep_den,
                       rows, mask);
    return hipGetLastError();
  }
  int n2max = 1;
  while (n2max < p.nKB) n2max <<= 1;
  const size_t seg = (12 * (size_t)n2max + (size_t)p.nKB + 15) & ~(size_t)15;  // per wave
  const int wpg = (int)std::max<size_t>(1, std::min<size_t>(4, 65536 / seg));   // waves per group
  hipLaunchKernelGGL(k_topk_select, dim3((unsigned)((rows + wpg - 1) / wpg)), dim3(64 * wpg),
                     wpg * seg, s, scores, p.nQB, p.nKB, n2max, seg, p.causal, (long long)keep_num,
                     (long long)keep_den, rows, mask);
  return hipGetLastError();
}

}  // namespace steel
