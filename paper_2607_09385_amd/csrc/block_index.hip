// Live-block index build on gfx950.
//
// Section IV-A of the paper has every core track the coordinates (i, j) of a
// score tile and either skip it (fully masked), process it as is (unmasked)
// or mask it locally (partially masked).  Here that classification runs once
// per call over the 64x64 block grid and is stored as a compressed list per
// query block: row_ptr (exclusive prefix sum of live counts) and col (live kb,
// bit 31 = partial).  Section IV-C balances the masked work across the
// pipelines; the GPU analogue is a work order that hands out the heaviest
// query blocks first (stable counting sort by live count).
//
// Kernels, in launch order:
//   classify : one wave per row: live count; head-pack uniformity flag
//   hist     : per chunk of 256 items: histogram of count bins (LDS atomics)
//   scan     : one workgroup: row_ptr, and the chunk bases of each work list
//   fill     : one wave per row: the live kb list with partial flags
//   scatter  : per chunk: stable placement of each item in its work order
#include "internal.h"

namespace steel {

__device__ __forceinline__ bool causal_dead(const Problem& p, int qb, int kb) {
  const int last_row = min((qb + 1) * kBlk, p.S_q) - 1;
  return p.causal && (long long)kb * kBlk > (long long)last_row + p.delta;
}

__device__ __forceinline__ bool partial_tile(const Problem& p, int qb, int kb) {
  return (p.causal && (long long)(kb + 1) * kBlk - 1 > (long long)qb * kBlk + p.delta) ||
         (long long)(kb + 1) * kBlk > p.S_k;
}

__device__ __forceinline__ bool tile_live(const Problem& p, const uint8_t* mrow, int qb, int kb) {
  return kb < p.nKB && (mrow == nullptr || mrow[kb] != 0) && !causal_dead(p, qb, kb);
}

__global__ __launch_bounds__(256) void k_classify(Problem p, const uint8_t* __restrict__ mask,
                                                  int32_t* __restrict__ cnt,
                                                  uint8_t* __restrict__ uni) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r = blockIdx.x * 4 + wave;
  if (r >= p.R) return;
  const int qb = r % p.nQB;
  const int h = (r / p.nQB) % p.Hq;
  const uint8_t* mrow = mask ? mask + (size_t)r * p.nKB : nullptr;
  int c = 0;
  for (int kb0 = 0; kb0 < p.nKB; kb0 += 64)
    c += __popcll(__ballot(tile_live(p, mrow, qb, kb0 + lane)));
  if (lane == 0) cnt[r] = c;
  if (p.pack > 1 && h % p.pack == 0) {
    bool same = true;
    if (mrow) {
      for (int j = 1; j < p.pack && same; ++j) {
        const uint8_t* mj = mrow + (size_t)j * p.nQB * p.nKB;
        for (int kb0 = 0; kb0 < p.nKB; kb0 += 64) {
          const int kb = kb0 + lane;
          const bool diff = tile_live(p, mrow, qb, kb) != tile_live(p, mj, qb, kb);
          if (__ballot(diff)) { same = false; break; }
        }
      }
    }
    if (lane == 0) uni[(size_t)((r / p.nQB) / p.pack) * p.nQB + qb] = same ? 1 : 0;
  }
}

// Item of a work list: list 0 holds single query-head rows that are not part
// of a uniform head pack, list 1 holds uniform head packs.
__device__ __forceinline__ bool item_info(const Problem& p, const int32_t* cnt, const uint8_t* uni,
                                          int list, int item, int* bin) {
  int row;
  if (list == 0) {
    if (item >= p.R) return false;
    if (p.pack > 1) {
      const int qb = item % p.nQB;
      const int pid = ((item / p.nQB) / p.pack) * p.nQB + qb;
      if (uni[pid]) return false;
    }
    row = item;
  } else {
    if (item >= p.NP) return false;
    if (!uni[item]) return false;
    const int qb = item % p.nQB;
    row = (item / p.nQB) * p.pack * p.nQB + qb;
  }
  *bin = cnt[row] >> p.bin_shift;
  return true;
}

__global__ __launch_bounds__(256) void k_hist(Problem p, const int32_t* __restrict__ cnt,
                                              const uint8_t* __restrict__ uni,
                                              int32_t* __restrict__ hist, int list, int nch) {
  __shared__ int32_t h[kMaxBins];
  for (int i = threadIdx.x; i < p.nbins; i += 256) h[i] = 0;
  __syncthreads();
  int bin;
  if (item_info(p, cnt, uni, list, blockIdx.x * kChunk + threadIdx.x, &bin)) atomicAdd(&h[bin], 1);
  __syncthreads();
  // bin-major with bins descending, so one linear scan yields heaviest-first bases
  for (int i = threadIdx.x; i < p.nbins; i += 256)
    hist[(size_t)(p.nbins - 1 - i) * nch + blockIdx.x] = h[i];
}

// Exclusive scan of n ints in place (or src -> dst) by one 1024-thread
// workgroup; returns the total to every thread.
__device__ int block_exclusive_scan(const int32_t* src, int32_t* dst, long long n, int32_t* sh) {
  const int t = threadIdx.x;
  const long long per = (n + 1023) / 1024;
  const long long lo = min((long long)t * per, n), hi = min(lo + per, n);
  int s = 0;
  for (long long i = lo; i < hi; ++i) s += src[i];
  sh[t] = s;
  __syncthreads();
  for (int off = 1; off < 1024; off <<= 1) {
    const int v = t >= off ? sh[t - off] : 0;
    __syncthreads();
    sh[t] += v;
    __syncthreads();
  }
  int run = sh[t] - s;  // exclusive prefix of this segment
  const int total = sh[1023];
  __syncthreads();
  for (long long i = lo; i < hi; ++i) {
    const int x = src[i];
    dst[i] = run;
    run += x;
  }
  return total;
}

__global__ __launch_bounds__(1024) void k_scan(Problem p, const int32_t* __restrict__ cnt,
                                               int32_t* __restrict__ row_ptr,
                                               int32_t* hist_s, long long nh_s,
                                               int32_t* hist_p, long long nh_p,
                                               int32_t* __restrict__ n_items) {
  __shared__ int32_t sh[1024];
  const int tot = block_exclusive_scan(cnt, row_ptr, p.R, sh);
  if (threadIdx.x == 0) row_ptr[p.R] = tot;
  __syncthreads();
  const int ns = block_exclusive_scan(hist_s, hist_s, nh_s, sh);
  __syncthreads();
  const int np = nh_p > 0 ? block_exclusive_scan(hist_p, hist_p, nh_p, sh) : 0;
  if (threadIdx.x == 0) {
    n_items[0] = ns;
    n_items[1] = np;
    n_items[2] = kPlanMagic;
    n_items[3] = p.R;
    n_items[4] = p.nKB;
    n_items[5] = p.pack;
    n_items[6] = p.causal;
    n_items[7] = p.delta;
  }
}

__global__ __launch_bounds__(256) void k_fill(Problem p, const uint8_t* __restrict__ mask,
                                              const int32_t* __restrict__ row_ptr,
                                              uint32_t* __restrict__ col) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r = blockIdx.x * 4 + wave;
  if (r >= p.R) return;
  const int qb = r % p.nQB;
  const uint8_t* mrow = mask ? mask + (size_t)r * p.nKB : nullptr;
  int pos = row_ptr[r];
  const unsigned long long below = (1ull << lane) - 1ull;
  for (int kb0 = 0; kb0 < p.nKB; kb0 += 64) {
    const int kb = kb0 + lane;
    const bool live = tile_live(p, mrow, qb, kb);
    const unsigned long long bal = __ballot(live);
    if (live)
      col[pos + __popcll(bal & below)] =
          (uint32_t)kb | (partial_tile(p, qb, kb) ? 0x80000000u : 0u);
    pos += __popcll(bal);
  }
}

__global__ __launch_bounds__(256) void k_scatter(Problem p, const int32_t* __restrict__ cnt,
                                                 const uint8_t* __restrict__ uni,
                                                 const int32_t* __restrict__ base, int list,
                                                 int nch, int32_t* __restrict__ order) {
  __shared__ int32_t bins[kChunk];
  const int t = threadIdx.x;
  const int item = blockIdx.x * kChunk + t;
  int bin = -1;
  const bool present = item_info(p, cnt, uni, list, item, &bin);
  bins[t] = present ? bin : -1;
  __syncthreads();
  if (!present) return;
  int rank = 0;
  for (int j = 0; j < t; ++j) rank += bins[j] == bin;
  order[base[(size_t)(p.nbins - 1 - bin) * nch + blockIdx.x] + rank] = item;
}

hipError_t launch_block_index(const Problem& p, const uint8_t* mask, const IndexBuffers& w,
                              hipStream_t s) {
  const int nch_s = nchunks(p.R);
  const int nch_p = p.pack > 1 ? nchunks(p.NP) : 0;
  const int rows_grid = (p.R + 3) / 4;
  hipLaunchKernelGGL(k_classify, dim3(rows_grid), dim3(256), 0, s, p, mask, w.cnt, w.uni);
  hipLaunchKernelGGL(k_hist, dim3(nch_s), dim3(256), 0, s, p, w.cnt, w.uni, w.hist_s, 0, nch_s);
  if (nch_p)
    hipLaunchKernelGGL(k_hist, dim3(nch_p), dim3(256), 0, s, p, w.cnt, w.uni, w.hist_p, 1, nch_p);
  hipLaunchKernelGGL(k_scan, dim3(1), dim3(1024), 0, s, p, w.cnt, w.row_ptr, w.hist_s,
                     (long long)p.nbins * nch_s, w.hist_p, (long long)p.nbins * nch_p, w.n_items);
  hipLaunchKernelGGL(k_fill, dim3(rows_grid), dim3(256), 0, s, p, mask, w.row_ptr, w.col);
  hipLaunchKernelGGL(k_scatter, dim3(nch_s), dim3(256), 0, s, p, w.cnt, w.uni, w.hist_s, 0, nch_s,
                     w.order_s);
  if (nch_p)
    hipLaunchKernelGGL(k_scatter, dim3(nch_p), dim3(256), 0, s, p, w.cnt, w.uni, w.hist_p, 1,
                       nch_p, w.order_p);
  return hipGetLastError();
}

}  // namespace steel
