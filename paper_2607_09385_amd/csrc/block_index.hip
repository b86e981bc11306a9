// Live-block index build on gfx950.
//
// Section IV-A of the paper has every core track the coordinates (i, j) of a
// score tile and either skip it (fully masked), process it as is (unmasked)
// or mask it locally (partially masked).  Here that classification runs once
// per call over the 64x64 block grid and is stored as a compressed list per
// query block: row_ptr (exclusive prefix sum of live counts) and col (live kb,
// bit 31 = partial).  Section IV-C balances the masked work across the
// pipelines; the GPU analogue is a work order that hands out the heaviest
// query blocks first: a stable counting sort by count_bin of the live count.
//
// Three launches in the common case (R <= kFastRows rows):
//   classify     one wave per row, 4 mask bytes per lane: live count, plus
//                kUniformBit on the first row of a head pack whose members
//                all have the same live set
//   scan_small   one workgroup, in LDS: row_ptr, and per work list the
//                per-chunk bin histograms turned into scatter bases
//   fill_scatter one wave per row writes its live list; one workgroup per
//                chunk of 256 items places them in the work order
// Larger problems build the histograms with one workgroup per chunk and scan
// them in a separate single-workgroup kernel.
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

// Live bits of tiles (qb, kb0 .. kb0+3) of one row (bit e = tile kb0 + e).
// wide: the row holds whole 4-byte words (nKB % 4 == 0, aligned mask).
// Without a mask tensor every block is in the mask, or, in the structured
// mode (p.win_blocks > 0), the window and sink blocks of the coordinates.
__device__ __forceinline__ uint32_t live_quad(const Problem& p, const uint8_t* mrow, bool wide,
                                              int qb, int kb0) {
  uint32_t bytes;
  if (mrow == nullptr) {
    if (p.win_blocks > 0) {
      bytes = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int kb = kb0 + e;
        const bool in = (kb <= qb && kb > qb - p.win_blocks) || kb < p.sink_blocks;
        bytes |= (uint32_t)in << (8 * e);
      }
    } else {
      bytes = 0x01010101u;
    }
  } else if (wide) {
    bytes = kb0 < p.nKB ? *(const uint32_t*)(mrow + kb0) : 0u;
  } else {
    bytes = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (kb0 + e < p.nKB) bytes |= (uint32_t)(mrow[kb0 + e] != 0) << (8 * e);
  }
  uint32_t bits = 0;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int kb = kb0 + e;
    const bool live = kb < p.nKB && ((bytes >> (8 * e)) & 0xffu) != 0 && !causal_dead(p, qb, kb);
    bits |= (uint32_t)live << e;
  }
  return bits;
}

__global__ __launch_bounds__(256) void k_classify(Problem p, const uint8_t* __restrict__ mask,
                                                  int wide, int32_t* __restrict__ cnt) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r = blockIdx.x * 4 + wave;
  if (r >= p.R) return;
  const int qb = r % p.nQB;
  const int h = (r / p.nQB) % p.Hq;
  const uint8_t* mrow = mask ? mask + (size_t)r * p.nKB : nullptr;
  const bool leader = p.pack > 1 && h % p.pack == 0;
  int c = 0;
  bool same = true;
  for (int kb0 = 4 * lane; kb0 < p.nKB; kb0 += 256) {
    const uint32_t bits = live_quad(p, mrow, wide, qb, kb0);
    c += __popc(bits);
    if (leader && mrow)
      for (int j = 1; j < p.pack; ++j)
        same &= live_quad(p, mrow + (size_t)j * p.nQB * p.nKB, wide, qb, kb0) == bits;
  }
  for (int off = 32; off > 0; off >>= 1) c += __shfl_xor(c, off);
  const bool uniform = leader && __ballot(!same) == 0ull;
  if (lane == 0) cnt[r] = c | (uniform ? (int)kUniformBit : 0);
}

// Item of a work list: list 0 holds the rows that are not in a uniform head
// pack, list 1 the uniform packs (item = pack index, its row = its first
// head's).  Returns false when the item is not in the list.
__device__ __forceinline__ bool item_info(const Problem& p, const int32_t* cnt, int list, int item,
                                          int* bin) {
  int c;
  if (list == 0) {
    if (item >= p.R) return false;
    c = cnt[item];
    if (p.pack > 1) {
      const int bh = item / p.nQB, qb = item - bh * p.nQB;
      if (cnt[(bh & ~(p.pack - 1)) * p.nQB + qb] & (int)kUniformBit) return false;
    }
  } else {
    if (item >= p.NP) return false;
    const int bh = item / p.nQB, qb = item - bh * p.nQB;
    c = cnt[bh * p.pack * p.nQB + qb];
    if (!(c & (int)kUniformBit)) return false;
  }
  *bin = count_bin(c & ~(int)kUniformBit);
  return true;
}

// Exclusive scan of one value per thread over a 1024-thread workgroup; the
// sum of all values goes to total.  sh needs 32 ints.
__device__ int wg_exclusive_scan(int x, int* sh, int& total) {
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  int incl = x;
  for (int off = 1; off < 64; off <<= 1) {
    const int y = __shfl_up(incl, off);
    if (lane >= off) incl += y;
  }
  if (lane == 63) sh[wave] = incl;
  __syncthreads();
  if (wave == 0) {
    int w = lane < 16 ? sh[lane] : 0;
    for (int off = 1; off < 16; off <<= 1) {
      const int y = __shfl_up(w, off);
      if (lane >= off) w += y;
    }
    if (lane < 16) sh[16 + lane] = w;  // inclusive wave totals
  }
  __syncthreads();
  const int base = wave > 0 ? sh[16 + wave - 1] : 0;
  total = sh[31];
  __syncthreads();  // sh is free again
  return base + incl - x;
}

// In-place exclusive scan of a[0 .. n) (LDS or global) by a 1024-thread
// workgroup, contiguous segments per thread; returns the total.  The segment
// length is odd, so the 64 lanes of a wave walking their segments in step hit
// 64 different LDS banks (an even length put up to 8 lanes on one bank).
__device__ int wg_scan_array(int* a, long long n, int* sh) {
  const long long per = ((n + 1023) / 1024) | 1;
  const long long lo = min((long long)threadIdx.x * per, n), hi = min(lo + per, n);
  int s = 0;
  for (long long i = lo; i < hi; ++i) s += a[i];
  int total;
  int run = wg_exclusive_scan(s, sh, total);
  for (long long i = lo; i < hi; ++i) {
    const int x = a[i];
    a[i] = run;
    run += x;
  }
  __syncthreads();
  return total;
}

__device__ __forceinline__ void write_header(const Problem& p, int32_t* n_items) {
  int32_t* h = n_items + kPlanAt;
  h[kPfMagic] = kPlanMagic;
  h[kPfR] = p.R;
  h[kPfNKB] = p.nKB;
  h[kPfPack] = p.pack;
  h[kPfCausal] = p.causal;
  h[kPfDelta] = p.delta;
  h[kPfB] = p.B;
  h[kPfHq] = p.Hq;
  h[kPfHkv] = p.Hkv;
  h[kPfSq] = p.S_q;
  h[kPfSk] = p.S_k;
  n_items[kPackItems] = n_items[1];  // k_bucket may take them over
}

// Histogram index of (bin, chunk): bins descending from the list's top bin,
// then chunks, so one exclusive scan yields heaviest-first, stable scatter
// bases.  n_items[kTopBin + list] holds the top bin of each list.
__device__ __forceinline__ int hist_at(int bin, int chunk, int nch, int top) {
  return (top - bin) * nch + chunk;
}

// Common case: one workgroup does the row_ptr scan and the work-order
// histograms and bases in LDS.
__global__ __launch_bounds__(1024) void k_scan_small(Problem p, const int32_t* __restrict__ cnt_g,
                                                     int32_t* __restrict__ row_ptr,
                                                     int32_t* __restrict__ hist_s,
                                                     int32_t* __restrict__ hist_p,
                                                     int32_t* __restrict__ n_items) {
  __shared__ int cnt[kFastRows];
  __shared__ int hist[kBins * (kFastRows / kChunk)];
  __shared__ int sh[32];
  constexpr int kPerThread = kFastRows / 1024;
  const int t = threadIdx.x;
  const int R = p.R;
  {
    int v[kPerThread];
#pragma unroll
    for (int j = 0; j < kPerThread; ++j) {
      const int i = t + 1024 * j;
      v[j] = i < R ? cnt_g[i] : 0;
    }
#pragma unroll
    for (int j = 0; j < kPerThread; ++j)
      if (t + 1024 * j < R) cnt[t + 1024 * j] = v[j];
  }
  __syncthreads();

  // row_ptr: prefix sums in hist (free so far), then stored coalesced
  for (int i = t; i < R; i += 1024) hist[i] = cnt[i] & ~(int)kUniformBit;
  __syncthreads();
  const int total = wg_scan_array(hist, R, sh);
  for (int i = t; i < R; i += 1024) row_ptr[i] = hist[i];
  if (t == 0) row_ptr[R] = total;
  __syncthreads();

  const int pmask = ~(p.pack - 1);  // pack is 1, 2 or 4
  const int dq = 1024 / p.nQB, dr = 1024 % p.nQB;
  for (int list = 0; list < 2; ++list) {
    const int n_all = list == 0 ? R : (p.pack > 1 ? p.NP : 0);
    const int nch = nchunks(n_all);
    // items t, t+1024, ...: (bh, qb) stepped by (dq, dr) instead of divided;
    // first the top bin of the list, then the histogram below it
    auto walk = [&](auto&& fn) {
      int bh = t / p.nQB, qb = t - bh * p.nQB;
      for (int i = t; i < n_all; i += 1024) {
        int c;
        bool present;
        if (list == 0) {
          c = cnt[i];
          present = p.pack == 1 || !(cnt[(bh & pmask) * p.nQB + qb] & (int)kUniformBit);
        } else {
          c = cnt[bh * p.pack * p.nQB + qb];
          present = (c & (int)kUniformBit) != 0;
        }
        fn(i, present ? count_bin(c & ~(int)kUniformBit) : -1);  // -1: not in this list
        qb += dr;
        bh += dq;
        if (qb >= p.nQB) {
          qb -= p.nQB;
          ++bh;
        }
      }
    };
    int top = -1;
    walk([&](int, int bin) { top = max(top, bin); });
    for (int off = 32; off > 0; off >>= 1) top = max(top, __shfl_xor(top, off));
    if ((t & 63) == 0) sh[t >> 6] = top;
    __syncthreads();
    top = -1;
    for (int w = 0; w < 16; ++w) top = max(top, sh[w]);
    __syncthreads();
    if (top < 0) {  // no item in this list
      if (t == 0) {
        n_items[list] = 0;
        n_items[kTopBin + list] = -1;
      }
      continue;
    }
    const int E = (top + 1) * nch;
    for (int i = t; i < E; i += 1024) hist[i] = 0;
    __syncthreads();
    // a wave's 64 items are consecutive rows in one chunk, whose bins come in
    // runs: the first lane of each run of equal entries adds the run's length
    // (the active lanes are a prefix of the wave)
    walk([&](int i, int bin) {
      const int at = bin >= 0 ? hist_at(bin, i / kChunk, nch, top) : -1;
      const int ln = t & 63;
      const int prev = __shfl_up(at, 1);
      const unsigned long long act = __ballot(true);
      const bool first = ln == 0 || prev != at;
      const unsigned long long starts = __ballot(first);
      if (first && at >= 0) {
        const unsigned long long above = ln == 63 ? 0ull : starts & (~0ull << (ln + 1));
        const int end = above != 0 ? __builtin_ctzll(above) : 64 - __builtin_clzll(act);
        atomicAdd(&hist[at], end - ln);
      }
    });
    __syncthreads();
    const int n = wg_scan_array(hist, E, sh);
    int32_t* g = list == 0 ? hist_s : hist_p;
    for (int i = t; i < E; i += 1024) g[i] = hist[i];
    if (t == 0) {
      n_items[list] = n;
      n_items[kTopBin + list] = top;
    }
    __syncthreads();
  }
  if (t == 0) write_header(p, n_items);
}

// Larger problems: per-chunk histograms ...
__global__ __launch_bounds__(256) void k_hist(Problem p, const int32_t* __restrict__ cnt,
                                              int32_t* __restrict__ hist, int list, int nch) {
  __shared__ int h[kBins];
  for (int i = threadIdx.x; i < kBins; i += 256) h[i] = 0;
  __syncthreads();
  int bin;
  if (item_info(p, cnt, list, blockIdx.x * kChunk + threadIdx.x, &bin)) atomicAdd(&h[bin], 1);
  __syncthreads();
  for (int i = threadIdx.x; i < kBins; i += 256) hist[hist_at(i, blockIdx.x, nch, kBins - 1)] = h[i];
}

// ... and one workgroup scanning them and the counts in global memory.
__global__ __launch_bounds__(1024) void k_scan_large(Problem p, const int32_t* __restrict__ cnt,
                                                     int32_t* __restrict__ row_ptr,
                                                     int32_t* hist_s, long long nh_s,
                                                     int32_t* hist_p, long long nh_p,
                                                     int32_t* __restrict__ n_items) {
  __shared__ int sh[32];
  for (long long i = threadIdx.x; i < p.R; i += 1024) row_ptr[i] = cnt[i] & ~(int)kUniformBit;
  __syncthreads();
  const int tot = wg_scan_array(row_ptr, p.R, sh);
  const int ns = wg_scan_array(hist_s, nh_s, sh);
  const int np = nh_p > 0 ? wg_scan_array(hist_p, nh_p, sh) : 0;
  if (threadIdx.x == 0) {
    row_ptr[p.R] = tot;
    n_items[0] = ns;
    n_items[1] = np;
    n_items[kTopBin] = kBins - 1;
    n_items[kTopBin + 1] = kBins - 1;
    write_header(p, n_items);
  }
}

// Workgroups [0, rows_grid): one wave per row writes the live list of the
// row at row_ptr[r].  The rest: one workgroup per chunk of 256 items of a
// work list puts each present item at its bin's base for the chunk plus its
// rank among the chunk's earlier items of the same bin.
__global__ __launch_bounds__(256) void k_fill_scatter(
    Problem p, const uint8_t* __restrict__ mask, int wide, const int32_t* __restrict__ cnt,
    const int32_t* __restrict__ row_ptr, uint32_t* __restrict__ col,
    const int32_t* __restrict__ hist_s, const int32_t* __restrict__ hist_p,
    const int32_t* __restrict__ n_items, int32_t* __restrict__ order_s,
    int32_t* __restrict__ order_p, int rows_grid, int nch_s) {
  __shared__ int bins[kChunk];
  const int t = threadIdx.x;
  if ((int)blockIdx.x < rows_grid) {
    const int wave = t >> 6, lane = t & 63;
    const int r = blockIdx.x * 4 + wave;
    if (r >= p.R) return;
    const int qb = r % p.nQB;
    const uint8_t* mrow = mask ? mask + (size_t)r * p.nKB : nullptr;
    int pos = row_ptr[r];
    for (int kb0 = 4 * lane; kb0 - 4 * lane < p.nKB; kb0 += 256) {
      const uint32_t bits = kb0 < p.nKB ? live_quad(p, mrow, wide, qb, kb0) : 0u;
      // this 256-block's entries in kb order: lane-major, 4 per lane; the
      // entries of earlier lanes counted per bit position (one ballot and
      // one masked bit count each)
      int before = 0, total = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const unsigned long long m = __ballot((bits >> e) & 1u);
        before += (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                                 __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
        total += __popcll(m);
      }
      int k = pos + before;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if ((bits >> e) & 1u) {
          const int kb = kb0 + e;
          col[k++] = (uint32_t)kb | (partial_tile(p, qb, kb) ? 0x80000000u : 0u);
        }
      pos += total;
    }
    return;
  }
  int c = (int)blockIdx.x - rows_grid;
  int list = 0, nch = nch_s;
  if (c >= nch_s) {
    list = 1;
    c -= nch_s;
    nch = nchunks(p.NP);
  }
  const int top = n_items[kTopBin + list];
  const int item = c * kChunk + t;
  int bin = -1;
  const bool present = top >= 0 && item_info(p, cnt, list, item, &bin);
  bins[t] = present ? bin : -1;
  __syncthreads();
  if (!present) return;
  int rank = 0;
  const int4* b4 = reinterpret_cast<const int4*>(bins);
  for (int j = 0; j < (t >> 2); ++j) {
    const int4 v = b4[j];
    rank += (v.x == bin) + (v.y == bin) + (v.z == bin) + (v.w == bin);
  }
  for (int j = t & ~3; j < t; ++j) rank += bins[j] == bin;
  const int32_t* base = list == 0 ? hist_s : hist_p;
  int32_t* order = list == 0 ? order_s : order_p;
  order[base[hist_at(bin, c, nch, top)] + rank] = item;
}

// Stable partition of the single-head work order into the XCD buckets.  The
// bucket of row r is g % 8, with g = r / (nQB*G) = b*Hkv + (key/value head).
// Within a bucket the items go head by head: the bucket's heads g = mb,
// mb + 8, ... fall into bucket_ranges(p) consecutive ranges (one head per
// range when a bucket holds at most kBucketRanges heads), the ranges in
// increasing g, and within a range the items keep the heaviest-first order.
// The workgroups an XCD runs at one time then read the key/value tiles of
// one head, which its L2 keeps, instead of those of all the bucket's heads.
// One 1024-thread workgroup per (bucket, range).  Each takes the order in
// slices of kSlice rounds of 1024 items (one per thread and round, the loads
// of a slice issued together; a 12,288-item order is one slice, loaded
// once).  A first pass counts the items before its range (lower buckets, and
// lower ranges of its bucket) and its own.  Then, per slice: one ballot per
// round gives each wave's count of own items, one wave scans the (round,
// wave) counts into bases, and every own item goes to its base plus the
// count of its wave's earlier lanes.
__global__ __launch_bounds__(1024) void k_bucket(Problem p, const int32_t* __restrict__ order,
                                                 const int32_t* __restrict__ order_p,
                                                 int32_t* __restrict__ n_items,
                                                 int32_t* __restrict__ bucket) {
  constexpr int kSlice = 16;        // rounds of 1024 items per slice
  __shared__ int tab[kSlice * 16];  // (round, wave) counts, then bases
  __shared__ int red[3][16];
  __shared__ int slice_total;
  const int nkey = bucket_ranges(p);
  const int mb = (int)blockIdx.x / nkey;  // this workgroup's bucket
  const int kk = (int)blockIdx.x % nkey;  // and head range
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int n = n_items[0];
  const int rows_per_g = p.nQB * p.G;
  const int nsub = (p.B * p.Hkv + kBuckets - 1) / kBuckets;  // heads of a bucket, at most
  const int per = (nsub + nkey - 1) / nkey;                  // heads per range
  // r / rows_per_g without an integer division (a long instruction sequence
  // per item): the double quotient is within one of the truth for r < 2^31,
  // and one correction step makes it exact
  const double inv_g = 1.0 / (double)rows_per_g;
  auto group_of = [&](int it) {
    int q = (int)((double)it * inv_g);
    const int rem = it - q * rows_per_g;
    q += (rem >= rows_per_g) - (rem < 0);
    return q;
  };
  // head range of group g within its bucket: (g / 8) / per = g / (8 per),
  // the same corrected double quotient
  const int range_div = kBuckets * per;
  const double inv_range = 1.0 / (double)range_div;
  auto range_of = [&](int g) {
    int q = (int)((double)g * inv_range);
    const int rem = g - q * range_div;
    q += (rem >= range_div) - (rem < 0);
    return q;
  };
  // A short head-pack list (fewer than kDemotePacks items) joins a long
  // single-head list (at least kDemoteMinSingle items, so the single-head
  // kernel runs): wave 0 takes one pack item per lane; the pack rows of a
  // bucket go after its single-head items, placed by its last range's
  // workgroup.
  const int np = n_items[1];
  const bool demote = p.pack > 1 && !p.heads_share_mask && np > 0 && np < kDemotePacks &&
                      n >= kDemoteMinSingle;
  int d_item = -1, d_below = 0, d_own = 0, d_rank = 0;
  if (demote && wave == 0) {
    d_item = lane < np ? order_p[lane] : -1;
    const int bh0 = d_item < 0 ? 0 : (d_item / p.nQB) * p.pack;  // b*Hq + first head
    const int bk = (bh0 / p.G) & (kBuckets - 1);                 // bucket of b*Hkv + g
    const unsigned long long mine = __ballot(d_item >= 0 && bk == mb);
    d_below = __popcll(__ballot(d_item >= 0 && bk < mb));
    d_own = __popcll(mine);
    d_rank = __popcll(mine & ((1ull << lane) - 1));
    if (!(d_item >= 0 && bk == mb)) d_item = -1;
  }
  if (blockIdx.x == 0 && t == 0 && demote) n_items[kPackItems] = 0;  // the pack kernels take none
  // item[r]: the order entry of round r; own[r]: it is in this range
  int item[kSlice], own[kSlice];
  int below_b = 0, below_r = 0;  // items of lower buckets, of lower ranges of this one
  auto load = [&](int s0, bool count) {
#pragma unroll
    for (int r = 0; r < kSlice; ++r) {
      const int i = s0 + 1024 * r + t;
      item[r] = i < n ? order[i] : -1;
    }
#pragma unroll
    for (int r = 0; r < kSlice; ++r) {
      const int g = item[r] < 0 ? -1 : group_of(item[r]);
      const int bk = g & (kBuckets - 1);
      const bool in_b = g >= 0 && bk == mb;
      const int key = in_b ? range_of(g) : -1;
      if (count) {
        below_b += g >= 0 && bk < mb;
        below_r += in_b && key < kk;
      }
      own[r] = in_b && key == kk;
    }
  };
  const bool one = n <= kSlice * 1024;  // the whole order stays in registers
  // pass 1: items before this range, and its own
  int mine = 0;
  for (int s0 = 0; s0 < n; s0 += kSlice * 1024) {
    load(s0, true);
#pragma unroll
    for (int r = 0; r < kSlice; ++r) mine += own[r];
  }
  for (int off = 32; off > 0; off >>= 1) {
    below_b += __shfl_xor(below_b, off);
    below_r += __shfl_xor(below_r, off);
    mine += __shfl_xor(mine, off);
  }
  if (lane == 0) {
    red[0][wave] = below_b;
    red[1][wave] = below_r;
    red[2][wave] = mine;
  }
  __syncthreads();
  int lower = p.pack * d_below, before = 0, total = 0;
  for (int w = 0; w < 16; ++w) {
    lower += red[0][w];
    before += red[1][w];
    total += red[2][w];
  }
  const int start = lower + before;  // list position of this range's first item
  int32_t* list = bucket + kBuckets + 1;
  if (kk == 0 && t == 0) bucket[mb] = lower;
  if (kk == nkey - 1) {  // the bucket's pack rows follow its last range
    const int at = start + total;
    if (d_item >= 0) {
      const int qb = d_item % p.nQB, bh0 = (d_item / p.nQB) * p.pack;
      for (int h = 0; h < p.pack; ++h) list[at + d_rank * p.pack + h] = (bh0 + h) * p.nQB + qb;
    }
    if (mb == kBuckets - 1 && t == 0) bucket[kBuckets] = at + p.pack * d_own;
  }
  // pass 2: this range's items in order, one slice at a time
  int run = start;
  for (int s0 = 0; s0 < n; s0 += kSlice * 1024) {
    if (!one) load(s0, false);
#pragma unroll
    for (int r = 0; r < kSlice; ++r) {
      const unsigned long long m = __ballot(own[r] != 0);
      if (lane == 0) tab[r * 16 + wave] = __popcll(m);
    }
    __syncthreads();
    if (wave == 0) {  // exclusive scan of the 256 counts in (round, wave) order
      int v[4], sum = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        v[j] = sum;
        sum += tab[4 * lane + j];
      }
      int incl = sum;  // inclusive scan of the lane sums
      for (int off = 1; off < 64; off <<= 1) {
        const int y = __shfl_up(incl, off);
        if (lane >= off) incl += y;
      }
      const int excl = run + incl - sum;
#pragma unroll
      for (int j = 0; j < 4; ++j) tab[4 * lane + j] = excl + v[j];
      if (lane == 63) slice_total = incl;
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kSlice; ++r) {
      const bool sel = own[r] != 0;
      const unsigned long long m = __ballot(sel);
      if (sel) list[tab[r * 16 + wave] + __popcll(m & ((1ull << lane) - 1))] = item[r];
    }
    run += slice_total;
    __syncthreads();  // tab and slice_total are rewritten by the next slice
  }
}

hipError_t launch_block_index(const Problem& p, const uint8_t* mask, const IndexBuffers& w,
                              hipStream_t s) {
  const int wide = mask == nullptr || ((p.nKB % 4) == 0 && ((uintptr_t)mask & 3u) == 0);
  const int rows_grid = (p.R + 3) / 4;
  const int nch_s = nchunks(p.R);
  const int nch_p = p.pack > 1 ? nchunks(p.NP) : 0;
  hipLaunchKernelGGL(k_classify, dim3(rows_grid), dim3(256), 0, s, p, mask, wide, w.cnt);
  if (p.R <= kFastRows) {
    hipLaunchKernelGGL(k_scan_small, dim3(1), dim3(1024), 0, s, p, w.cnt, w.row_ptr, w.hist_s,
                       w.hist_p, w.n_items);
  } else {
    hipLaunchKernelGGL(k_hist, dim3(nch_s), dim3(256), 0, s, p, w.cnt, w.hist_s, 0, nch_s);
    if (nch_p)
      hipLaunchKernelGGL(k_hist, dim3(nch_p), dim3(256), 0, s, p, w.cnt, w.hist_p, 1, nch_p);
    hipLaunchKernelGGL(k_scan_large, dim3(1), dim3(1024), 0, s, p, w.cnt, w.row_ptr, w.hist_s,
                       (long long)kBins * nch_s, w.hist_p, (long long)kBins * nch_p, w.n_items);
  }
  hipLaunchKernelGGL(k_fill_scatter, dim3(rows_grid + nch_s + nch_p), dim3(256), 0, s, p, mask,
                     wide, w.cnt, w.row_ptr, w.col, w.hist_s, w.hist_p, w.n_items, w.order_s,
                     w.order_p, rows_grid, nch_s);
  if (w.bucket != nullptr)
    hipLaunchKernelGGL(k_bucket, dim3(kBuckets * bucket_ranges(p)), dim3(1024), 0, s, p, w.order_s,
                       w.order_p, w.n_items, w.bucket);
  return hipGetLastError();
}

}  // namespace steel
