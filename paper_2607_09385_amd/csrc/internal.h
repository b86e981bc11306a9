// Internal interfaces between the C ABI layer and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace steel {

constexpr int kBlk = 64;          // mask block edge = tile edge
constexpr int kMaxBins = 4096;    // work-order histogram bins
constexpr int kChunk = 256;       // items per work-order chunk

// Problem description shared by the index build and the attention kernels.
struct Problem {
  int B, Hq, Hkv, S_q, S_k, D;
  int G;        // Hq / Hkv
  int pack;     // query heads of one group processed together (1, 2 or 4)
  int nQB, nKB;
  int causal;
  int delta;    // S_k - S_q
  int R;        // B*Hq*nQB rows of the live-block list
  int NP;       // B*(Hq/pack)*nQB head packs (0 when pack == 1)
  int bin_shift;
  int nbins;
};

// Device workspace of one call.
struct IndexBuffers {
  int32_t* cnt;        // [R]   live blocks per row
  uint8_t* uni;        // [NP]  1 if the pack's rows have identical live lists
  int32_t* hist_s;     // [nbins * nchunk_s]  per-chunk bin counts, then bases
  int32_t* hist_p;     // [nbins * nchunk_p]
  int32_t* row_ptr;    // [R+1]
  uint32_t* col;       // [R*nKB] capacity
  int32_t* order_s;    // [R]   single-head items, heaviest first
  int32_t* order_p;    // [NP]  head-pack items, heaviest first
  int32_t* n_items;    // [8]   {single items, pack items, plan header ...}
};

// Plan header written after the two item counts; the attention kernels check
// it against their own arguments before touching the index.
constexpr int kPlanMagic = 0x5354454c;  // "STEL"
constexpr int kHeaderInts = 8;

inline int nchunks(int n) { return (n + kChunk - 1) / kChunk; }

// Enqueue the index build.  With p.pack == 1 every row is a single-head item.
hipError_t launch_block_index(const Problem& p, const uint8_t* mask, const IndexBuffers& w,
                              hipStream_t stream);

// Enqueue the fused attention over both item lists.
hipError_t launch_attention(const Problem& p, const void* q, const void* k, const void* v,
                            float* out, float scale, const IndexBuffers& w, hipStream_t stream);

}  // namespace steel
