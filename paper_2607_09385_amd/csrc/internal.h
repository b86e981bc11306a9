// Internal interfaces between the C ABI layer and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace steel {

constexpr int kBlk = 64;          // mask block edge = tile edge
constexpr int kBins = 512;        // work-order bins (count_bin < kBins)
constexpr int kChunk = 256;       // items per work-order chunk

// Work-order bin of a live count c in [0, 2^31): c itself below 128; above,
// 16 bins per octave, 128 + 16*(e - 7) + (the 4 bits below the leading one),
// e = floor(log2 c).  Monotone in c, exact where the counts are small, and
// within 1/16 of the count where they are large.
__host__ __device__ inline int count_bin(int c) {
  if (c < 128) return c;
  const int e = 31 - __builtin_clz((unsigned)c);
  return 128 + 16 * (e - 7) + ((c >> (e - 4)) & 15);
}

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
  // Block mask from coordinates instead of a mask tensor (win_blocks > 0):
  // block (qb, kb) is in the mask iff qb - win_blocks < kb <= qb (a window
  // of win_blocks blocks ending at the block diagonal) or kb < sink_blocks.
  // The index kernels then read no mask (the paper generates masks on the
  // core rather than fetching them, Section III-B; windowed attention is the
  // masking scheme Section IV-A names).
  int win_blocks, sink_blocks;
  // Set by the fused calls when every query head has the same block mask (no
  // mask tensor, or the structured mask): with pack > 1 every head pack is
  // then uniform and the single-head list is empty, so it is not launched.
  int heads_share_mask;
  int out_bf16;  // output in bf16 (RNE of the fp32 result) instead of fp32
  int fp8;       // operand precision of the products: a Prec value
};

// Operand precision of Algorithm 1's two products: bf16 (the paper's AIE
// datapath, Section II-C), E4M3 for P V only, or E4M3 for both (see
// Fp8Buffers); accumulation is fp32 in every case.
enum Prec { kBf16 = 0, kFp8Pv = 1, kFp8All = 2 };

// Operands of the fp8 form, written by the pre-pass (quant_fp8.hip) and read
// by the attention kernels.  Both tensors are cut into the 64-key tiles of
// the mask, tile (b*Hkv + g, kb) at byte (b*Hkv + g) * nKB * 64 * D +
// kb * 64 * D, keys past S_k zero; each tile is stored exactly as the
// kernels keep it in LDS, so one straight copy moves it:
//   k8  row r (key 64 kb + r) of D bytes E4M3(K s_k); its 16-byte chunk c
//       (dims 16c .. 16c + 15) at chunk slot c ^ kswz(r) of the row;
//   v8  row d of 64 bytes E4M3(V s_v) over the tile's keys in the order of
//       the P operand (byte j = 32 h + b holds key 32 (b/16) + 8 ((b%16)/4)
//       + 4 h + b%4); its chunk c at slot c ^ ((d >> 2) & 3).
// The swizzles keep the 16-byte operand reads of 16 lanes on distinct LDS
// banks.  scale: per (b*Hkv + g) the two inverse scales {1/s_k, 1/s_v};
// part: the per-chunk maxima the scales come from.  k8 is nullptr when
// only P V takes E4M3 operands.
struct Fp8Buffers {
  uint8_t* k8;
  uint8_t* v8;
  float* part;   // [B*Hkv][kFp8Chunks][2]
  float* scale;  // [B*Hkv][2]
};
constexpr int kFp8Chunks = 128;
constexpr float kE4M3Max = 448.f;

template <int D>
__host__ __device__ inline int kswz8(int r) {
  return D == 128 ? (r >> 1) & 7 : (r >> 2) & 3;
}

// Power-of-two scale 2^floor(log2(448 / amax)) of a tensor whose largest
// magnitude is amax (1 for 0 or a non-finite amax).
__host__ __device__ inline float e4m3_scale(float amax) {
  if (!(amax > 0.f) || !(amax <= 3.4e38f)) return 1.f;
  const float x = kE4M3Max / amax;  // >= 1.3e-36: a normal float
  uint32_t bits;
  __builtin_memcpy(&bits, &x, 4);
  bits &= 0x7f800000u;              // 2^floor(log2 x)
  if (bits == 0x7f800000u) bits = 0x7f000000u;  // x overflowed: 2^127
  float sc;
  __builtin_memcpy(&sc, &bits, 4);
  return sc;
}

// Device workspace of one call.
struct IndexBuffers {
  int32_t* cnt;        // [R]   live blocks per row (| kUniformBit, see below)
  int32_t* hist_s;     // [kBins * nchunk_s]  per-chunk bin counts, then bases
  int32_t* hist_p;     // [kBins * nchunk_p]
  int32_t* row_ptr;    // [R+1]
  uint32_t* col;       // [R*nKB] capacity
  int32_t* order_s;    // [R]   single-head items, heaviest first
  int32_t* order_p;    // [NP]  head-pack items, heaviest first
  int32_t* n_items;    // [kHeaderInts] {single items, pack items, plan header,
                       //   top bins of the two lists, pack items the pack
                       //   kernels take} (see kPlanAt, kTopBin, kPackItems)
  // single-head items dealt to the 8 XCDs by key/value head (nullptr: none):
  // [kBuckets + 1] bucket starts, then the items of order_s stably
  // partitioned by bucket
  int32_t* bucket;
};

// XCD buckets of single-head items: bucket (b*Hkv + g) % kBuckets, so that the
// workgroups of one XCD read the key/value tensors of only a few heads and
// its L2 keeps them.
constexpr int kBuckets = 8;

// Head ranges of a bucket: its key/value heads g = mb, mb + 8, ... (at most
// ceil(B*Hkv / 8)) split into at most kBucketRanges consecutive ranges.
constexpr int kBucketRanges = 8;
__host__ __device__ inline int bucket_ranges(const Problem& p) {
  const int nsub = (p.B * p.Hkv + kBuckets - 1) / kBuckets;
  return nsub < kBucketRanges ? nsub : kBucketRanges;
}

// Plan header written after the two item counts; the attention kernels check
// it against their own arguments before touching the index, so a run with
// other sizes, another causal limit or another head packing than the plan
// leaves its output untouched.  Layout of n_items: [0] single-head items,
// [1] head-pack items, [kPlanAt + f] field f of PlanField, [kTopBin + list]
// the top work-order bin of each list, [kPackItems] the head-pack items the
// pack kernels take (n_items[1], or 0 when k_bucket hands a short pack list
// to the single-head kernel, see kDemotePacks).
constexpr int kPlanMagic = 0x5354454c;  // "STEL"
enum PlanField { kPfMagic, kPfR, kPfNKB, kPfPack, kPfCausal, kPfDelta, kPfB, kPfHq, kPfHkv,
                 kPfSq, kPfSk, kPlanFields };
constexpr int kPlanAt = 2;
constexpr int kTopBin = kPlanAt + kPlanFields;
constexpr int kPackItems = kTopBin + 2;
constexpr int kHeaderInts = kPackItems + 1;

// A head-pack list shorter than kDemotePacks (a quarter of the CUs) is run
// by the single-head kernel, as pack-many rows per item, when that kernel
// has at least kDemoteMinSingle items of its own: a pack kernel for a few
// items would add one item's latency to the run while most CUs idle, and the
// single-head kernel absorbs the rows.  The rows of a uniform pack have one
// live list, so either kernel computes the same rows.
constexpr int kDemotePacks = 64;
constexpr int kDemoteMinSingle = 1024;

__host__ __device__ inline int nchunks(int n) { return (n + kChunk - 1) / kChunk; }

// Set in cnt[r] of the first row of a head pack whose rows all have the same
// live list (counts are below 2^30: R * nKB < 2^31).
constexpr uint32_t kUniformBit = 1u << 30;

// Up to this many rows one workgroup scans the counts and the work-order
// histograms in LDS (4 + 4 * kBins / kChunk = 12 bytes per row: 144 KiB).
constexpr int kFastRows = 12288;

// Size of the fixed per-device scratch array of steel_attn_fwd_noalloc (the
// live-block index of one call: counts, histograms, row_ptr, the list
// capacity R * nKB and the work orders).  Equals STEEL_NOALLOC_SCRATCH_BYTES.
constexpr size_t kNoAllocBytes = (size_t)32 << 20;

// Device address of this device's copy of that array (looked up on the
// first call for a device, with the device made current, then cached).
hipError_t noalloc_scratch(int dev, char** ptr);

// Enqueue the index build.  With p.pack == 1 every row is a single-head item.
hipError_t launch_block_index(const Problem& p, const uint8_t* mask, const IndexBuffers& w,
                              hipStream_t stream);

// Enqueue the top-k mean-pooled block selection (block_select.hip): writes the
// whole block mask [B][Hq][nQB][nKB].  qm, km, scores: float64 workspace of
// B*Hq*nQB*D, B*Hkv*nKB*D and B*Hq*nQB*nKB values.  Needs nKB <= 4096.
hipError_t launch_topk_mask(const Problem& p, const __bf16* q, const __bf16* k, int keep_num,
                            int keep_den, uint8_t* mask, double* qm, double* km, double* scores,
                            hipStream_t stream);

// Enqueue the fp8 pre-pass: per (b, g) maxima of |K| and |V|, their scales
// and the E4M3 tiles of Fp8Buffers.
hipError_t launch_fp8_prepass(const Problem& p, const void* k, const void* v, const Fp8Buffers& f,
                              hipStream_t stream);

// Enqueue the fused attention over both item lists; lse (nullable) receives
// the row log-sum-exp [B][Hq][S_q].  f: the fp8 operands when p.fp8, else
// ignored.
hipError_t launch_attention(const Problem& p, const void* q, const void* k, const void* v,
                            float* out, float* lse, float scale, const IndexBuffers& w,
                            const Fp8Buffers& f, hipStream_t stream);

// Enqueue the merge of n_parts partial results over disjoint key sets
// (attn_merge.hip): o_parts [n_parts][rows][D], lse_parts [n_parts][rows].
hipError_t launch_merge(const float* o_parts, const float* lse_parts, int n_parts, long long rows,
                        int D, float* out, float* lse_out, hipStream_t stream);

}  // namespace steel
