// Pieces shared by the gfx950 attention kernels: kernel arguments, the LDS
// tile layout, the global -> LDS copy, the wave-level helpers and the
// XCD-aware placement of work items.
#pragma once

#include <climits>

#include "internal.h"

namespace steel {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

struct AttnArgs {
  const __bf16* q;
  const __bf16* k;
  const __bf16* v;
  float* out;
  float* lse;               // [B][Hq][S_q] row log-sum-exp, or nullptr
  int out_bf16;             // out holds bf16 (round to nearest even), not fp32
  const int32_t* row_ptr;
  const uint32_t* col;
  const int32_t* order;
  const int32_t* n_items;   // this list's item count
  const int32_t* header;    // plan header (after the two counts)
  const int32_t* bucket;    // single-head list by XCD bucket, or nullptr
  const uint8_t* k8;        // fp8 form: E4M3 tiles of K and V (Fp8Buffers),
  const uint8_t* v8;        //   nullptr in the bf16 form
  const float* f8_scale;    //   and the per-(b, g) inverse scales {1/s_k, 1/s_v}
  int B, Hq, Hkv, S_q, S_k, nQB, nKB, G, causal, delta, R, pack;
  float c;  // scale * log2(e)
};

typedef const __attribute__((address_space(4))) int32_t* cint_p;

// The plan header (written by the index build) describes the same problem as
// the kernel's arguments: every size, the causal limit and the head packing.
// Every field is read unconditionally (no short circuit), so the compiler
// fetches the header with one scalar load instead of one load per field.
__device__ __forceinline__ bool plan_matches(const AttnArgs& a) {
  const cint_p h = (cint_p)a.header;
  const bool ok = (h[kPfMagic] == kPlanMagic) & (h[kPfR] == a.R) & (h[kPfNKB] == a.nKB) &
                  (h[kPfPack] == a.pack) & (h[kPfCausal] == a.causal) & (h[kPfDelta] == a.delta) &
                  (h[kPfB] == a.B) & (h[kPfHq] == a.Hq) & (h[kPfHkv] == a.Hkv) & (h[kPfSq] == a.S_q) &
                  (h[kPfSk] == a.S_k);
  return ok;
}

__device__ __forceinline__ float other_half_max(float x) {
  const unsigned u = __float_as_uint(x);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Sum of the two lanes l and l^32, added in the same order on both.
__device__ __forceinline__ float half_pair_sum(float x) {
  const unsigned u = __float_as_uint(x);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// LDS tile layout: 64 rows (keys) x D bf16, no padding, 16-byte chunks
// XOR-swizzled within a row: chunk c of row r sits at chunk slot
// c ^ swz(r).  swz is linear over the row bits it reads (D = 128: bits 0-3;
// D = 64: bits 1-3), which makes both the 16-byte K reads (32 consecutive
// rows, same chunk) and the transposed V reads (4 rows x 4 chunks per
// 32 lanes) free of LDS bank conflicts on 64 banks, and lets every lane keep
// its read offsets in a few registers.
template <int D>
__device__ __forceinline__ int swz(int r) {
  if constexpr (D == 128) return ((r & 3) << 2) | ((r >> 2) & 3);
  else return (((r >> 1) & 1) << 2) | ((r >> 2) & 3);
}

template <int D>
__device__ __forceinline__ int tile_elem(int r, int c) {  // bf16 offset of (row, chunk)
  return (r * (D / 8) + (c ^ swz<D>(r))) * 8;
}

// s_waitcnt vmcnt(N) with the other counters left alone: waits until at most
// N of this wave's vector memory operations (here: global -> LDS copies) are
// still in flight.  vmcnt is split over bits [3:0] and [15:14].
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0F70);
}

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) void glob_void;

// One 16-byte global -> LDS copy per lane (global_load_lds_dwordx4, SGPR
// base + 32-bit VGPR offset): lane i writes LDS bytes
// [lds_base + 16 i, lds_base + 16 i + 16).  Issued as inline assembly so the
// compiler does not treat every later LDS read as possibly aliasing the copy
// (it would insert a full vmcnt wait before each one); the kernel itself
// waits (wait_vm) and barriers before any wave reads the data.
__device__ __forceinline__ void copy16_to_lds(const void* sbase, uint32_t voff, uint32_t lds_base) {
  // the base pointer and the LDS address are wave-uniform: keep them in SGPRs
  // (readfirstlane returns int: widen through uint32_t so the low half is not
  // sign-extended into the high half)
  const uint64_t p = (uint64_t)(uintptr_t)sbase;
  const uint64_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(p >> 32));
  const uint64_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)p);
  const uint64_t ps = (hi << 32) | lo;
  // The base comes from v_readfirstlane just before the statement: a VMEM
  // instruction may read an SGPR only 5 wait states after a VALU wrote it,
  // and the compiler pads only the instructions it emits itself, so the
  // statement pads its own (s_mov + s_nop 4; also covers the M0 write).
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 4\n\tglobal_load_lds_dwordx4 %1, %2"
               :
               : "s"(__builtin_amdgcn_readfirstlane(lds_base)), "v"(voff), "s"(ps)
               : "memory", "m0");
}

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// Workgroups are dealt to the 8 XCDs round-robin (workgroup b runs on XCD
// b % 8).  Work-order position of workgroup b: the order is cut into groups
// of kXcdGroup consecutive items, group g goes to XCD g % 8, and each XCD
// takes its groups in order.  Neighbouring items of one head pack (adjacent
// query blocks, mostly the same key/value tiles) then share one XCD's L2,
// while every XCD still works from the heavy end of the order first.  The
// grid is a multiple of 8 * kXcdGroup; positions past the item count exit.
constexpr int kXcdGroup = 16;
template <int GROUP = kXcdGroup>
__device__ __forceinline__ int xcd_slot(int b) {
  const int x = b & 7, j = b >> 3;
  return ((j / GROUP) * 8 + x) * GROUP + j % GROUP;
}
inline int xcd_grid(int n) {
  const int m = 8 * kXcdGroup;
  return (n + m - 1) / m * m;
}

typedef const __attribute__((address_space(4))) uint32_t* cuint_p;
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

template <int P> struct Par { static constexpr int value = P; };

// Head packs of 4 at D = 128: two waves per head (scores and softmax; P V and
// output), persistent (attn_ws.hip); prec: a Prec value.
hipError_t launch_attention_ws(const AttnArgs& a, int prec, hipStream_t s);


}  // namespace steel
