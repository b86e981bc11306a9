// Fused sparse attention forward for head packs of 4 on gfx950: one wave per
// query head, 64 rows per wave, software-pipelined, persistent.
//
// Same mathematics as k_attn (the online-softmax recurrence of Algorithm 1
// over the live tiles of a query block, Section IV-A masking, Section IV-C
// work order), with a different schedule:
//
// * Each wave owns all 64 rows of its head (two 32-row MFMA N-tiles), so
//   every K or V fragment read from LDS feeds two MFMAs: half the LDS read
//   traffic of 32-row waves.  One wave per SIMD; O and the Q fragments live
//   in AGPRs (the O MFMAs are issued as inline assembly on AGPR
//   accumulators), S in VGPRs where the softmax reads it.
// * Software pipeline over the tiles i of an item: iteration i runs the
//   softmax of S_i on the VALU while the matrix core computes O += V_{i-1}
//   P_{i-1}, the two interleaved in 32 slots of one MFMA each, then
//   S_{i+1} = K_{i+1} Q^T (the paper's pipeline stages, Algorithm 1, running
//   concurrently inside one wavefront).
// * K/V tiles flow through a 5-stage LDS ring (160 KiB) in one stream across
//   the workgroup's items: while an item finishes, the first tiles of the
//   next one are already being copied, and its Q rows are loaded before
//   the item's last O update.
// * One workgroup per CU; each takes one item per round of its XCD's share
//   of the work order (the same XCD-aware placement as k_attn), serpentine
//   over rounds.
//
// Ring: during iteration i the tiles i-1 (V), i (V, next iteration) and i+1
// (K now, V later) are live; the stage of tile i-2 is refilled with tile i+3,
// which is first read (K) in iteration i+2.  Every wave waits for its own
// copies before the barrier that ends an iteration.
#include <utility>

#include "attn_common.h"

namespace steel {

namespace {

// f(Par<0>{}), f(Par<1>{}), ..., f(Par<N-1>{}): a loop whose index is a
// compile-time constant in every copy of the body.
template <typename F, int... S>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, S...>) {
  (f(Par<S>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

constexpr int kW64Stages = 5;
// GROUP: items of the work order dealt to each XCD in groups of this many
// (see xcd_slot), chosen per launch.  With few items per workgroup, groups of
// 4 spread the heavy end of the order over the XCDs more evenly (S = 4096
// causal, 32/8 heads, 2 items per workgroup: 167 us and 283 MB read with
// groups of 16, 151 us and 159 MB with 4).  With many, groups of 16 keep a
// pack's neighbouring query blocks, which read mostly the same key/value
// tiles, in one XCD's L2 (window/sink S = 16384, 8 items per workgroup: the
// same time either way, 311 MB read with 16 and 471 MB with 4).

// s_waitcnt vmcnt(n) for a count known at run time (n <= 2 tiles of copies);
// larger values wait for everything.
__device__ __forceinline__ void wait_vm_upto(int n) {
  switch (n) {
    case 8: wait_vm<8>(); break;
    case 16: wait_vm<16>(); break;
    default: wait_vm<0>(); break;
  }
}

// Read one accumulator element where it is used: the scores stay in AGPRs
// and only the values a softmax step needs pass through VGPRs.
__device__ __forceinline__ float acc_read(float x) {
  float r;
  asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(r) : "a"(x));
  return r;
}
__device__ __forceinline__ float acc_write(float v) {
  float r;
  asm volatile("v_accvgpr_write_b32 %0, %1" : "=a"(r) : "v"(v));
  return r;
}

// O += A B on the matrix core with the accumulator in AGPRs.  The scores
// use the compiler's MFMA (built with VGPR accumulators, read by the
// softmax), the output accumulator stays in AGPRs: it is only read by the
// rescale and the epilogue, through acc_read after explicit waits.  In-place
// accumulation chains are at least 8 MFMAs apart.
// Four 16-byte global -> LDS copies per lane from one SGPR base: copy j
// writes LDS bytes [lds + 1024 j + 16 lane, +16) from base + off_j.  The
// nops: 5 wait states between a VALU write of an SGPR the copies read and
// the first copy (the compiler pads only its own instructions), and 1 after
// each M0 write.
__device__ __forceinline__ void copy4_to_lds(uint64_t base, uint32_t lds, uint32_t o0, uint32_t o1,
                                             uint32_t o2, uint32_t o3) {
  asm volatile(
      "s_mov_b32 m0, %0\n\t"
      "s_nop 4\n\t"
      "global_load_lds_dwordx4 %2, %1\n\t"
      "s_add_u32 m0, m0, 0x400\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %3, %1\n\t"
      "s_add_u32 m0, m0, 0x400\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %4, %1\n\t"
      "s_add_u32 m0, m0, 0x400\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %5, %1"
      :
      : "s"(lds), "s"(base), "v"(o0), "v"(o1), "v"(o2), "v"(o3)
      : "memory", "m0", "scc");
}

__device__ __forceinline__ void mfma_acc(f32x16& acc, const bf16x8& a, const bf16x8& b) {
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
}

}  // namespace

// RAGGED: S_k is not a multiple of the block, so the last key block is cut
// short and its copies clamp their rows.  Without it that path is compiled
// out (its address arithmetic would otherwise run on every tile).
template <int D, bool RAGGED, int GROUP>
__global__ __launch_bounds__(256, 1) void k_attn_w64(AttnArgs a) {
  constexpr int kGroup = GROUP;
  constexpr int NW = 4;             // waves = query heads of the pack
  constexpr int C = D / 8;          // 16-byte chunks per row
  constexpr int TE = kBlk * D;      // bf16 elements per tile
  constexpr int TB = TE * 2;        // bytes per tile
  constexpr int LPW = C / NW;       // copies per lane per tile and tensor
  constexpr int KS = D / 16;        // k-steps of S^T = K Q^T
  constexpr int DT = D / 32;        // d tiles of O^T
  constexpr int ST = kW64Stages;
  constexpr int CPT = 2 * LPW;      // copy instructions per lane per tile
  constexpr float TAU = 8.0f;       // rescale only when a row max grows by > 2^8
  static_assert(D == 128 && CPT == 8, "tuned for D = 128");
  static_assert(2 * KS * 2 == 32 && 4 * DT * 2 == 32, "32 slots of one QK and one PV MFMA");
  __shared__ __attribute__((aligned(1024))) __bf16 smem[2 * ST * TE];

  if (!plan_matches(a)) return;  // index planned for another problem: out untouched
  const int n_all = ((cint_p)a.n_items)[0];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // in an SGPR
  const int n = lane & 31, hf = lane >> 5;
  const int xb = (int)blockIdx.x & 7, wb = (int)blockIdx.x >> 3, nwb = (int)gridDim.x >> 3;
  const uint32_t lds0 = __builtin_amdgcn_readfirstlane(lds_addr(smem));

  // copy plan: copy j of this lane fills tile slot (wave*LPW + j)*64 + lane,
  // i.e. row (wave*LPW + j)*64/C + lane/C, chunk lane%C (C divides 64)
  static_assert(64 % C == 0, "whole rows per copy instruction");
  const int cp_r0 = lane / C, cp_c = lane % C;
  auto cp_row = [&](int j) __attribute__((always_inline)) { return (wave * LPW + j) * (64 / C) + cp_r0; };
  auto cp_off = [&](int j) __attribute__((always_inline)) {
    const int r = cp_row(j);
    return (uint32_t)((r * D + (cp_c ^ swz<D>(r)) * 8) * 2);
  };
  // LDS read offsets (bytes within a tile): K fragment (sg, ks) and the two
  // transposed halves of V fragment (chunk, dt)
  uint32_t koff[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) koff[ks] = (uint32_t)tile_elem<D>(n, 2 * ks + hf) * 2;
  const int tg = lane >> 4, tr = (lane >> 2) & 3, tq = lane & 3;
  uint32_t voff[2][DT];
#pragma unroll
  for (int cc = 0; cc < 2; ++cc)
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const int row = 8 * cc + 4 * (tg >> 1) + tr;
      voff[cc][dt] = (uint32_t)(tile_elem<D>(row, 4 * dt + 2 * (tg & 1) + (tq >> 1)) + 4 * (tq & 1)) * 2;
    }

  // ---- work items ----
  struct Item {
    int L, beg, qb, b, h0;
    const __bf16* kg;
    const __bf16* vg;
  };
  // This workgroup's items: in round r it takes position
  // r*nwb + w (even r) or r*nwb + (nwb-1-w) (odd r) of its XCD's share of the
  // work order (serpentine: the share is sorted heaviest first, so a
  // workgroup that takes a heavy item in one round takes a light one in the
  // next).  It runs its rounds in the order K-1, 0, 1, ..., K-2: the same
  // items, but the lightest round first, so that workgroups whose items all
  // have the same length do not all reach their item boundaries (Q loads,
  // output stores) at the same moment.
  const int n_x = (n_all / (8 * kGroup)) * kGroup +
                  min(max(n_all % (8 * kGroup) - kGroup * xb, 0), kGroup);
  const int K = (n_x + nwb - 1) / nwb;  // rounds of this XCD
  auto round_pos = [&](int k) __attribute__((always_inline)) -> int {  // -1: none
    if (k >= K) return -1;
    const int r = k == 0 ? K - 1 : k - 1;
    const int p = r * nwb + ((r & 1) ? nwb - 1 - wb : wb);
    return p < n_x ? p : -1;
  };
  // The items are fetched 64 at a time with vector loads: lane t of w_item,
  // w_beg, w_end holds item 64*iw + t (-1 if none) and the bounds of its
  // live list, so decoding an item at an item boundary is register work
  // (scalar loads there would share their wait counter with the LDS reads
  // of the last O update and stall it).
  int iw = -1;
  int w_item = -1, w_beg = 0, w_end = 0;
  auto load_items = [&](int win) __attribute__((always_inline)) {
    const int p = round_pos(64 * win + lane);
    const int idx = p < 0 ? n_all : xcd_slot<kGroup>(8 * p + xb);
    w_item = -1;
    w_beg = 0;
    w_end = 0;
    if (idx < n_all) {
      w_item = a.order[idx];
      const int r0 = (w_item / a.nQB) * 4 * a.nQB + w_item % a.nQB;
      w_beg = a.row_ptr[r0];
      w_end = a.row_ptr[r0 + 1];
    }
    // wait here (once per 64 items), not at every later use
    asm volatile("" ::"v"(w_item), "v"(w_beg), "v"(w_end));
    iw = win;
  };
  auto decode = [&](int k, Item& it) __attribute__((always_inline)) -> bool {
    if ((k >> 6) != iw) load_items(k >> 6);
    const int item = __builtin_amdgcn_readlane(w_item, k & 63);
    if (item < 0) return false;
    it.qb = item % a.nQB;
    const int bh0 = (item / a.nQB) * 4;
    it.b = bh0 / a.Hq;
    const int h0 = bh0 % a.Hq;
    it.h0 = h0;
    it.beg = __builtin_amdgcn_readlane(w_beg, k & 63);
    it.L = __builtin_amdgcn_readlane(w_end, k & 63) - it.beg;
    const size_t kvoff = ((size_t)it.b * a.Hkv + h0 / a.G) * a.S_k * D;
    it.kg = a.k + kvoff;
    it.vg = a.v + kvoff;
    return true;
  };

  // this lane's byte offsets of its four 16-byte chunks of a tile
  static_assert(LPW == 4, "four copies per lane, tile and tensor");
  const uint32_t co0 = cp_off(0), co1 = cp_off(1), co2 = cp_off(2), co3 = cp_off(3);
  auto issue_copy = [&](const __bf16* src, uint32_t dst, int kb) __attribute__((always_inline)) {
    const uint32_t lbase = lds0 + dst + (uint32_t)(wave * LPW) * 1024u;
    if (!RAGGED || (kb + 1) * kBlk <= a.S_k) {
      // the item's pointers may sit in VGPRs: the base goes to an SGPR pair
      const uint64_t p = (uint64_t)(uintptr_t)(src + (size_t)kb * kBlk * D);
      const uint64_t ps = ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(p >> 32)) << 32) |
                          (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)p);
      copy4_to_lds(ps, __builtin_amdgcn_readfirstlane(lbase), co0, co1, co2, co3);
    } else {
#pragma unroll
      for (int j = 0; j < LPW; ++j) {
        const int key = min(kb * kBlk + cp_row(j), a.S_k - 1);
        const uint32_t off = cp_off(j) + (uint32_t)((key - cp_row(j)) * D * 2);
        copy16_to_lds(src, off, lbase + j * 1024u);
      }
    }
  };
  auto issue_tile = [&](const Item& it, int stage, int kb) __attribute__((always_inline)) {
    issue_copy(it.kg, (uint32_t)(2 * stage) * TB, kb);
    issue_copy(it.vg, (uint32_t)(2 * stage + 1) * TB, kb);
  };
  // live-list entry t of an item (t < 64 for the look-ahead of the next
  // item; the current item keeps a 128-entry window in two VGPRs)
  auto load_entry_vec = [&](const Item& it, int base) __attribute__((always_inline)) -> uint32_t {
    return base + lane < it.L ? a.col[it.beg + base + lane] : 0u;
  };

  bf16x8 qf[2][KS];
  auto load_q = [&](const Item& it) __attribute__((always_inline)) {
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      const int row = min(it.qb * kBlk + 32 * nt + n, a.S_q - 1);
      const __bf16* qp = a.q + (((size_t)it.b * a.Hq + it.h0 + wave) * a.S_q + row) * D + 8 * hf;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) qf[nt][ks] = *(const bf16x8*)(qp + 16 * ks);
    }
  };
  // Q fragments are only MFMA operands: keep them in AGPRs (the VGPRs hold
  // the softmax state, P and the LDS fragments)
  auto q_to_agpr = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int nt = 0; nt < 2; ++nt)
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) asm volatile("" : "+a"(qf[nt][ks]));
  };

  f32x16 o[2][DT];
  bf16x8 pa[2][4];  // P of one tile: [nt][chunk]
  float m[2], l[2];
#pragma unroll
  for (int nt = 0; nt < 2; ++nt) {
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) o[nt][dt] = f32x16{};
    m[nt] = -INFINITY;
    l[nt] = 0.f;
  }

  const char* lds_bytes = (const char*)smem;
  auto k_frag = [&](uint32_t kbase, int q) __attribute__((always_inline)) -> bf16x8 {  // q = 2*ks + sg
    return *(const bf16x8*)(lds_bytes + kbase + (q & 1) * 32 * D * 2 + koff[q >> 1]);
  };
  auto v_frag = [&](uint32_t vbase, int q) __attribute__((always_inline)) -> bf16x8 {  // q = 4*chunk + dt
    const int ch = q >> 2, dt = q & 3;
    const char* base = lds_bytes + vbase + (32 * (ch >> 1) + 16 * (ch & 1)) * D * 2;
    const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(base + voff[0][dt]));
    const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(base + voff[1][dt]));
    return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
  };
  auto stage_bytes = [](int s) __attribute__((always_inline)) -> uint32_t { return (uint32_t)(2 * s) * TB; };

  // ---- first item ----
  int j = 0;  // round of the current item
  Item cur, nxt;
  if (!decode(j, cur)) {  // no item in the lightest round: start with the next
    j = 1;
    if (!decode(j, cur)) return;
  }
  bool have_next = decode(j + 1, nxt);
  int pos = 0;          // stream position of cur's tile 0
  int issued_cur = 0;   // tiles of cur already copied
  int issued_next = 0;  // tiles of nxt already copied
  uint32_t win0 = load_entry_vec(cur, 0), win1 = load_entry_vec(cur, 64);
  uint32_t nwin = have_next ? load_entry_vec(nxt, 0) : 0u;
  load_q(cur);
  asm volatile("" ::"v"(win0), "v"(win1), "v"(nwin));
  q_to_agpr();
  wait_vm<0>();
  int wbase = 0;  // the window holds entries wbase .. wbase+127 of cur
  auto entry = [&](int t) __attribute__((always_inline)) -> uint32_t {
    const int off = t - wbase;
    return (uint32_t)__builtin_amdgcn_readlane((int)(off < 64 ? win0 : win1), off & 63);
  };

  f32x16 sc[2][2];  // S of the current tile: [nt][sg]

  while (true) {
    const int L = cur.L;
    // catch up on the copies of cur's first tiles that the previous item did
    // not get to (its stream ended early, or this is the first item)
    for (; issued_cur < min(L, ST - 2); ++issued_cur)
      issue_tile(cur, (pos + issued_cur) % ST, (int)(entry(issued_cur) & 0x7fffffffu));
    wait_vm<0>();
    __syncthreads();

    // S_t = K_t Q^T: 32 MFMAs, the K fragments read two ahead.  On a
    // partial tile (Section IV-A case iii) the elements beyond the causal
    // limit or the last key are then set to -inf (rare: the diagonal tile).
    auto qk_phase = [&](int t) __attribute__((always_inline)) {
      const uint32_t kbase = stage_bytes((pos + t) % ST);
      bf16x8 kf[3];
      kf[0] = k_frag(kbase, 0);
      kf[1] = k_frag(kbase, 1);
      static_for<32>([&](auto slot) __attribute__((always_inline)) {
        constexpr int s = decltype(slot)::value;
        constexpr int q = s >> 1, nt = s & 1;
        if constexpr (nt == 0 && q + 2 < 16) kf[(q + 2) % 3] = k_frag(kbase, q + 2);
        sc[nt][q & 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            kf[q % 3], qf[nt][q >> 1], q < 2 ? f32x16{} : sc[nt][q & 1], 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
      });
      const uint32_t cw = entry(t);
      if (cw >> 31) {
        const int kb = (int)(cw & 0x7fffffffu);
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) {
          const int lim_abs = min(a.causal ? cur.qb * kBlk + 32 * nt + n + a.delta : INT_MAX - kBlk,
                                  a.S_k - 1);
          const int lim = lim_abs - (kb * kBlk + 4 * hf);
#pragma unroll
          for (int sg = 0; sg < 2; ++sg)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              const int off = 32 * sg + 8 * (r >> 2) + (r & 3);
              const unsigned dead = (unsigned)((lim - off) >> 31);
              sc[nt][sg][r] = __uint_as_float((dead & 0xff800000u) |
                                              (~dead & __float_as_uint(sc[nt][sg][r])));
            }
        }
      }
    };

    // Half of chunk (t, ch) of P = 2^(S c - m): 4 exponentials, rounded to
    // bf16; the second half also adds the chunk's bf16 values to l.  The
    // empty statement pins the chunk to its slot (without a use there the
    // compiler sinks the exponentials below the MFMAs they overlap).
    float msafe[2];
    auto p_chunk = [&](auto tv, auto chv, auto hv) __attribute__((always_inline)) {
      constexpr int t = decltype(tv)::value, ch = decltype(chv)::value, h = decltype(hv)::value;
      constexpr int sg = ch >> 1, half = ch & 1;
#pragma unroll
      for (int e = 4 * h; e < 4 * h + 4; ++e)
        pa[t][ch][e] = (__bf16)__builtin_amdgcn_exp2f(
            __builtin_fmaf(sc[t][sg][8 * half + e], a.c, -msafe[t]));
      if constexpr (h == 1) {
        const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
        for (int e = 0; e < 8; e += 2)
          l[t] = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{pa[t][ch][e], pa[t][ch][e + 1]}, ones,
                                                 l[t], false);
        asm volatile("" ::"v"(pa[t][ch]), "v"(l[t]));
      }
    };

    // Softmax of S_i into P_i on the VALU, interleaved with O += V_{i-1}
    // P_{i-1} on the matrix core when PV is set (every tile but the first).
    // P has one buffer: the PV MFMAs of slots 8c .. 8c+7 read chunk c of
    // P_{i-1}, so chunk c of P_i is written after them (chunks 0-2 here,
    // chunk 3 by p_tail once the phase is over).
    auto soft_phase = [&](int i, auto pv_flag) __attribute__((always_inline)) {
      constexpr bool do_pv = decltype(pv_flag)::value != 0;
      const uint32_t vbase = stage_bytes((pos + i + ST - 1) % ST) + TB;
      float mx[2] = {-INFINITY, -INFINITY};
      bf16x8 vf[3];
      if constexpr (do_pv) {
        vf[0] = v_frag(vbase, 0);
        vf[1] = v_frag(vbase, 1);
      }
      bool grow = false;
      float alpha[2] = {1.f, 1.f};
      static_for<32>([&](auto slot) __attribute__((always_inline)) {
        constexpr int s = decltype(slot)::value;
        constexpr int q = s >> 1, nt = s & 1;
        if constexpr (do_pv) {
          if constexpr (nt == 0 && q + 2 < 16) vf[(q + 2) % 3] = v_frag(vbase, q + 2);
          mfma_acc(o[nt][q & 3], vf[q % 3], pa[nt][q >> 2]);
        }
        if constexpr (s < 8) {
          // slots 0..7: row maxima, 8 scores per slot (N-tile s/4)
          constexpr int t = s >> 2, sg = (s >> 1) & 1, r0 = 8 * (s & 1);
#pragma unroll
          for (int r = r0; r < r0 + 8; ++r) mx[t] = fmaxf(mx[t], sc[t][sg][r]);
          asm volatile("" ::"v"(mx[t]));
        } else if constexpr (s == 8) {
#pragma unroll
          for (int t = 0; t < 2; ++t) {
            const float x = other_half_max(mx[t]);
            mx[t] = x == -INFINITY ? -INFINITY : x * a.c;
            grow |= mx[t] > m[t] + TAU;
          }
        } else if constexpr (s == 9) {
          const bool any = __builtin_amdgcn_ballot_w64(grow) != 0;
#pragma unroll
          for (int t = 0; t < 2; ++t) {
            if (any) {
              const float mnew = fmaxf(m[t], mx[t]);
              alpha[t] = mnew == -INFINITY ? 1.f : __builtin_amdgcn_exp2f(m[t] - mnew);
              l[t] *= alpha[t];
              m[t] = mnew;
            }
            msafe[t] = m[t] == -INFINITY ? 0.f : m[t];
          }
          grow = any;
        } else if constexpr (s >= 10 && s < 14) {
          p_chunk(Par<((s - 10) >> 1)>{}, Par<0>{}, Par<((s - 10) & 1)>{});
        } else if constexpr (s >= 16 && s < 20) {
          p_chunk(Par<((s - 16) >> 1)>{}, Par<1>{}, Par<((s - 16) & 1)>{});
        } else if constexpr (s >= 24 && s < 28) {
          p_chunk(Par<((s - 24) >> 1)>{}, Par<2>{}, Par<((s - 24) & 1)>{});
        }
        __builtin_amdgcn_sched_barrier(0);
      });
      // O holds sums relative to the old maxima: rescale before P_i enters it
      // (rare: only when some row max grew by more than TAU; O is still 0 on
      // the first tile)
      if constexpr (do_pv) {
        if (grow) {
          // element by element through one VGPR each (O stays in AGPRs);
          // the nops keep the reads clear of the last MFMA's write
          asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7");
#pragma unroll
          for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int dt = 0; dt < DT; ++dt)
#pragma unroll
              for (int r = 0; r < 16; ++r) o[t][dt][r] = acc_write(acc_read(o[t][dt][r]) * alpha[t]);
        }
      }
    };
    // the last chunk of P_i, after every PV MFMA of the phase
    auto p_tail = [&]() __attribute__((always_inline)) {
      p_chunk(Par<0>{}, Par<3>{}, Par<0>{});
      p_chunk(Par<0>{}, Par<3>{}, Par<1>{});
      p_chunk(Par<1>{}, Par<3>{}, Par<0>{});
      p_chunk(Par<1>{}, Par<3>{}, Par<1>{});
    };

    // copy of stream position pos + i + 3: tile i+3 of cur or a first tile
    // of nxt; returns whether one was issued
    auto copy_ahead = [&](int i) __attribute__((always_inline)) -> bool {
      const int t3 = i + ST - 2;
      const int cstage = (pos + t3) % ST;
      if (t3 < L && t3 >= wbase + 128) {  // slide the window (once per 64 tiles)
        wbase += 64;
        win0 = win1;
        win1 = load_entry_vec(cur, wbase + 64);
        asm volatile("" ::"v"(win1));
      }
      const bool in_cur = t3 < L;
      const bool in_next = !in_cur && have_next && t3 - L == issued_next && issued_next < nxt.L;
      if (in_cur)
        issue_tile(cur, cstage, (int)(entry(t3) & 0x7fffffffu));
      else if (in_next)
        issue_tile(nxt, cstage,
                   (int)((uint32_t)__builtin_amdgcn_readlane((int)nwin, issued_next) & 0x7fffffffu));
      // counters updated outside the branches (kept in SGPRs)
      issued_cur += in_cur ? 1 : 0;
      issued_next += in_next ? 1 : 0;
      return in_cur || in_next;
    };
    // tile i+2 (read as K in the next iteration) must have landed: only the
    // copy issued in this iteration may still be in flight
    auto end_iteration = [&](bool copied) __attribute__((always_inline)) {
      wait_vm_upto(copied ? CPT : 0);
      __syncthreads();
    };
    // middle tile i (0 < i < L-1): softmax(i) with PV(i-1), then S_{i+1}
    auto middle = [&](int i, auto) __attribute__((always_inline)) {
      const bool copied = copy_ahead(i);
      soft_phase(i, Par<1>{});
      p_tail();
      qk_phase(i + 1);
      end_iteration(copied);
    };

    if (L > 0) {
      qk_phase(0);
      // tile 0: softmax only (O is still empty), then S_1
      {
        const bool copied = copy_ahead(0);
        soft_phase(0, Par<0>{});
        p_tail();
        if (L > 1) qk_phase(1);
        end_iteration(copied);
      }
      int i = 1;
      for (; i + 1 < L; ++i) middle(i, Par<0>{});
      // last tile i = L-1 (> 0): softmax(i) with PV(i-1), no further S
      if (i == L - 1 && i > 0) {
        const bool copied = copy_ahead(i);
        soft_phase(i, Par<1>{});
        p_tail();
        end_iteration(copied);
      }
    }

    // Next item: its Q rows are loaded now (qf is free: the last S was
    // computed in iteration L-2), then O += V_{L-1} P_{L-1} and the output.
    // The live-list windows of the next two items are loaded here too,
    // ahead of the output stores, so that waiting for them does not wait
    // for the stores.
    const bool more = have_next;
    Item after;
    bool have_after = false;
    uint32_t win1_next = 0u, nwin_next = 0u;
    if (more) {
      have_after = decode(j + 2, after);
      load_q(nxt);
      win1_next = load_entry_vec(nxt, 64);
      nwin_next = have_after ? load_entry_vec(after, 0) : 0u;
    }
    if (L > 0) {
      // V fragments read two ahead, as in the soft phase
      const uint32_t vbase = stage_bytes((pos + L - 1) % ST) + TB;
      bf16x8 vf[3];
      vf[0] = v_frag(vbase, 0);
      vf[1] = v_frag(vbase, 1);
      static_for<16>([&](auto qv) __attribute__((always_inline)) {
        constexpr int q = decltype(qv)::value;
        if constexpr (q + 2 < 16) vf[(q + 2) % 3] = v_frag(vbase, q + 2);
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) mfma_acc(o[nt][q & 3], vf[q % 3], pa[nt][q >> 2]);
      });
    }
    // Output O / l, staged through LDS so that every store instruction
    // writes two whole 512-byte rows (in the accumulator layout a lane holds
    // 16-byte pieces of one row, and one store would touch 32 rows).  The
    // stages of stream positions pos+L+3 and pos+L+4 are free here: the
    // first was last read in iteration L-2, the second (tile L-1) once every
    // wave has done the O update above, and neither is refilled before the
    // next item's first barrier.  Each wave stages 32 rows (16 KiB) at a
    // time, 16-byte chunk c of row r at chunk c ^ r (conflict-free both
    // ways); it reads back only what it wrote, so no barrier separates the
    // two halves.
    __syncthreads();
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7");  // O reads after the last MFMA
    {
      char* const stg = (char*)smem + stage_bytes((pos + L + 3 + (wave >> 1)) % ST) +
                        (uint32_t)(wave & 1) * 16384u;
      const size_t ob = ((size_t)cur.b * a.Hq + cur.h0 + wave) * a.S_q * D;  // element offset
      const int rr = lane >> 5, cc = lane & 31;  // read-back: row 2k + rr, chunk cc
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const float lt = half_pair_sum(l[t]);
        const float inv = lt > 0.f ? 1.f / lt : 0.f;
        // row log-sum-exp (m + log2 l) ln 2, one lane per row
        if (a.lse != nullptr && hf == 0) {
          const int qrow = cur.qb * kBlk + 32 * t + n;
          if (qrow < a.S_q)
            a.lse[((size_t)cur.b * a.Hq + cur.h0 + wave) * a.S_q + qrow] =
                lt > 0.f ? (m[t] + log2f(lt)) * 0.69314718055994531f : -INFINITY;
        }
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
          for (int gq = 0; gq < 4; ++gq) {
            const f32x4 w = {acc_read(o[t][dt][4 * gq]) * inv, acc_read(o[t][dt][4 * gq + 1]) * inv,
                             acc_read(o[t][dt][4 * gq + 2]) * inv, acc_read(o[t][dt][4 * gq + 3]) * inv};
            const int chunk = 8 * dt + 2 * gq + hf;  // columns 4 * chunk .. 4 * chunk + 3 of row n
            *(f32x4*)(stg + n * 512 + ((chunk ^ n) << 4)) = w;
          }
        const int qrow0 = cur.qb * kBlk + 32 * t;
        if (qrow0 + 32 <= a.S_q) {
          // every row exists: all 16 reads first, then the stores
          f32x4 w[16];
#pragma unroll
          for (int k = 0; k < 16; ++k) {
            const int r = 2 * k + rr;
            w[k] = *(const f32x4*)(stg + r * 512 + ((cc ^ r) << 4));
          }
          if (a.out_bf16) {
#pragma unroll
            for (int k = 0; k < 16; ++k)
              *(bf16x4*)((__bf16*)a.out + ob + (size_t)(qrow0 + 2 * k + rr) * D + 4 * cc) =
                  bf16x4{(__bf16)w[k][0], (__bf16)w[k][1], (__bf16)w[k][2], (__bf16)w[k][3]};
          } else {
#pragma unroll
            for (int k = 0; k < 16; ++k) *(f32x4*)(a.out + ob + (size_t)(qrow0 + 2 * k + rr) * D + 4 * cc) = w[k];
          }
        } else {
#pragma unroll
          for (int k = 0; k < 16; ++k) {
            const int r = 2 * k + rr;
            const f32x4 w = *(const f32x4*)(stg + r * 512 + ((cc ^ r) << 4));
            if (qrow0 + r < a.S_q) {
              const size_t at = ob + (size_t)(qrow0 + r) * D + 4 * cc;
              if (a.out_bf16)
                *(bf16x4*)((__bf16*)a.out + at) = bf16x4{(__bf16)w[0], (__bf16)w[1], (__bf16)w[2], (__bf16)w[3]};
              else
                *(f32x4*)(a.out + at) = w;
            }
          }
        }
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[t][dt][r] = acc_write(0.f);
        m[t] = -INFINITY;
        l[t] = 0.f;
      }
    }
    if (!more) break;
    pos += L;
    cur = nxt;
    issued_cur = issued_next;
    issued_next = 0;
    have_next = have_after;
    if (have_after) nxt = after;
    j += 1;
    wbase = 0;
    win0 = nwin;
    win1 = win1_next;
    nwin = nwin_next;
    asm volatile("" ::"v"(win0), "v"(win1), "v"(nwin));
    q_to_agpr();
  }
}

hipError_t launch_attention_w64(const AttnArgs& a, hipStream_t s) {
  // the pack list has at most NP items (one per head pack and query block)
  const long long np = (long long)a.R / 4;
  const bool few = np <= 4ll * 256;
  if (a.S_k % kBlk != 0) {
    if (few) hipLaunchKernelGGL((k_attn_w64<128, true, 4>), dim3(256), dim3(256), 0, s, a);
    else hipLaunchKernelGGL((k_attn_w64<128, true, 16>), dim3(256), dim3(256), 0, s, a);
  } else {
    if (few) hipLaunchKernelGGL((k_attn_w64<128, false, 4>), dim3(256), dim3(256), 0, s, a);
    else hipLaunchKernelGGL((k_attn_w64<128, false, 16>), dim3(256), dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace steel
