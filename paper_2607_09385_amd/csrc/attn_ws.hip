// Fused sparse attention forward for head packs of 4 at D = 128 on gfx950,
// wave-specialized: per query head one wave computes S = K Q^T and the online
// softmax, a second wave on the same SIMD accumulates O += V P and writes the
// output.
//
// Same mathematics as k_attn (the online-softmax recurrence of Algorithm 1
// over the live tiles of a query block, Section IV-A masking, Section IV-C
// work order).  The schedule is built around how a CDNA4 SIMD issues: a
// wave issues in order, one VALU instruction every 8-16 cycles on its own,
// and an MFMA waits for the SIMD's matrix core, so a wave that mixes score
// MFMAs into its softmax stalls whenever another wave's MFMAs hold the
// matrix core.  Kept apart, one wave's softmax runs while the matrix core
// serves the other wave's MFMAs.  Algorithm 1 has three stages
// (scores, softmax, P V); the paper places them on separate AIE cores, here
// they go to two waves of one SIMD that hand P over through LDS:
//
// * S-wave (waves 0-3, one per head of the pack, 64 query rows): K fragments
//   from LDS, S^T = K Q^T on the matrix core (Q in registers), element mask on
//   partial tiles, row maxima, the rescale decision, P = 2^(S c - m) rounded
//   to bf16; P and the per-row rescale factor go to LDS.
// * O-wave (waves 4-7, same heads, same SIMDs): O^T += V^T P^T on the matrix
//   core (O in registers, V^T through ds_read_b64_tr_b16, P from LDS), the row
//   sums l from the same bf16 P, rescales O and l when the S-wave asks, the
//   output O / l, and every global -> LDS tile copy of the workgroup.
// * One barrier per step.  In step g the S-waves work on tile g of the
//   workgroup's tile stream and the O-waves on tile g - 1, so the two waves of
//   a SIMD share the matrix core and each fills the other's VALU cycles.
//
// The stream is the concatenation of the workgroup's items (a query block of
// a pack of 4 heads sharing one live list), taken in the same XCD-aware,
// heaviest-first, serpentine order as the other kernels; item boundaries need
// no pipeline drain: the O-waves write an item's output while the S-waves
// already compute the next item's first tile.
//
// LDS (152 KiB): a 3-stage K ring and a 2-stage V ring (16 KiB tiles, the
// swizzled layout of attn_common.h), P double-buffered per head (8 KiB), and
// per head and buffer 64 lanes x {alpha[2], m[2]} (1 KiB).  Tile g's V is
// copied during step g and read in step g + 1; tile g's K is copied two steps
// ahead of its use.
//
// The fp8 forms (PREC, see internal.h) keep this schedule and change the
// operands: V (and, with kFp8All, K) come as the pre-pass's E4M3 tiles (8
// KiB, stored in their LDS layout, copied straight), the S-wave rounds P to
// E4M3 (4 KiB per head and buffer) under an exact running maximum and keeps
// the row sums itself (handed over with {alpha, m}), and both products run on
// v_mfma_f32_32x32x64_f8f6f4 (Q quantized per row at each item's start).
#include <utility>

#include "attn_common.h"

namespace steel {

namespace {

template <typename F, int... S>
__device__ __forceinline__ void ws_static_for_impl(F&& f, std::integer_sequence<int, S...>) {
  (f(Par<S>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void ws_static_for(F&& f) {
  ws_static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// Four 16-byte global -> LDS copies per lane from one SGPR base: copy j writes
// LDS bytes [lds + 1024 j + 16 lane, +16) from base + off_j.  The nops: 5 wait
// states between a VALU write of an SGPR the copies read and the first copy
// (the compiler pads only its own instructions), and 1 after each M0 write.
__device__ __forceinline__ void ws_copy4(uint64_t base, uint32_t lds, uint32_t o0, uint32_t o1,
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


// Two 16-byte global -> LDS copies per lane (an 8 KiB E4M3 tile over the
// four O-waves): copy j writes LDS bytes [lds + 1024 j + 16 lane, +16).
__device__ __forceinline__ void ws_copy2(uint64_t base, uint32_t lds, uint32_t o0, uint32_t o1) {
  asm volatile(
      "s_mov_b32 m0, %0\n\t"
      "s_nop 4\n\t"
      "global_load_lds_dwordx4 %2, %1\n\t"
      "s_add_u32 m0, m0, 0x400\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %3, %1"
      :
      : "s"(lds), "s"(base), "v"(o0), "v"(o1)
      : "memory", "m0", "scc");
}

typedef int i32x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ f32x16 ws_mfma_e4m3(const i32x8& a, const i32x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
}

// 32 bytes of E4M3 operand from two 16-byte LDS reads.
__device__ __forceinline__ i32x8 ws_lds_pair(const char* p0, const char* p1) {
  const u32x4 lo = *(const u32x4*)p0, hi = *(const u32x4*)p1;
  return __builtin_bit_cast(i32x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

__device__ __forceinline__ int ws_pack_e4m3(float a, float b, float c, float d) {
  int w = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0, false);
  return __builtin_amdgcn_cvt_pk_fp8_f32(c, d, w, true);
}

__device__ __forceinline__ void wait_lgkm0() { __builtin_amdgcn_s_waitcnt(0xC07F); }

// Workgroup barrier ordering LDS accesses only: the fences keep the compiler
// from moving LDS reads and writes across it and wait for this wave's LDS
// operations, but not for its global loads, stores or tile copies (those are
// waited for explicitly with vmcnt).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

}  // namespace

// RAGGED: S_k is not a multiple of the block (the last key block's copies
// clamp their rows); without it that path is compiled out.
template <bool RAGGED, int GROUP, int PREC>
__global__ __launch_bounds__(512, 1) void k_attn_ws(AttnArgs a) {
  constexpr bool QK8 = PREC == kFp8All;  // S = K Q^T from E4M3 operands
  constexpr bool PV8 = PREC != kBf16;    // O += V P from E4M3 operands
  constexpr int D = 128;
  constexpr int C = D / 8;           // 16-byte chunks per bf16 row
  constexpr int TB = kBlk * D * 2;   // bytes per bf16 K or V tile
  constexpr int TB8 = kBlk * D;      // bytes per E4M3 tile
  constexpr int TBK = QK8 ? TB8 : TB, TBV = PV8 ? TB8 : TB;
  constexpr int KCP = QK8 ? 2 : 4;   // copy instructions per lane of one K tile
  constexpr int KS = D / 16;         // k-steps of S^T = K Q^T (bf16)
  constexpr int KS8 = D / 64;        // k-steps of S^T = K Q^T (E4M3)
  constexpr int DT = D / 32;         // d tiles of O^T
  // bf16 P: rescale only when a row max grows by > 2^8; E4M3 P: on every
  // growth (its weights 2^(S - m + 8) need the exact maximum)
  constexpr float TAU = PV8 ? 0.0f : 8.0f;
  constexpr int PB = PV8 ? 4096 : 8192;  // P bytes per head and buffer
  constexpr int AB = PV8 ? 2048 : 1024;  // {alpha, m} (and l) bytes per head and buffer
  constexpr uint32_t K_AT = 0;                 // K ring: 3 stages
  constexpr uint32_t V_AT = 3 * TBK;           // V ring: 2 stages
  constexpr uint32_t P_AT = V_AT + 2 * TBV;    // P: [2 buffers][4 heads]
  constexpr uint32_t A_AT = P_AT + 8 * PB;     // {alpha, m (, l)}: [2][4]
  constexpr uint32_t LDS_BYTES = A_AT + 8 * AB;
  static_assert(LDS_BYTES <= 160 * 1024, "LDS budget");
  __shared__ __attribute__((aligned(1024))) char smem[LDS_BYTES];

  if (!plan_matches(a)) return;  // index planned for another problem: out untouched
  const int n_all = ((cint_p)a.n_items)[0];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool s_role = wave < 4;
  const int h = wave & 3;                       // head of the pack
  const int n = lane & 31, hf = lane >> 5;
  const int xb = (int)blockIdx.x & 7, wb = (int)blockIdx.x >> 3, nwb = (int)gridDim.x >> 3;
  const uint32_t lds0 = __builtin_amdgcn_readfirstlane(lds_addr(smem));
  const char* lds_bytes = (const char*)smem;

  // ---- work items (decoded identically by every wave) ----
  struct Item {
    int L, beg, qb, b, h0;
  };
  const int n_x = (n_all / (8 * GROUP)) * GROUP +
                  min(max(n_all % (8 * GROUP) - GROUP * xb, 0), GROUP);
  const int K = (n_x + nwb - 1) / nwb;  // rounds of this XCD
  // round k of this workgroup: position r*nwb + w (even r) or r*nwb + nwb-1-w
  // (odd r) of the XCD's share of the work order, rounds in the order K-1,
  // 0, 1, ..., K-2 (lightest first, so that workgroups with equal items do
  // not all reach their item boundaries together)
  auto round_pos = [&](int k) __attribute__((always_inline)) -> int {
    if (k >= K) return -1;
    const int r = k == 0 ? K - 1 : k - 1;
    const int p = r * nwb + ((r & 1) ? nwb - 1 - wb : wb);
    return p < n_x ? p : -1;
  };
  int iw = -1;
  int w_item = -1, w_beg = 0, w_end = 0;
  auto load_items = [&](int win) __attribute__((always_inline)) {
    const int p = round_pos(64 * win + lane);
    const int idx = p < 0 ? n_all : xcd_slot<GROUP>(8 * p + xb);
    w_item = -1;
    w_beg = 0;
    w_end = 0;
    if (idx < n_all) {
      w_item = a.order[idx];
      const int r0 = (w_item / a.nQB) * 4 * a.nQB + w_item % a.nQB;
      w_beg = a.row_ptr[r0];
      w_end = a.row_ptr[r0 + 1];
    }
    asm volatile("" ::"v"(w_item), "v"(w_beg), "v"(w_end));
    iw = win;
  };
  // item of round k; false when the round has none
  auto decode = [&](int k, Item& it) __attribute__((always_inline)) -> bool {
    if (k >= K) return false;
    if ((k >> 6) != iw) load_items(k >> 6);
    const int item = __builtin_amdgcn_readlane(w_item, k & 63);
    if (item < 0) return false;
    it.qb = item % a.nQB;
    const int bh0 = (item / a.nQB) * 4;
    it.b = bh0 / a.Hq;
    it.h0 = bh0 % a.Hq;
    it.beg = __builtin_amdgcn_readlane(w_beg, k & 63);
    it.L = __builtin_amdgcn_readlane(w_end, k & 63) - it.beg;
    return true;
  };
  auto load_entry_vec = [&](const Item& it, int base) __attribute__((always_inline)) -> uint32_t {
    return base + lane < it.L ? a.col[it.beg + base + lane] : 0u;
  };
  auto kv_tile8 = [&](const Item& it) __attribute__((always_inline)) -> size_t {
    return ((size_t)it.b * a.Hkv + it.h0 / a.G) * a.nKB;
  };
  auto out_row_base = [&](const Item& it) __attribute__((always_inline)) -> size_t {
    return ((size_t)it.b * a.Hq + it.h0 + h) * a.S_q;  // row index of the head's row 0
  };

  // Walk of the item sequence shared by both roles: X is the item whose
  // tiles the S-waves work on, Y the next item with at least one tile (empty
  // items in between are handed to on_empty, in order).
  int jx = 0;
  Item X{}, Y{};
  bool have_x = false, have_y = false;
  int jy = 0;
  auto next_nonempty = [&](int from, Item& it, int& jit, auto&& on_empty) __attribute__((always_inline)) -> bool {
    for (int k = from; k < K; ++k) {
      if (!decode(k, it)) continue;
      if (it.L > 0) {
        jit = k;
        return true;
      }
      on_empty(it);
    }
    return false;
  };

  if (s_role) {
    // ===================== S-wave =====================
    uint32_t koff[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) koff[ks] = (uint32_t)tile_elem<D>(n, 2 * ks + hf) * 2;
    auto k_frag = [&](uint32_t kbase, int q) __attribute__((always_inline)) -> bf16x8 {  // q = 2*ks + sg
      return *(const bf16x8*)(lds_bytes + kbase + (q & 1) * 32 * D * 2 + koff[q >> 1]);
    };
    // E4M3 K fragment (sg, ks): row 32*sg + n, logical chunks 4*ks + 2*hf + {0, 1}
    uint32_t koff8[QK8 ? KS8 : 1][2];
#pragma unroll
    for (int ks = 0; ks < (QK8 ? KS8 : 1); ++ks)
#pragma unroll
      for (int u = 0; u < 2; ++u) koff8[ks][u] = (uint32_t)(n * D + 16 * ((4 * ks + 2 * hf + u) ^ kswz8<D>(n)));
    auto k_frag8 = [&](uint32_t kbase, int sg, int ks) __attribute__((always_inline)) -> i32x8 {
      const char* base = lds_bytes + kbase + sg * 32 * D;
      return ws_lds_pair(base + koff8[ks][0], base + koff8[ks][1]);
    };
    // bf16: Q rows as the B operand (lane: row 32*nt + n, d = 16*ks + 8*hf + 0..7).
    // E4M3: the raw rows (lane: d = 64*ks + 32*hf + 0..31) are quantized at
    // the item's first step, with the row's own power-of-two scale.
    bf16x8 qf[2][QK8 ? 8 : KS];
    i32x8 q8[2][QK8 ? KS8 : 1];
    float crow[2] = {a.c, a.c};  // per row: scores (MFMA units) to log2 units
    auto load_q = [&](const Item& it) __attribute__((always_inline)) {
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) {
        const int row = min(it.qb * kBlk + 32 * nt + n, a.S_q - 1);
        const __bf16* qr = a.q + (((size_t)it.b * a.Hq + it.h0 + h) * a.S_q + row) * D;
        if constexpr (QK8) {
#pragma unroll
          for (int u = 0; u < 8; ++u) qf[nt][u] = *(const bf16x8*)(qr + 64 * (u >> 2) + 32 * hf + 8 * (u & 3));
        } else {
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) qf[nt][ks] = *(const bf16x8*)(qr + 8 * hf + 16 * ks);
        }
      }
    };
    auto quant_q = [&](const Item& it) __attribute__((always_inline)) {
      const float dk = a.f8_scale[2 * ((size_t)it.b * a.Hkv + it.h0 / a.G)];
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) {
        float amax = 0.f;
#pragma unroll
        for (int u = 0; u < 8; ++u)
#pragma unroll
          for (int e = 0; e < 8; ++e) amax = fmaxf(amax, fabsf((float)qf[nt][u][e]));
        const float sq = e4m3_scale(other_half_max(amax));
#pragma unroll
        for (int ks = 0; ks < KS8; ++ks)
#pragma unroll
          for (int w = 0; w < 8; ++w) {
            const bf16x8& x = qf[nt][4 * ks + (w >> 1)];
            const int e = 4 * (w & 1);
            q8[nt][ks][w] = ws_pack_e4m3((float)x[e] * sq, (float)x[e + 1] * sq, (float)x[e + 2] * sq,
                                         (float)x[e + 3] * sq);
          }
        crow[nt] = a.c / sq * dk;
      }
    };
    // bf16: Q rows scaled by c = scale * log2(e) and rounded to bf16 at the
    // item's first tile, so the score MFMAs yield log2 units directly, and
    // the accumulators start from -m (the row's running maximum, 0 while it
    // is -inf; nm holds it as a full accumulator tile per N-tile and changes
    // only when m moves): the common tile needs no per-element fma before
    // its exponentials
    constexpr bool MFOLD = PREC == kBf16;
    f32x16 nm[2];
    auto scale_q = [&]() __attribute__((always_inline)) {
#pragma unroll
      for (int nt = 0; nt < 2; ++nt)
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
          for (int e = 0; e < 8; ++e) qf[nt][ks][e] = (__bf16)((float)qf[nt][ks][e] * a.c);
    };
    auto skip = [&](const Item&) __attribute__((always_inline)) {};
    have_x = next_nonempty(0, X, jx, skip);
    if (have_x) have_y = next_nonempty(jx + 1, Y, jy, skip);
    if (have_x) load_q(X);
    uint32_t win0 = 0u, win1 = 0u;
    int wbase = 0;
    if (have_x) {
      win0 = load_entry_vec(X, 0);
      win1 = load_entry_vec(X, 64);
    }
    asm volatile("" ::"v"(win0), "v"(win1));
    lds_barrier();  // prologue: the first K tiles are in

    f32x16 sc[2][2];
    bf16x8 pa[2][4];
    float m[2] = {-INFINITY, -INFINITY};
    float ls[2] = {0.f, 0.f};  // E4M3 P: the row sums, kept here
    int g = 0;     // step
    int ks3 = 0;   // g % 3: K stage
    while (have_x) {
      const int L = X.L;
      for (int t = 0; t < L; ++t) {
        if (t >= wbase + 128) {  // slide the live-list window (once per 64 tiles)
          wbase += 64;
          win0 = win1;
          win1 = load_entry_vec(X, wbase + 64);
          asm volatile("" ::"v"(win1));
        }
        const int off = t - wbase;
        const uint32_t cw = (uint32_t)__builtin_amdgcn_readlane((int)(off < 64 ? win0 : win1), off & 63);
        const uint32_t kbase = K_AT + (uint32_t)ks3 * TBK;
        if (t == 0) {
          m[0] = -INFINITY;
          m[1] = -INFINITY;
          ls[0] = 0.f;
          ls[1] = 0.f;
          if constexpr (QK8) quant_q(X);
          if constexpr (MFOLD) {
            scale_q();
            nm[0] = f32x16{};
            nm[1] = f32x16{};
          }
        }
        // S^T = K Q^T: for each K fragment (keys 32 sg .. +31, k-step ks) the
        // two N-tiles; fragments read two ahead
        if constexpr (QK8) {
#pragma unroll
          for (int sg = 0; sg < 2; ++sg)
#pragma unroll
            for (int ks = 0; ks < KS8; ++ks) {
              const i32x8 kf = k_frag8(kbase, sg, ks);
#pragma unroll
              for (int nt = 0; nt < 2; ++nt)
                sc[nt][sg] = ws_mfma_e4m3(kf, q8[nt][ks], ks == 0 ? f32x16{} : sc[nt][sg]);
            }
        } else {
          bf16x8 kf[3];
          kf[0] = k_frag(kbase, 0);
          kf[1] = k_frag(kbase, 1);
          ws_static_for<32>([&](auto slot) __attribute__((always_inline)) {
            constexpr int s = decltype(slot)::value;
            constexpr int q = s >> 1, nt = s & 1;  // q = 2*ks + sg
            if constexpr (nt == 0 && q + 2 < 16) kf[(q + 2) % 3] = k_frag(kbase, q + 2);
            sc[nt][q & 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                kf[q % 3], qf[nt][q >> 1], q < 2 ? (MFOLD ? nm[nt] : f32x16{}) : sc[nt][q & 1], 0, 0, 0);
          });
        }
        // the item's last tile: Q of the next item (its loads run under the
        // softmax of this tile)
        if (t == L - 1 && have_y) load_q(Y);
        // element mask of a partial tile (Section IV-A case iii)
        if (cw >> 31) {
          const int kb = (int)(cw & 0x7fffffffu);
#pragma unroll
          for (int nt = 0; nt < 2; ++nt) {
            const int lim_abs = min(a.causal ? X.qb * kBlk + 32 * nt + n + a.delta : INT_MAX - kBlk,
                                    a.S_k - 1);
            const int lim = lim_abs - (kb * kBlk + 4 * hf);
#pragma unroll
            for (int sg = 0; sg < 2; ++sg)
#pragma unroll
              for (int r = 0; r < 16; ++r) {
                const int o = 32 * sg + 8 * (r >> 2) + (r & 3);
                const unsigned dead = (unsigned)((lim - o) >> 31);
                sc[nt][sg][r] = __uint_as_float((dead & 0xff800000u) | (~dead & __float_as_uint(sc[nt][sg][r])));
              }
          }
        }
        // row maxima and the rescale decision: m moves only when some row's
        // maximum grew by more than TAU (then P <= 2^TAU; m cancels in O / l)
        float alpha[2] = {1.f, 1.f}, msafe[2];
        {
          bool grow = false;
          float mx[2];
#pragma unroll
          for (int nt = 0; nt < 2; ++nt) {
            float x = -INFINITY;
#pragma unroll
            for (int sg = 0; sg < 2; ++sg)
#pragma unroll
              for (int r = 0; r < 16; ++r) x = fmaxf(x, sc[nt][sg][r]);
            x = other_half_max(x);
            if constexpr (MFOLD)  // scores relative to msafe, in log2 units
              mx[nt] = x == -INFINITY ? -INFINITY : x + (m[nt] == -INFINITY ? 0.f : m[nt]);
            else
              mx[nt] = x == -INFINITY ? -INFINITY : x * crow[nt];
            grow |= mx[nt] > m[nt] + TAU;
          }
          const bool any = __builtin_amdgcn_ballot_w64(grow) != 0;
          float mold[2];
#pragma unroll
          for (int nt = 0; nt < 2; ++nt) {
            mold[nt] = m[nt] == -INFINITY ? 0.f : m[nt];
            if (any) {
              const float mnew = fmaxf(m[nt], mx[nt]);
              alpha[nt] = mnew == -INFINITY ? 1.f : __builtin_amdgcn_exp2f(m[nt] - mnew);
              m[nt] = mnew;
              if constexpr (PV8) ls[nt] *= alpha[nt];
            }
            msafe[nt] = m[nt] == -INFINITY ? 0.f : m[nt];
          }
          if constexpr (MFOLD) {
            if (any) {  // rare: the scores move to the new maximum, and so does nm
#pragma unroll
              for (int nt = 0; nt < 2; ++nt) {
                const float d = mold[nt] - msafe[nt];
#pragma unroll
                for (int sg = 0; sg < 2; ++sg) sc[nt][sg] += d;
                nm[nt] = -msafe[nt] + f32x16{};
              }
            }
          }
        }
        if constexpr (PV8) {
          // P = 2^(S c - m + 8), at most 2^8 (m is the exact running
          // maximum), rounded to E4M3 in the operand's byte order (byte
          // 16*sg + r of the lane's 32 = register r of sub-tile sg); the row
          // sums add the unrounded weights
          const int pb = g & 1;
          char* ad = (char*)smem + A_AT + (uint32_t)(pb * 4 + h) * AB + lane * 16;
          *(f32x4*)ad = f32x4{alpha[0], alpha[1], m[0], m[1]};
          char* pdst = (char*)smem + P_AT + (uint32_t)(pb * 4 + h) * PB + lane * 16;
#pragma unroll
          for (int nt = 0; nt < 2; ++nt) {
            const float mo = 8.f - msafe[nt];
#pragma unroll
            for (int sg = 0; sg < 2; ++sg) {
              float pv[16];
#pragma unroll
              for (int r = 0; r < 16; ++r)
                pv[r] = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[nt][sg][r], crow[nt], mo));
#pragma unroll
              for (int r = 0; r < 16; ++r) ls[nt] += pv[r];
              const u32x4 w = {(uint32_t)ws_pack_e4m3(pv[0], pv[1], pv[2], pv[3]),
                               (uint32_t)ws_pack_e4m3(pv[4], pv[5], pv[6], pv[7]),
                               (uint32_t)ws_pack_e4m3(pv[8], pv[9], pv[10], pv[11]),
                               (uint32_t)ws_pack_e4m3(pv[12], pv[13], pv[14], pv[15])};
              *(u32x4*)(pdst + (nt * 2 + sg) * 1024) = w;
              __builtin_amdgcn_sched_barrier(0);
            }
          }
          *(f32x4*)(ad + 1024) = f32x4{ls[0], ls[1], 0.f, 0.f};
        } else
        // P = 2^(S c - m), rounded to bf16 (the PV operand layout), each
        // 16-byte chunk handed to the O-wave as soon as it is computed, so
        // the LDS writes run under the remaining exponentials
        {
          const int pb = g & 1;
          *(f32x4*)((char*)smem + A_AT + (uint32_t)(pb * 4 + h) * 1024u + lane * 16) =
              f32x4{alpha[0], alpha[1], m[0], m[1]};
          char* pdst = (char*)smem + P_AT + (uint32_t)(pb * 4 + h) * 8192u + lane * 16;
#pragma unroll
          for (int nt = 0; nt < 2; ++nt)
#pragma unroll
            for (int ch = 0; ch < 4; ++ch) {
#pragma unroll
              for (int e = 0; e < 8; ++e)
                pa[nt][ch][e] = (__bf16)__builtin_amdgcn_exp2f(
                    MFOLD ? sc[nt][ch >> 1][8 * (ch & 1) + e]
                          : __builtin_fmaf(sc[nt][ch >> 1][8 * (ch & 1) + e], a.c, -msafe[nt]));
              *(bf16x8*)(pdst + (nt * 4 + ch) * 1024) = pa[nt][ch];
              __builtin_amdgcn_sched_barrier(0);
            }
        }
        lds_barrier();
        ++g;
        ks3 = ks3 == 2 ? 0 : ks3 + 1;
      }
      // next item
      if (!have_y) break;
      X = Y;
      jx = jy;
      have_y = next_nonempty(jx + 1, Y, jy, skip);
      wbase = 0;
      win0 = load_entry_vec(X, 0);
      win1 = load_entry_vec(X, 64);
      asm volatile("" ::"v"(win0), "v"(win1));
    }
    return;
  }

  // ===================== O-wave =====================
  const int ow = wave - 4;  // copy share and head
  // copy plan: copy j of this lane fills tile slot (ow*4 + j)*64 + lane, i.e.
  // row (ow*4 + j)*4 + lane/16, chunk lane%16 (source chunk swizzled)
  const int cp_r0 = lane / C, cp_c = lane % C;
  auto cp_row = [&](int j) __attribute__((always_inline)) { return (ow * 4 + j) * (64 / C) + cp_r0; };
  auto cp_off = [&](int j) __attribute__((always_inline)) {
    const int r = cp_row(j);
    return (uint32_t)((r * D + (cp_c ^ swz<D>(r)) * 8) * 2);
  };
  const uint32_t co0 = cp_off(0), co1 = cp_off(1), co2 = cp_off(2), co3 = cp_off(3);
  auto issue_copy = [&](const __bf16* src, uint32_t dst, int kb) __attribute__((always_inline)) {
    const uint32_t lbase = lds0 + dst + (uint32_t)(ow * 4) * 1024u;
    if (!RAGGED || (kb + 1) * kBlk <= a.S_k) {
      const uint64_t p = (uint64_t)(uintptr_t)(src + (size_t)kb * kBlk * D);
      const uint64_t ps = ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(p >> 32)) << 32) |
                          (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)p);
      ws_copy4(ps, __builtin_amdgcn_readfirstlane(lbase), co0, co1, co2, co3);
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int key = min(kb * kBlk + cp_row(j), a.S_k - 1);
        const uint32_t off = cp_off(j) + (uint32_t)((key - cp_row(j)) * D * 2);
        copy16_to_lds(src, off, lbase + j * 1024u);
      }
    }
  };
  auto kv_base = [&](const Item& it) __attribute__((always_inline)) -> size_t {
    return ((size_t)it.b * a.Hkv + it.h0 / a.G) * a.S_k * D;
  };
  // E4M3 tile kb of an item's key/value head (stored as it sits in LDS, keys
  // past S_k zero): two straight 16-byte pieces per lane
  const uint32_t c8o0 = (uint32_t)(((ow * 2) * 64 + lane) * 16), c8o1 = (uint32_t)(((ow * 2 + 1) * 64 + lane) * 16);
  auto issue_copy8 = [&](const uint8_t* src8, uint32_t dst, const Item& it, int kb) __attribute__((always_inline)) {
    const uint64_t p = (uint64_t)(uintptr_t)(src8 + (kv_tile8(it) + (size_t)kb) * TB8);
    const uint64_t ps = ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(p >> 32)) << 32) |
                        (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)p);
    ws_copy2(ps, __builtin_amdgcn_readfirstlane(lds0 + dst + (uint32_t)(ow * 2) * 1024u), c8o0, c8o1);
  };
  auto copy_k = [&](uint32_t dst, const Item& it, int kb) __attribute__((always_inline)) {
    if constexpr (QK8) issue_copy8(a.k8, dst, it, kb);
    else issue_copy(a.k + kv_base(it), dst, kb);
  };
  // V^T fragment (chunk, dt) of a V stage: the two transposed halves
  const int tg = lane >> 4, tr = (lane >> 2) & 3, tq = lane & 3;
  uint32_t voff[2][DT];
#pragma unroll
  for (int cc = 0; cc < 2; ++cc)
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const int row = 8 * cc + 4 * (tg >> 1) + tr;
      voff[cc][dt] = (uint32_t)(tile_elem<D>(row, 4 * dt + 2 * (tg & 1) + (tq >> 1)) + 4 * (tq & 1)) * 2;
    }
  // E4M3 V^T fragment dt: row 32*dt + n of the transposed tile, logical
  // chunks 2*hf + {0, 1}
  uint32_t voff8[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) voff8[u] = (uint32_t)(n * kBlk + 16 * ((2 * hf + u) ^ ((n >> 2) & 3)));
  auto v_frag8 = [&](uint32_t vbase, int dt) __attribute__((always_inline)) -> i32x8 {
    const char* base = lds_bytes + vbase + dt * 32 * kBlk;
    return ws_lds_pair(base + voff8[0], base + voff8[1]);
  };
  auto v_frag = [&](uint32_t vbase, int q) __attribute__((always_inline)) -> bf16x8 {  // q = 4*chunk + dt
    const int ch = q >> 2, dt = q & 3;
    const char* base = lds_bytes + vbase + (32 * (ch >> 1) + 16 * (ch & 1)) * D * 2;
    const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(base + voff[0][dt]));
    const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(base + voff[1][dt]));
    return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
  };

  // output rows of an item from the accumulators: O / l (0 for rows with no
  // visible key), fp32 or bf16, and the row log-sum-exp
  f32x16 o[2][DT];
  float l[2] = {0.f, 0.f};
  auto write_rows = [&](const Item& it, const float* mz, bool zero) __attribute__((always_inline)) {
    const size_t rb = out_row_base(it);
    // E4M3 forms: V's scale divided out here; the weights carry an extra 2^8
    const float dvw = PV8 ? a.f8_scale[2 * ((size_t)it.b * a.Hkv + it.h0 / a.G) + 1] : 1.f;
    constexpr float m_off = PV8 ? 8.f : 0.f;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const float lt = zero ? 0.f : half_pair_sum(l[t]);
      const float inv = lt > 0.f ? dvw / lt : 0.f;
      const int row = it.qb * kBlk + 32 * t + n;
      if (a.lse != nullptr && hf == 0 && row < a.S_q)
        a.lse[rb + row] = lt > 0.f ? (mz[t] - m_off + log2f(lt)) * 0.69314718055994531f : -INFINITY;
      const size_t at = (rb + (size_t)min(row, a.S_q - 1)) * D + 4 * hf;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int gq = 0; gq < 4; ++gq) {
          f32x4 w;
          if (zero) {
            w = f32x4{0.f, 0.f, 0.f, 0.f};
          } else {
            w = f32x4{o[t][dt][4 * gq] * inv, o[t][dt][4 * gq + 1] * inv, o[t][dt][4 * gq + 2] * inv,
                      o[t][dt][4 * gq + 3] * inv};
          }
          if (row < a.S_q) {
            if (a.out_bf16)
              *(bf16x4*)((__bf16*)a.out + at + 32 * dt + 8 * gq) =
                  bf16x4{(__bf16)w[0], (__bf16)w[1], (__bf16)w[2], (__bf16)w[3]};
            else
              *(f32x4*)(a.out + at + 32 * dt + 8 * gq) = w;
          }
        }
    }
  };
  const float minf2[2] = {-INFINITY, -INFINITY};
  auto zero_item = [&](const Item& it) __attribute__((always_inline)) { write_rows(it, minf2, true); };

  have_x = next_nonempty(0, X, jx, zero_item);
  if (have_x) have_y = next_nonempty(jx + 1, Y, jy, zero_item);
  uint32_t win0 = 0u, win1 = 0u, nwin = 0u;
  int wbase = 0;
  if (have_x) {
    win0 = load_entry_vec(X, 0);
    win1 = load_entry_vec(X, 64);
  }
  if (have_y) nwin = load_entry_vec(Y, 0);
  asm volatile("" ::"v"(win0), "v"(win1), "v"(nwin));
  // K tile of stream position p (relative to X's first position) if X or Y
  // holds it: entry of X (window) or of Y (first 64 entries)
  auto k_entry = [&](int p, int& kb, bool& in_y) __attribute__((always_inline)) -> bool {
    if (p < X.L) {
      const int off = p - wbase;
      if (off >= 128) return false;  // beyond the window: copied after the slide
      kb = (int)(((uint32_t)__builtin_amdgcn_readlane((int)(off < 64 ? win0 : win1), off & 63)) & 0x7fffffffu);
      in_y = false;
      return true;
    }
    const int py = p - X.L;
    if (!have_y || py >= Y.L || py >= 64) return false;
    kb = (int)(((uint32_t)__builtin_amdgcn_readlane((int)nwin, py)) & 0x7fffffffu);
    in_y = true;
    return true;
  };
  // prologue: K tiles of positions 0 and 1
  int pk = 0;  // next stream position (relative to X) whose K tile is to be copied
  if (have_x) {
    for (int p = 0; p < 2; ++p) {
      int kb;
      bool in_y;
      if (!k_entry(p, kb, in_y)) break;
      copy_k(K_AT + (uint32_t)p * TBK, in_y ? Y : X, kb);
      ++pk;
    }
  }
  wait_vm<0>();
  lds_barrier();

  Item W{};           // item of the tile the O-wave works on
  int wu = -1;        // its tile index (-1: none yet)
  float mz[2] = {-INFINITY, -INFINITY};
  int g = 0;
  int kring = 0;      // K stage of position pk (absolute position mod 3)
  // (absolute position of pk = X's first position + pk)
  {
    // kring tracks (first(X) + pk) % 3; first(X) = 0 here
    kring = pk % 3;
  }
  // PV of the previous step's S tile (item W, tile wu) and, on its last tile,
  // the output of W
  // PV of the previous step's S tile (item W, tile wu): P and {alpha, m}
  // from LDS, the rescale of O and l when asked (rare; not on an item's first
  // tile, whose output starts from zero), O += V P with the V^T fragments
  // read two ahead, the row sums of the bf16 P the MFMAs consumed, and on the
  // item's last tile its output.
  auto pv_mfmas = [&](uint32_t vbase, const bf16x8 (&pa)[2][4], auto first_v) __attribute__((always_inline)) {
    constexpr bool FIRST = decltype(first_v)::value != 0;
    bf16x8 vf[3];
    vf[0] = v_frag(vbase, 0);
    vf[1] = v_frag(vbase, 1);
    ws_static_for<32>([&](auto slot) __attribute__((always_inline)) {
      constexpr int s = decltype(slot)::value;
      constexpr int q = s >> 1, nt = s & 1;  // q = 4*chunk + dt
      if constexpr (nt == 0 && q + 2 < 16) vf[(q + 2) % 3] = v_frag(vbase, q + 2);
      o[nt][q & 3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
          vf[q % 3], pa[nt][q >> 2], (FIRST && (q >> 2) == 0) ? f32x16{} : o[nt][q & 3], 0, 0, 0);
    });
  };
  auto pv_mfmas8 = [&](uint32_t vbase, const i32x8 (&p8)[2], auto first_v) __attribute__((always_inline)) {
    constexpr bool FIRST = decltype(first_v)::value != 0;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const i32x8 vf = v_frag8(vbase, dt);
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) o[nt][dt] = ws_mfma_e4m3(vf, p8[nt], FIRST ? f32x16{} : o[nt][dt]);
    }
  };
  auto pv_step8 = [&](int gprev) __attribute__((always_inline)) {
    const int pb = gprev & 1;
    const char* ab = lds_bytes + A_AT + (uint32_t)(pb * 4 + h) * AB + lane * 16;
    const f32x4 am = *(const f32x4*)ab;
    i32x8 p8[2];
    const char* psrc = lds_bytes + P_AT + (uint32_t)(pb * 4 + h) * PB + lane * 16;
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) p8[nt] = ws_lds_pair(psrc + (nt * 2) * 1024, psrc + (nt * 2 + 1) * 1024);
    const uint32_t vbase = V_AT + (uint32_t)(gprev & 1) * TBV;
    if (wu == 0) {
      pv_mfmas8(vbase, p8, Par<1>{});
    } else {
      if (__builtin_amdgcn_ballot_w64(am[0] != 1.f || am[1] != 1.f) != 0) {
        // O holds sums relative to the old maxima (the S-wave rescales l)
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) o[t][dt] *= am[t];
      }
      pv_mfmas8(vbase, p8, Par<0>{});
    }
    mz[0] = am[2];
    mz[1] = am[3];
    if (wu == W.L - 1) {
      const f32x4 al = *(const f32x4*)(ab + 1024);
      l[0] = al[0];
      l[1] = al[1];
      write_rows(W, mz, false);
    }
  };
  auto pv_step = [&](int gprev) __attribute__((always_inline)) {
    if constexpr (PV8) {
      pv_step8(gprev);
      return;
    }
    const int pb = gprev & 1;
    const f32x4 am = *(const f32x4*)(lds_bytes + A_AT + (uint32_t)(pb * 4 + h) * 1024u + lane * 16);
    bf16x8 pa[2][4];
    const char* psrc = lds_bytes + P_AT + (uint32_t)(pb * 4 + h) * 8192u + lane * 16;
#pragma unroll
    for (int nt = 0; nt < 2; ++nt)
#pragma unroll
      for (int ch = 0; ch < 4; ++ch) pa[nt][ch] = *(const bf16x8*)(psrc + (nt * 4 + ch) * 1024);
    const uint32_t vbase = V_AT + (uint32_t)(gprev & 1) * TB;
    if (wu == 0) {
      l[0] = 0.f;
      l[1] = 0.f;
      pv_mfmas(vbase, pa, Par<1>{});
    } else {
      if (__builtin_amdgcn_ballot_w64(am[0] != 1.f || am[1] != 1.f) != 0) {
        // O and l hold sums relative to the old maxima
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          l[t] *= am[t];
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) o[t][dt] *= am[t];
        }
      }
      pv_mfmas(vbase, pa, Par<0>{});
    }
    mz[0] = am[2];
    mz[1] = am[3];
    const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
    for (int nt = 0; nt < 2; ++nt)
#pragma unroll
      for (int ch = 0; ch < 4; ++ch)
#pragma unroll
        for (int e = 0; e < 8; e += 2)
          l[nt] = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{pa[nt][ch][e], pa[nt][ch][e + 1]}, ones, l[nt], false);
    if (wu == W.L - 1) write_rows(W, mz, false);
  };

  while (have_x) {
    const int L = X.L;
    for (int t = 0; t < L; ++t) {
      // slide X's live-list window when a copy position would leave it
      if (pk < L && pk >= wbase + 128) {
        wbase += 64;
        win0 = win1;
        win1 = load_entry_vec(X, wbase + 64);
        asm volatile("" ::"v"(win1));
      }
      // V of this step's S tile (position t of X): read in the next step
      {
        const int off = t - wbase;
        const int kb = (int)(((uint32_t)__builtin_amdgcn_readlane((int)(off < 64 ? win0 : win1), off & 63)) & 0x7fffffffu);
        if constexpr (PV8) issue_copy8(a.v8, V_AT + (uint32_t)(g & 1) * TBV, X, kb);
        else issue_copy(a.v + kv_base(X), V_AT + (uint32_t)(g & 1) * TB, kb);
      }
      // K tiles up to position t + 2 (two steps ahead; a position in the item
      // after Y is copied once that item is Y).  Before the barrier this
      // step's V copy and every K copy up to position t + 1 must have landed:
      // the memory counter completes in issue order, so waiting until at
      // most kpend operations are outstanding (the copy of position t + 2,
      // when it was the last one issued; the output stores come later and
      // are waited for too) is enough.
      int kpend = 0;
      while (pk <= t + 2) {
        int kb;
        bool in_y;
        if (!k_entry(pk, kb, in_y)) break;
        copy_k(K_AT + (uint32_t)kring * TBK, in_y ? Y : X, kb);
        kpend = pk == t + 2 ? KCP : 0;
        ++pk;
        kring = kring == 2 ? 0 : kring + 1;
      }
      if (wu >= 0) pv_step(g - 1);
      // this step's S tile becomes the O-wave's next tile
      if (t == 0) W = X;
      wu = t;
      if (kpend != 0) wait_vm<KCP>();
      else wait_vm<0>();
      lds_barrier();
      ++g;
    }
    if (!have_y) break;
    // next item: positions continue into Y
    pk -= L;
    X = Y;
    jx = jy;
    have_y = next_nonempty(jx + 1, Y, jy, zero_item);
    wbase = 0;
    win0 = nwin;
    win1 = load_entry_vec(X, 64);
    nwin = have_y ? load_entry_vec(Y, 0) : 0u;
    asm volatile("" ::"v"(win0), "v"(win1), "v"(nwin));
  }
  // drain: the last S tile
  if (wu >= 0) pv_step(g - 1);
}

template <int PREC>
static void launch_ws(const AttnArgs& a, hipStream_t s) {
  const long long np = (long long)a.R / 4;
  const bool few = np <= 4ll * 256;
  // E4M3 tiles are padded with zero keys: only bf16 K or V tiles clamp
  if (PREC != kFp8All && a.S_k % kBlk != 0) {
    if (few) hipLaunchKernelGGL((k_attn_ws<true, 4, PREC>), dim3(256), dim3(512), 0, s, a);
    else hipLaunchKernelGGL((k_attn_ws<true, 16, PREC>), dim3(256), dim3(512), 0, s, a);
  } else {
    if (few) hipLaunchKernelGGL((k_attn_ws<false, 4, PREC>), dim3(256), dim3(512), 0, s, a);
    else hipLaunchKernelGGL((k_attn_ws<false, 16, PREC>), dim3(256), dim3(512), 0, s, a);
  }
}

hipError_t launch_attention_ws(const AttnArgs& a, int prec, hipStream_t s) {
  if (prec == kFp8All) launch_ws<kFp8All>(a, s);
  else if (prec == kFp8Pv) launch_ws<kFp8Pv>(a, s);
  else launch_ws<kBf16>(a, s);
  return hipGetLastError();
}

}  // namespace steel
