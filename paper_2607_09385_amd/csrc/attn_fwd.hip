// Fused sparse attention forward on gfx950 (bf16 MFMA, fp32 softmax state).
//
// The math is the online-softmax recurrence of Algorithm 1 (Section IV):
// for each live key block j of a query block i,
//   S = Q_i K_j^T (scaled by scale*log2 e, so exp becomes exp2),
//   element mask on partial tiles (Section IV-A, case iii),
//   m' = max(m, rowmax S);  P = 2^(S - m');  a = 2^(m - m');
//   l = a*l + rowsum P;  O = a*O + P V_j;  m = m'
// and finally O = O / l.  The three pipeline stages the paper maps onto three
// AIE cores become three phases of one wavefront here; the key/value
// broadcast of Section IV-B becomes one LDS copy of each K/V tile shared by
// every wave of the workgroup.
//
// Layout.  Each wave owns 32 query rows.  The score tile is computed
// transposed, S^T = K Q^T, with v_mfma_f32_32x32x16_bf16: A = K rows from
// LDS, B = Q rows held in VGPRs.  In the accumulator, lane l then holds query
// row l%32 and 16 of the 32 keys of a sub-tile (key 8*(r/4) + 4*(l/32) + r%4
// for register r), so a row's max and sum need one cross-half exchange
// (v_permlane32_swap) instead of a 32-lane reduction, and the per-row scale
// factors live in the same lane as the output row.  P in that layout is
// already the B operand of O^T += V^T P^T, with the keys of each 16-key step
// taken in the order (4 keys of this half, then the same 4 keys 8 further);
// V^T is read from the row-major V tile with ds_read_b64_tr_b16, whose
// 16-lane 4x16 -> 16x4 transpose delivers exactly those keys per d column.
//
// A workgroup handles one work item: either one (b, h, qb) query block
// (4 waves: two row halves times two key halves of every tile) or a pack of
// PACK query heads of one key/value group that share the same live list
// (2*PACK waves), so each K/V tile is loaded once for up to 256 query rows.
#include <climits>

#include "attn_common.h"

namespace steel {

// Depth of the K/V ring (stages of one K tile and one V tile each).  A
// single-head workgroup has only two waves, so it keeps the ring short and
// leaves LDS for more workgroups per CU.
template <int PACK>
constexpr int stages_for() { return PACK == 1 ? 2 : 4; }

// Key halves per row half: a single head in bf16 splits every tile's keys
// over two wave pairs (see k_attn); everything else keeps whole tiles per
// wave.
template <int D, int PACK, int PREC, bool RAGGED>
constexpr int key_halves() { return PACK == 1 && PREC == kBf16 ? 2 : 1; }
template <int D, int PACK, int PREC, bool RAGGED>
constexpr int attn_threads() { return 128 * PACK * key_halves<D, PACK, PREC, RAGGED>(); }
// Waves per SIMD the register allocation must allow: the key-split D = 64
// kernel is built for four (128 VGPRs), so that four of its workgroups (16
// waves, the 2-stage rings filling 128 KiB of LDS) share a CU; 1 leaves the
// allocation free.
template <int D, int PACK, int PREC, bool RAGGED>
constexpr int attn_min_waves() { return D == 64 && key_halves<D, PACK, PREC, RAGGED>() == 2 ? 4 : 1; }

typedef int i32x8 __attribute__((ext_vector_type(8)));

// Four values rounded to E4M3 (nearest even), packed in memory order.
__device__ __forceinline__ int pack_e4m3(float a, float b, float c, float d) {
  int w = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0, false);
  return __builtin_amdgcn_cvt_pk_fp8_f32(c, d, w, true);
}

// 32 bytes of E4M3 operand from two 16-byte LDS reads.
__device__ __forceinline__ i32x8 lds_pair(const char* p0, const char* p1) {
  const u32x4 lo = *(const u32x4*)p0, hi = *(const u32x4*)p1;
  return __builtin_bit_cast(i32x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

__device__ __forceinline__ f32x16 mfma_e4m3(const i32x8& a, const i32x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
}

// End of a key-split single-head workgroup: the waves of the two key halves of
// one row half hold (m_h, l_h, O_h) over their keys, with O_h = sum 2^(s - m_h) v
// and l_h the sum of the same weights.  With M = max(m_0, m_1) and
// w_h = 2^(m_h - M) (0 for a half that saw no key) the row's state is
// l = w_0 l_0 + w_1 l_1, O = w_0 O_0 + w_1 O_1.  Each wave finishes half of the
// d tiles: it leaves the other half of its O, its m and its row sum in LDS
// (free once the loop's last barrier has passed), and reads its partner's.
// LDS per record: [field][lane] floats, record (row half, key half).
template <int D>
__device__ __forceinline__ void merge_halves(const AttnArgs& a, f32x16 (&o)[D / 32], float m,
                                             float l, int kh, int rh, int lane, float* xs, int b,
                                             int head, int qrow0, int hf) {
  constexpr int DT = D / 32, HD = DT / 2;  // d tiles, d tiles finished per wave
  constexpr int F = 2 + 16 * HD;           // fields per record
  const float lt = half_pair_sum(l);
  float* mine = xs + (rh * 2 + kh) * F * 64 + lane;
  const float* part = xs + (rh * 2 + (kh ^ 1)) * F * 64 + lane;
  // d tiles [0, HD) are finished by key half 0, [HD, DT) by key half 1 (the
  // register array is only indexed by constants: selects, not scratch)
  mine[0] = m;
  mine[64] = lt;
#pragma unroll
  for (int j = 0; j < HD; ++j) {
    const f32x16 give = kh ? o[j] : o[HD + j];
#pragma unroll
    for (int r = 0; r < 16; ++r) mine[(2 + 16 * j + r) * 64] = give[r];
  }
  __syncthreads();
  const float mp = part[0], ltp = part[64];
  const float M = fmaxf(m, mp);
  const float w = m == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m - M);
  const float wp = mp == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mp - M);
  const float ls = w * lt + wp * ltp;
  const float inv = ls > 0.f ? 1.f / ls : 0.f;
  const int qrow = qrow0;
  if (qrow >= a.S_q) return;
  // log sum_j exp(scale s_ij) = (M + log2 l) ln 2 (Algorithm 1's statistics)
  if (a.lse != nullptr && hf == 0 && kh == 0)
    a.lse[((size_t)b * a.Hq + head) * a.S_q + qrow] =
        ls > 0.f ? (M + log2f(ls)) * 0.69314718055994531f : -INFINITY;
  const size_t at = (((size_t)b * a.Hq + head) * a.S_q + qrow) * D + 4 * hf;
#pragma unroll
  for (int j = 0; j < HD; ++j) {
    const int dt = kh * HD + j;
    const f32x16 keep = kh ? o[HD + j] : o[j];
#pragma unroll
    for (int gq = 0; gq < 4; ++gq) {
      f32x4 v;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = 4 * gq + e;
        v[e] = (w * keep[r] + wp * part[(2 + 16 * j + r) * 64]) * inv;
      }
      if (a.out_bf16) {
        const bf16x4 vb = {(__bf16)v[0], (__bf16)v[1], (__bf16)v[2], (__bf16)v[3]};
        *(bf16x4*)((__bf16*)a.out + at + 32 * dt + 8 * gq) = vb;
      } else {
        *(f32x4*)(a.out + at + 32 * dt + 8 * gq) = v;
      }
    }
  }
}

// Workgroup = PACK heads x 64 query rows.  Each wave owns 32 query rows (one
// 32-row MFMA N-tile) of one head, two waves per head, so that two waves
// share each SIMD and one can issue MFMAs while the other computes
// exponentials.  A single head at D = 128 (whose register use allows one
// such workgroup per SIMD pair only) would leave one wave per SIMD, so there
// the keys of every tile are split as well: waves 0-1 take keys 0-31, waves
// 2-3 keys 32-63, each with its own softmax state, and the two states of a
// row are merged at the end (the split-key form of the same recurrence, exact
// up to rounding).  A single head at D = 64 splits its keys the same way:
// each wave then holds half the scores and fits in 128 VGPRs, so four waves
// share each SIMD (twice the softmax issue of the two-wave form, whose four
// workgroups per CU left two per SIMD).
// RAGGED: S_k is not a multiple of the block (the
// tail block's copies clamp their rows); without it that path is compiled out.
template <int D, int PACK, bool RAGGED, int PREC>
__global__ __launch_bounds__((attn_threads<D, PACK, PREC, RAGGED>()))
__attribute__((amdgpu_waves_per_eu(attn_min_waves<D, PACK, PREC, RAGGED>()))) void k_attn(AttnArgs a) {
  constexpr bool QK8 = PREC == kFp8All;  // S = K Q^T from E4M3 operands
  constexpr bool PV8 = PREC != kBf16;    // O += V P from E4M3 operands
  constexpr int NT = 1;            // 32-row N-tiles per wave
  constexpr int KH = key_halves<D, PACK, PREC, RAGGED>();  // key halves (waves per 32 rows)
  constexpr int NSG = 2 / KH;      // 32-key sub-tiles per wave and tile
  constexpr int NW = PACK * 2 * KH;  // waves
  constexpr int C = D / 8;         // 16-byte chunks per bf16 row
  constexpr int TE = kBlk * D;     // elements per tile
  constexpr int TB8 = TE;          // bytes of an E4M3 tile
  constexpr int TBK = QK8 ? TB8 : 2 * TE, TBV = PV8 ? TB8 : 2 * TE;  // K, V tile bytes
  constexpr int SB = TBK + TBV;    // bytes per ring stage
  // 16-byte copies per lane per tile: bf16 tiles LPW from every wave; E4M3
  // tiles LPW8 from the first CW8 waves
  constexpr int LPW = C / NW;
  constexpr int LPW8 = TB8 / 16 >= 64 * NW ? TB8 / 16 / (64 * NW) : 1;
  constexpr int CW8 = TB8 / 16 / (64 * LPW8);
  // copy instructions per lane per tile of waves below CW8 and of the others
  constexpr int CPT_LO = (QK8 ? LPW8 : LPW) + (PV8 ? LPW8 : LPW);
  constexpr int CPT_HI = (QK8 ? 0 : LPW) + (PV8 ? 0 : LPW);
  constexpr int KS = D / 16;       // k-steps of S^T = K Q^T (bf16)
  constexpr int KS8 = D / 64;      // k-steps of S^T = K Q^T (fp8)
  constexpr int DT = D / 32;       // d tiles of O^T
  // bf16 P: rescale only when the row max grows by > 2^8; E4M3 P: on every
  // growth (its weights need the exact maximum, see the P step)
  constexpr float TAU = PV8 ? 0.0f : 8.0f;
  static_assert(LPW >= 1 && C % NW == 0 && CW8 >= 1 && CW8 <= NW && CW8 * 64 * LPW8 * 16 == TB8,
                "tile copy split");
  // A ring of ST stages, each holding the K and the V tile of one key block:
  // tiles i+1 .. i+ST-1 are being copied in while tile i is computed on.
  constexpr int ST = stages_for<PACK>();
  __shared__ __attribute__((aligned(1024))) char smem[ST * SB];

  // index data is read-only during the kernel: scalar loads
  int item;
  if (PACK == 1 && a.bucket != nullptr) {
    // single-head items: workgroup b runs on XCD b % 8 and takes the
    // (b / 8)-th item of that XCD's bucket (heaviest first within it).  The
    // bucket bounds (always present) and the plan header are read together,
    // so that the many workgroups past a short bucket leave after one load.
    const cint_p bk = (cint_p)a.bucket;
    const int x = (int)blockIdx.x & (kBuckets - 1), j = (int)blockIdx.x / kBuckets;
    const int lo = bk[x], hi = bk[x + 1];
    const bool ok = plan_matches(a);
    if (j >= hi - lo) return;
    if (!ok) return;  // index planned for another problem: out untouched
    item = bk[kBuckets + 1 + lo + j];
    if ((unsigned)item >= (unsigned)a.R) return;  // never for a well-formed index
  } else {
    if (!plan_matches(a)) return;  // index planned for another problem: out untouched
    const int idx = xcd_slot((int)blockIdx.x);
    if (idx >= ((cint_p)a.n_items)[0]) return;
    item = ((cint_p)a.order)[idx];
  }
  const int qb = item % a.nQB;
  const int bh0 = (item / a.nQB) * PACK;  // b*Hq + first head
  const int b = bh0 / a.Hq;
  const int h0 = bh0 % a.Hq;
  const int g = h0 / a.G;

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int kh = KH == 1 ? 0 : wave >> 1;  // key half of this wave
  const int head = h0 + (KH == 1 ? wave >> 1 : 0);
  const int n = lane & 31, hf = lane >> 5;
  const int qrow0 = qb * kBlk + (wave & 1) * 32 + n;  // N-tile nt holds row qrow0 + 32*nt

  const int r0 = bh0 * a.nQB + qb;
  const int beg = ((cint_p)a.row_ptr)[r0];
  const int L = ((cint_p)a.row_ptr)[r0 + 1] - beg;
  const cuint_p colp = (cuint_p)a.col + beg;
  const size_t kvoff = ((size_t)b * a.Hkv + g) * a.S_k * D;
  const __bf16* kg = a.k + kvoff;
  const __bf16* vg = a.v + kvoff;
  const uint32_t lds0 = __builtin_amdgcn_readfirstlane(lds_addr(smem));

  // copy plan: copy j of this lane fills tile slot (wave*LPW + j)*64 + lane,
  // i.e. row r = slot / C, chunk slot % C, which holds source chunk
  // (slot % C) ^ swz(r) of key row r.
  uint32_t cp_off[LPW];
  int cp_row[LPW];
#pragma unroll
  for (int j = 0; j < LPW; ++j) {
    const int slot = (wave * LPW + j) * 64 + lane;
    const int r = slot / C;
    cp_row[j] = r;
    cp_off[j] = (uint32_t)((r * D + ((slot % C) ^ swz<D>(r)) * 8) * 2);
  }
  // Copy key block kb of K (or V) into the tile buffer at LDS byte offset
  // dst.  Rows past S_k (the tail block) read the last key row instead.
  auto issue_copy = [&](const __bf16* src, uint32_t dst, int kb) {
    const uint32_t lbase = lds0 + dst + (uint32_t)(wave * LPW) * 1024u;
    if (!RAGGED || (kb + 1) * kBlk <= a.S_k) {
      const __bf16* sb = src + (size_t)kb * kBlk * D;
#pragma unroll
      for (int j = 0; j < LPW; ++j) copy16_to_lds(sb, cp_off[j], lbase + j * 1024u);
    } else {
#pragma unroll
      for (int j = 0; j < LPW; ++j) {
        const int key = min(kb * kBlk + cp_row[j], a.S_k - 1);
        const uint32_t off = cp_off[j] + (uint32_t)((key - cp_row[j]) * D * 2);
        copy16_to_lds(src, off, lbase + j * 1024u);
      }
    }
  };
  // E4M3 tiles are stored as they sit in LDS (keys past S_k zero), so a
  // straight copy by the first CW8 waves, LPW8 16-byte pieces per lane
  const size_t tile8 = ((size_t)b * a.Hkv + g) * a.nKB;  // first tile of this head
  auto issue_copy8 = [&](const uint8_t* src, uint32_t dst, int kb) {
    if (wave < CW8) {
      const uint8_t* sb = src + (tile8 + kb) * TB8;
      const uint32_t lbase = lds0 + dst + (uint32_t)(wave * LPW8) * 1024u;
#pragma unroll
      for (int j = 0; j < LPW8; ++j)
        copy16_to_lds(sb, (uint32_t)(((wave * LPW8 + j) * 64 + lane) * 16), lbase + j * 1024u);
    }
  };
  // K and V tiles of key block kb into ring stage st (K at st*SB, V after it)
  auto copy_kv = [&](int st, int kb) {
    const uint32_t at = (uint32_t)st * SB;
    if constexpr (QK8) issue_copy8(a.k8, at, kb);
    else issue_copy(kg, at, kb);
    if constexpr (PV8) issue_copy8(a.v8, at + TBK, kb);
    else issue_copy(vg, at + TBK, kb);
  };

  // Per-lane LDS read offsets in bytes (tile buffer base and the row block of
  // each fragment are compile-time immediates; a key-half wave adds its half):
  //   K fragment (sg, ks): row 32*sg + n, chunk (2*ks + hf)
  //   V fragment (sg, t, cc, dt): row 32*sg + 16*t + 8*cc + 4*(tg>>1) + tr,
  //                               chunk 4*dt + 2*(tg&1) + (tq>>1), half tq&1
  const uint32_t half_off = (uint32_t)(kh * 32 * D * 2);
  uint32_t koff[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) koff[ks] = (uint32_t)tile_elem<D>(n, 2 * ks + hf) * 2 + half_off;
  const int tg = lane >> 4, tr = (lane >> 2) & 3, tq = lane & 3;
  uint32_t voff[2][DT];
#pragma unroll
  for (int cc = 0; cc < 2; ++cc)
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const int row = 8 * cc + 4 * (tg >> 1) + tr;
      voff[cc][dt] =
          (uint32_t)(tile_elem<D>(row, 4 * dt + 2 * (tg & 1) + (tq >> 1)) + 4 * (tq & 1)) * 2 + half_off;
    }

  // Prologue.  Tile 0 is copied in while Q is fetched; the Q fragments are
  // then consumed by an empty asm statement, which makes the compiler wait for
  // its Q loads here, before the loop (and with them for tile 0, issued
  // earlier).  Left to itself it would put that wait at the first use inside
  // the loop, where it would drain every in-flight copy on each iteration.
  // Only then are tiles 1 .. ST-2 put in flight.  Stage s holds K at byte
  // offset s*SB and V at s*SB + TBK.
  if (L > 0) copy_kv(0, (int)(colp[0] & 0x7fffffffu));

  // Q rows as the B operand: N-tile nt, lane holds row 32*nt + n, d = 16*ks + 8*hf + 0..7
  bf16x8 qf[QK8 ? 1 : NT][QK8 ? 1 : KS];
  // fp8: lane holds row 32*nt + n, dims 64*ks8 + 32*hf + 0..31 as E4M3 of
  // Q * s_q with the row's own power-of-two scale s_q; cr is the row's
  // factor from the MFMA scores to log2 units, scale*log2(e) / (s_q s_k)
  i32x8 q8[NT][QK8 ? KS8 : 1];
  float cr[NT];
  const float dv = PV8 ? a.f8_scale[2 * ((size_t)b * a.Hkv + g) + 1] : 1.f;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const __bf16* qrow =
        a.q + (((size_t)b * a.Hq + head) * a.S_q + min(qrow0 + 32 * nt, a.S_q - 1)) * D;
    if constexpr (QK8) {
      bf16x8 x[KS8][4];
      float amax = 0.f;
#pragma unroll
      for (int ks = 0; ks < KS8; ++ks)
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          x[ks][u] = *(const bf16x8*)(qrow + 64 * ks + 32 * hf + 8 * u);
#pragma unroll
          for (int e = 0; e < 8; ++e) amax = fmaxf(amax, fabsf((float)x[ks][u][e]));
        }
      const float sq = e4m3_scale(other_half_max(amax));
#pragma unroll
      for (int ks = 0; ks < KS8; ++ks)
#pragma unroll
        for (int w = 0; w < 8; ++w) {
          const bf16x8& xv = x[ks][w >> 1];
          const int e = 4 * (w & 1);
          q8[nt][ks][w] = pack_e4m3((float)xv[e] * sq, (float)xv[e + 1] * sq, (float)xv[e + 2] * sq,
                                    (float)xv[e + 3] * sq);
        }
      cr[nt] = a.c / sq * a.f8_scale[2 * ((size_t)b * a.Hkv + g)];
    } else {
      cr[nt] = a.c;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) qf[nt][ks] = *(const bf16x8*)(qrow + 8 * hf + 16 * ks);
    }
  }
  // The live list is kept in two VGPRs (entries 64j .. 64j+127, one per
  // lane) and entries are extracted with v_readlane.  Scalar loads inside the
  // loop would make every LDS wait an lgkmcnt(0) wait for them.
  const uint32_t* colv = a.col + beg;
  auto load_win = [&](int base) -> uint32_t {
    return base + lane < L ? colv[base + lane] : 0u;
  };
  int wbase = 0;
  uint32_t win0 = load_win(0), win1 = load_win(64);
  auto entry = [&](int k) -> uint32_t {  // k in [wbase, wbase + 128)
    const int off = k - wbase;
    return (uint32_t)__builtin_amdgcn_readlane((int)(off < 64 ? win0 : win1), off & 63);
  };
  if constexpr (!QK8) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) asm volatile("" ::"v"(qf[nt][ks]));
  }
  asm volatile("" ::"v"(win0), "v"(win1));
  wait_vm<0>();

#pragma unroll
  for (int s = 1; s < ST - 1; ++s)
    if (s < L) copy_kv(s, (int)(colp[s] & 0x7fffffffu));

  f32x16 o[NT][DT];
  float m[NT], l[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
#pragma unroll
    for (int t = 0; t < DT; ++t) o[nt][t] = f32x16{};
    m[nt] = -INFINITY;
    l[nt] = 0.f;
  }

  const char* lds_bytes = (const char*)smem;
  auto ld_k = [&](int S, int sg, int ks) -> bf16x8 {
    return *(const bf16x8*)(lds_bytes + S * SB + sg * 32 * D * 2 + koff[ks]);
  };
  auto ld_v = [&](int S, int sg, int t, int dt) -> bf16x8 {
    const char* base = lds_bytes + S * SB + TBK + (32 * sg + 16 * t) * D * 2;
    const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(base + voff[0][dt]));
    const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(base + voff[1][dt]));
    return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
  };
  // fp8 operand reads (layouts of Fp8Buffers): K fragment (sg, ks8) = row
  // 32*sg + n, logical chunks 4*ks8 + 2*hf + {0, 1}; V fragment dt = row
  // 32*dt + n of the transposed tile, logical chunks 2*hf + {0, 1}
  uint32_t koff8[QK8 ? KS8 : 1][2], voff8[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
#pragma unroll
    for (int ks = 0; ks < (QK8 ? KS8 : 1); ++ks)
      koff8[ks][u] = (uint32_t)(n * D + 16 * ((4 * ks + 2 * hf + u) ^ kswz8<D>(n)));
    voff8[u] = (uint32_t)(n * kBlk + 16 * ((2 * hf + u) ^ ((n >> 2) & 3)));
  }
  auto ld_k8 = [&](int S, int sg, int ks) -> i32x8 {
    const char* base = lds_bytes + S * SB + sg * 32 * D;
    return lds_pair(base + koff8[ks][0], base + koff8[ks][1]);
  };
  auto ld_v8 = [&](int S, int dt) -> i32x8 {
    const char* base = lds_bytes + S * SB + TBK + dt * 32 * kBlk;
    return lds_pair(base + voff8[0], base + voff8[1]);
  };

  // tile 0 has landed (waited for with Q); make it visible to every wave
  if (L > 0) __syncthreads();

  // One iteration for tile i.  S = i % ST is a compile-time constant (the
  // loop is unrolled ST times), so every LDS offset folds into an
  // instruction immediate.
  auto step = [&](int i, auto stage) {
    constexpr int S = decltype(stage)::value;
    // slide the list window when entry i + ST - 1 would leave it (once per
    // 64 tiles; the load is waited for at once)
    if (i + ST - 1 >= wbase + 128) {
      wbase += 64;
      win0 = win1;
      win1 = load_win(wbase + 64);
      asm volatile("" ::"v"(win1));
    }
    const uint32_t cw = entry(i);
    const int kb = (int)(cw & 0x7fffffffu);
    const bool partial = (cw >> 31) != 0;
    // refill the stage tile i-1 used (free since the barrier that ended it)
    const bool refill = i + ST - 1 < L;
    if (refill) {
      constexpr int SN = (S + ST - 1) % ST;
      copy_kv(SN, (int)(entry(i + ST - 1) & 0x7fffffffu));
    }

    // S^T = K Q^T; K fragments read one step ahead of their MFMAs
    f32x16 sc[NT][NSG];
    if constexpr (QK8) {
#pragma unroll
      for (int sg = 0; sg < NSG; ++sg)
#pragma unroll
        for (int ks = 0; ks < KS8; ++ks) {
          const i32x8 kf = ld_k8(S, sg, ks);
#pragma unroll
          for (int nt = 0; nt < NT; ++nt)
            sc[nt][sg] = mfma_e4m3(kf, q8[nt][ks], ks == 0 ? f32x16{} : sc[nt][sg]);
        }
    } else {
      bf16x8 kf[2][NSG];
#pragma unroll
      for (int sg = 0; sg < NSG; ++sg) kf[0][sg] = ld_k(S, sg, 0);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const int cb = ks & 1;
        if (ks + 1 < KS) {
#pragma unroll
          for (int sg = 0; sg < NSG; ++sg) kf[cb ^ 1][sg] = ld_k(S, sg, ks + 1);
        }
#pragma unroll
        for (int sg = 0; sg < NSG; ++sg)
#pragma unroll
          for (int nt = 0; nt < NT; ++nt) {
            if (ks == 0) sc[nt][sg] = f32x16{};
            sc[nt][sg] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[cb][sg], qf[nt][ks], sc[nt][sg], 0, 0, 0);
          }
      }
    }

    if (partial) {
      // Element mask from coordinates (Section IV-A case iii): key j of the
      // tile is visible to row i iff j <= i + delta (causal) and j < S_k.
      // One threshold per row; each element is kept or set to -inf with an
      // arithmetic select (no per-element condition registers).
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const int lim_abs = min(a.causal ? qrow0 + 32 * nt + a.delta : INT_MAX - kBlk, a.S_k - 1);
        const int lim = lim_abs - (kb * kBlk + 4 * hf + 32 * kh);
#pragma unroll
        for (int sg = 0; sg < NSG; ++sg)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int off = 32 * sg + 8 * (r >> 2) + (r & 3);
            const unsigned dead = (unsigned)((lim - off) >> 31);  // all ones if off > lim
            sc[nt][sg][r] = __uint_as_float((dead & 0xff800000u) |
                                            (~dead & __float_as_uint(sc[nt][sg][r])));
          }
      }
    }

    float mt[NT];
    bool grow = false;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      float mx = -INFINITY;
#pragma unroll
      for (int sg = 0; sg < NSG; ++sg)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sc[nt][sg][r]);
      mx = other_half_max(mx);
      mt[nt] = mx == -INFINITY ? -INFINITY : mx * cr[nt];
      grow |= mt[nt] > m[nt] + TAU;
    }
    // Rescale only when some row's maximum grew by more than TAU (log2
    // units): P = 2^(S - m) then stays below 2^TAU, and m cancels in O / l.
    if (__builtin_amdgcn_ballot_w64(grow)) {
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const float mnew = fmaxf(m[nt], mt[nt]);
        const float alpha = mnew == -INFINITY ? 1.f : __builtin_amdgcn_exp2f(m[nt] - mnew);
        l[nt] *= alpha;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) o[nt][dt] *= alpha;
        m[nt] = mnew;
      }
    }
    float msafe[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) msafe[nt] = m[nt] == -INFINITY ? 0.f : m[nt];

    if constexpr (PV8) {
      // P = 2^(S - m + 8) in (0, 2^8] (m is the exact running maximum):
      // rounded to E4M3 for the product, summed before rounding into l; the
      // lane's 32 weights in the operand's byte order b = 16*sg + r
      i32x8 p8[NT];
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const float mo = 8.f - msafe[nt];
        float pv[32];
#pragma unroll
        for (int sg = 0; sg < NSG; ++sg)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            pv[16 * sg + r] = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[nt][sg][r], cr[nt], mo));
#pragma unroll
        for (int j = 0; j < 32; ++j) l[nt] += pv[j];
#pragma unroll
        for (int w = 0; w < 8; ++w) p8[nt][w] = pack_e4m3(pv[4 * w], pv[4 * w + 1], pv[4 * w + 2], pv[4 * w + 3]);
      }
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const i32x8 vf = ld_v8(S, dt);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) o[nt][dt] = mfma_e4m3(vf, p8[nt], o[nt][dt]);
      }
    } else {

    // P.V in 2*NSG phases, one per 16-key chunk k = (sg, t): phase k runs the
    // MFMAs of chunk k while the exponentials of chunk k+1 are computed and
    // the V fragments of chunk k+1 are read.  The row sums add the
    // bf16-rounded P that the MFMAs consume (v_dot2 against (1, 1)), so
    // O / l weights the value rows exactly as used.
    const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
    auto exps = [&](int k, bf16x8* p) {
      const int sg = k >> 1, t = k & 1;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
#pragma unroll
        for (int e = 0; e < 8; ++e)
          p[nt][e] = (__bf16)__builtin_amdgcn_exp2f(__builtin_fmaf(sc[nt][sg][8 * t + e], a.c, -msafe[nt]));
#pragma unroll
        for (int e = 0; e < 8; e += 2)
          l[nt] = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{p[nt][e], p[nt][e + 1]}, ones, l[nt], false);
      }
    };
    bf16x8 vf[2][DT], pa[2][NT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) vf[0][dt] = ld_v(S, 0, 0, dt);
    exps(0, pa[0]);
    constexpr int NCH = 2 * NSG;
#pragma unroll
    for (int k = 0; k < NCH; ++k) {
      const int cur = k & 1, nx = cur ^ 1;
      if (k + 1 < NCH) {
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) vf[nx][dt] = ld_v(S, (k + 1) >> 1, (k + 1) & 1, dt);
        exps(k + 1, pa[nx]);
      }
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
          o[nt][dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[cur][dt], pa[cur][nt], o[nt][dt], 0, 0, 0);
    }
    }

    // tile i+1 must have landed before the barrier: newer copies (tiles
    // i+2 .. i+ST-1, the wave's CPT_LO or CPT_HI instructions each) may stay
    // in flight
    if (i + 1 < L) {
      if (i + ST - 1 < L) {
        if (CPT_LO == CPT_HI || wave < CW8) wait_vm<(ST - 2) * CPT_LO>();
        else wait_vm<(ST - 2) * CPT_HI>();
      } else {
        wait_vm<0>();
      }
    }
    __syncthreads();  // tile i's stage may be refilled from here on
  };

  int i = 0;
  for (; i + ST <= L; i += ST) {
#pragma unroll
    for (int u = 0; u < ST; ++u) {
      if (u == 0) step(i, Par<0>{});
      if (u == 1) step(i + 1, Par<(1 % ST)>{});
      if (u == 2 && ST > 2) step(i + 2, Par<(2 % ST)>{});
      if (u == 3 && ST > 3) step(i + 3, Par<(3 % ST)>{});
    }
  }
  // the last L % ST tiles (i is a multiple of ST here)
  if constexpr (ST == 2) {
    if (i < L) step(i, Par<0>{});
  } else {
    for (int u = 0; i < L; ++i, ++u) {
      if (u == 0) step(i, Par<0>{});
      else if (u == 1) step(i, Par<(1 % ST)>{});
      else if (u == 2) step(i, Par<(2 % ST)>{});
    }
  }

  if constexpr (KH == 2) {
    merge_halves<D>(a, o[0], m[0], l[0], kh, wave & 1, lane, (float*)smem, b, head, qrow0, hf);
    return;
  }
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int qrow = qrow0 + 32 * nt;
    const float lt = half_pair_sum(l[nt]);
    // fp8: the value scale s_v is divided out here (dv = 1/s_v)
    const float inv = lt > 0.f ? dv / lt : 0.f;
    // log sum_j exp(scale s_ij) = (m + log2 l) ln 2: m in log2 units, l the
    // row sum relative to 2^m (Algorithm 1's statistics; the fp8 weights
    // carry an extra 2^8)
    constexpr float m_off = PV8 ? 8.f : 0.f;
    if (a.lse != nullptr && hf == 0 && qrow < a.S_q)
      a.lse[((size_t)b * a.Hq + head) * a.S_q + qrow] =
          lt > 0.f ? (m[nt] - m_off + log2f(lt)) * 0.69314718055994531f : -INFINITY;
    if (qrow < a.S_q) {
      const size_t at = (((size_t)b * a.Hq + head) * a.S_q + qrow) * D + 4 * hf;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int gq = 0; gq < 4; ++gq) {
          f32x4 w = {o[nt][dt][4 * gq] * inv, o[nt][dt][4 * gq + 1] * inv,
                     o[nt][dt][4 * gq + 2] * inv, o[nt][dt][4 * gq + 3] * inv};
          if (a.out_bf16) {
            const bf16x4 wb = {(__bf16)w[0], (__bf16)w[1], (__bf16)w[2], (__bf16)w[3]};
            *(bf16x4*)((__bf16*)a.out + at + 32 * dt + 8 * gq) = wb;
          } else {
            *(f32x4*)(a.out + at + 32 * dt + 8 * gq) = w;
          }
        }
    }
  }
}

template <int D, int PACK, int PREC>
static void launch_one(const AttnArgs& a, int grid, hipStream_t s) {
  if (grid <= 0) return;
  // the bucket-dealt single-head list: grid is already 8 x (largest bucket)
  const int g = PACK == 1 && a.bucket != nullptr ? grid : xcd_grid(grid);
  // E4M3 tiles are padded with zero keys: with both tensors in E4M3 no copy
  // clamps.  The whole-tile D = 64 kernels keep the ragged copy for every
  // S_k: without it they need fewer registers, a third wave fits on each
  // SIMD, and the two-wave single-head kernel ran 4.6% slower that way on
  // the 24-head S = 32768 workload.  The key-split single-head D = 64 kernel
  // has its own register budget.
  constexpr bool kRaggedAlways = D == 64 && !(PACK == 1 && PREC == kBf16);
  if constexpr (PREC == kFp8All)
    hipLaunchKernelGGL((k_attn<D, PACK, false, PREC>), dim3(g),
                       dim3(attn_threads<D, PACK, PREC, false>()), 0, s, a);
  else if (kRaggedAlways || a.S_k % kBlk != 0)
    hipLaunchKernelGGL((k_attn<D, PACK, true, PREC>), dim3(g),
                       dim3(attn_threads<D, PACK, PREC, true>()), 0, s, a);
  else
    hipLaunchKernelGGL((k_attn<D, PACK, false, PREC>), dim3(g),
                       dim3(attn_threads<D, PACK, PREC, false>()), 0, s, a);
}

template <int D, int PREC>
static hipError_t launch_d(const Problem& p, AttnArgs a, const IndexBuffers& w, hipStream_t s) {
  if (p.pack > 1) {
    AttnArgs ap = a;
    ap.order = w.order_p;
    ap.n_items = w.n_items + kPackItems;  // 0 when k_bucket handed them to the single-head list
    if (p.pack == 2) {
      launch_one<D, 2, PREC>(ap, p.NP, s);
    } else if (D == 128 && (size_t)p.S_q * D * 4 < (1ull << 31)) {
      const hipError_t e = launch_attention_ws(ap, PREC, s);
      if (e != hipSuccess) return e;
    } else {
      launch_one<D, 4, PREC>(ap, p.NP, s);
    }
  }
  if (p.pack > 1 && p.heads_share_mask) return hipGetLastError();  // no single-head item
  a.order = w.order_s;
  a.n_items = w.n_items;
  a.bucket = w.bucket;
  int grid = p.R;
  if (w.bucket != nullptr) {
    // at most the rows of the key/value heads of one bucket: nQB * G rows per
    // head, ceil(B*Hkv / 8) heads per bucket
    const long long per = (long long)p.nQB * p.G * ((p.B * p.Hkv + kBuckets - 1) / kBuckets);
    grid = (int)(kBuckets * per);
  }
  launch_one<D, 1, PREC>(a, grid, s);
  return hipGetLastError();
}

hipError_t launch_attention(const Problem& p, const void* q, const void* k, const void* v,
                            float* out, float* lse, float scale, const IndexBuffers& w,
                            const Fp8Buffers& f, hipStream_t s) {
  AttnArgs a;
  a.q = (const __bf16*)q;
  a.k = (const __bf16*)k;
  a.v = (const __bf16*)v;
  a.out = out;
  a.lse = lse;
  a.out_bf16 = p.out_bf16;
  a.row_ptr = w.row_ptr;
  a.col = w.col;
  a.order = nullptr;
  a.n_items = nullptr;
  a.header = w.n_items + kPlanAt;
  a.bucket = nullptr;
  a.k8 = p.fp8 ? f.k8 : nullptr;
  a.v8 = p.fp8 ? f.v8 : nullptr;
  a.f8_scale = p.fp8 ? f.scale : nullptr;
  a.nKB = p.nKB;
  a.B = p.B;
  a.R = p.R;
  a.pack = p.pack;
  a.Hq = p.Hq;
  a.Hkv = p.Hkv;
  a.S_q = p.S_q;
  a.S_k = p.S_k;
  a.nQB = p.nQB;
  a.G = p.G;
  a.causal = p.causal;
  a.delta = p.delta;
  a.c = scale * 1.4426950408889634f;
  if (p.fp8 == kFp8All) return p.D == 64 ? launch_d<64, kFp8All>(p, a, w, s) : launch_d<128, kFp8All>(p, a, w, s);
  if (p.fp8 == kFp8Pv) return p.D == 64 ? launch_d<64, kFp8Pv>(p, a, w, s) : launch_d<128, kFp8Pv>(p, a, w, s);
  return p.D == 64 ? launch_d<64, kBf16>(p, a, w, s) : launch_d<128, kBf16>(p, a, w, s);
}

}  // namespace steel
