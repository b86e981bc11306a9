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
// (2 waves, 64 rows) or a pack of PACK query heads of one key/value group
// that share the same live list (2*PACK waves), so each K/V tile is loaded
// once for up to 256 query rows.
#include "internal.h"

namespace steel {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
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
  const int32_t* row_ptr;
  const uint32_t* col;
  const int32_t* order;
  const int32_t* n_items;   // this list's item count
  const int32_t* header;    // plan header (after the two counts)
  int Hq, Hkv, S_q, S_k, nQB, nKB, G, causal, delta, R, pack;
  float c;  // scale * log2(e)
};

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

template <int D, int PACK>
__global__ __launch_bounds__(128 * PACK) void k_attn(AttnArgs a) {
  constexpr int NT = 128 * PACK;   // threads
  constexpr int ST = D + 8;        // LDS row stride (bf16): 16-byte pad
  constexpr int KS = D / 16;       // k-steps of S^T = K Q^T
  constexpr int DT = D / 32;       // d tiles of O^T
  constexpr int CH = kBlk * D / 8; // 16-byte chunks per tile
  __shared__ __attribute__((aligned(16))) __bf16 sK[kBlk * ST];
  __shared__ __attribute__((aligned(16))) __bf16 sV[kBlk * ST];

  const int32_t* hd = a.header;
  if (hd[0] != kPlanMagic || hd[1] != a.R || hd[2] != a.nKB || hd[3] != a.pack ||
      hd[4] != a.causal || hd[5] != a.delta)
    return;  // index was planned for another problem: leave out untouched
  if ((int)blockIdx.x >= a.n_items[0]) return;
  const int item = a.order[blockIdx.x];
  const int qb = item % a.nQB;
  const int bh0 = (item / a.nQB) * PACK;  // b*Hq + first head
  const int b = bh0 / a.Hq;
  const int h0 = bh0 % a.Hq;
  const int g = h0 / a.G;

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int head = h0 + (wave >> 1);
  const int n = lane & 31, hf = lane >> 5;
  const int qrow = qb * kBlk + (wave & 1) * 32 + n;

  // Q rows as the B operand: lane holds row n, d = 16*ks + 8*hf + 0..7
  bf16x8 qf[KS];
  {
    const __bf16* qp = a.q + (((size_t)b * a.Hq + head) * a.S_q + qrow) * D + 8 * hf;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      if (qrow < a.S_q) qf[ks] = *(const bf16x8*)(qp + 16 * ks);
      else qf[ks] = bf16x8{};
    }
  }

  f32x16 o[DT];
#pragma unroll
  for (int t = 0; t < DT; ++t) o[t] = f32x16{};
  float m = -INFINITY, l = 0.f;

  const int r0 = bh0 * a.nQB + qb;
  const int beg = a.row_ptr[r0], end = a.row_ptr[r0 + 1];
  const size_t kvoff = ((size_t)b * a.Hkv + g) * a.S_k * D;
  const __bf16* kg = a.k + kvoff;
  const __bf16* vg = a.v + kvoff;

  // lane constants of the transposed V read (16-lane groups)
  const int tg = lane >> 4, tr = (lane >> 2) & 3, tq = lane & 3;
  const int v_lane_off = (4 * (tg >> 1) + tr) * ST + 16 * (tg & 1) + 4 * tq;
  const int k_lane_off = n * ST + 8 * hf;

  for (int it = beg; it < end; ++it) {
    const uint32_t cw = a.col[it];
    const int kb = (int)(cw & 0x7fffffffu);
    const bool partial = (cw >> 31) != 0;

    __syncthreads();  // previous tile fully consumed
#pragma unroll
    for (int c = tid; c < CH; c += NT) {
      const int row = c / (D / 8), c8 = c % (D / 8);
      const int key = kb * kBlk + row;
      u32x4 kk = u32x4{0, 0, 0, 0}, vv = u32x4{0, 0, 0, 0};
      if (key < a.S_k) {
        kk = *(const u32x4*)(kg + (size_t)key * D + c8 * 8);
        vv = *(const u32x4*)(vg + (size_t)key * D + c8 * 8);
      }
      *(u32x4*)(sK + row * ST + c8 * 8) = kk;
      *(u32x4*)(sV + row * ST + c8 * 8) = vv;
    }
    __syncthreads();

    // S^T = K Q^T for two 32-key sub-tiles
    f32x16 s[2];
#pragma unroll
    for (int sg = 0; sg < 2; ++sg) {
      s[sg] = f32x16{};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x8 ka = *(const bf16x8*)(sK + k_lane_off + sg * 32 * ST + 16 * ks);
        s[sg] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qf[ks], s[sg], 0, 0, 0);
      }
    }

    if (partial) {
#pragma unroll
      for (int sg = 0; sg < 2; ++sg)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = kb * kBlk + 32 * sg + 8 * (r >> 2) + 4 * hf + (r & 3);
          const bool vis = key < a.S_k && (!a.causal || key <= qrow + a.delta);
          if (!vis) s[sg][r] = -INFINITY;
        }
    }

    float mx = -INFINITY;
#pragma unroll
    for (int sg = 0; sg < 2; ++sg)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[sg][r]);
    mx = other_half_max(mx);
    const float mt = mx == -INFINITY ? -INFINITY : mx * a.c;
    const float mnew = fmaxf(m, mt);
    const float msafe = mnew == -INFINITY ? 0.f : mnew;
    const float alpha = __builtin_amdgcn_exp2f(m - msafe);

    float rs = 0.f;
    bf16x8 pb[2][2];
#pragma unroll
    for (int sg = 0; sg < 2; ++sg)
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float pv = __builtin_amdgcn_exp2f(__builtin_fmaf(s[sg][8 * t + e], a.c, -msafe));
          rs += pv;
          pb[sg][t][e] = (__bf16)pv;
        }
    l = alpha * l + rs;
    m = mnew;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) o[dt] *= alpha;

    // O^T += V^T P^T
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int sg = 0; sg < 2; ++sg)
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          const __bf16* base = sV + v_lane_off + (32 * sg + 16 * t) * ST + 32 * dt;
          const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(base));
          const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(base + 8 * ST));
          const s16x8 both = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
          o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, both),
                                                          pb[sg][t], o[dt], 0, 0, 0);
        }
  }

  const float lt = half_pair_sum(l);
  const float inv = lt > 0.f ? 1.f / lt : 0.f;
  if (qrow < a.S_q) {
    float* op = a.out + (((size_t)b * a.Hq + head) * a.S_q + qrow) * D + 4 * hf;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int gq = 0; gq < 4; ++gq) {
        f32x4 w = {o[dt][4 * gq] * inv, o[dt][4 * gq + 1] * inv, o[dt][4 * gq + 2] * inv,
                   o[dt][4 * gq + 3] * inv};
        *(f32x4*)(op + 32 * dt + 8 * gq) = w;
      }
  }
}

template <int D, int PACK>
static void launch_one(const AttnArgs& a, int grid, hipStream_t s) {
  if (grid > 0) hipLaunchKernelGGL((k_attn<D, PACK>), dim3(grid), dim3(128 * PACK), 0, s, a);
}

template <int D>
static void launch_d(const Problem& p, AttnArgs a, const IndexBuffers& w, hipStream_t s) {
  if (p.pack > 1) {
    AttnArgs ap = a;
    ap.order = w.order_p;
    ap.n_items = w.n_items + 1;
    if (p.pack == 2) launch_one<D, 2>(ap, p.NP, s);
    else launch_one<D, 4>(ap, p.NP, s);
  }
  a.order = w.order_s;
  a.n_items = w.n_items;
  launch_one<D, 1>(a, p.R, s);
}

hipError_t launch_attention(const Problem& p, const void* q, const void* k, const void* v,
                            float* out, float scale, const IndexBuffers& w, hipStream_t s) {
  AttnArgs a;
  a.q = (const __bf16*)q;
  a.k = (const __bf16*)k;
  a.v = (const __bf16*)v;
  a.out = out;
  a.row_ptr = w.row_ptr;
  a.col = w.col;
  a.order = nullptr;
  a.n_items = nullptr;
  a.header = w.n_items + 2;
  a.nKB = p.nKB;
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
  if (p.D == 64) launch_d<64>(p, a, w, s);
  else launch_d<128>(p, a, w, s);
  return hipGetLastError();
}

}  // namespace steel
