/*
 * libsteel -- sparsity-aware fused attention forward for AMD Instinct MI355X
 * (gfx950).  C ABI: plain pointers and sizes, no C++ or framework types.
 *
 * What it computes (Section II-A, Eq. 1 of the STEEL paper, with the masking
 * of Section IV-A):  for every batch b and query head h, with key/value head
 * g = h / (Hq / Hkv),
 *
 *     O[b,h,i,:] = sum_j softmax_j( scale * Q[b,h,i,:] . K[b,g,j,:] + M[b,h,i,j] ) V[b,g,j,:]
 *
 * where M is 0 where element (i, j) is visible and -inf elsewhere.  (i, j) is
 * visible iff its 64x64 block (i/64, j/64) is live in ``block_mask`` and, when
 * ``causal`` is nonzero, j <= i + (S_k - S_q) (bottom-right aligned causal
 * structure; plain lower-triangular when S_q == S_k).  A query row with no
 * visible key has output 0.
 *
 * The pass is fused (Section II-A; Algorithm 1): scores, the running row
 * maximum and row sum, and the rescaled accumulation of P.V stay on chip; only
 * Q, K, V, the mask and O touch device memory.  Key blocks that are dead
 * (mask byte 0, or entirely above the causal diagonal) are never loaded;
 * partially masked blocks get the element mask from their coordinates;
 * unmasked blocks run without it (the three tile cases of Section IV-A).
 *
 * All calls are asynchronous on the given HIP stream (a hipStream_t passed as
 * ``void*``; NULL means the default stream) and return once the work is
 * enqueued.  Argument checks run before any HIP call; on a non-OK status
 * nothing has been enqueued and no output has been written.  Kernel faults
 * surface at the caller's next synchronisation, as usual for HIP.
 *
 * Thread safety: calls may be made concurrently from several threads and on
 * several streams.  The fused calls keep their index in a scratch buffer
 * that belongs to the calling stream (one per device and stream, allocated on
 * the stream's first call, grown when a call needs more, kept until the
 * process ends): calls on one stream reuse it in stream order, and calls on
 * different streams use different buffers, so they never wait for each
 * other.  Two threads enqueueing on the same stream take turns while they
 * enqueue (a short host lock per stream).  Besides these buffers the only
 * process-wide state is the thread-local error text and the fixed array of
 * steel_attn_fwd_noalloc.
 */
#ifndef STEEL_H
#define STEEL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum steel_status {
  STEEL_OK = 0,
  STEEL_ERR_INVALID_ARGUMENT = 1, /* bad pointer, shape, alignment or scale    */
  STEEL_ERR_UNSUPPORTED = 2,      /* valid but not built: D not 64/128, blk != 64 */
  STEEL_ERR_HIP = 3               /* HIP runtime error; see steel_last_error()  */
} steel_status;

/*
 * Fused attention forward (Section II-A Eq. 1; Algorithm 1; Section IV-A).
 *
 *   q          bf16 [B][Hq][S_q][D], device memory, row-major, 16-byte aligned
 *   k, v       bf16 [B][Hkv][S_k][D], device memory, row-major, 16-byte aligned
 *   block_mask uint8 [B][Hq][ceil(S_q/blk)][ceil(S_k/blk)], device memory,
 *              nonzero = live block; NULL = every block live
 *   out        fp32 [B][Hq][S_q][D], device memory, 16-byte aligned; every
 *              element is written
 *   B, Hq, Hkv, S_q, S_k >= 1;  Hq % Hkv == 0
 *   D          head dimension: 64 or 128 (others: STEEL_ERR_UNSUPPORTED)
 *   blk        block edge of the mask: 64 (others: STEEL_ERR_UNSUPPORTED)
 *   scale      multiplies Q.K^T; finite and > 0 (1/sqrt(D) in the paper)
 *   causal     0 or 1
 *   stream     hipStream_t as void*, or NULL
 *
 * Inputs and output are owned by the caller; the library keeps no pointer to
 * them after it returns.  Internal workspace (the compressed live-block list
 * and the work order) lives in the calling stream's scratch buffer, which the
 * library allocates on the stream's first call and grows (hipMalloc,
 * synchronous; the stream's earlier calls are waited for) when a call needs
 * more than it holds; it is kept until the process ends.  Results are
 * bitwise reproducible run to run.
 */
int steel_attn_fwd(const void* q, const void* k, const void* v,
                   const uint8_t* block_mask, void* out,
                   int B, int Hq, int Hkv, int S_q, int S_k, int D, int blk,
                   float scale, int causal, void* stream);

/*
 * Live-block index (Section IV-A tile classes, as a compressed list; Section
 * IV-C balance, as a work order).  Rows are r = (b*Hq + h)*nQB + qb with
 * nQB = ceil(S_q/blk), nKB = ceil(S_k/blk).
 *
 *   A block (qb, kb) is dead if its mask byte is 0, or if causal and
 *   kb*blk > min((qb+1)*blk, S_q) - 1 + (S_k - S_q).  A live block is partial
 *   if causal and (kb+1)*blk - 1 > qb*blk + (S_k - S_q), or if
 *   (kb+1)*blk > S_k.
 *
 *   row_ptr  int32 [R+1], device: exclusive prefix sum of the live counts
 *   col      uint32 [capacity], device: for row r, entries
 *            row_ptr[r] .. row_ptr[r+1]-1 hold the live kb in increasing
 *            order, bit 31 set for a partial block.  Capacity must be at
 *            least R*nKB (the live total is only known on the device).
 *   order    int32 [R], device: the rows sorted by the bin of their live
 *            count, heaviest first, equal bins in increasing row order.  The
 *            bin of a count c is c itself when c < 128; above, with
 *            e = floor(log2 c), it is 128 + 16*(e - 7) + ((c >> (e - 4)) & 15)
 *            (16 bins per octave, all bins below 512).
 *
 * The arguments shared with steel_attn_fwd mean the same and are checked the
 * same way; D and the tensors are not needed here.
 */
int steel_block_index(const uint8_t* block_mask, int B, int Hq, int S_q, int S_k,
                      int blk, int causal, int32_t* row_ptr, uint32_t* col,
                      int32_t* order, void* stream);

/*
 * Two-phase form of steel_attn_fwd for callers that reuse one mask over many
 * calls (for example every layer of a model): steel_attn_plan builds the
 * live-block index once into caller-owned device workspace, steel_attn_run
 * runs the fused pass over it.  plan + run computes exactly what
 * steel_attn_fwd computes.
 *
 *   steel_attn_workspace_bytes  size of the workspace for these sizes, or 0
 *                               after an argument error (see
 *                               steel_last_error())
 *   workspace                   device memory, 256-byte aligned, at least
 *                               that many bytes, owned by the caller; run
 *                               only reads it, so several runs may share one
 *                               plan concurrently
 *
 * run must be given the same B, Hq, Hkv, S_q, S_k, blk and causal as the plan:
 * the plan writes a header with every one of them (and the head packing and
 * causal limit derived from them) into the workspace, the attention kernels
 * compare it with their own arguments, and on any mismatch they return
 * without writing out (the call itself still returns STEEL_OK: the header is
 * only readable on the device).  run must be ordered after the plan on the
 * device (same stream, or an event).  Arguments mean what they mean for
 * steel_attn_fwd.
 */
size_t steel_attn_workspace_bytes(int B, int Hq, int Hkv, int S_q, int S_k, int blk);

int steel_attn_plan(const uint8_t* block_mask, int B, int Hq, int Hkv, int S_q, int S_k,
                    int blk, int causal, void* workspace, size_t workspace_bytes, void* stream);

int steel_attn_run(const void* q, const void* k, const void* v, void* out,
                   int B, int Hq, int Hkv, int S_q, int S_k, int D, int blk,
                   float scale, int causal, const void* workspace, size_t workspace_bytes,
                   void* stream);

/*
 * steel_attn_fwd with two additions for work split over key chunks
 * (chunked prefill, keys held on several devices):
 *
 *   lse            float [B][Hq][S_q] device buffer, or NULL: receives each
 *                  query row's log sum_j exp(scale * q_i . k_j) over its
 *                  visible keys (natural log; -inf when no key is visible).
 *                  It is the row statistic Algorithm 1 carries (running
 *                  maximum m and sum l: lse = m + log l).
 *   causal_offset  when causal, key j is visible to query i iff
 *                  j <= i + causal_offset (steel_attn_fwd uses S_k - S_q);
 *                  a chunk [k0, k1) of a sequence of S_k_total keys is passed
 *                  as its own K, V with causal_offset = S_k_total - S_q - k0.
 *                  Ignored when causal == 0; otherwise within [-2^30, 2^30].
 *   flags          0 or an OR of:
 *     STEEL_OUT_BF16  out is bf16, each value the round-to-nearest-even of
 *                     the fp32 result (half the output bytes); without it
 *                     out is fp32 [B][Hq][S_q][D] as for steel_attn_fwd.
 *     STEEL_FP8_PV    the fp8 form for P V only: the scores come from bf16
 *                     Q and K as without flags; V and the softmax weights
 *                     are rounded to E4M3 as described under STEEL_FP8.
 *     STEEL_FP8       the fp8 form: both products of Algorithm 1 take E4M3
 *                     operands (OCP 8-bit float: 4 exponent bits, 3 mantissa
 *                     bits, largest value 448) instead of the bf16 operands
 *                     of the paper's datapath (Section II-C), accumulating in
 *                     fp32 as before.  Q is rounded per query row after a
 *                     power-of-two scale that maps the row's largest |value|
 *                     into (224, 448]; K and V likewise with one scale each
 *                     per (batch, key/value head), found by a pre-pass over
 *                     K and V; the softmax weights 2^(s - m + 8) (m the exact
 *                     running row maximum, so the weights lie in (0, 256])
 *                     are rounded for P V, while the row sum adds them
 *                     unrounded.  Scales are divided out exactly.  The
 *                     result follows the same recurrence with larger
 *                     rounding: its error against exact attention is the
 *                     form's own budget, measured per workload in the
 *                     library's design notes, not the bf16 tolerance.  The
 *                     E4M3 copies of K and V (B*Hkv*ceil(S_k/64)*64*D bytes
 *                     each) live in the calling stream's scratch buffer.
 *                     Scores of large magnitude (sharply peaked attention)
 *                     lose the most: their absolute error grows with |s|,
 *                     and STEEL_FP8_PV keeps them at bf16 precision.
 *                     STEEL_FP8 together with STEEL_FP8_PV is STEEL_FP8.
 *
 * Other flag bits: STEEL_ERR_INVALID_ARGUMENT.  Everything else as
 * steel_attn_fwd; with lse == NULL, causal_offset = S_k - S_q and flags == 0
 * the output is bitwise that of steel_attn_fwd.
 */
#define STEEL_OUT_BF16 1
#define STEEL_FP8 2
#define STEEL_FP8_PV 4
int steel_attn_fwd_ex(const void* q, const void* k, const void* v,
                      const uint8_t* block_mask, void* out, float* lse,
                      int B, int Hq, int Hkv, int S_q, int S_k, int D, int blk,
                      float scale, int causal, int causal_offset, int flags,
                      void* stream);

/*
 * Merge of partial results over disjoint key sets: with n_parts outputs O_c
 * and row log-sum-exps lse_c (from steel_attn_fwd_ex over each key chunk),
 *   out = sum_c exp(lse_c - L) O_c / sum_c exp(lse_c - L),   L = max_c lse_c
 *   lse_out = L + log sum_c exp(lse_c - L)
 * per row; rows with every lse_c = -inf get out = 0 and lse_out = -inf.
 *
 *   o_parts    float [n_parts][rows][D] device, 16-byte aligned
 *   lse_parts  float [n_parts][rows] device
 *   rows       rows per part (B*Hq*S_q for attention outputs), >= 1
 *   D          positive multiple of 4
 *   out        float [rows][D] device, 16-byte aligned (may not alias a part)
 *   lse_out    float [rows] device, or NULL
 *
 * Invalid arguments: STEEL_ERR_INVALID_ARGUMENT before any HIP call.  The
 * call only enqueues; it allocates nothing.
 */
int steel_attn_merge(const float* o_parts, const float* lse_parts, int n_parts, long long rows,
                     int D, float* out, float* lse_out, void* stream);

/*
 * Structured-mask forms: the block mask is generated from block coordinates
 * instead of read from a tensor (the paper builds masks on the core rather
 * than fetching them, Section III-B, and names windowed attention among the
 * masking schemes its coordinate tracking covers, Section IV-A).  Block
 * (qb, kb) is in the mask iff
 *     qb - window_blocks < kb <= qb      (window ending at the block diagonal)
 *  or kb < sink_blocks                   (sink blocks at the start)
 * and the causal structure is then applied exactly as for a mask tensor.  The
 * result equals steel_attn_fwd / steel_attn_plan given that mask as a
 * [B][Hq][nQB][nKB] tensor; no mask is read.  Every query head shares the
 * pattern, so head packs always run together.
 *
 *   window_blocks  >= 1 (STEEL_ERR_INVALID_ARGUMENT otherwise)
 *   sink_blocks    >= 0
 *
 * All other arguments, the workspace (same size as for steel_attn_plan),
 * ownership and error behaviour are those of steel_attn_fwd and
 * steel_attn_plan; a window plan is run with steel_attn_run.
 */
int steel_attn_fwd_window(const void* q, const void* k, const void* v, void* out,
                          int B, int Hq, int Hkv, int S_q, int S_k, int D, int blk,
                          float scale, int causal, int window_blocks, int sink_blocks,
                          void* stream);

int steel_attn_plan_window(int B, int Hq, int Hkv, int S_q, int S_k, int blk, int causal,
                           int window_blocks, int sink_blocks, void* workspace,
                           size_t workspace_bytes, void* stream);

/*
 * Block-mask producer run ahead of the pass: top-k key blocks per query block
 * by mean-pooled score, plus the diagonal block.  (The paper generates masks
 * on the compute core rather than fetching them, Section III-B, and any block
 * mask then goes through the tile classes of Section IV-A.)  For every
 * (b, query head h, query block qb), with g = h / (Hq/Hkv):
 *   mean_q(qb)  float64 mean of the block's rows of Q[b][h] (a ragged last
 *               block averages the rows it has); mean_k(kb) likewise of
 *               K[b][g]
 *   score(kb)   dot(mean_q(qb), mean_k(kb)) in float64
 *   candidates  kb < min(qb + 1, nKB) when causal, kb < nKB otherwise
 *   kept        the ceil(keep_num / keep_den * #candidates) candidates with
 *               the largest scores (equal scores: the smaller kb first), and
 *               kb = qb when qb < nKB
 * block_mask[b][h][qb][kb] = 1 for kept blocks and 0 for all others (every
 * byte of the [B][Hq][nQB][nKB] mask is written).  The float64 operation
 * order is fixed (rows summed in increasing order, mean = sum / row count,
 * products summed in increasing d without fused multiply-add), so the mask is
 * reproducible bit for bit.
 *
 *   q, k        bf16 device tensors laid out as for steel_attn_fwd
 *   D           64 or 128; blk 64; nKB <= 4096 (STEEL_ERR_UNSUPPORTED)
 *   keep_num, keep_den   1 <= keep_num <= keep_den (1 and 10: 10%)
 *   block_mask  uint8 device buffer of B*Hq*nQB*nKB bytes, caller-owned
 *
 * Float64 workspace for the block means and scores lives in the calling
 * stream's scratch buffer (as for steel_attn_fwd); the call only enqueues,
 * unless the buffer must grow.  Errors as for steel_attn_fwd.
 */
int steel_topk_block_mask(const void* q, const void* k, int B, int Hq, int Hkv, int S_q,
                          int S_k, int D, int blk, int causal, int keep_num, int keep_den,
                          uint8_t* block_mask, void* stream);

/*
 * steel_attn_fwd for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same computation, arguments, checks and kernels, bitwise the same
 * output, but the live-block index is built in a fixed array of
 * STEEL_NOALLOC_SCRATCH_BYTES that the library holds on each device it runs on
 * (a file-scope device array, present from the library's load until the
 * process ends).  The call allocates nothing: no hipMalloc, hipFree or
 * allocating library routine.  The first call on a device looks up that
 * device's copy of the array (hipGetSymbolAddress); later calls only enqueue.
 *
 *   Limit: the index of the problem must fit the array.  It needs about
 *   4 * R * (nKB + 4) bytes plus 2 KiB per 256 rows (R = B*Hq*ceil(S_q/64),
 *   nKB = ceil(S_k/64)): 24.3 MiB for 24 heads at S = 32768, 8.2 MiB for
 *   32 heads at S = 16384 (steel_attn_workspace_bytes gives the exact
 *   figure).  A larger problem returns STEEL_ERR_UNSUPPORTED before any HIP
 *   call (use steel_attn_fwd or plan/run).
 *
 *   Every call on one device shares that device's array, which keeps the last
 *   call's index: calls that overlap on one device (concurrent streams, or
 *   threads enqueueing on different streams) race on it and must be ordered
 *   by the caller; calls queued on one stream are ordered by the stream.
 *   Nothing in the array needs to start at zero (each call writes all it
 *   reads).
 */
#define STEEL_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)

int steel_attn_fwd_noalloc(const void* q, const void* k, const void* v,
                           const uint8_t* block_mask, void* out,
                           int B, int Hq, int Hkv, int S_q, int S_k, int D, int blk,
                           float scale, int causal, void* stream);

/* Text of the last non-OK status returned on the calling thread ("" if none). */
const char* steel_last_error(void);

/* Library version string. */
const char* steel_version(void);

#ifdef __cplusplus
}
#endif

#endif /* STEEL_H */
