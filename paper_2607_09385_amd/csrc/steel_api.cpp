// C ABI of libsteel: argument checks, workspace, launches.
//
// Every check runs before the first HIP call, so an invalid call enqueues
// nothing and writes no output.  The fused calls keep the live-block index in
// a scratch buffer owned by the calling stream (one per device and stream,
// kept for the life of the process): calls on one stream reuse it in stream
// order, calls on different streams never share it, so a call only enqueues
// and calls on different streams overlap.  The two-phase plan/run form takes
// caller-owned workspace instead, and steel_attn_fwd_noalloc a fixed
// per-device array (noalloc.hip) that no call allocates.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <memory>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/steel.h"
#include "internal.h"

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(STEEL_ERR_HIP, "HIP error in %s: %s (%d)", what, hipGetErrorString(e), (int)e);
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

constexpr int kMaxDevices = 64;

// Scratch of the fused calls (the live-block index; the means and scores of
// the mask producer): one buffer per (device, stream), kept for the life of
// the process and grown when a call needs more.  Work on one stream runs in
// issue order, so a stream's buffer is reused without any wait; buffers of
// different streams are distinct, so calls on different streams never wait
// for each other.  A slot's lock is held from scratch_begin to scratch_end,
// so two host threads enqueueing on the same stream do not interleave their
// kernels over one buffer.  Each use records an event that the next use of
// the slot waits for on its stream: that keeps the order if a stream is
// destroyed and a new one gets the same handle.  A (stream-ordered) pool
// allocation per call was not used: it made every call wait on the host for
// the previous one's release.
struct StreamScratch {
  hipStream_t stream = nullptr;
  std::mutex mu;
  char* ptr = nullptr;
  size_t bytes = 0;
  hipEvent_t done = nullptr;  // completion of the last call that used ptr
  bool recorded = false;
};
struct DeviceScratch {
  std::mutex mu;  // guards the list (slots are never removed)
  std::vector<std::unique_ptr<StreamScratch>> slots;
};
DeviceScratch g_scratch[kMaxDevices];

StreamScratch* stream_slot(int dev, hipStream_t s) {
  DeviceScratch& d = g_scratch[dev];
  std::lock_guard<std::mutex> g(d.mu);
  for (auto& sl : d.slots)
    if (sl->stream == s) return sl.get();
  d.slots.emplace_back(new StreamScratch);
  d.slots.back()->stream = s;
  return d.slots.back().get();
}

// Selects dev for the calls in its scope and restores the caller's device.
struct DeviceScope {
  int prev = -1;
  hipError_t err = hipSuccess;
  explicit DeviceScope(int dev) {
    err = hipGetDevice(&prev);
    if (err == hipSuccess && prev != dev) err = hipSetDevice(dev);
  }
  ~DeviceScope() {
    if (prev >= 0) (void)hipSetDevice(prev);
  }
};

int scratch_begin(int dev, hipStream_t s, size_t need, std::unique_lock<std::mutex>* lk,
                  StreamScratch** slot, char** out) {
  StreamScratch& d = *stream_slot(dev, s);
  *lk = std::unique_lock<std::mutex>(d.mu);
  *slot = &d;
  DeviceScope scope(dev);
  if (scope.err != hipSuccess) return hip_fail(scope.err, "selecting the stream's device");
  hipError_t e = hipSuccess;
  if (!d.done && (e = hipEventCreateWithFlags(&d.done, hipEventDisableTiming)) != hipSuccess)
    return hip_fail(e, "creating the scratch event");
  if (need > d.bytes) {
    if (d.ptr) {
      // only this stream's earlier calls can still read the old buffer
      if (d.recorded && (e = hipEventSynchronize(d.done)) != hipSuccess)
        return hip_fail(e, "waiting for the previous user of the scratch buffer");
      if ((e = hipFree(d.ptr)) != hipSuccess) return hip_fail(e, "releasing the scratch buffer");
      d.ptr = nullptr;
      d.bytes = 0;
      d.recorded = false;
    }
    const size_t grow = (need + need / 4 + ((size_t)1 << 20) - 1) & ~(((size_t)1 << 20) - 1);
    if ((e = hipMalloc(reinterpret_cast<void**>(&d.ptr), grow)) != hipSuccess) {
      d.ptr = nullptr;
      return hip_fail(e, "allocating the scratch buffer");
    }
    d.bytes = grow;
  }
  if (d.recorded && (e = hipStreamWaitEvent(s, d.done, 0)) != hipSuccess)
    return hip_fail(e, "ordering after the previous user of the scratch buffer");
  *out = d.ptr;
  return STEEL_OK;
}

// After the call's work is enqueued on s (slot lock still held).
int scratch_end(StreamScratch* slot, int dev, hipStream_t s) {
  DeviceScope scope(dev);
  if (scope.err != hipSuccess) return hip_fail(scope.err, "selecting the stream's device");
  hipError_t e = hipEventRecord(slot->done, s);
  if (e != hipSuccess) {
    slot->recorded = false;
    return hip_fail(e, "recording the scratch buffer's use");
  }
  slot->recorded = true;
  return STEEL_OK;
}

// Shape checks shared by both entry points; fills the Problem on success.
int check_shape(int B, int Hq, int Hkv, int S_q, int S_k, int blk, int causal,
                steel::Problem* p) {
  if (B < 1 || Hq < 1 || Hkv < 1 || S_q < 1 || S_k < 1)
    return fail(STEEL_ERR_INVALID_ARGUMENT,
                "sizes must be >= 1 (B=%d Hq=%d Hkv=%d S_q=%d S_k=%d)", B, Hq, Hkv, S_q, S_k);
  if (Hq % Hkv != 0)
    return fail(STEEL_ERR_INVALID_ARGUMENT, "Hq (%d) must be a multiple of Hkv (%d)", Hq, Hkv);
  if (causal != 0 && causal != 1)
    return fail(STEEL_ERR_INVALID_ARGUMENT, "causal must be 0 or 1 (got %d)", causal);
  if (blk != steel::kBlk)
    return fail(STEEL_ERR_UNSUPPORTED, "blk=%d not supported (only %d)", blk, steel::kBlk);
  const long long nQB = (S_q + (long long)blk - 1) / blk;
  const long long nKB = (S_k + (long long)blk - 1) / blk;
  const long long R = (long long)B * Hq * nQB;
  if (R > INT32_MAX / 2 || R * nKB >= (1ll << 31))
    return fail(STEEL_ERR_UNSUPPORTED,
                "block grid too large: %lld rows x %lld key blocks exceeds 2^31 list entries", R,
                nKB);
  p->B = B;
  p->Hq = Hq;
  p->Hkv = Hkv;
  p->S_q = S_q;
  p->S_k = S_k;
  p->G = Hq / Hkv;
  p->nQB = (int)nQB;
  p->nKB = (int)nKB;
  p->causal = causal;
  p->delta = S_k - S_q;
  p->R = (int)R;
  p->pack = 1;
  p->NP = 0;
  return STEEL_OK;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

struct Layout {
  size_t cnt, hist_s, hist_p, row_ptr, col, order_s, order_p, n_items, bucket, total;
  bool has_bucket;  // the single-head list is also dealt into XCD buckets
  size_t k8, v8, f8_part, f8_scale;  // fp8 operands (when Problem::fp8)
};

Layout layout(const steel::Problem& p, bool with_rowptr_col_order) {
  Layout L{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t at = off;
    off += align256(bytes);
    return at;
  };
  const size_t nch_s = steel::nchunks(p.R);
  const size_t nch_p = p.pack > 1 ? steel::nchunks(p.NP) : 0;
  L.cnt = take(sizeof(int32_t) * p.R);
  L.hist_s = take(sizeof(int32_t) * steel::kBins * nch_s);
  L.hist_p = take(sizeof(int32_t) * (nch_p ? steel::kBins * nch_p : 1));
  L.n_items = take(sizeof(int32_t) * steel::kHeaderInts);
  L.order_p = take(sizeof(int32_t) * (p.NP > 0 ? p.NP : 1));
  if (with_rowptr_col_order) {
    L.row_ptr = take(sizeof(int32_t) * (p.R + 1));
    L.col = take(sizeof(uint32_t) * (size_t)p.R * p.nKB);
    L.order_s = take(sizeof(int32_t) * p.R);
    L.bucket = take(sizeof(int32_t) * ((size_t)p.R + steel::kBuckets + 1));
    L.has_bucket = true;
  }
  if (p.fp8) {
    const size_t tiles = (size_t)p.B * p.Hkv * p.nKB * steel::kBlk * p.D;  // bytes per tensor
    L.k8 = p.fp8 == steel::kFp8All ? take(tiles) : 0;
    L.v8 = take(tiles);
    L.f8_part = take(sizeof(float) * 2 * steel::kFp8Chunks * p.B * p.Hkv);
    L.f8_scale = take(sizeof(float) * 2 * p.B * p.Hkv);
  }
  L.total = off;
  return L;
}

int stream_device(hipStream_t s, int* dev) {
  hipError_t e = s ? hipStreamGetDevice(s, dev) : hipGetDevice(dev);
  if (e != hipSuccess) return hip_fail(e, "querying the stream's device");
  if (*dev < 0 || *dev >= kMaxDevices) return fail(STEEL_ERR_HIP, "device %d out of range", *dev);
  return STEEL_OK;
}

// Argument checks of the fused pass (everything but the workspace).
int check_attn(const void* q, const void* k, const void* v, const void* out, int B, int Hq,
               int Hkv, int S_q, int S_k, int D, int blk, float scale, int causal,
               steel::Problem* p) {
  if (!q || !k || !v || !out)
    return fail(STEEL_ERR_INVALID_ARGUMENT, "q, k, v and out must be non-NULL device pointers");
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out))
    return fail(STEEL_ERR_INVALID_ARGUMENT, "q, k, v and out must be 16-byte aligned");
  if (!std::isfinite(scale) || !(scale > 0.f))
    return fail(STEEL_ERR_INVALID_ARGUMENT, "scale must be finite and > 0 (got %g)", (double)scale);
  int rc = check_shape(B, Hq, Hkv, S_q, S_k, blk, causal, p);
  if (rc != STEEL_OK) return rc;
  if (D != 64 && D != 128) return fail(STEEL_ERR_UNSUPPORTED, "D=%d not supported (64 or 128)", D);
  p->D = D;
  return STEEL_OK;
}

// Head packing: query heads of one key/value group that share a live list run
// in one workgroup (up to 4).
void set_pack(steel::Problem* p) {
  p->pack = (p->G % 4 == 0) ? 4 : (p->G % 2 == 0) ? 2 : 1;
  p->NP = p->pack > 1 ? p->R / p->pack : 0;
}

// Structured mask (window of window_blocks blocks ending at the block
// diagonal, plus the first sink_blocks key blocks) in place of a mask tensor.
int set_window(steel::Problem* p, int window_blocks, int sink_blocks) {
  if (window_blocks < 1)
    return fail(STEEL_ERR_INVALID_ARGUMENT, "window_blocks must be >= 1 (got %d)", window_blocks);
  if (sink_blocks < 0)
    return fail(STEEL_ERR_INVALID_ARGUMENT, "sink_blocks must be >= 0 (got %d)", sink_blocks);
  p->win_blocks = window_blocks;
  p->sink_blocks = sink_blocks;
  return STEEL_OK;
}

steel::IndexBuffers carve(char* ws, const Layout& L) {
  steel::IndexBuffers w{};
  w.cnt = reinterpret_cast<int32_t*>(ws + L.cnt);
  w.hist_s = reinterpret_cast<int32_t*>(ws + L.hist_s);
  w.hist_p = reinterpret_cast<int32_t*>(ws + L.hist_p);
  w.n_items = reinterpret_cast<int32_t*>(ws + L.n_items);
  w.order_p = reinterpret_cast<int32_t*>(ws + L.order_p);
  w.row_ptr = reinterpret_cast<int32_t*>(ws + L.row_ptr);
  w.col = reinterpret_cast<uint32_t*>(ws + L.col);
  w.order_s = reinterpret_cast<int32_t*>(ws + L.order_s);
  w.bucket = L.has_bucket ? reinterpret_cast<int32_t*>(ws + L.bucket) : nullptr;
  return w;
}

int check_workspace(const void* ws, size_t bytes, const Layout& L) {
  if (!ws) return fail(STEEL_ERR_INVALID_ARGUMENT, "workspace must be a non-NULL device pointer");
  if ((reinterpret_cast<uintptr_t>(ws) & 255u) != 0)
    return fail(STEEL_ERR_INVALID_ARGUMENT, "workspace must be 256-byte aligned");
  if (bytes < L.total)
    return fail(STEEL_ERR_INVALID_ARGUMENT, "workspace of %zu bytes is smaller than the %zu needed",
                bytes, L.total);
  return STEEL_OK;
}

// The fused call once the arguments are checked: the device's scratch buffer,
// index build, attention.
int fused_call(const steel::Problem& p, const void* q, const void* k, const void* v,
               const uint8_t* block_mask, void* out, float* lse, float scale, void* stream) {
  int rc;
  hipStream_t s = static_cast<hipStream_t>(stream);
  int dev = 0;
  if ((rc = stream_device(s, &dev)) != STEEL_OK) return rc;
  const Layout L = layout(p, true);
  std::unique_lock<std::mutex> lk;
  StreamScratch* slot = nullptr;
  char* ws = nullptr;
  if ((rc = scratch_begin(dev, s, L.total, &lk, &slot, &ws)) != STEEL_OK) return rc;
  const steel::IndexBuffers w = carve(ws, L);
  steel::Fp8Buffers f{};
  if (p.fp8) {
    f.k8 = p.fp8 == steel::kFp8All ? reinterpret_cast<uint8_t*>(ws + L.k8) : nullptr;
    f.v8 = reinterpret_cast<uint8_t*>(ws + L.v8);
    f.part = reinterpret_cast<float*>(ws + L.f8_part);
    f.scale = reinterpret_cast<float*>(ws + L.f8_scale);
  }
  hipError_t e = steel::launch_block_index(p, block_mask, w, s);
  if (e == hipSuccess && p.fp8) e = steel::launch_fp8_prepass(p, k, v, f, s);
  if (e == hipSuccess)
    e = steel::launch_attention(p, q, k, v, static_cast<float*>(out), lse, scale, w, f, s);
  const int re = scratch_end(slot, dev, s);
  if (e != hipSuccess) return hip_fail(e, "launching kernels");
  return re;
}

}  // namespace

extern "C" {

const char* steel_version(void) { return "libsteel 0.1.0 (gfx950)"; }

const char* steel_last_error(void) { return g_err.c_str(); }

int steel_attn_fwd(const void* q, const void* k, const void* v, const uint8_t* block_mask,
                   void* out, int B, int Hq, int Hkv, int S_q, int S_k, int D, int blk,
                   float scale, int causal, void* stream) {
  g_err.clear();
  steel::Problem p{};
  int rc = check_attn(q, k, v, out, B, Hq, Hkv, S_q, S_k, D, blk, scale, causal, &p);
  if (rc != STEEL_OK) return rc;
  set_pack(&p);
  p.heads_share_mask = block_mask == nullptr;
  return fused_call(p, q, k, v, block_mask, out, nullptr, scale, stream);
}

int steel_attn_fwd_window(const void* q, const void* k, const void* v, void* out, int B, int Hq,
                          int Hkv, int S_q, int S_k, int D, int blk, float scale, int causal,
                          int window_blocks, int sink_blocks, void* stream) {
  g_err.clear();
  steel::Problem p{};
  int rc = check_attn(q, k, v, out, B, Hq, Hkv, S_q, S_k, D, blk, scale, causal, &p);
  if (rc != STEEL_OK) return rc;
  if ((rc = set_window(&p, window_blocks, sink_blocks)) != STEEL_OK) return rc;
  set_pack(&p);
  p.heads_share_mask = 1;
  return fused_call(p, q, k, v, nullptr, out, nullptr, scale, stream);
}

int steel_attn_fwd_ex(const void* q, const void* k, const void* v, const uint8_t* block_mask,
                      void* out, float* lse, int B, int Hq, int Hkv, int S_q, int S_k, int D,
                      int blk, float scale, int causal, int causal_offset, int flags,
                      void* stream) {
  g_err.clear();
  steel::Problem p{};
  int rc = check_attn(q, k, v, out, B, Hq, Hkv, S_q, S_k, D, blk, scale, causal, &p);
  if (rc != STEEL_OK) return rc;
  if (causal) {
    if (causal_offset < -(1 << 30) || causal_offset > (1 << 30))
      return fail(STEEL_ERR_INVALID_ARGUMENT, "causal_offset %d outside [-2^30, 2^30]", causal_offset);
    p.delta = causal_offset;
  }
  if (flags & ~(STEEL_OUT_BF16 | STEEL_FP8 | STEEL_FP8_PV))
    return fail(STEEL_ERR_INVALID_ARGUMENT,
                "flags may hold only STEEL_OUT_BF16, STEEL_FP8 and STEEL_FP8_PV (got %d)", flags);
  p.out_bf16 = (flags & STEEL_OUT_BF16) != 0;
  p.fp8 = (flags & STEEL_FP8) ? steel::kFp8All : (flags & STEEL_FP8_PV) ? steel::kFp8Pv : steel::kBf16;
  set_pack(&p);
  p.heads_share_mask = block_mask == nullptr;
  return fused_call(p, q, k, v, block_mask, out, lse, scale, stream);
}

int steel_attn_fwd_noalloc(const void* q, const void* k, const void* v,
                           const uint8_t* block_mask, void* out, int B, int Hq, int Hkv, int S_q,
                           int S_k, int D, int blk, float scale, int causal, void* stream) {
  g_err.clear();
  steel::Problem p{};
  int rc = check_attn(q, k, v, out, B, Hq, Hkv, S_q, S_k, D, blk, scale, causal, &p);
  if (rc != STEEL_OK) return rc;
  set_pack(&p);
  p.heads_share_mask = block_mask == nullptr;
  const Layout L = layout(p, true);
  if (L.total > steel::kNoAllocBytes)
    return fail(STEEL_ERR_UNSUPPORTED,
                "the index of this problem needs %zu bytes of scratch; steel_attn_fwd_noalloc "
                "holds %zu (use steel_attn_fwd or plan/run)",
                L.total, steel::kNoAllocBytes);
  hipStream_t s = static_cast<hipStream_t>(stream);
  int dev = 0;
  if ((rc = stream_device(s, &dev)) != STEEL_OK) return rc;
  char* ws = nullptr;
  hipError_t e = steel::noalloc_scratch(dev, &ws);
  if (e != hipSuccess) return hip_fail(e, "looking up the fixed scratch array");
  const steel::IndexBuffers w = carve(ws, L);
  e = steel::launch_block_index(p, block_mask, w, s);
  if (e == hipSuccess)
    e = steel::launch_attention(p, q, k, v, static_cast<float*>(out), nullptr, scale, w,
                                steel::Fp8Buffers{}, s);
  if (e != hipSuccess) return hip_fail(e, "launching kernels");
  return STEEL_OK;
}

int steel_attn_merge(const float* o_parts, const float* lse_parts, int n_parts, long long rows,
                     int D, float* out, float* lse_out, void* stream) {
  g_err.clear();
  if (!o_parts || !lse_parts || !out)
    return fail(STEEL_ERR_INVALID_ARGUMENT, "o_parts, lse_parts and out must be non-NULL");
  if (!aligned16(o_parts) || !aligned16(out))
    return fail(STEEL_ERR_INVALID_ARGUMENT, "o_parts and out must be 16-byte aligned");
  if (n_parts < 1 || rows < 1)
    return fail(STEEL_ERR_INVALID_ARGUMENT, "n_parts (%d) and rows (%lld) must be >= 1", n_parts,
                rows);
  if (D < 4 || D % 4 != 0)
    return fail(STEEL_ERR_INVALID_ARGUMENT, "D=%d must be a positive multiple of 4", D);
  if (rows * (D / 4) >= (1ll << 40))
    return fail(STEEL_ERR_UNSUPPORTED, "%lld rows of %d values is too large", rows, D);
  hipError_t e = steel::launch_merge(o_parts, lse_parts, n_parts, rows, D, out, lse_out,
                                     static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "launching the merge");
  return STEEL_OK;
}

size_t steel_attn_workspace_bytes(int B, int Hq, int Hkv, int S_q, int S_k, int blk) {
  g_err.clear();
  steel::Problem p{};
  if (check_shape(B, Hq, Hkv, S_q, S_k, blk, 0, &p) != STEEL_OK) return 0;
  set_pack(&p);
  return layout(p, true).total;
}

int steel_attn_plan(const uint8_t* block_mask, int B, int Hq, int Hkv, int S_q, int S_k,
                    int blk, int causal, void* workspace, size_t workspace_bytes, void* stream) {
  g_err.clear();
  steel::Problem p{};
  int rc = check_shape(B, Hq, Hkv, S_q, S_k, blk, causal, &p);
  if (rc != STEEL_OK) return rc;
  set_pack(&p);
  const Layout L = layout(p, true);
  if ((rc = check_workspace(workspace, workspace_bytes, L)) != STEEL_OK) return rc;
  hipError_t e = steel::launch_block_index(p, block_mask, carve(static_cast<char*>(workspace), L),
                                           static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "launching the index build");
  return STEEL_OK;
}

int steel_attn_plan_window(int B, int Hq, int Hkv, int S_q, int S_k, int blk, int causal,
                           int window_blocks, int sink_blocks, void* workspace,
                           size_t workspace_bytes, void* stream) {
  g_err.clear();
  steel::Problem p{};
  int rc = check_shape(B, Hq, Hkv, S_q, S_k, blk, causal, &p);
  if (rc != STEEL_OK) return rc;
  if ((rc = set_window(&p, window_blocks, sink_blocks)) != STEEL_OK) return rc;
  set_pack(&p);
  const Layout L = layout(p, true);
  if ((rc = check_workspace(workspace, workspace_bytes, L)) != STEEL_OK) return rc;
  hipError_t e = steel::launch_block_index(p, nullptr, carve(static_cast<char*>(workspace), L),
                                           static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "launching the index build");
  return STEEL_OK;
}

int steel_attn_run(const void* q, const void* k, const void* v, void* out, int B, int Hq,
                   int Hkv, int S_q, int S_k, int D, int blk, float scale, int causal,
                   const void* workspace, size_t workspace_bytes, void* stream) {
  g_err.clear();
  steel::Problem p{};
  int rc = check_attn(q, k, v, out, B, Hq, Hkv, S_q, S_k, D, blk, scale, causal, &p);
  if (rc != STEEL_OK) return rc;
  set_pack(&p);
  const Layout L = layout(p, true);
  if ((rc = check_workspace(workspace, workspace_bytes, L)) != STEEL_OK) return rc;
  hipError_t e = steel::launch_attention(
      p, q, k, v, static_cast<float*>(out), nullptr, scale,
      carve(const_cast<char*>(static_cast<const char*>(workspace)), L), steel::Fp8Buffers{},
      static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "launching the attention kernels");
  return STEEL_OK;
}

int steel_topk_block_mask(const void* q, const void* k, int B, int Hq, int Hkv, int S_q, int S_k,
                          int D, int blk, int causal, int keep_num, int keep_den,
                          uint8_t* block_mask, void* stream) {
  g_err.clear();
  if (!q || !k || !block_mask)
    return fail(STEEL_ERR_INVALID_ARGUMENT, "q, k and block_mask must be non-NULL device pointers");
  if (!aligned16(q) || !aligned16(k))
    return fail(STEEL_ERR_INVALID_ARGUMENT, "q and k must be 16-byte aligned");
  if (keep_num < 1 || keep_den < 1 || keep_num > keep_den)
    return fail(STEEL_ERR_INVALID_ARGUMENT,
                "keep fraction %d/%d must satisfy 1 <= keep_num <= keep_den", keep_num, keep_den);
  steel::Problem p{};
  int rc = check_shape(B, Hq, Hkv, S_q, S_k, blk, causal, &p);
  if (rc != STEEL_OK) return rc;
  if (D != 64 && D != 128) return fail(STEEL_ERR_UNSUPPORTED, "D=%d not supported (64 or 128)", D);
  p.D = D;
  if (p.nKB > 4096)
    return fail(STEEL_ERR_UNSUPPORTED, "%d key blocks: the selection ranks at most 4096", p.nKB);
  hipStream_t s = static_cast<hipStream_t>(stream);
  int dev = 0;
  if ((rc = stream_device(s, &dev)) != STEEL_OK) return rc;
  const size_t n_qm = (size_t)B * Hq * p.nQB * D, n_km = (size_t)B * Hkv * p.nKB * D;
  const size_t n_sc = (size_t)B * Hq * p.nQB * p.nKB;
  const size_t o_km = align256(n_qm * sizeof(double)), o_sc = o_km + align256(n_km * sizeof(double));
  const size_t total = o_sc + align256(n_sc * sizeof(double));
  std::unique_lock<std::mutex> lk;
  StreamScratch* slot = nullptr;
  char* ws = nullptr;
  if ((rc = scratch_begin(dev, s, total, &lk, &slot, &ws)) != STEEL_OK) return rc;
  hipError_t e = steel::launch_topk_mask(
      p, static_cast<const __bf16*>(q), static_cast<const __bf16*>(k), keep_num, keep_den,
      block_mask, reinterpret_cast<double*>(ws), reinterpret_cast<double*>(ws + o_km),
      reinterpret_cast<double*>(ws + o_sc), s);
  const int re = scratch_end(slot, dev, s);
  if (e != hipSuccess) return hip_fail(e, "launching kernels");
  return re;
}

int steel_block_index(const uint8_t* block_mask, int B, int Hq, int S_q, int S_k, int blk,
                      int causal, int32_t* row_ptr, uint32_t* col, int32_t* order, void* stream) {
  g_err.clear();
  if (!row_ptr || !col || !order)
    return fail(STEEL_ERR_INVALID_ARGUMENT, "row_ptr, col and order must be non-NULL");
  steel::Problem p{};
  int rc = check_shape(B, Hq, Hq, S_q, S_k, blk, causal, &p);
  if (rc != STEEL_OK) return rc;
  p.D = 0;

  hipStream_t s = static_cast<hipStream_t>(stream);
  int dev = 0;
  if ((rc = stream_device(s, &dev)) != STEEL_OK) return rc;
  const Layout L = layout(p, false);
  std::unique_lock<std::mutex> lk;
  StreamScratch* slot = nullptr;
  char* ws = nullptr;
  if ((rc = scratch_begin(dev, s, L.total, &lk, &slot, &ws)) != STEEL_OK) return rc;
  steel::IndexBuffers w{};
  w.cnt = reinterpret_cast<int32_t*>(ws + L.cnt);
  w.hist_s = reinterpret_cast<int32_t*>(ws + L.hist_s);
  w.hist_p = reinterpret_cast<int32_t*>(ws + L.hist_p);
  w.n_items = reinterpret_cast<int32_t*>(ws + L.n_items);
  w.order_p = reinterpret_cast<int32_t*>(ws + L.order_p);
  w.row_ptr = row_ptr;
  w.col = col;
  w.order_s = order;
  hipError_t e = steel::launch_block_index(p, block_mask, w, s);
  const int re = scratch_end(slot, dev, s);
  if (e != hipSuccess) return hip_fail(e, "launching kernels");
  return re;
}

}  // extern "C"
