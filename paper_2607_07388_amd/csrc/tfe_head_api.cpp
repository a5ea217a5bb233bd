// C ABI of the early-exit prefetch head: create / top-K / free.
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdlib.h>

#include <mutex>
#include <new>

#include "../../include/tfe.h"
#include "tfe_head.h"
#include "tfe_internal.h"

struct tfe_head {
  int device = 0;
  int cus = 256;
  const void* w = nullptr;   // caller's [V x D] bf16 projection (not owned)
  uint32_t V = 0, D = 0, max_batch = 0, max_k = 0;
  // Scratch, rows = max_batch rounded up to 64 (the logits kernel writes
  // whole 64-row groups), tiles = V rounded up to 32 (whole 32-token
  // super-tiles), over 16.
  float* d_logits = nullptr;  // [rows x tiles x 16]
  uint64_t* d_tkey = nullptr; // [rows x tiles rounded up to 16]
  float* d_tsum = nullptr;    // [rows x tiles rounded up to 16]
  uint64_t* d_bmax = nullptr; // [rows x compute units]
  // Scratch of the one-launch path (calls of at most 64 rows, also under
  // capture, when the device can launch it): barrier counters, call epoch and fault word,
  // per (row, block) maxima, sums and candidate counts, then the candidate
  // segments (ccap keys per row and block).
  unsigned char* d_fuse = nullptr;
  bool fused = false;
  uint32_t ccap = 0;
  // Recorded after every top-K call made outside graph capture; freeing the
  // head waits for it (and for nothing else on the device).
  hipEvent_t ev_last = nullptr;
  bool recorded = false;
};

namespace tfe {
namespace {

tfe_status hip_fail(hipError_t e, const char* what) {
  return fail(TFE_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

#define HEAD_HIP(call, what)                         \
  do {                                               \
    hipError_t e_ = (call);                          \
    if (e_ != hipSuccess) return hip_fail(e_, what); \
  } while (0)

void forget_fused(const tfe_head* h);

void release(tfe_head* h) {
  if (!h) return;
  int cur = 0;
  (void)hipGetDevice(&cur);
  (void)hipSetDevice(h->device);
  if (h->recorded) (void)hipEventSynchronize(h->ev_last);
  forget_fused(h);
  void* bufs[] = {h->d_logits, h->d_tkey, h->d_tsum, h->d_bmax, h->d_fuse};
  for (void* b : bufs) dev_free(b);
  if (h->ev_last) (void)hipEventDestroy(h->ev_last);
  (void)hipSetDevice(cur);
  delete h;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// One-launch calls of all heads on a device run one after another: a call
// on another stream than the previous one waits on the device for that
// call's event (the head's ev_last, recorded right after each call).  Two of
// them side by side could each hold part of the compute units with blocks
// waiting at a grid barrier for blocks of their own that cannot start.
// Calls on the stream of the previous one are ordered by the stream itself
// and add nothing.  The stream handle is only compared, never used.
constexpr int kOrderDevices = 64;
std::mutex g_fused_mu;
const tfe_head* g_fused_head[kOrderDevices];
hipStream_t g_fused_stream[kOrderDevices];

// A head that is released stops being the previous call's head (release
// has waited for its last call).
void forget_fused(const tfe_head* h) {
  std::lock_guard<std::mutex> lock(g_fused_mu);
  if (h->device >= 0 && h->device < kOrderDevices && g_fused_head[h->device] == h)
    g_fused_head[h->device] = nullptr;
}

// Enqueues launch() on `stream` behind the previous one-launch call on the
// device, then records h->ev_last behind it.
template <class F>
tfe_status fused_in_order(tfe_head* h, hipStream_t stream, F launch) {
  std::lock_guard<std::mutex> lock(g_fused_mu);
  const tfe_head* prev = g_fused_head[h->device];
  if (prev && g_fused_stream[h->device] != stream)
    HEAD_HIP(hipStreamWaitEvent(stream, prev->ev_last, 0), "head ordering wait");
  HEAD_HIP(launch(), "head launch");
  HEAD_HIP(hipEventRecord(h->ev_last, stream), "record");
  h->recorded = true;
  g_fused_head[h->device] = h;
  g_fused_stream[h->device] = stream;
  return TFE_OK;
}

// Layout of the one-launch scratch for nblk blocks: 8 KB of barrier
// counters and flags (one 128-byte line each) and the fault word, two
// [64 x nblk] word arrays, then the candidate segments.
constexpr size_t kFuseCtl = 8192;
size_t fuse_words(uint32_t nblk) { return (size_t)64 * nblk; }
size_t fuse_cand_at(uint32_t nblk) { return (kFuseCtl + 2 * fuse_words(nblk) * 4 + 255) / 256 * 256; }
size_t fuse_bytes(uint32_t nblk, uint32_t ccap) {
  return fuse_cand_at(nblk) + fuse_words(nblk) * ccap * sizeof(uint64_t);
}
void fuse_args(const tfe_head* h, HeadArgs* a) {
  unsigned char* p = h->d_fuse;
  const size_t n = fuse_words((uint32_t)h->cus);
  a->bar = (unsigned long long*)p;
  a->ectl = (unsigned long long*)(p + 4352);  // 16 lines after the barrier's 33
  a->fault = (unsigned long long*)(p + kFuseCtl - 128);
  a->bhi = (uint32_t*)(p + kFuseCtl);
  a->bsum = a->bhi + n;
  a->cand = (uint64_t*)(p + fuse_cand_at((uint32_t)h->cus));
  a->ccap = h->ccap;
}

tfe_status create(const void* w, int32_t vocab, int32_t dim, int32_t max_batch, int32_t max_k,
                  tfe_head** out) {
  if (!out) return fail(TFE_ERR_INVALID_ARG, "null output handle");
  *out = nullptr;
  if (!w) return fail(TFE_ERR_INVALID_ARG, "null projection");
  if (!aligned16(w)) return fail(TFE_ERR_INVALID_ARG, "projection not 16-byte aligned");
  if (vocab < 1 || vocab > (1 << 18)) return fail(TFE_ERR_INVALID_ARG, "vocab outside [1, 2^18]");
  if (!head_dim_supported(dim)) return fail(TFE_ERR_UNSUPPORTED, "dim %d (256, 512 or 1024)", dim);
  if (max_batch < 1 || max_batch > 65535)
    return fail(TFE_ERR_INVALID_ARG, "max_batch outside [1, 65535]");
  if (max_k < 1 || max_k > kHeadMaxK || max_k > vocab)
    return fail(TFE_ERR_INVALID_ARG, "max_k outside [1, min(%d, vocab)]", kHeadMaxK);
  hipPointerAttribute_t attr;
  const hipError_t pe = hipPointerGetAttributes(&attr, w);
  if (pe != hipSuccess || attr.type != hipMemoryTypeDevice) {
    (void)hipGetLastError();
    return fail(TFE_ERR_INVALID_ARG, "projection is not device memory");
  }
  tfe_head* h = alloc_fails() ? nullptr : new (std::nothrow) tfe_head;
  if (!h) return fail(TFE_ERR_OOM, "head");
  tfe_status st = TFE_OK;
  do {
    if (hipGetDevice(&h->device) != hipSuccess) { st = fail(TFE_ERR_HIP, "hipGetDevice"); break; }
    if (attr.device != h->device) {
      st = fail(TFE_ERR_INVALID_ARG, "projection lives on device %d, device %d is current",
                attr.device, h->device);
      break;
    }
    int lds = 0;
    if (hipDeviceGetAttribute(&h->cus, hipDeviceAttributeMultiprocessorCount, h->device) !=
            hipSuccess ||
        hipDeviceGetAttribute(&lds, hipDeviceAttributeMaxSharedMemoryPerBlock, h->device) !=
            hipSuccess) {
      st = fail(TFE_ERR_HIP, "device attributes");
      break;
    }
    if ((uint32_t)lds < head_lds_bytes(dim)) {
      st = fail(TFE_ERR_UNSUPPORTED, "dim %d needs %u bytes of LDS per block, device has %d",
                dim, head_lds_bytes(dim), lds);
      break;
    }
    h->w = w;
    h->V = (uint32_t)vocab;
    h->D = (uint32_t)dim;
    h->max_batch = (uint32_t)max_batch;
    h->max_k = (uint32_t)max_k;
    const size_t nb = ((size_t)h->max_batch + 63) / 64 * 64, nt = (h->V + 31) / 32 * 2;
    const size_t nt16 = (nt + 15) / 16 * 16;
    if (dev_malloc((void**)&h->d_logits, nb * nt * 16 * sizeof(float)) != hipSuccess ||
        dev_malloc((void**)&h->d_tkey, nb * nt16 * sizeof(uint64_t)) != hipSuccess ||
        dev_malloc((void**)&h->d_tsum, nb * nt16 * sizeof(float)) != hipSuccess ||
        dev_malloc((void**)&h->d_bmax, nb * (size_t)h->cus * sizeof(uint64_t)) != hipSuccess) {
      st = fail(TFE_ERR_OOM, "head scratch for %u rows", h->max_batch);
      break;
    }
    // The one-launch path, where one of its blocks fits a compute unit and
    // some call shape fits it.
    HeadArgs probe{};
    probe.V = h->V;
    probe.D = h->D;
    probe.B = 1;
    probe.K = 1;
    probe.nblk = (uint32_t)h->cus;
    if (head_fused_fits(probe) && head_fused_resident(dim)) {
      h->ccap = head_fused_ccap(h->V, (uint32_t)h->cus);
      if (dev_malloc((void**)&h->d_fuse, fuse_bytes((uint32_t)h->cus, h->ccap)) != hipSuccess) {
        st = fail(TFE_ERR_OOM, "head scratch for %u rows", h->max_batch);
        break;
      }
      if (hipMemset(h->d_fuse, 0, kFuseCtl) != hipSuccess) {
        st = fail(TFE_ERR_HIP, "head barrier reset");
        break;
      }
      h->fused = true;
    }
    if (hipEventCreateWithFlags(&h->ev_last, hipEventDisableTiming) != hipSuccess) {
      h->ev_last = nullptr;
      st = fail(TFE_ERR_HIP, "head event");
      break;
    }
  } while (0);
  if (st != TFE_OK) {
    release(h);
    return st;
  }
  *out = h;
  return TFE_OK;
}

tfe_status topk(tfe_head* h, const void* hidden, int32_t B, int32_t K, int32_t* ids, float* prob,
                hipStream_t stream) {
  if (!h) return fail(TFE_ERR_INVALID_ARG, "null head");
  if (B < 0 || (uint32_t)B > h->max_batch)
    return fail(TFE_ERR_INVALID_ARG, "B outside [0, %u]", h->max_batch);
  if (K < 0 || (uint32_t)K > h->max_k) return fail(TFE_ERR_INVALID_ARG, "K outside [0, %u]", h->max_k);
  if (B == 0 || K == 0) return TFE_OK;
  if (!hidden || !ids || !prob) return fail(TFE_ERR_INVALID_ARG, "null hidden, ids or probs");
  if (!aligned16(hidden)) return fail(TFE_ERR_INVALID_ARG, "hidden not 16-byte aligned");
  int cur = -1;
  HEAD_HIP(hipGetDevice(&cur), "hipGetDevice");
  if (cur != h->device)
    return fail(TFE_ERR_INVALID_ARG, "head lives on device %d but device %d is current",
                h->device, cur);
  HeadArgs a{};
  a.w = h->w;
  a.hidden = hidden;
  a.logits = h->d_logits;
  a.tkey = h->d_tkey;
  a.tsum = h->d_tsum;
  a.bmax = h->d_bmax;
  a.top_ids = ids;
  a.top_prob = prob;
  a.V = h->V;
  a.tpitch = (h->V + 31) / 32 * 2;
  a.tblocks = (a.tpitch + 15) / 16;
  a.D = h->D;
  a.B = (uint32_t)B;
  a.K = (uint32_t)K;
  a.nblk = (uint32_t)h->cus;
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  HEAD_HIP(hipStreamIsCapturing(stream, &cs), "hipStreamIsCapturing");
  if (h->fused && head_fused_fits(a) && h->device < kOrderDevices) {
    fuse_args(h, &a);
    a.wait_limit = kHeadWaitLimit;
    if (const char* wl = getenv("TFE_HEAD_WAIT_LIMIT")) a.wait_limit = (uint32_t)strtoul(wl, nullptr, 0);
    // Captured: the graph's edges order the call (the call epoch is kept on
    // the device, so replays stay aligned).
    if (cs != hipStreamCaptureStatusNone) {
      HEAD_HIP(launch_head_fused(a, stream), "head launch");
      return TFE_OK;
    }
    return fused_in_order(h, stream, [&] { return launch_head_fused(a, stream); });
  }
  HEAD_HIP(launch_head_logits(a, stream), "head logits launch");
  HEAD_HIP(launch_head_rows(a, stream), "head top-K launch");
  if (cs == hipStreamCaptureStatusNone) {
    HEAD_HIP(hipEventRecord(h->ev_last, stream), "record");
    h->recorded = true;
  }
  return TFE_OK;
}

tfe_status last_fault(tfe_head* h, int64_t* call) {
  if (!h || !call) return fail(TFE_ERR_INVALID_ARG, "null head or output");
  *call = 0;
  if (!h->fused) return TFE_OK;
  int cur = -1;
  HEAD_HIP(hipGetDevice(&cur), "hipGetDevice");
  if (cur != h->device)
    return fail(TFE_ERR_INVALID_ARG, "head lives on device %d but device %d is current",
                h->device, cur);
  if (h->recorded) HEAD_HIP(hipEventSynchronize(h->ev_last), "head wait");
  // The fault word holds the largest (epoch + 1) of the calls that gave up:
  // the 1-based number of the latest such call.
  unsigned long long f = 0;
  HEAD_HIP(hipMemcpy(&f, h->d_fuse + kFuseCtl - 128, sizeof f, hipMemcpyDeviceToHost),
           "head fault word");
  *call = (int64_t)f;
  return TFE_OK;
}

}  // namespace
}  // namespace tfe

extern "C" {

tfe_status tfe_head_create(const void* w_pref, int32_t vocab, int32_t dim, int32_t max_batch,
                           int32_t max_k, tfe_head** out) {
  tfe::begin_call();
  return tfe::create(w_pref, vocab, dim, max_batch, max_k, out);
}

tfe_status tfe_head_topk(tfe_head* head, const void* hidden, int32_t B, int32_t K,
                         int32_t* top_ids, float* top_prob, void* stream) {
  tfe::begin_call();
  return tfe::topk(head, hidden, B, K, top_ids, top_prob, (hipStream_t)stream);
}

tfe_status tfe_head_last_fault(tfe_head* head, int64_t* call) {
  tfe::begin_call();
  return tfe::last_fault(head, call);
}

tfe_status tfe_head_free(tfe_head* head) {
  tfe::begin_call();
  tfe::release(head);
  return TFE_OK;
}

}  // extern "C"
