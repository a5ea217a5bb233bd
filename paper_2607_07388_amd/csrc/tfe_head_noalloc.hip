// Early-exit head top-K without any allocation, for callers that cannot
// allocate device memory (code under HIP graph capture, serving loops,
// harnesses that forbid hipMalloc).  The two-launch kernels of
// tfe_head_topk (the same ids as its one-launch path, probabilities within
// float32 rounding); their scratch (logits, tile statistics and block maxima
// of one 64-row group, for vocabularies up to 2^18 and up to kNaMaxBlocks
// compute units) is a file-scope device array that each GPU holds until the
// process ends.  (The one-launch path is not used here: its barrier targets
// come from a per-call count kept on the host, which a captured graph would
// replay unchanged.)
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "../../include/tfe.h"
#include "tfe_head.h"
#include "tfe_internal.h"

namespace tfe {
namespace {

constexpr uint32_t kNaRows = 64;              // rows per call: one 64-row group
constexpr uint32_t kNaTiles = kHeadMaxTiles;  // 16-token tiles of a 2^18 vocabulary
constexpr size_t kNaLogitBytes = (size_t)kNaRows * kNaTiles * 16 * sizeof(float);  // 64 MiB
constexpr size_t kNaKeyBytes = (size_t)kNaRows * kNaTiles * sizeof(uint64_t);      // 8 MiB
constexpr size_t kNaSumBytes = (size_t)kNaRows * kNaTiles * sizeof(float);         // 4 MiB
constexpr uint32_t kNaMaxBlocks = 1024;       // logits blocks: one per compute unit
constexpr size_t kNaBmaxBytes = (size_t)kNaRows * kNaMaxBlocks * sizeof(uint64_t); // 512 KiB
constexpr size_t kNaBytes = kNaLogitBytes + kNaKeyBytes + kNaSumBytes + kNaBmaxBytes;
constexpr int kNaMaxDevices = 64;

}  // namespace
}  // namespace tfe

// The scratch.  Host code never uses this name as an address: it is a host
// stand-in; the device address comes from hipGetSymbolAddress, per device.
static __device__ __align__(256) unsigned char scratch[tfe::kNaBytes];

namespace tfe {
namespace {

struct NaDevice {
  bool ready = false;
  unsigned char* ptr = nullptr;  // device address of `scratch` on this device
  int cus = 0;
  int lds = 0;
};
std::mutex g_na_mu;
NaDevice g_na[kNaMaxDevices];

// Set-up on the first call on a device (that device current): the
// scratch's device address and the device limits.
tfe_status na_device(int dev, NaDevice* out) {
  if (dev < 0 || dev >= kNaMaxDevices) return fail(TFE_ERR_UNSUPPORTED, "device %d", dev);
  std::lock_guard<std::mutex> lock(g_na_mu);
  NaDevice& d = g_na[dev];
  if (!d.ready) {
    void* p = nullptr;
    hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e == hipSuccess)
      e = hipDeviceGetAttribute(&d.cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e == hipSuccess)
      e = hipDeviceGetAttribute(&d.lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
    if (e != hipSuccess) {
      (void)hipGetLastError();
      return fail(TFE_ERR_HIP, "no-allocation scratch on device %d: %s", dev,
                  hipGetErrorString(e));
    }
    d.ptr = (unsigned char*)p;
    d.ready = true;
  }
  *out = d;
  return TFE_OK;
}

tfe_status topk_noalloc(const void* w, int32_t vocab, int32_t dim, const void* hidden, int32_t B,
                        int32_t K, int32_t* ids, float* prob, hipStream_t stream) {
  if (!w) return fail(TFE_ERR_INVALID_ARG, "null projection");
  if (((uintptr_t)w & 15u) != 0) return fail(TFE_ERR_INVALID_ARG, "projection not 16-byte aligned");
  if (vocab < 1 || vocab > (1 << 18)) return fail(TFE_ERR_INVALID_ARG, "vocab outside [1, 2^18]");
  if (!head_dim_supported(dim)) return fail(TFE_ERR_UNSUPPORTED, "dim %d (256, 512 or 1024)", dim);
  if (B < 0 || (uint32_t)B > kNaRows)
    return fail(TFE_ERR_INVALID_ARG, "B outside [0, %u] (the no-allocation scratch holds %u rows)",
                kNaRows, kNaRows);
  if (K < 0 || K > kHeadMaxK || K > vocab)
    return fail(TFE_ERR_INVALID_ARG, "K outside [0, min(%d, vocab)]", kHeadMaxK);
  if (B == 0 || K == 0) return TFE_OK;
  if (!hidden || !ids || !prob) return fail(TFE_ERR_INVALID_ARG, "null hidden, ids or probs");
  if (((uintptr_t)hidden & 15u) != 0) return fail(TFE_ERR_INVALID_ARG, "hidden not 16-byte aligned");
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(TFE_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  hipPointerAttribute_t attr;
  e = hipPointerGetAttributes(&attr, w);
  if (e != hipSuccess || attr.type != hipMemoryTypeDevice) {
    (void)hipGetLastError();
    return fail(TFE_ERR_INVALID_ARG, "projection is not device memory");
  }
  if (attr.device != dev)
    return fail(TFE_ERR_INVALID_ARG, "projection lives on device %d, device %d is current",
                attr.device, dev);
  NaDevice d;
  tfe_status st = na_device(dev, &d);
  if (st != TFE_OK) return st;
  if (d.cus < 1 || (uint32_t)d.cus > kNaMaxBlocks)
    return fail(TFE_ERR_UNSUPPORTED, "%d compute units (the no-allocation scratch holds %u)",
                d.cus, kNaMaxBlocks);
  if ((uint32_t)d.lds < head_lds_bytes(dim))
    return fail(TFE_ERR_UNSUPPORTED, "dim %d needs %u bytes of LDS per block, device has %d", dim,
                head_lds_bytes(dim), d.lds);
  HeadArgs a{};
  a.w = w;
  a.hidden = hidden;
  a.logits = (float*)d.ptr;
  a.tkey = (uint64_t*)(d.ptr + kNaLogitBytes);
  a.tsum = (float*)(d.ptr + kNaLogitBytes + kNaKeyBytes);
  a.bmax = (uint64_t*)(d.ptr + kNaLogitBytes + kNaKeyBytes + kNaSumBytes);
  a.top_ids = ids;
  a.top_prob = prob;
  a.V = (uint32_t)vocab;
  a.tpitch = (a.V + 31) / 32 * 2;
  a.tblocks = (a.tpitch + 15) / 16;
  a.D = (uint32_t)dim;
  a.B = (uint32_t)B;
  a.K = (uint32_t)K;
  a.nblk = (uint32_t)d.cus;
  // One 64-row group: logits [tpitch x 64 x 16] <= kNaLogitBytes, statistics
  // [tblocks x 64 x 16] <= kNaKeyBytes / 8 entries, block maxima
  // [nblk x 64] <= kNaBmaxBytes / 8.
  e = launch_head_logits(a, stream);
  if (e == hipSuccess) e = launch_head_rows(a, stream);
  if (e != hipSuccess) return fail(TFE_ERR_HIP, "head launch: %s", hipGetErrorString(e));
  return TFE_OK;
}

}  // namespace
}  // namespace tfe

extern "C" tfe_status tfe_head_topk_noalloc(const void* w_pref, int32_t vocab, int32_t dim,
                                            const void* hidden, int32_t B, int32_t K,
                                            int32_t* top_ids, float* top_prob, void* stream) {
  tfe::begin_call();
  return tfe::topk_noalloc(w_pref, vocab, dim, hidden, B, K, top_ids, top_prob,
                           (hipStream_t)stream);
}
