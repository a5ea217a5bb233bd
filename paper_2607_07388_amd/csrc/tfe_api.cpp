// C ABI of libtfe: table load/free, lookup + inject, prefetch, statistics.
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <stddef.h>

#include <new>
#include <vector>

#include "../../include/tfe.h"
#include "tfe_internal.h"

namespace tfe {

hipError_t dev_malloc(void** p, size_t n) {
  *p = nullptr;
  if (alloc_fails()) return hipErrorOutOfMemory;
  const hipError_t e = hipMalloc(p, n);
  if (e != hipSuccess) {
    *p = nullptr;
    (void)hipGetLastError();
    return e;
  }
  note_alloc(*p, n, false);
  return hipSuccess;
}

void dev_free(void* p) {
  if (!p) return;
  note_free(p);
  (void)hipFree(p);
}

hipError_t pinned_malloc(void** p, size_t n, unsigned flags) {
  *p = nullptr;
  if (alloc_fails()) return hipErrorOutOfMemory;
  const hipError_t e = hipHostMalloc(p, n, flags);
  if (e != hipSuccess) {
    *p = nullptr;
    (void)hipGetLastError();
    return e;
  }
  note_alloc(*p, n, true);
  return hipSuccess;
}

void pinned_free(void* p) {
  if (!p) return;
  note_free(p);
  (void)hipHostFree(p);
}

tfe_status refuse_capture(hipStream_t stream, const char* what) {
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  const hipError_t e = hipStreamIsCapturing(stream, &cs);
  if (e != hipSuccess) return fail(TFE_ERR_HIP, "%s: hipStreamIsCapturing: %s", what,
                                   hipGetErrorString(e));
  if (cs != hipStreamCaptureStatusNone)
    return fail(TFE_ERR_UNSUPPORTED, "%s cannot be captured into a graph", what);
  return TFE_OK;
}

static tfe_status hip_fail(hipError_t e, const char* what) {
  return fail(TFE_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

#define TFE_HIP(call, what)                                   \
  do {                                                        \
    hipError_t e_ = (call);                                   \
    if (e_ != hipSuccess) return hip_fail(e_, what);          \
  } while (0)

static size_t elem_size(int dtype) { return dtype == TFE_F32 ? 4 : 2; }

// Host threads that stage pageable rows of one tiered table (each serves
// about four rows per microsecond).
constexpr int kStageThreads = 4;

// Waits on the host for the work this table has enqueued -- its last
// lookup, a pending prefetch, its own stream (uploads, side-stream fills) --
// and for nothing else on the device.  A lookup still being captured into a
// graph has not run yet and is not waited for.
static tfe_status sync_table(const tfe_table* ct) {
  tfe_table* t = const_cast<tfe_table*>(ct);  // events are recorded, nothing observable changes
  if (t->lookup_recorded && t->ev_lookup) {
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    TFE_HIP(hipStreamIsCapturing(t->last_stream, &cs), "hipStreamIsCapturing");
    if (cs == hipStreamCaptureStatusNone) {
      TFE_HIP(hipEventRecord(t->ev_lookup, t->last_stream), "record");
      TFE_HIP(hipEventSynchronize(t->ev_lookup), "wait for the last lookup");
    }
  }
  if (t->prefetch_pending && t->ev_prefetch)
    TFE_HIP(hipEventSynchronize(t->ev_prefetch), "wait for the prefetch");
  if (t->pf_counted_pending && t->ev_prefetch) {
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    TFE_HIP(hipStreamIsCapturing(t->pf_stream, &cs), "hipStreamIsCapturing");
    if (cs == hipStreamCaptureStatusNone) {
      TFE_HIP(hipEventRecord(t->ev_prefetch, t->pf_stream), "record");
      TFE_HIP(hipEventSynchronize(t->ev_prefetch), "wait for the prefetch");
    }
  }
  if (t->own_stream) TFE_HIP(hipStreamSynchronize(t->own_stream), "wait for the table stream");
  return TFE_OK;
}

static void release(tfe_table* t) {
  if (!t) return;
  // Teardown is best effort: errors here have no one to report to.
  int cur = 0;
  (void)hipGetDevice(&cur);
  (void)hipSetDevice(t->device);
  (void)sync_table(t);
  tfe::stager_stop(t->stager);  // after the table's kernels, the only ones that post to it
  void* dev_bufs[] = {t->d_slots, t->d_values, t->d_cache, t->d_where, t->d_owner, t->d_stamp,
                      t->d_pref, t->d_ring, t->d_ring2, t->d_ctl, t->d_row_of,
                      t->d_slot_of, t->d_phase, t->d_jobs, t->d_hit_ctr, t->d_hkey, t->d_hpos, t->d_hval, t->d_blk, t->d_spare, t->d_pf_row_of,
                      t->d_pf_slot_of, t->d_pf_phase, t->d_pf_jobs, t->d_stage_ack};
  for (void* b : dev_bufs)
    dev_free(b);
  if (t->own_h_values && t->h_values) pinned_free(t->h_values);
  if (t->own_stream) (void)hipStreamDestroy(t->own_stream);
  hipEvent_t evs[] = {t->ev_resolved, t->ev_filled, t->ev_lookup, t->ev_prefetch};
  for (hipEvent_t e : evs)
    if (e) (void)hipEventDestroy(e);
  (void)hipSetDevice(cur);
  delete t;
}

static tfe_status check_device(const tfe_table* t) {
  int cur = -1;
  TFE_HIP(hipGetDevice(&cur), "hipGetDevice");
  if (cur != t->device)
    return fail(TFE_ERR_INVALID_ARG, "table lives on device %d but device %d is current",
                t->device, cur);
  return TFE_OK;
}

static tfe_status load_resident(tfe_table* t, const tfe_table_desc* d, hipStream_t stream) {
  const size_t ctr_bytes = (size_t)kHitCounters * kHitStride * sizeof(unsigned long long);
  if (dev_malloc((void**)&t->d_hit_ctr, ctr_bytes) != hipSuccess) {
    t->d_hit_ctr = nullptr;
    return fail(TFE_ERR_OOM, "hit counters (%zu bytes)", ctr_bytes);
  }
  TFE_HIP(hipMemsetAsync(t->d_hit_ctr, 0, ctr_bytes, stream), "hit counters");
  TFE_HIP(hipStreamSynchronize(stream), "hit counters");
  if (d->n_phrases == 0) return TFE_OK;
  const size_t vbytes = (size_t)d->n_phrases * d->dim * elem_size(d->dtype);
  if (dev_malloc(&t->d_values, vbytes) != hipSuccess)
    return fail(TFE_ERR_OOM, "device values (%zu bytes)", vbytes);
  TFE_HIP(hipMemcpyAsync(t->d_values, d->values, vbytes,
                         d->values_on_device ? hipMemcpyDeviceToDevice : hipMemcpyHostToDevice,
                         stream),
          "values upload");
  TFE_HIP(hipStreamSynchronize(stream), "values upload");
  return TFE_OK;
}

template <class T>
static tfe_status dev_alloc(T** p, size_t n, const char* what) {
  if (dev_malloc((void**)p, n * sizeof(T) + (n == 0)) != hipSuccess)
    return fail(TFE_ERR_OOM, "%s (%zu bytes)", what, n * sizeof(T));
  return TFE_OK;
}

#define TFE_TRY(x)                   \
  do {                               \
    tfe_status st_ = (x);            \
    if (st_ != TFE_OK) return st_;   \
  } while (0)

static tfe::TierArgs tier_args(tfe_table* t) {
  tfe::TierArgs a = {};
  a.host_values = t->h_values_dev;
  a.pinned_rows = (uint32_t)t->pinned_rows;
  if (t->stager) {
    a.stage = tfe::stager_queue(t->stager);
    a.stage_rows = tfe::stager_rows(t->stager);
    a.stage_ack = t->d_stage_ack;
  }
  a.cache = t->d_cache;
  a.where = t->d_where;
  a.owner = t->d_owner;
  a.stamp = t->d_stamp;
  a.pref = t->d_pref;
  a.ring = t->d_ring;
  a.ring_mask = t->ring_cap - 1;
  a.ctl = t->d_ctl;
  a.row_of = t->d_row_of;
  a.slot_of = t->d_slot_of;
  a.phase = t->d_phase;
  a.jobs = t->d_jobs;
  a.hkey = t->d_hkey;
  a.hpos = t->d_hpos;
  a.hval = t->d_hval;
  a.hmask = 2 * (uint64_t)t->scratch_cap - 1;
  a.blk = t->d_blk;
  a.spare = t->d_spare;
  a.clock = t->clock;
  a.row_bytes = (uint32_t)(t->dim * elem_size(t->dtype));
  a.fill_inline = t->fill_mode == TFE_FILL_INLINE ? 1u : 0u;
  a.look.slots = t->d_slots;
  a.look.bucket_mask = (uint64_t)(t->capacity / TFE_SLOTS_PER_BUCKET - 1);
  a.look.n_min = t->n_min;
  a.look.n_max = t->n_max;
  a.look.vocab = t->vocab;
  return a;
}

// Orders the kernels enqueued next on `s` after the counted work submitted
// so far -- every one-launch decode call (lk) and every one-block prefetch's
// copy blocks (pf) -- with one waiting wave.
static tfe_status order_after_counted(tfe_table* t, hipStream_t s, bool lk, bool pf) {
  tfe::TierArgs a = tier_args(t);
  a.wait_lk = lk ? t->decodes_issued : 0;
  a.wait_pf = pf ? t->fills_issued : 0;
  if (!a.wait_lk && !a.wait_pf) return TFE_OK;
  TFE_HIP(tfe::launch_tier_wait(a, s), "ordering wait");
  return TFE_OK;
}

static uint64_t pow2_at_least(uint64_t n) {
  uint64_t c = 1;
  while (c < n) c <<= 1;
  return c;
}

// Tiered load: value rows in pinned host memory (the caller's, or a copy),
// an HBM cache of hbm_cache_rows rows with rows [0, prefill_rows) preloaded,
// and the residency / recency state of every slot.
static tfe_status load_tiered(tfe_table* t, const tfe_table_desc* d, hipStream_t stream) {
  const int64_t P = d->n_phrases, C = d->hbm_cache_rows;
  const size_t row_bytes = (size_t)d->dim * elem_size(d->dtype);
  // Rows [0, Ppin) are pinned; rows [Ppin, P) stay in the caller's pageable
  // memory behind the staging queue.
  const int64_t Ppin = d->pinned_rows > 0 ? d->pinned_rows : P;
  t->pinned_rows = Ppin;
  t->cache_rows = C;
  t->prefill_rows = d->prefill_rows;
  t->fill_mode = d->miss_fill;
  if (P > 0 && d->adopt_host_values) {
    hipPointerAttribute_t attr;
    const hipError_t pe = hipPointerGetAttributes(&attr, d->values);
    if (pe != hipSuccess) (void)hipGetLastError();  // unknown memory: clear the error state
    if (pe != hipSuccess || attr.type != hipMemoryTypeHost)
      return fail(TFE_ERR_INVALID_ARG, "adopted values are not pinned host memory (hipHostMalloc)");
    t->h_values = const_cast<void*>(d->values);
  } else if (P > 0) {
    if (pinned_malloc(&t->h_values, (size_t)Ppin * row_bytes) != hipSuccess) {
      t->h_values = nullptr;
      return fail(TFE_ERR_OOM, "pinned host values (%zu bytes)", (size_t)Ppin * row_bytes);
    }
    t->own_h_values = true;
    TFE_HIP(hipMemcpy(t->h_values, d->values, (size_t)Ppin * row_bytes,
                      d->values_on_device ? hipMemcpyDeviceToHost : hipMemcpyHostToHost),
            "values to pinned host memory");
  }
  if (Ppin < P) {
    TFE_TRY(dev_alloc(&t->d_stage_ack, tfe::kStageSlots, "staging acknowledgements"));
    TFE_HIP(hipMemsetAsync(t->d_stage_ack, 0, tfe::kStageSlots * sizeof(unsigned long long),
                           stream),
            "init");
    TFE_TRY(tfe::stager_start(d->pageable_values, Ppin, P, row_bytes, kStageThreads, &t->stager));
  }
  if (t->h_values) {
    void* dp = nullptr;
    TFE_HIP(hipHostGetDevicePointer(&dp, t->h_values, 0), "hipHostGetDevicePointer");
    t->h_values_dev = dp;
  }
  // Physical cache slots: C rows of the cache plus kDecodeMaxT spare slots
  // that the one-launch decode writes missed rows into and swaps with its
  // victims (never in the recency order, never mapped by a row).
  const size_t slots = (size_t)C + tfe::kDecodeMaxT;
  TFE_TRY(dev_alloc((char**)&t->d_cache, slots * row_bytes, "HBM cache"));
  // At least one entry: the resolve kernels read entry 0 unconditionally.
  const size_t where_n = P > 0 ? (size_t)P : 1;
  TFE_TRY(dev_alloc(&t->d_where, where_n, "residency map"));
  TFE_TRY(dev_alloc(&t->d_owner, slots, "slot owners"));
  TFE_TRY(dev_alloc(&t->d_stamp, slots, "slot stamps"));
  TFE_TRY(dev_alloc(&t->d_pref, slots, "prefetch flags"));
  TFE_TRY(dev_alloc(&t->d_spare, (size_t)tfe::kDecodeMaxT, "spare slots"));
  t->ring_cap = pow2_at_least((uint64_t)C * 4 < 4096 ? 4096 : (uint64_t)C * 4);
  TFE_TRY(dev_alloc(&t->d_ring, t->ring_cap, "recency ring"));
  TFE_TRY(dev_alloc(&t->d_ring2, t->ring_cap, "recency ring"));
  TFE_TRY(dev_alloc(&t->d_ctl, 1, "tier control block"));

  TFE_HIP(hipMemsetAsync(t->d_where, 0xFF, where_n * sizeof(int32_t), stream), "init");
  TFE_HIP(hipMemsetAsync(t->d_ctl, 0, sizeof(tfe::TierCtl), stream), "init");
  tfe::TierArgs a = tier_args(t);
  TFE_HIP(tfe::launch_tier_init(a, (uint32_t)C, (uint32_t)d->prefill_rows, stream), "init launch");
  const int64_t pre_pinned = d->prefill_rows < Ppin ? d->prefill_rows : Ppin;
  if (pre_pinned > 0)
    TFE_HIP(hipMemcpyAsync(t->d_cache, t->h_values, (size_t)pre_pinned * row_bytes,
                           hipMemcpyHostToDevice, stream),
            "cache prefill");
  if (d->prefill_rows > Ppin)  // from pageable memory (a staged copy by the runtime)
    TFE_HIP(hipMemcpyAsync((char*)t->d_cache + (size_t)Ppin * row_bytes, d->pageable_values,
                           (size_t)(d->prefill_rows - Ppin) * row_bytes, hipMemcpyHostToDevice,
                           stream),
            "cache prefill");
  t->ring_bound = (uint64_t)C;
  // Test hook: TFE_TIER_CLOCK_START starts the recency clock elsewhere than
  // 0 (the tests start it just below the 32-bit wrap).  Stamps start at 0,
  // below any clock a call uses.
  if (const char* cs = getenv("TFE_TIER_CLOCK_START")) t->clock = (uint32_t)strtoul(cs, nullptr, 0);
  TFE_HIP(hipStreamSynchronize(stream), "tiered init");
  return TFE_OK;
}

// Grows the per-call scratch (rows, slots, phases, fill jobs, the call-wide
// row table) to n entries.  The new buffers are allocated first: if one
// fails, the others are returned and the table keeps its old scratch.  The
// old buffers are freed after the table's pending work that may still use
// them.
static tfe_status ensure_scratch(tfe_table* t, uint32_t n) {
  if (n <= t->scratch_cap) return TFE_OK;
  const uint64_t cap = pow2_at_least(n < 1024 ? 1024 : n);
  int32_t *row_of = nullptr, *slot_of = nullptr;
  uint8_t* phase = nullptr;
  tfe::TierJob* jobs = nullptr;
  uint64_t *hkey = nullptr, *hpos = nullptr, *hval = nullptr;
  uint64_t* blk = nullptr;
  tfe_status st = TFE_OK;
  if ((st = dev_alloc(&row_of, cap, "scratch")) == TFE_OK &&
      (st = dev_alloc(&slot_of, cap, "scratch")) == TFE_OK &&
      (st = dev_alloc(&phase, cap, "scratch")) == TFE_OK &&
      (st = dev_alloc(&jobs, cap, "scratch")) == TFE_OK &&
      (st = dev_alloc(&hkey, 2 * cap, "scratch")) == TFE_OK &&
      (st = dev_alloc(&hpos, 2 * cap, "scratch")) == TFE_OK &&
      (st = dev_alloc(&hval, 2 * cap, "scratch")) == TFE_OK)
    st = dev_alloc(&blk, cap / 1024 + 1, "scratch");
  void* fresh[] = {row_of, slot_of, phase, jobs, hkey, hpos, hval, blk};
  if (st == TFE_OK) st = sync_table(t);
  if (st != TFE_OK) {
    for (void* b : fresh) dev_free(b);
    return st;
  }
  void* olds[] = {t->d_row_of, t->d_slot_of, t->d_phase, t->d_jobs, t->d_hkey, t->d_hpos,
                  t->d_hval, t->d_blk};
  for (void* b : olds) dev_free(b);
  t->d_row_of = row_of;
  t->d_slot_of = slot_of;
  t->d_phase = phase;
  t->d_jobs = jobs;
  t->d_hkey = hkey;
  t->d_hpos = hpos;
  t->d_hval = hval;
  t->d_blk = blk;
  // Clock 0 tags every entry of the call-wide row table as empty (calls use
  // clocks from 1).
  TFE_HIP(hipMemsetAsync(t->d_hkey, 0, 2 * cap * sizeof(uint64_t), t->own_stream), "scratch");
  TFE_HIP(hipMemsetAsync(t->d_hpos, 0, 2 * cap * sizeof(uint64_t), t->own_stream), "scratch");
  TFE_HIP(hipMemsetAsync(t->d_hval, 0, 2 * cap * sizeof(uint64_t), t->own_stream), "scratch");
  TFE_HIP(hipStreamSynchronize(t->own_stream), "scratch");
  t->scratch_cap = (uint32_t)cap;
  return TFE_OK;
}

// Grows the prefetches' own per-call scratch to n entries, in the same way.
static tfe_status ensure_pf_scratch(tfe_table* t, uint64_t n) {
  if (n <= t->pf_cap) return TFE_OK;
  const uint64_t cap = pow2_at_least(n < 1024 ? 1024 : n);
  int32_t *row_of = nullptr, *slot_of = nullptr;
  uint8_t* phase = nullptr;
  tfe::TierJob* jobs = nullptr;
  tfe_status st = TFE_OK;
  if ((st = dev_alloc(&row_of, cap, "prefetch scratch")) == TFE_OK &&
      (st = dev_alloc(&slot_of, cap, "prefetch scratch")) == TFE_OK &&
      (st = dev_alloc(&phase, cap, "prefetch scratch")) == TFE_OK)
    st = dev_alloc(&jobs, cap, "prefetch scratch");
  void* fresh[] = {row_of, slot_of, phase, jobs};
  if (st == TFE_OK) st = sync_table(t);
  if (st != TFE_OK) {
    for (void* b : fresh) dev_free(b);
    return st;
  }
  void* olds[] = {t->d_pf_row_of, t->d_pf_slot_of, t->d_pf_phase, t->d_pf_jobs};
  for (void* b : olds) dev_free(b);
  t->d_pf_row_of = row_of;
  t->d_pf_slot_of = slot_of;
  t->d_pf_phase = phase;
  t->d_pf_jobs = jobs;
  t->pf_cap = (uint32_t)cap;
  return TFE_OK;
}

// Before a call that appends at most `appends` recency entries: drops the
// dead entries when the ring could overflow (every slot keeps exactly one
// live entry, so afterwards the ring holds cache_rows entries), growing the
// ring if even that would not leave room.
// `lk`, `pf`: counted work that the kernels of this call on `stream` still
// have to follow (a compaction launched here waits for it first).
static tfe_status reserve_ring(tfe_table* t, uint64_t appends, hipStream_t stream, bool lk,
                               bool pf) {
  if (t->ring_bound + appends <= t->ring_cap) {
    t->ring_bound += appends;
    return TFE_OK;
  }
  TFE_TRY(order_after_counted(t, stream, lk, pf));
  const uint64_t need = (uint64_t)t->cache_rows + appends;
  tfe::TierArgs a = tier_args(t);
  if (need > t->ring_cap) {
    const uint64_t cap = pow2_at_least(2 * need);
    uint64_t *r1 = nullptr, *r2 = nullptr;
    TFE_TRY(dev_alloc(&r1, cap, "recency ring"));
    if (dev_alloc(&r2, cap, "recency ring") != TFE_OK) {
      dev_free(r1);
      return TFE_ERR_OOM;
    }
    TFE_HIP(tfe::launch_ring_compact(a, r1, cap - 1, false, stream), "ring compaction");
    TFE_HIP(hipStreamSynchronize(stream), "ring regrow");
    dev_free(t->d_ring);
    dev_free(t->d_ring2);
    t->d_ring = r1;
    t->d_ring2 = r2;
    t->ring_cap = cap;
  } else {
    TFE_HIP(tfe::launch_ring_compact(a, t->d_ring2, t->ring_cap - 1, false, stream),
            "ring compaction");
    uint64_t* tmp = t->d_ring;
    t->d_ring = t->d_ring2;
    t->d_ring2 = tmp;
  }
  t->ring_bound = (uint64_t)t->cache_rows + appends;
  return TFE_OK;
}

// Starts the next call's recency clock.  Stamps and the call-wide row
// table hold 32-bit clocks; before the clock would wrap, every live recency
// entry and slot stamp restart at 0 (order kept) and the row table is
// cleared, so clocks 1, 2, ... can be used again.
static tfe_status advance_clock(tfe_table* t, uint64_t appends, hipStream_t stream, bool lk,
                                bool pf) {
  if (t->clock == 0xFFFFFFFFu) {
    TFE_TRY(order_after_counted(t, stream, lk, pf));
    tfe::TierArgs a = tier_args(t);
    TFE_HIP(tfe::launch_ring_compact(a, t->d_ring2, t->ring_cap - 1, true, stream),
            "clock restart");
    uint64_t* tmp = t->d_ring;
    t->d_ring = t->d_ring2;
    t->d_ring2 = tmp;
    t->ring_bound = (uint64_t)t->cache_rows + appends;  // this call's reservation
    if (t->scratch_cap) {
      TFE_HIP(hipMemsetAsync(t->d_hkey, 0, 2 * (size_t)t->scratch_cap * sizeof(uint64_t), stream),
              "clock restart");
      TFE_HIP(hipMemsetAsync(t->d_hpos, 0, 2 * (size_t)t->scratch_cap * sizeof(uint64_t), stream),
              "clock restart");
      TFE_HIP(hipMemsetAsync(t->d_hval, 0, 2 * (size_t)t->scratch_cap * sizeof(uint64_t), stream),
              "clock restart");
    }
    t->clock = 0;
  }
  t->clock++;
  return TFE_OK;
}

static tfe_status lookup_tiered(tfe_table* t, const LookupArgs& look, hipStream_t stream) {
  TFE_TRY(ensure_scratch(t, look.T));
  // Calls on one table are ordered: after the previous lookup (when it ran
  // on another stream) and after a pending prefetch.
  if (t->lookup_recorded && stream != t->last_stream) {
    TFE_HIP(hipEventRecord(t->ev_lookup, t->last_stream), "record");
    TFE_HIP(hipStreamWaitEvent(stream, t->ev_lookup, 0), "wait lookup");
  }
  // A pending prefetch and the previous call's side-stream cache fill use
  // the same per-call scratch (matched rows, fill list), the recency ring
  // and the residency state as everything below, so every kernel of this
  // call -- ring compaction and the probe included -- waits for them.
  // (The pending flag is cleared once this call has been enqueued.)
  if (t->prefetch_pending) TFE_HIP(hipStreamWaitEvent(stream, t->ev_prefetch, 0), "wait prefetch");
  if (t->fill_recorded) TFE_HIP(hipStreamWaitEvent(stream, t->ev_filled, 0), "wait fill");
  // A one-block prefetch on another stream is followed without HIP events:
  // the one-launch decode waits for its copy blocks itself; any other
  // kernel of this call is preceded by a waiting wave.
  const bool pf = t->pf_counted_pending && stream != t->pf_stream;
  const bool decode = t->fill_mode == TFE_FILL_INLINE && look.T <= tfe::kDecodeMaxT;
  if (pf && !decode) TFE_TRY(order_after_counted(t, stream, false, true));
  const bool pf_kernel = pf && decode;  // still to be awaited by the decode kernel
  TFE_TRY(reserve_ring(t, look.T, stream, false, pf_kernel));
  TFE_TRY(advance_clock(t, look.T, stream, false, pf_kernel));
  // Everything after this call follows it, and through it the prefetches.
  t->pf_counted_pending = false;
  t->prefetch_pending = false;
  tfe::TierArgs a = tier_args(t);
  a.look = look;
  if (decode) {
    // The whole call in one launch (probe, inject, residency).
    a.wait_pf = pf_kernel ? t->fills_issued : 0;
    // Counting (a release of the residency writes and one addition) is only
    // needed once prefetches follow decodes on this table.
    a.count_lookup = t->counting ? 1u : 0u;
    TFE_HIP(tfe::launch_tier_decode(a, t->dtype, t->dim, stream), "tiered decode");
    if (t->counting) t->decodes_issued += 1;
    t->last_lookup_counted = t->counting;
    t->lookup_recorded = true;
    t->last_stream = stream;
    return TFE_OK;
  }
  t->last_lookup_counted = false;
  const bool fused = tfe::lookup_resolve_fused(look.T);
  if (!fused) TFE_HIP(tfe::launch_tier_probe(a, stream), "tier probe");
  if (fused)
    TFE_HIP(tfe::launch_lookup_resolve_small(a, stream), "tier probe + resolve");
  else
    TFE_HIP(tfe::launch_resolve_lookup(a, stream), "tier resolve");
  if (t->fill_mode == TFE_FILL_SIDE_STREAM) {
    // Missed rows are copied into their new cache slots on the side stream,
    // overlapped with the injection, which reads them from host memory.
    TFE_HIP(hipEventRecord(t->ev_resolved, stream), "record");
    TFE_HIP(hipStreamWaitEvent(t->own_stream, t->ev_resolved, 0), "wait resolve");
    TFE_HIP(tfe::launch_fill(a, t->dtype, t->dim, look.T, t->own_stream), "tier fill");
    TFE_HIP(hipEventRecord(t->ev_filled, t->own_stream), "record");
    t->fill_recorded = true;
  }
  // Inline fill: the injection writes each missed row into its slot.
  TFE_HIP(tfe::launch_tier_inject(a, t->dtype, t->dim, stream), "inject");
  t->lookup_recorded = true;
  t->last_stream = stream;
  return TFE_OK;
}

static tfe_status prefetch_tiered(tfe_table* t, const int32_t* tail, int32_t tail_len,
                                  const int32_t* cand, const float* prob, int32_t B, int32_t K,
                                  int32_t budget, hipStream_t side) {
  const uint64_t N = (uint64_t)B * K;
  if (N == 0) return TFE_OK;
  if (N > 0x7FFFFFFFull) return fail(TFE_ERR_UNSUPPORTED, "B * K above 2^31 - 1");
  TFE_TRY(check_device(t));
  TFE_TRY(refuse_capture(side, "a prefetch"));
  const bool one_block = N <= tfe::prefetch_fused_max();
  // The one-block prefetch keeps one probe result per (candidate, length)
  // in its scratch; the scored resolution uses the call-wide row table of
  // the lookups' scratch (never run by two calls at once).
  TFE_TRY(ensure_pf_scratch(t, one_block ? N * (uint64_t)(t->n_max - t->n_min + 1) : N));
  TFE_TRY(ensure_scratch(t, (uint32_t)N));
  t->counting = true;  // later decodes count themselves for the prefetches
  // After the table's last lookup, its cache fill, and any earlier
  // prefetch.  A one-launch decode lookup and a one-block prefetch are
  // followed on the device (counters in the control block) instead of with
  // HIP events; the other kernels use events.
  const bool other_stream = t->lookup_recorded && side != t->last_stream;
  const bool lk = one_block && other_stream && t->last_lookup_counted;
  if (other_stream && !lk) {
    TFE_HIP(hipEventRecord(t->ev_lookup, t->last_stream), "record");
    TFE_HIP(hipStreamWaitEvent(side, t->ev_lookup, 0), "wait lookup");
  }
  if (t->fill_recorded) TFE_HIP(hipStreamWaitEvent(side, t->ev_filled, 0), "wait fill");
  // (The pending flag is cleared once this call has been enqueued: if it
  // fails on the way, later calls still wait for the earlier prefetch.)
  if (t->prefetch_pending) TFE_HIP(hipStreamWaitEvent(side, t->ev_prefetch, 0), "wait prefetch");
  // A counted prefetch on another stream shares this one's scratch: this
  // whole call (its probe too) waits for it.
  const bool pf = t->pf_counted_pending && side != t->pf_stream;
  if (pf) TFE_TRY(order_after_counted(t, side, false, true));
  if (!one_block) TFE_TRY(order_after_counted(t, side, lk, false));
  TFE_TRY(reserve_ring(t, N, side, lk, false));
  TFE_TRY(advance_clock(t, N, side, lk, false));
  tfe::TierArgs a = tier_args(t);
  a.prefetch = 1;
  a.row_of = t->d_pf_row_of;
  a.slot_of = t->d_pf_slot_of;
  a.phase = t->d_pf_phase;
  a.jobs = t->d_pf_jobs;
  if (one_block) {
    // The probe runs before this wait: it touches only the index, the
    // candidates and the prefetch scratch.
    a.wait_lk = lk ? t->decodes_issued : 0;
    TFE_HIP(tfe::launch_prefetch_fused(a, tail, tail_len, cand, (uint32_t)B, (uint32_t)K, prob,
                                       (uint32_t)budget, side),
            "prefetch");
    a.wait_lk = a.wait_pf = 0;
    a.count_fill = 1;
    TFE_HIP(tfe::launch_fill(a, t->dtype, t->dim, (uint32_t)N, side), "prefetch fill");
    t->fills_issued += tfe::fill_blocks((uint32_t)N);
    t->prefetch_pending = false;
    t->pf_counted_pending = true;
    t->pf_stream = side;
    return TFE_OK;
  }
  TFE_HIP(tfe::launch_prefetch_probe(a, tail, tail_len, cand, (uint32_t)B, (uint32_t)K, side),
          "prefetch probe");
  if (prob) {
    TFE_HIP(tfe::launch_resolve_prefetch_scored(a, (uint32_t)N, prob, (uint32_t)budget, side),
            "prefetch resolve");
  } else {
    // The candidates are referenced like a lookup's positions.
    a.look.T = (uint32_t)N;
    TFE_HIP(tfe::launch_resolve_lookup(a, side), "prefetch resolve");
  }
  TFE_HIP(tfe::launch_fill(a, t->dtype, t->dim, (uint32_t)N, side), "prefetch fill");
  TFE_HIP(hipEventRecord(t->ev_prefetch, side), "record");
  t->prefetch_pending = true;
  t->pf_counted_pending = false;  // this prefetch follows the counted ones
  return TFE_OK;
}

static tfe_status load(const tfe_table_desc* d, hipStream_t stream, tfe_table** out) {
  if (!d || !out) return fail(TFE_ERR_INVALID_ARG, "null desc or out");
  *out = nullptr;
  if (d->dtype != TFE_F32 && d->dtype != TFE_BF16) return fail(TFE_ERR_INVALID_ARG, "bad dtype");
  if (!dim_supported(d->dtype, d->dim))
    return fail(TFE_ERR_UNSUPPORTED, "dim %d not supported for dtype %d", d->dim, d->dtype);
  double lf = d->max_load_factor == 0.0 ? 0.5 : d->max_load_factor;
  if (!(lf > 0.0 && lf <= 0.9)) return fail(TFE_ERR_INVALID_ARG, "max_load_factor not in (0, 0.9]");
  if (d->hbm_cache_rows < 0) return fail(TFE_ERR_INVALID_ARG, "hbm_cache_rows < 0");
  if (d->hbm_cache_rows > (1ll << 30) - 1024)
    return fail(TFE_ERR_UNSUPPORTED, "hbm_cache_rows above 2^30 - 1024");
  if (d->prefill_rows < 0 || d->prefill_rows > d->hbm_cache_rows ||
      d->prefill_rows > d->n_phrases)
    return fail(TFE_ERR_INVALID_ARG, "prefill_rows outside [0, min(hbm_cache_rows, n_phrases)]");
  if (d->miss_fill != TFE_FILL_INLINE && d->miss_fill != TFE_FILL_SIDE_STREAM)
    return fail(TFE_ERR_INVALID_ARG, "miss_fill must be TFE_FILL_INLINE or TFE_FILL_SIDE_STREAM");
  if (d->adopt_host_values && (d->hbm_cache_rows == 0 || d->values_on_device))
    return fail(TFE_ERR_INVALID_ARG, "adopt_host_values needs a tiered table and host values");
  if (d->pinned_rows < 0 || d->pinned_rows > d->n_phrases)
    return fail(TFE_ERR_INVALID_ARG, "pinned_rows outside [0, n_phrases]");
  if (d->pinned_rows > 0 && d->pinned_rows < d->n_phrases &&
      (d->hbm_cache_rows == 0 || d->values_on_device || !d->pageable_values))
    return fail(TFE_ERR_INVALID_ARG,
                "pinned_rows < n_phrases needs a tiered table, host values and pageable_values");
  tfe_status st = validate_phrases(d->phrase_tokens, d->phrase_len, d->n_phrases, d->n_min,
                                   d->n_max, d->vocab);
  if (st != TFE_OK) return st;
  if (d->n_phrases > 0 && !d->values) return fail(TFE_ERR_INVALID_ARG, "null values");

  const int64_t cap = index_capacity(d->n_phrases, lf);
  std::vector<tfe_slot> slots;
  try {
    if (alloc_fails()) throw std::bad_alloc();
    slots.resize((size_t)cap);
  } catch (const std::bad_alloc&) {
    return fail(TFE_ERR_OOM, "host index of %lld slots", (long long)cap);
  }
  st = build_index(d->phrase_tokens, d->phrase_len, d->n_phrases, d->n_max, slots.data(), cap);
  if (st != TFE_OK) return st;

  tfe_table* t = alloc_fails() ? nullptr : new (std::nothrow) tfe_table;
  if (!t) return fail(TFE_ERR_OOM, "table object");
  if (hipGetDevice(&t->device) != hipSuccess ||
      hipDeviceGetAttribute(&t->cus, hipDeviceAttributeMultiprocessorCount, t->device) !=
          hipSuccess) {
    delete t;
    return fail(TFE_ERR_HIP, "device query");
  }
  t->n_phrases = d->n_phrases;
  t->n_min = d->n_min;
  t->n_max = d->n_max;
  t->vocab = d->vocab;
  t->dim = d->dim;
  t->dtype = d->dtype;
  t->capacity = cap;
  {
    hipError_t ce = hipStreamCreateWithFlags(&t->own_stream, hipStreamNonBlocking);
    hipEvent_t* evs[] = {&t->ev_resolved, &t->ev_filled, &t->ev_lookup, &t->ev_prefetch};
    for (hipEvent_t* ev : evs)
      if (ce == hipSuccess) ce = hipEventCreateWithFlags(ev, hipEventDisableTiming);
    if (ce != hipSuccess) {
      release(t);
      return hip_fail(ce, "table stream and events");
    }
  }

  const size_t slot_bytes = (size_t)cap * sizeof(tfe_slot);
  if (dev_malloc((void**)&t->d_slots, slot_bytes) != hipSuccess) {
    release(t);
    return fail(TFE_ERR_OOM, "device index (%zu bytes)", slot_bytes);
  }
  hipError_t e = hipMemcpyAsync(t->d_slots, slots.data(), slot_bytes, hipMemcpyHostToDevice, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  if (e != hipSuccess) {
    release(t);
    return hip_fail(e, "index upload");
  }
  st = d->hbm_cache_rows > 0 ? load_tiered(t, d, stream) : load_resident(t, d, stream);
  if (st != TFE_OK) {
    release(t);
    return st;
  }
  *out = t;
  return TFE_OK;
}

static tfe_status lookup_inject(tfe_table* t, const int32_t* tokens, int32_t B, int32_t ctx,
                                int32_t S, const void* hin, void* hout, uint8_t* hit,
                                int32_t* slot, uint8_t* len, int32_t gate, float scale,
                                hipStream_t stream, int32_t weighting = -1) {
  const bool multi = weighting >= 0;
  if (!t) return fail(TFE_ERR_INVALID_ARG, "null table");
  if (B < 0 || ctx < 0 || S < 0) return fail(TFE_ERR_INVALID_ARG, "negative B, ctx or S");
  if (gate != TFE_GATE_SIGMOID && gate != TFE_GATE_CONST) return fail(TFE_ERR_INVALID_ARG, "bad gate");
  if (!isfinite(scale)) return fail(TFE_ERR_INVALID_ARG, "scale is not finite");
  const int64_t T = (int64_t)B * S;
  if ((int64_t)ctx + S > 0x7FFFFFFFll) return fail(TFE_ERR_INVALID_ARG, "ctx + S overflows");
  if (T > 0x7FFFFFFFll) return fail(TFE_ERR_UNSUPPORTED, "B * S above 2^31 - 1 positions");
  if (multi && weighting != TFE_WEIGHT_LENGTH && weighting != TFE_WEIGHT_UNIFORM)
    return fail(TFE_ERR_INVALID_ARG, "bad weighting");
  if (multi && t->cache_rows > 0)
    return fail(TFE_ERR_UNSUPPORTED, "multi-match lookup on a tiered table");
  // The recency clock, the ring bound and the cross-stream events of a
  // tiered table live on the host and change with every call: a replayed
  // graph would reuse them.  Refused before anything is counted.
  if (t->cache_rows > 0) TFE_TRY(refuse_capture(stream, "a lookup on a tiered table"));
  if (T == 0) return TFE_OK;
  if (!tokens || !hin || !hout || !hit || !slot)
    return fail(TFE_ERR_INVALID_ARG, "null tokens, hidden, mask or slot_ids");
  tfe_status st = check_device(t);
  if (st != TFE_OK) return st;
  LookupArgs a;
  a.slots = t->d_slots;
  a.bucket_mask = (uint64_t)(t->capacity / TFE_SLOTS_PER_BUCKET - 1);
  a.values = t->d_values;
  a.tokens = tokens;
  a.T = (uint32_t)T;
  a.S = S;
  a.ctx = ctx;
  a.W = ctx + S;
  a.n_min = t->n_min;
  a.n_max = t->n_max;
  a.vocab = t->vocab;
  a.hin = hin;
  a.hout = hout;
  a.inplace = hin == hout;
  a.hit = hit;
  a.slot_out = slot;
  a.len_out = len;
  a.gate = gate;
  a.scale = scale;
  a.inv_d = 1.0f / (float)t->dim;
  a.inv_sqrt_d = (float)(1.0 / sqrt((double)t->dim));
  a.weighting = weighting;
  a.hit_ctr = t->cache_rows > 0 ? nullptr : t->d_hit_ctr;
  if (multi) {
    a.len_out = nullptr;
    TFE_HIP(launch_lookup_inject_multi(a, t->dtype, t->dim, stream), "lookup_inject_multi launch");
    t->stats.positions += (uint64_t)T;
    t->lookup_recorded = true;
    t->last_stream = stream;
    return TFE_OK;
  }
  if (t->cache_rows > 0) return lookup_tiered(t, a, stream);
  TFE_HIP(launch_lookup_inject(a, t->dtype, t->dim, stream), "lookup_inject launch");
  t->stats.positions += (uint64_t)T;
  t->lookup_recorded = true;
  t->last_stream = stream;
  return TFE_OK;
}

}  // namespace tfe

extern "C" {

tfe_status tfe_table_load(const tfe_table_desc* desc, void* stream, tfe_table** out) {
  tfe::begin_call();
  return tfe::load(desc, (hipStream_t)stream, out);
}

tfe_status tfe_table_free(tfe_table* table) {
  tfe::begin_call();
  tfe::release(table);
  return TFE_OK;
}

tfe_status tfe_lookup_inject(tfe_table* table, const int32_t* tokens, int32_t B, int32_t ctx,
                             int32_t S, const void* hidden_in, void* hidden_out,
                             uint8_t* hit_mask, int32_t* slot_ids, uint8_t* match_len,
                             int32_t gate, float scale, void* stream) {
  tfe::begin_call();
  const tfe_status st = tfe::lookup_inject(table, tokens, B, ctx, S, hidden_in, hidden_out,
                                           hit_mask, slot_ids, match_len, gate, scale,
                                           (hipStream_t)stream);
  if (st == TFE_OK) table->stats.calls++;
  return st;
}

tfe_status tfe_lookup_inject_multi(tfe_table* table, const int32_t* tokens, int32_t B,
                                   int32_t ctx, int32_t S, const void* hidden_in,
                                   void* hidden_out, uint8_t* match_mask, int32_t* slot_ids,
                                   int32_t weighting, int32_t gate, float scale, void* stream) {
  tfe::begin_call();
  if (weighting < 0) return tfe::fail(TFE_ERR_INVALID_ARG, "bad weighting");
  const tfe_status st = tfe::lookup_inject(table, tokens, B, ctx, S, hidden_in, hidden_out,
                                           match_mask, slot_ids, nullptr, gate, scale,
                                           (hipStream_t)stream, weighting);
  if (st == TFE_OK) table->stats.calls++;
  return st;
}

tfe_status tfe_prefetch(tfe_table* table, const int32_t* tail, int32_t tail_len,
                        const int32_t* candidates, int32_t B, int32_t K, void* side_stream) {
  tfe::begin_call();
  if (!table) return tfe::fail(TFE_ERR_INVALID_ARG, "null table");
  if (tail_len < 0 || B < 0 || K < 0) return tfe::fail(TFE_ERR_INVALID_ARG, "negative size");
  if ((int64_t)B * K > 0 && (!candidates || (tail_len > 0 && !tail)))
    return tfe::fail(TFE_ERR_INVALID_ARG, "null tail or candidates");
  if (table->cache_rows == 0) return TFE_OK;  // resident tables have nothing to prefetch
  return tfe::prefetch_tiered(table, tail, tail_len, candidates, nullptr, B, K, 0,
                              (hipStream_t)side_stream);
}

tfe_status tfe_prefetch_scored(tfe_table* table, const int32_t* tail, int32_t tail_len,
                               const int32_t* candidates, const float* cand_prob, int32_t B,
                               int32_t K, int32_t budget, void* side_stream) {
  tfe::begin_call();
  if (!table) return tfe::fail(TFE_ERR_INVALID_ARG, "null table");
  if (tail_len < 0 || B < 0 || K < 0) return tfe::fail(TFE_ERR_INVALID_ARG, "negative size");
  if (budget < 0 || budget > (int32_t)tfe::scored_prefetch_budget_max())
    return tfe::fail(TFE_ERR_INVALID_ARG, "budget outside [0, %u]",
                     tfe::scored_prefetch_budget_max());
  if ((int64_t)B * K > 0 && (!candidates || !cand_prob || (tail_len > 0 && !tail)))
    return tfe::fail(TFE_ERR_INVALID_ARG, "null tail, candidates or probabilities");
  if (table->cache_rows == 0) return TFE_OK;
  return tfe::prefetch_tiered(table, tail, tail_len, candidates, cand_prob, B, K, budget,
                              (hipStream_t)side_stream);
}

tfe_status tfe_get_stats(const tfe_table* table, tfe_stats* out) {
  tfe::begin_call();
  if (!table || !out) return tfe::fail(TFE_ERR_INVALID_ARG, "null table or out");
  tfe_status st = tfe::sync_table(table);
  if (st != TFE_OK) return st;
  tfe_stats s = table->stats;
  if (table->cache_rows > 0) {
    tfe::TierCtl c;
    hipError_t e = hipMemcpyAsync(&c, table->d_ctl, sizeof c, hipMemcpyDeviceToHost,
                                  table->own_stream);
    if (e == hipSuccess) e = hipStreamSynchronize(table->own_stream);
    if (e != hipSuccess) return tfe::fail(TFE_ERR_HIP, "stats: %s", hipGetErrorString(e));
    s.positions = c.stats.positions;
    s.hits = c.stats.hits;
    s.cache_hits = c.stats.cache_hits;
    s.cache_misses = c.stats.cache_misses;
    s.prefetch_keys = c.stats.prefetch_keys;
    s.prefetch_found = c.stats.prefetch_found;
    s.prefetch_filled = c.stats.prefetch_filled;
    s.prefetch_used = c.stats.prefetch_used;
    s.host_bytes = c.stats.host_bytes;
    s.prefetch_dropped = c.stats.prefetch_dropped;
    if (c.wait_timeouts)
      return tfe::fail(TFE_ERR_HIP, "%u device-side ordering waits hit their bound",
                       c.wait_timeouts);
  } else if (table->d_hit_ctr) {
    std::vector<unsigned long long> ctr((size_t)tfe::kHitCounters * tfe::kHitStride);
    hipError_t e = hipMemcpyAsync(ctr.data(), table->d_hit_ctr, ctr.size() * sizeof ctr[0],
                                  hipMemcpyDeviceToHost, table->own_stream);
    if (e == hipSuccess) e = hipStreamSynchronize(table->own_stream);
    if (e != hipSuccess) return tfe::fail(TFE_ERR_HIP, "stats: %s", hipGetErrorString(e));
    s.hits = 0;
    for (int i = 0; i < tfe::kHitCounters; ++i) s.hits += ctr[i * tfe::kHitStride];
  }
  *out = s;
  return TFE_OK;
}

tfe_status tfe_reset_stats(tfe_table* table) {
  tfe::begin_call();
  if (!table) return tfe::fail(TFE_ERR_INVALID_ARG, "null table");
  tfe_status st = tfe::sync_table(table);
  if (st != TFE_OK) return st;
  table->stats = tfe_stats{};
  hipError_t e = hipSuccess;
  if (table->cache_rows > 0)
    e = hipMemsetAsync((char*)table->d_ctl + offsetof(tfe::TierCtl, stats), 0,
                       sizeof(tfe::TierStats), table->own_stream);
  else if (table->d_hit_ctr)
    e = hipMemsetAsync(table->d_hit_ctr, 0,
                       sizeof(unsigned long long) * tfe::kHitCounters * tfe::kHitStride,
                       table->own_stream);
  if (e == hipSuccess) e = hipStreamSynchronize(table->own_stream);
  if (e != hipSuccess) return tfe::fail(TFE_ERR_HIP, "reset stats: %s", hipGetErrorString(e));
  return TFE_OK;
}

tfe_status tfe_residency(const tfe_table* table, const int32_t* rows, int64_t n, int32_t* out,
                         void* stream) {
  tfe::begin_call();
  if (!table) return tfe::fail(TFE_ERR_INVALID_ARG, "null table");
  if (n < 0 || n > 0x7FFFFFFF00ll) return tfe::fail(TFE_ERR_INVALID_ARG, "bad n");
  if (n > 0 && (!rows || !out)) return tfe::fail(TFE_ERR_INVALID_ARG, "null rows or out");
  tfe_status st = tfe::check_device(table);
  if (st != TFE_OK) return st;
  if (n == 0) return TFE_OK;
  hipStream_t s = (hipStream_t)stream;
  tfe_table* t = const_cast<tfe_table*>(table);  // events only
  if (t->cache_rows > 0) {
    // After the table's last lookup and a pending prefetch.
    if (t->lookup_recorded && s != t->last_stream) {
      hipError_t e = hipEventRecord(t->ev_lookup, t->last_stream);
      if (e == hipSuccess) e = hipStreamWaitEvent(s, t->ev_lookup, 0);
      if (e != hipSuccess) return tfe::fail(TFE_ERR_HIP, "residency: %s", hipGetErrorString(e));
    }
    if (t->prefetch_pending) {
      const hipError_t e = hipStreamWaitEvent(s, t->ev_prefetch, 0);
      if (e != hipSuccess) return tfe::fail(TFE_ERR_HIP, "residency: %s", hipGetErrorString(e));
    }
    if (t->pf_counted_pending && s != t->pf_stream) {
      st = tfe::order_after_counted(t, s, false, true);
      if (st != TFE_OK) return st;
    }
  }
  const hipError_t e = tfe::launch_residency(t->cache_rows > 0 ? t->d_where : nullptr,
                                             t->n_phrases, rows, n, out, s);
  if (e != hipSuccess) return tfe::fail(TFE_ERR_HIP, "residency: %s", hipGetErrorString(e));
  return TFE_OK;
}


}  // extern "C"
