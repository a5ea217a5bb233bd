// Internal declarations of libtfe (not part of the C ABI).
#pragma once
#include <stdarg.h>
#include <stdint.h>

#include "../../include/tfe.h"
#include "tfe_index.h"

#if defined(__HIPCC__) || defined(__HIP_PLATFORM_AMD__)
#include <hip/hip_runtime_api.h>
#endif

namespace tfe {

// Thread-local error message; fail() formats it and returns the status.
tfe_status fail(tfe_status st, const char* fmt, ...);
// Clears the message; every C-ABI call starts with it, which also restarts
// the call's allocation count.
void clear_error();
const char* last_error();

// Staging of pageable host rows.  Rows at or beyond a tiered table's pinned
// rows live in pageable host memory, which the GPU cannot address; a wave
// that needs one takes a ticket, and slot ticket mod kStageSlots of a queue
// in coherent pinned host memory carries the request to the table's host
// threads, which copy the row into the slot's staging row.  A requester
// posts into a slot only once the slot's previous ticket has been read
// (acknowledged in a word of its own, which only requesters use), so a
// staging row is never overwritten while it is read.
struct StageSlot {
  unsigned long long req;   // requester: ((ticket + 1) mod 2^32) << 32 | row, one store
  unsigned long long done;  // host: ticket + 1 once the staging row holds the row
};
constexpr uint32_t kStageSlots = 4096;  // requests in flight at most

// The request word of `ticket` for row id `row` (0 never is one).
TFE_HD unsigned long long stage_request(unsigned long long ticket, int32_t row) {
  return (((ticket + 1) & 0xFFFFFFFFull) << 32) | (uint32_t)row;
}

// The serving loop of one host thread: tickets first, first + step, ... in
// order, until *stop.  Row r >= first_row is copied from
// pageable + (r - first_row) * row_bytes into rows + slot * row_bytes; other
// ids (never asked for) read as zeros.
void stage_serve(StageSlot* q, char* rows, const char* pageable, int64_t first_row,
                 int64_t n_rows, size_t row_bytes, uint64_t first, uint64_t step,
                 const volatile bool* stop);

// Allocation-failure hook: with TFE_FAIL_ALLOC=k in the environment, the
// k-th allocation of a library call (counted from its clear_error) fails as
// if memory had run out.  Every allocation asks this first.
bool alloc_fails();
// Device and pinned-host bytes the library holds, across all tables.
void note_alloc(const void* p, size_t n, bool pinned);
void note_free(const void* p);
void memory_held(int64_t* device_bytes, int64_t* pinned_bytes);

int64_t index_capacity(int64_t n, double lf);
tfe_status validate_phrases(const int32_t* tokens, const uint8_t* lens, int64_t P, int n_min,
                            int n_max, int vocab);
tfe_status build_index(const int32_t* tokens, const uint8_t* lens, int64_t P, int n_max,
                       tfe_slot* slots, int64_t cap);

#if defined(__HIPCC__) || defined(__HIP_PLATFORM_AMD__)

// TFE_ERR_UNSUPPORTED if `stream` is being captured into a graph (for calls
// that keep per-call host state or synchronise), TFE_ERR_HIP if the query
// fails, else TFE_OK.
tfe_status refuse_capture(hipStream_t stream, const char* what);

// Starts a C-ABI call that uses the HIP runtime: clears the message and the
// call's allocation count, and discards an error status that HIP calls made
// outside the library left on this thread (launches are checked with
// hipGetLastError, which would report it as theirs).
inline void begin_call() {
  clear_error();
  (void)hipGetLastError();
}

// The library's only ways to get and give back device and pinned host
// memory: they honour the failure hook and keep the held-memory count.
hipError_t dev_malloc(void** p, size_t n);
void dev_free(void* p);
hipError_t pinned_malloc(void** p, size_t n, unsigned flags = hipHostMallocDefault);
void pinned_free(void* p);

// Host side of the pageable-row staging: a coherent pinned queue of
// kStageSlots slots and staging rows, served by host threads that copy the
// requested rows out of the caller's pageable memory.
struct Stager;
struct StageSlot;
// Starts the queue and `threads` host threads for rows [pinned_rows, P) at
// `pageable` (row_bytes each); *out owns them.
tfe_status stager_start(const void* pageable, int64_t pinned_rows, int64_t n_phrases,
                        size_t row_bytes, int threads, Stager** out);
// Device addresses of the queue and of the staging rows.
StageSlot* stager_queue(const Stager* s);
const void* stager_rows(const Stager* s);
// Stops and joins the threads and frees the queue (the table's work that
// may still post requests must be finished).
void stager_stop(Stager* s);

// Per-call arguments of the lookup + inject kernels.
struct LookupArgs {
  const tfe_slot* slots;
  uint64_t bucket_mask;       // buckets - 1
  const void* values;         // resident value rows [P x dim]
  const int32_t* tokens;      // [B x W]
  uint32_t T;                 // B * S (< 2^31)
  int32_t S, ctx, W;          // W = ctx + S
  int32_t n_min, n_max, vocab;
  const void* hin;
  void* hout;
  int32_t inplace;
  uint8_t* hit;
  int32_t* slot_out;
  uint8_t* len_out;           // may be null
  int32_t gate;
  float scale;
  float inv_d;                // 1 / dim
  float inv_sqrt_d;           // 1 / sqrt(dim)
  int32_t weighting;          // multi-match kernel: tfe_weighting
  // Resident tables: matched-position counters, kHitCounters of them
  // kHitStride words apart; null for tiered tables, whose resolve kernels
  // count their own.  Blocks add to counter blockIdx mod kHitCounters, so a
  // launch's additions are spread thin (with 64 counters, same-address
  // additions cost 2% of the stacked decode launch; with 4096, 0.5%).
  unsigned long long* hit_ctr;
};
constexpr int kHitCounters = 4096;
constexpr int kHitStride = 1;

// Device-side bookkeeping of a tiered table (see tfe_tiered.hip).
struct TierStats {
  unsigned long long positions, hits, cache_hits, cache_misses, prefetch_keys, prefetch_found,
      prefetch_filled, prefetch_used, host_bytes, prefetch_dropped;
};
struct TierCtl {
  unsigned long long head, tail;  // recency ring cursors (monotone)
  unsigned long long njobs;       // host -> cache copies of the current call
  unsigned long long call_head;   // long calls: ring head before the call's appends
  unsigned int arrive;            // one-launch decode: waves done with their position
  unsigned int wait_timeouts;     // device-side ordering waits that hit their bound
  // Device-side ordering of decode lookups and prefetches (no HIP events):
  unsigned long long lk_done;     // decode calls done with the shared state (monotone)
  unsigned long long pf_done;     // prefetch copy blocks done (monotone)
  unsigned long long stage_ticket;  // pageable rows: staging requests issued (monotone)
  TierStats stats;
};

struct TierJob {
  int32_t row, slot;
};
struct TierArgs {
  LookupArgs look;            // probe and inject arguments of the call
  const void* host_values;    // device address of the pinned host rows [P x dim]
  void* cache;                // HBM cache [C x dim]
  int32_t* where;             // [P]  slot or -1
  int32_t* owner;             // [C + kDecodeMaxT]  row or -1 (physical slots)
  uint32_t* stamp;            // [C + kDecodeMaxT]  clock of the last reference
  uint8_t* pref;              // [C]  filled by a prefetch and not used yet
  uint64_t* ring;             // recency ring of (slot << 32 | stamp)
  uint64_t ring_mask;
  TierCtl* ctl;
  int32_t* row_of;            // [cap] matched row per position / candidate
  int32_t* slot_of;           // [cap]
  uint8_t* phase;             // [cap]
  TierJob* jobs;              // [cap]
  uint64_t* hkey;             // [2 cap] long calls: call-wide row table (clock << 32 | row)
  uint64_t* hpos;             // [2 cap] its first positions (clock << 32 | ~position)
  uint64_t* hval;             // [2 cap] scored prefetch: best score (clock << 32 | bits)
  uint64_t hmask;             // 2 cap - 1
  uint64_t* blk;              // [cap / 1024 + 1] per-block first-position counts
  int32_t* spare;             // one-launch decode: [kDecodeMaxT] spare cache slot of each
                              // position (slots C .. C + kDecodeMaxT - 1 at load)
  uint32_t clock;
  uint32_t row_bytes;
  uint32_t fill_inline;       // the inject writes missed rows into their slots
  uint32_t prefetch;          // resolve kernels: the call is a prefetch (fills are marked
                              // prefetched; prefetch counters instead of lookup counters)
  // Device-side ordering: wait until ctl->lk_done >= wait_lk and ctl->pf_done
  // >= wait_pf before touching the shared state (0: no wait); count_* make
  // a decode call and the copy blocks count themselves in when done.
  unsigned long long wait_lk, wait_pf;
  uint32_t count_lookup, count_fill;
  // Rows [pinned_rows, P) are pageable: read through the staging queue.
  uint32_t pinned_rows;       // P when every row is pinned
  StageSlot* stage;           // device address of the queue [kStageSlots]
  unsigned long long* stage_ack;  // [kStageSlots] device memory: ticket + 1 of the last read
  const void* stage_rows;     // device address of the staging rows [kStageSlots x dim]
};

// Phase bit of a position whose inject writes its row into slot_of (inline
// fill: the first position of each row filled by the call).
constexpr uint8_t kPhaseWrite = 0x10;

hipError_t launch_tier_init(const TierArgs& t, uint32_t C, uint32_t prefill, hipStream_t s);
hipError_t launch_ring_compact(const TierArgs& t, uint64_t* dst, uint64_t dst_mask,
                               bool restamp, hipStream_t s);
hipError_t launch_tier_probe(const TierArgs& t, hipStream_t s);
// Calls of at most lookup_resolve_one_block_max() positions: one block;
// longer calls: the multi-block pipeline (mark, first, pop, assign).
uint32_t lookup_resolve_one_block_max();
hipError_t launch_resolve_lookup(const TierArgs& t, hipStream_t s);
// Decode-sized lookups: probe + resolve in one single-block launch.
bool lookup_resolve_fused(uint32_t T);
// Decode-sized lookups with inline fill: the whole call (probe, inject,
// residency) in one launch, for T <= kDecodeMaxT.
constexpr uint32_t kDecodeMaxT = 64;
hipError_t launch_tier_decode(const TierArgs& t, int dtype, int dim, hipStream_t s);
hipError_t launch_lookup_resolve_small(const TierArgs& t, hipStream_t s);
hipError_t launch_prefetch_probe(const TierArgs& t, const int32_t* tail, int32_t tail_len,
                                 const int32_t* cand, uint32_t B, uint32_t K, hipStream_t s);
hipError_t launch_resolve_prefetch_scored(const TierArgs& t, uint32_t N, const float* prob,
                                         uint32_t budget, hipStream_t s);
uint32_t scored_prefetch_budget_max();
// Prefetches of at most prefetch_fused_max() candidates run as one
// single-block launch (probe, residency, copies).
uint32_t prefetch_fused_max();
hipError_t launch_prefetch_fused(const TierArgs& t, const int32_t* tail, int32_t tail_len,
                                 const int32_t* cand, uint32_t B, uint32_t K, const float* prob,
                                 uint32_t budget, hipStream_t s);
// out[i] = where[rows[i]] (where = null: rows[i]); -2 outside [0, P).
hipError_t launch_residency(const int32_t* where, int64_t P, const int32_t* rows, int64_t n,
                            int32_t* out, hipStream_t s);
hipError_t launch_fill(const TierArgs& t, int dtype, int dim, uint32_t max_jobs, hipStream_t s);
// Blocks of one fill launch (each counts itself into ctl->pf_done when
// t.count_fill is set).
uint32_t fill_blocks(uint32_t max_jobs);
// One wave that waits for ctl->lk_done >= t.wait_lk and ctl->pf_done >=
// t.wait_pf: orders the following kernels of its stream after them.
hipError_t launch_tier_wait(const TierArgs& t, hipStream_t s);
hipError_t launch_tier_inject(const TierArgs& t, int dtype, int dim, hipStream_t s);

// Launches the fused resident-table kernel; returns the launch error.
hipError_t launch_lookup_inject(const LookupArgs& a, int dtype, int dim, hipStream_t stream);
// Multi-match variant: `hit` receives the match mask, `slot_out` the
// [T x (n_max - n_min + 1)] row ids.
hipError_t launch_lookup_inject_multi(const LookupArgs& a, int dtype, int dim,
                                      hipStream_t stream);

// True if (dtype, dim) has a kernel instantiation.
bool dim_supported(int dtype, int dim);

#endif

}  // namespace tfe

#if defined(__HIPCC__) || defined(__HIP_PLATFORM_AMD__)
struct tfe_table {
  int device = 0;
  int cus = 256;                 // compute units of `device`
  int64_t n_phrases = 0;
  int32_t n_min = 2, n_max = 3, vocab = 0, dim = 0, dtype = 0;
  int64_t capacity = 0;          // index slots
  tfe_slot* d_slots = nullptr;   // [capacity]
  void* d_values = nullptr;      // resident: [P x dim]
  tfe_stats stats = {};          // host-side counters (calls, resident positions)
  unsigned long long* d_hit_ctr = nullptr;  // resident: [kHitCounters * kHitStride]
  hipStream_t own_stream = nullptr;  // the table's own stream: uploads, stats, fills

  // Tiered mode (cache_rows > 0).
  int64_t cache_rows = 0;
  int64_t prefill_rows = 0;
  int32_t fill_mode = 0;         // tfe_fill_mode
  void* h_values = nullptr;      // pinned host rows [pinned_rows x dim]
  const void* h_values_dev = nullptr;
  bool own_h_values = false;
  int64_t pinned_rows = 0;       // rows [pinned_rows, P) are pageable (caller's memory)
  tfe::Stager* stager = nullptr;  // queue and host threads of the pageable rows
  unsigned long long* d_stage_ack = nullptr;  // [kStageSlots] with a stager
  void* d_cache = nullptr;
  int32_t* d_where = nullptr;
  int32_t* d_owner = nullptr;
  uint32_t* d_stamp = nullptr;
  uint8_t* d_pref = nullptr;
  uint64_t* d_ring = nullptr;
  uint64_t* d_ring2 = nullptr;
  uint64_t ring_cap = 0;         // entries, power of two
  uint64_t ring_bound = 0;       // upper bound of ring occupancy (host view)
  tfe::TierCtl* d_ctl = nullptr;
  int32_t* d_row_of = nullptr;
  int32_t* d_slot_of = nullptr;
  uint8_t* d_phase = nullptr;
  tfe::TierJob* d_jobs = nullptr;
  uint64_t* d_hkey = nullptr;    // [2 scratch_cap]
  uint64_t* d_hpos = nullptr;    // [2 scratch_cap]
  uint64_t* d_hval = nullptr;    // [2 scratch_cap]
  uint64_t* d_blk = nullptr;     // [scratch_cap / 1024 + 1]
  int32_t* d_spare = nullptr;    // [kDecodeMaxT] spare slots of the one-launch decode
  // Per-call scratch of prefetches, apart from the lookups' (a prefetch's
  // probe runs while a decode lookup on another stream may still use its
  // own): matched row, matched length / phase, slot, fill list.
  int32_t* d_pf_row_of = nullptr;
  int32_t* d_pf_slot_of = nullptr;
  uint8_t* d_pf_phase = nullptr;
  tfe::TierJob* d_pf_jobs = nullptr;
  uint32_t pf_cap = 0;
  uint32_t scratch_cap = 0;
  uint32_t clock = 0;
  hipEvent_t ev_resolved = nullptr, ev_filled = nullptr, ev_lookup = nullptr,
             ev_prefetch = nullptr;
  bool lookup_recorded = false, prefetch_pending = false, fill_recorded = false;
  hipStream_t last_stream = nullptr;   // stream of the last lookup (lookup_recorded)
  // Device-side ordering of one-launch decode lookups and one-block
  // prefetches: totals submitted, compared by the kernels with ctl->lk_done
  // and ctl->pf_done.
  uint64_t decodes_issued = 0;   // one-launch decode calls submitted
  uint64_t fills_issued = 0;     // counted prefetch copy blocks submitted
  bool last_lookup_counted = false;  // the last lookup was a counted decode
  bool counting = false;             // decodes count themselves (from the first prefetch on)
  bool pf_counted_pending = false;   // a counted prefetch may still run
  hipStream_t pf_stream = nullptr;   // stream of the last counted prefetch
};
#endif
