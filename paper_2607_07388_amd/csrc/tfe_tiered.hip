// Tiered tables: HBM cache of value rows in front of pinned host memory
// (paper Sec. 4.3, Eq. 12; the SSD tier is not built), with exact
// least-recently-used replacement kept entirely on the device, and the
// prefetch of predicted next-token phrases (Sec. 4.4, Eq. 14-16).
//
// Residency (the second level of Eq. 10: phrase id -> tier and offset):
//   where[row]   cache slot holding the row, or -1 (host only)
//   owner[slot]  row held by the slot, or -1 (empty)
//   stamp[slot]  clock of the last call that referenced the slot
// Recency order: a ring of (slot, stamp) entries in the order the slots were
// last referenced.  An entry is live while stamp[slot] still equals its
// stamp; a slot referenced again gets a new entry and its old one dies.  The
// least recent slot is the first live entry from the tail.  Every slot has
// exactly one live entry, so compaction (dropping dead entries) leaves
// exactly `cache_rows` entries.
//
// A lookup call runs: probe (wide) -> resolve (one block: residency, victim
// choice, fill list, recency update, all in position order so the policy is
// deterministic) -> inject (wide; cached rows from HBM, the others straight
// from pinned host memory over PCIe).  A missed row given a slot is written
// into it either by the inject itself, from the copy it read (inline fill),
// or by a copy kernel on a side stream that reads it from host memory again;
// the next call waits for that copy, nothing in this call does.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tfe_device.h"
#include "tfe_internal.h"

namespace tfe {
namespace {

using dev::u32x4;

constexpr int kResolveThreads = 1024;
constexpr int kHashSize = 2048;  // open-addressing dedupe table in LDS

constexpr int kWaves = kResolveThreads / 64;

// Number of set bits of the ballot m in the lanes below this one.
__device__ __forceinline__ uint32_t lanes_below(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                   __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// Block-wide rank of a flag among the block's threads and its total, and
// the lowest thread index whose flag is set: the one-item forms of
// block_count_n (defined below).  All threads must call them.
template <int N>
__device__ __forceinline__ void block_count_n(const bool* f, uint32_t* rank, uint32_t* total,
                                              const bool* g = nullptr, uint32_t* first = nullptr);

__device__ __forceinline__ uint32_t block_count(bool f, uint32_t* total) {
  uint32_t rank;
  block_count_n<1>(&f, &rank, total, nullptr, nullptr);
  return rank;
}

__device__ __forceinline__ uint32_t block_first(bool f) {
  uint32_t rank, total, first;
  const bool none = false;
  block_count_n<1>(&none, &rank, &total, &f, &first);
  return first;
}

__device__ __forceinline__ uint64_t ring_entry(uint32_t slot, uint32_t stamp) {
  return ((uint64_t)slot << 32) | stamp;
}

// Device-scope (coherent across the XCDs' L2s) store and load.
__device__ __forceinline__ void st_dev(int32_t* p, int32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int32_t ld_dev(const int32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Waits until every memory operation this wave issued has completed
// (s_waitcnt vmcnt(0); the other counters left at their maximum).
__device__ __forceinline__ void wait_mem() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Device-side ordering between a one-launch decode lookup and a one-block
// prefetch on different streams, instead of HIP events (whose record and
// cross-stream wait cost about 20 us of host time per prefetch here).  A
// waiter only ever waits for work that the host submitted before it, so
// the waits end; each is bounded all the same (kWaitLimit sleeps, about a
// second), and a wait that hits the bound is counted in ctl->wait_timeouts
// (tfe_get_stats then reports an error).
constexpr uint32_t kWaitLimit = 1u << 22;

// One thread: waits until *ctr >= want.
__device__ __forceinline__ void wait_at_least(TierCtl* ctl, unsigned long long* ctr,
                                              unsigned long long want) {
  uint32_t n = 0;
  while (__hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < want) {
    __builtin_amdgcn_s_sleep(8);
    if (++n == kWaitLimit) {
      atomicAdd(&ctl->wait_timeouts, 1u);
      break;
    }
  }
}

// Called by every thread of a block: the block's thread 0 waits for
// ctl->lk_done >= t.wait_lk and ctl->pf_done >= t.wait_pf, then every wave
// drops its stale cache lines (agent-scope acquire) before reading state
// that the awaited kernels wrote.
__device__ __forceinline__ void wait_ordered_block(const TierArgs& t) {
  if (!t.wait_lk && !t.wait_pf) return;  // block-uniform
  if (threadIdx.x == 0) {
    if (t.wait_lk) wait_at_least(t.ctl, &t.ctl->lk_done, t.wait_lk);
    if (t.wait_pf) wait_at_least(t.ctl, &t.ctl->pf_done, t.wait_pf);
  }
  __syncthreads();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
}

// Reads a value row that is not cached.  Rows below t.pinned_rows are read
// straight from pinned host memory (zero-copy over PCIe; NT: non-temporal).
// Rows at or beyond it are pageable: the wave's first lane takes a ticket,
// waits until the ticket's queue slot is free (the slot's previous ticket
// has been read: its ack word in device memory), posts ticket and row in
// one word, and waits until a host thread has staged the row; the whole
// wave then reads the staged row and the first lane frees the slot.  The
// queue and the staged rows are coherent host memory, written, polled and
// read with system-scope accesses (sc0 sc1) that bypass the GPU caches; no
// fence is needed, and none is used: a system-scope acquire would
// invalidate the whole L2 once per staged row.  The polls back off -- about 0.4 us apart at first,
// then 1.7, 3.4 and at last 54 us -- so that the thousands of waves of a
// long call that wait behind each other in the queue do not crowd the host
// link with reads (polling every few microseconds, 2000 waves read about
// 40 GB/s and starve both the polls and the zero-copy row reads).
// The waits are bounded (seconds); one that runs out is counted in
// ctl->wait_timeouts (tfe_get_stats then reports an error) and the row
// reads as zeros.  `row` is wave-uniform.
constexpr uint32_t kStageWaitLimit = 1u << 17;  // polls: seconds at the longest interval

__device__ __forceinline__ bool wait_host_done(TierCtl* ctl, const unsigned long long* p,
                                               unsigned long long want) {
  for (uint32_t n = 0; n < kStageWaitLimit; ++n) {
    if (__hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM) == want) return true;
    if (n < 4) {
      __builtin_amdgcn_s_sleep(16);
    } else if (n < 16) {
      __builtin_amdgcn_s_sleep(64);
    } else if (n < 48) {
      __builtin_amdgcn_s_sleep(127);
    } else {
      for (int k = 0; k < 16; ++k) __builtin_amdgcn_s_sleep(127);
    }
  }
  atomicAdd(&ctl->wait_timeouts, 1u);
  return false;
}

__device__ __forceinline__ bool wait_slot_free(TierCtl* ctl, const unsigned long long* p,
                                               unsigned long long want) {
  for (uint32_t n = 0; n < kStageWaitLimit; ++n) {
    if (__hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == want) return true;
    __builtin_amdgcn_s_sleep(64);
  }
  atomicAdd(&ctl->wait_timeouts, 1u);
  return false;
}

template <int NCH, bool NT>
__device__ __forceinline__ void read_host_row(const TierArgs& t, int32_t row, u32x4* v,
                                              int lane) {
  constexpr int ROW_VECS = NCH * 64;
  if ((uint32_t)row < t.pinned_rows) {
    const u32x4* src = (const u32x4*)t.host_values + (size_t)row * ROW_VECS;
#pragma unroll
    for (int k = 0; k < NCH; ++k)
      v[k] = NT ? __builtin_nontemporal_load(src + k * 64 + lane) : src[k * 64 + lane];
    return;
  }
  unsigned long long tk = 0;
  uint32_t slot = 0, ok = 0;
  if (lane == 0) {
    tk = __hip_atomic_fetch_add(&t.ctl->stage_ticket, 1ull, __ATOMIC_RELAXED,
                                __HIP_MEMORY_SCOPE_AGENT);
    slot = (uint32_t)(tk % kStageSlots);
    ok = wait_slot_free(t.ctl, t.stage_ack + slot,
                        tk >= kStageSlots ? tk + 1 - kStageSlots : 0ull);
    if (ok) {
      __hip_atomic_store(&t.stage[slot].req, stage_request(tk, row), __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_SYSTEM);
      ok = wait_host_done(t.ctl, &t.stage[slot].done, tk + 1);
    }
  }
  slot = __builtin_amdgcn_readfirstlane(slot);
  ok = __builtin_amdgcn_readfirstlane(ok);
  // Buffer loads with cache policy sc0 | sc1 (= 1 | 16): read from host
  // memory, past the L2.  The resource covers the slot's staging row.
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
      (void*)((const u32x4*)t.stage_rows + (size_t)slot * ROW_VECS), (short)0, ROW_VECS * 16,
      0x00020000);
#pragma unroll
  for (int k = 0; k < NCH; ++k)
    v[k] = ok ? (u32x4)__builtin_amdgcn_raw_buffer_load_b128(rs, (k * 64 + lane) * 16, 0, 17)
              : u32x4{0u, 0u, 0u, 0u};
  wait_mem();
  if (lane == 0 && ok)
    __hip_atomic_store(t.stage_ack + slot, tk + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Takes up to `need` least-recent slots not referenced in this call (stamp
// below the call's clock) from the tail of the ring into vict[0..got).
// Dead entries passed on the way are dropped.  Returns got (block-uniform).
__device__ uint32_t pop_victims(const TierArgs& t, uint32_t need, uint32_t* vict) {
  __shared__ unsigned long long s_tail, s_head, s_last;
  __shared__ uint32_t s_got, s_stop;
  if (threadIdx.x == 0) {
    s_tail = t.ctl->tail;
    s_head = t.ctl->head;
    s_got = 0;
    s_stop = 0;
  }
  __syncthreads();
  for (;;) {
    const uint32_t got = s_got;
    const unsigned long long base = s_tail, head = s_head;
    if (got >= need || s_stop || base >= head) break;
    const unsigned long long i = base + threadIdx.x;
    const bool in = i < head;
    const uint64_t e = in ? t.ring[i & t.ring_mask] : 0;
    const uint32_t slot = (uint32_t)(e >> 32), st = (uint32_t)e;
    const bool cur = in && st == t.clock;  // entries of this call end the search
    const bool live = in && !cur && t.stamp[slot] == st;
    uint32_t nlive;
    const uint32_t rank = block_count(live, &nlive);
    const uint32_t first_cur = block_first(cur);
    const uint32_t take = nlive < need - got ? nlive : need - got;
    if (live && rank < take) {
      vict[got + rank] = slot;
      if (rank == take - 1) s_last = i;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      if (take > 0 && take == need - got) {
        s_tail = s_last + 1;
        s_got = need;
      } else {
        s_got = got + take;
        if (first_cur != 0xFFFFFFFFu) {
          s_tail = base + first_cur;
          s_stop = 1;
        } else {
          s_tail = head < base + kResolveThreads ? head : base + kResolveThreads;
        }
      }
    }
    __syncthreads();
  }
  const uint32_t got = s_got;
  if (threadIdx.x == 0) t.ctl->tail = s_tail;
  __syncthreads();
  return got;
}

// First occurrence of each row among the block's positions: returns true for
// the lowest position naming the row, and the row's entry index in the LDS
// table in *hidx (-1 for rows < 0), where callers keep per-row results.
__device__ bool first_of_row(int32_t r, uint32_t pos, int32_t* hkey, uint32_t* hpos, int* hidx) {
  for (int i = threadIdx.x; i < kHashSize; i += kResolveThreads) {
    hkey[i] = -1;
    hpos[i] = 0xFFFFFFFFu;
  }
  __syncthreads();
  int h = -1;
  if (r >= 0) {
    h = (int)(((uint32_t)r * 2654435761u) >> 21) & (kHashSize - 1);
    for (;;) {
      const int old = atomicCAS(&hkey[h], -1, r);
      if (old == -1 || old == r) break;
      h = (h + 1) & (kHashSize - 1);
    }
    atomicMin(&hpos[h], pos);
  }
  __syncthreads();
  const bool first = r >= 0 && hpos[h] == pos;
  *hidx = h;
  return first;
}

// Versions of the block helpers for N items per thread: item k of thread x
// stands for index k * kResolveThreads + x, and counts and minima follow
// that index order.
//
// Ranks of the set flags (rank[k] = set flags at lower indices) and their
// total.  All threads must call it.
//
// With g non-null, *first also receives the lowest index whose g flag is
// set (0xFFFFFFFF if none), from the same exchange.
template <int N>
__device__ __forceinline__ void block_count_n(const bool* f, uint32_t* rank, uint32_t* total,
                                              const bool* g, uint32_t* first) {
  static_assert(kWaves == 16, "one DPP row holds the per-wave counts");
  __shared__ uint32_t s_n[N][kWaves];
  __shared__ uint32_t s_f[kWaves];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  uint64_t m[N];
#pragma unroll
  for (int k = 0; k < N; ++k) {
    m[k] = __builtin_amdgcn_ballot_w64(f[k]);
    if (lane == 0) s_n[k][wave] = (uint32_t)__builtin_popcountll(m[k]);
  }
  if (g) {
    uint32_t best = 0xFFFFFFFFu;
#pragma unroll
    for (int k = N - 1; k >= 0; --k) {
      const uint64_t mg = __builtin_amdgcn_ballot_w64(g[k]);
      if (mg)
        best = (uint32_t)k * kResolveThreads + (uint32_t)wave * 64u +
               (uint32_t)__builtin_ctzll(mg);
    }
    if (lane == 0) s_f[wave] = best;
  }
  __syncthreads();
  if (g) {
    uint32_t x = lane < kWaves ? s_f[lane] : 0xFFFFFFFFu;
    uint32_t r = x;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) r = min(r, (uint32_t)__builtin_amdgcn_readlane((int)x, w));
    *first = r;
  }
  // Lane w < 16 holds wave w's count; an inclusive scan along the row
  // (DPP shifts by 1, 2, 4, 8) gives every wave's offset by readlane.
  uint32_t run = 0;
#pragma unroll
  for (int k = 0; k < N; ++k) {
    uint32_t x = lane < kWaves ? s_n[k][lane] : 0u;
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xF, 0xF, false);  // row_shr:1
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xF, 0xF, false);  // row_shr:2
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xF, 0xF, false);  // row_shr:4
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xF, 0xF, false);  // row_shr:8
    const uint32_t before = wave > 0 ? (uint32_t)__builtin_amdgcn_readlane((int)x, wave - 1) : 0u;
    const uint32_t all = (uint32_t)__builtin_amdgcn_readlane((int)x, kWaves - 1);
    rank[k] = run + before + lanes_below(m[k]);
    run += all;
  }
  __syncthreads();
  *total = run;
}

// pop_victims over windows of N kResolveThreads ring entries per round;
// out(i, slot, owner) receives victim i and the row its slot holds (read
// with its stamp).
template <int N, class Out>
__device__ __forceinline__ uint32_t pop_victims_n(const TierArgs& t, uint32_t need, Out out) {
  __shared__ unsigned long long s_tail, s_head, s_last;
  __shared__ uint32_t s_got, s_stop;
  if (threadIdx.x == 0) {
    s_tail = t.ctl->tail;
    s_head = t.ctl->head;
    s_got = 0;
    s_stop = 0;
  }
  __syncthreads();
  for (;;) {
    const uint32_t got = s_got;
    const unsigned long long base = s_tail, head = s_head;
    if (got >= need || s_stop || base >= head) break;
    // Unconditional loads (the ring index wraps in bounds; entries past the
    // head read slot 0's stamp), issued back to back.
    uint64_t e[N];
#pragma unroll
    for (int k = 0; k < N; ++k) {
      const unsigned long long i = base + (uint64_t)k * kResolveThreads + threadIdx.x;
      const uint64_t x = t.ring[i & t.ring_mask];
      e[k] = i < head ? x : 0;
    }
    uint32_t st_now[N];
    int32_t own[N];
#pragma unroll
    for (int k = 0; k < N; ++k) {
      st_now[k] = t.stamp[(uint32_t)(e[k] >> 32)];
      own[k] = t.owner[(uint32_t)(e[k] >> 32)];
    }
    bool live[N], cur[N];
#pragma unroll
    for (int k = 0; k < N; ++k) {
      const unsigned long long i = base + (uint64_t)k * kResolveThreads + threadIdx.x;
      const bool in = i < head;
      cur[k] = in && (uint32_t)e[k] == t.clock;  // entries of this call end the search
      live[k] = in && !cur[k] && st_now[k] == (uint32_t)e[k];
    }
    uint32_t rank[N], nlive, first_cur;
    block_count_n<N>(live, rank, &nlive, cur, &first_cur);
    const uint32_t take = nlive < need - got ? nlive : need - got;
#pragma unroll
    for (int k = 0; k < N; ++k) {
      if (live[k] && rank[k] < take) {
        out(got + rank[k], (uint32_t)(e[k] >> 32), own[k]);
        if (rank[k] == take - 1) s_last = base + (uint64_t)k * kResolveThreads + threadIdx.x;
      }
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      if (take > 0 && take == need - got) {
        s_tail = s_last + 1;
        s_got = need;
      } else {
        s_got = got + take;
        if (first_cur != 0xFFFFFFFFu) {
          s_tail = base + first_cur;
          s_stop = 1;
        } else {
          const unsigned long long end = base + (uint64_t)N * kResolveThreads;
          s_tail = head < end ? head : end;
        }
      }
    }
    __syncthreads();
  }
  const uint32_t got = s_got;
  if (threadIdx.x == 0) t.ctl->tail = s_tail;
  __syncthreads();
  return got;
}

// first_of_row for N positions per thread and an LDS table of HS entries
// (a power of two, at least twice the block's positions).
template <int N, int HS>
__device__ __forceinline__ void first_of_rows(const int32_t* r, const uint32_t* pos, int32_t* hkey,
                              uint32_t* hpos, int* hidx, bool* first) {
  static_assert((HS & (HS - 1)) == 0 && HS >= 2 * N * kResolveThreads, "hash size");
  constexpr int shift = 32 - __builtin_ctz(HS);
  for (int i = threadIdx.x; i < HS; i += kResolveThreads) {
    hkey[i] = -1;
    hpos[i] = 0xFFFFFFFFu;
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < N; ++k) {
    int h = -1;
    if (r[k] >= 0) {
      h = (int)(((uint32_t)r[k] * 2654435761u) >> shift);
      for (;;) {
        const int old = atomicCAS(&hkey[h], -1, r[k]);
        if (old == -1 || old == r[k]) break;
        h = (h + 1) & (HS - 1);
      }
      atomicMin(&hpos[h], pos[k]);
    }
    hidx[k] = h;
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < N; ++k) first[k] = r[k] >= 0 && hpos[hidx[k]] == pos[k];
}

// Number of set flags in the wave, added once per wave to an LDS counter
// (one atomic per wave instead of one per lane).
__device__ __forceinline__ void wave_tally(bool f, uint32_t* counter) {
  const uint64_t m = __builtin_amdgcn_ballot_w64(f);
  if ((threadIdx.x & 63) == 0 && m) atomicAdd(counter, (uint32_t)__builtin_popcountll(m));
}

// Residency resolution of a lookup call of at most kGroup positions, in one
// block (thread x handles positions k kResolveThreads + x).  A prefetch
// (t.prefetch) is resolved the same way, its candidates standing for the
// positions: it references its cached rows and fills the others, marked
// prefetched.  Per position:
// slot_of (cache slot or -1) and phase (0: cached when the call began, read
// from the cache; 1: filled in this call; 2: not cached, no slot given to
// it; 3: no match).  Rows of phases 1 and 2 are read from host memory by the
// inject; a phase-1 row is also written into its slot, by the inject of its
// first position (inline fill) or by a copy on the side stream.  Every
// cached row of the call marks its slot referenced before any victim is
// chosen, so no slot the call uses is evicted.
constexpr int kGroupItems = 4;
constexpr int kGroup = kGroupItems * kResolveThreads;
constexpr int kGroupHash = 2 * kGroup;

// Returns the number of rows filled (block-uniform); the fill list is
// jobs[0 .. filled).
__device__ uint32_t resolve_one_block(const TierArgs& t, uint32_t T) {
  constexpr int N = kGroupItems;
  __shared__ int32_t hkey[kGroupHash];
  __shared__ uint32_t hpos[kGroupHash];
  __shared__ int32_t hslot[kGroupHash];    // per row: its slot after this call (-1: none)
  __shared__ uint8_t hphase[kGroupHash];
  __shared__ uint32_t vict[kGroup];
  __shared__ int32_t vown[kGroup];  // row held by each victim slot
  __shared__ uint32_t s_cnt[4];  // hits, cache hits, prefetch used, host-served
  if (threadIdx.x < 4) s_cnt[threadIdx.x] = 0;
  const unsigned long long head0 = t.ctl->head;
  int32_t r[N];
  uint32_t pos[N];
#pragma unroll
  for (int k = 0; k < N; ++k) {
    pos[k] = k * kResolveThreads + threadIdx.x;
    const int32_t rr = t.row_of[pos[k] < T ? pos[k] : 0u];
    r[k] = pos[k] < T ? rr : -1;
  }
  int h[N];
  bool fb[N];
  first_of_rows<N, kGroupHash>(r, pos, hkey, hpos, h, fb);
  // First occurrences read the row's slot; a cached row's slot becomes
  // referenced (a stamp of this call keeps it from being a victim).  The
  // rows are distinct and so are their slots, so all reads go before the
  // writes; they are unconditional (index 0 where there is nothing to read)
  // so that they issue back to back.
  int32_t s0[N];
#pragma unroll
  for (int k = 0; k < N; ++k) {
    const int32_t w = t.where[(uint32_t)max(r[k], 0)];
    s0[k] = fb[k] ? w : -1;
  }
  uint32_t pf[N];
#pragma unroll
  for (int k = 0; k < N; ++k) pf[k] = t.pref[(uint32_t)max(s0[k], 0)];
  uint32_t f_app = 0, f_miss = 0;
#pragma unroll
  for (int k = 0; k < N; ++k) {
    bool used = false;
    if (s0[k] >= 0) {
      f_app |= 1u << k;
      t.stamp[s0[k]] = t.clock;
      hslot[h[k]] = s0[k];
      hphase[h[k]] = 0;
      if (pf[k] && !t.prefetch) {  // a lookup uses the prefetched row
        t.pref[s0[k]] = 0;
        used = true;
      }
    } else if (fb[k]) {
      f_miss |= 1u << k;
    }
    wave_tally(used, &s_cnt[2]);
  }
  __threadfence_block();  // this call's stamps, before the ring walk reads them
  __syncthreads();
  bool mb[N];
#pragma unroll
  for (int k = 0; k < N; ++k) mb[k] = (f_miss >> k) & 1u;
  uint32_t mrank[N], need;
  block_count_n<N>(mb, mrank, &need);
  const uint32_t got =
      need ? pop_victims_n<N>(t, need, [&](uint32_t i, uint32_t slot, int32_t own) {
        vict[i] = slot;
        vown[i] = own;
      }) : 0;
  uint32_t f_fill = 0;
#pragma unroll
  for (int k = 0; k < N; ++k) f_fill |= ((f_miss >> k) & 1u) && mrank[k] < got ? 1u << k : 0u;
#pragma unroll
  for (int k = 0; k < N; ++k) {
    if ((f_fill >> k) & 1u) {
      // Evicted rows were cached and filled rows were not: the two sets
      // are disjoint, so these writes never collide.  A victim is never a
      // slot of this call, so its owner is still the one the pop read.
      const uint32_t vk = vict[mrank[k]];
      const int32_t old = vown[mrank[k]];
      if (old >= 0) t.where[old] = -1;
      t.owner[vk] = r[k];
      t.where[r[k]] = (int32_t)vk;
      t.stamp[vk] = t.clock;
      t.pref[vk] = t.prefetch ? 1 : 0;
      t.jobs[mrank[k]] = TierJob{r[k], (int32_t)vk};
      hslot[h[k]] = (int32_t)vk;
      hphase[h[k]] = 1;
      f_app |= 1u << k;
    } else if ((f_miss >> k) & 1u) {
      hslot[h[k]] = -1;
      hphase[h[k]] = 2;
    }
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < N; ++k) {
    const bool valid = pos[k] < T;
    const bool m = r[k] >= 0;
    const int32_t s1 = m ? hslot[h[k]] : -1;
    const uint8_t ph = m ? hphase[h[k]] : 3;
    const bool writes = t.fill_inline && ((f_fill >> k) & 1u);
    if (valid) {
      t.slot_of[pos[k]] = s1;
      t.phase[pos[k]] = writes ? (uint8_t)(ph | kPhaseWrite) : ph;
    }
    wave_tally(m, &s_cnt[0]);
    wave_tally(m && ph == 0, &s_cnt[1]);
    wave_tally(m && ph != 0, &s_cnt[3]);
  }
  bool ab[N];
#pragma unroll
  for (int k = 0; k < N; ++k) ab[k] = (f_app >> k) & 1u;
  uint32_t arank[N], napp;
  block_count_n<N>(ab, arank, &napp);
#pragma unroll
  for (int k = 0; k < N; ++k)
    if ((f_app >> k) & 1u)
      t.ring[(head0 + arank[k]) & t.ring_mask] = ring_entry((uint32_t)hslot[h[k]], t.clock);
  if (threadIdx.x == 0) {
    t.ctl->head = head0 + napp;
    t.ctl->njobs = got;
    TierStats& st = t.ctl->stats;
    if (t.prefetch) {
      st.prefetch_keys += T;
      st.prefetch_found += s_cnt[0];
      st.prefetch_filled += got;
      st.host_bytes += (unsigned long long)got * t.row_bytes;
    } else {
      st.positions += T;
      st.hits += s_cnt[0];
      st.cache_hits += s_cnt[1];
      st.cache_misses += s_cnt[0] - s_cnt[1];
      st.prefetch_used += s_cnt[2];
      st.host_bytes += (unsigned long long)((t.fill_inline ? 0u : got) + s_cnt[3]) * t.row_bytes;
    }
  }
  return got;
}

__global__ __launch_bounds__(kResolveThreads) void k_resolve_lookup(const TierArgs t, uint32_t T) {
  (void)resolve_one_block(t, T);
}

// ---- Resolution of calls longer than kGroup positions, over many blocks.
// The same policy as k_resolve_lookup, in four launches of which only the
// victim pop is a single block:
//   k_res_mark    every position reads its row's slot; a cached row's slot is
//                 stamped referenced; the distinct rows of the block enter a
//                 call-wide hash table that keeps each row's first position;
//   k_res_first   first positions are found; per block, the number of first
//                 positions of cached rows and of missed rows; counters;
//   k_res_pop     those counts are scanned; the missed rows' victims are
//                 taken from the recency ring (least recent first, skipping
//                 referenced slots) into the fill list;
//   k_res_assign  a missed row's first position takes victim number (its
//                 rank among missed first positions) while any are left;
//                 residency and recency entries are written in first-position
//                 order, so the recency update equals the one-block kernel's.
// The hash table lives in the table's scratch and is never cleared: an
// entry holds (clock << 32 | row) and counts as empty unless its clock is
// this call's; the first position is kept as (clock << 32 | ~pos) under an
// atomic maximum, so a stale entry is replaced by any write of this call.
constexpr int kMarkThreads = kResolveThreads;

__device__ __forceinline__ uint64_t gh_home(int32_t r, uint64_t mask) {
  return ((uint64_t)(uint32_t)r * 0x9E3779B97F4A7C15ull >> 29) & mask;
}

__device__ __forceinline__ uint64_t gh_load(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Inserts row r (first seen at position p within its block) into the
// call-wide table.
__device__ void gh_insert(const TierArgs& t, int32_t r, uint32_t p) {
  const uint64_t tag = (uint64_t)t.clock << 32;
  const uint64_t want = tag | (uint32_t)r;
  uint64_t h = gh_home(r, t.hmask);
  for (;;) {
    uint64_t old = gh_load(t.hkey + h);
    // Entries only ever change from another call's to this call's, so a
    // failed exchange returns the entry's final value.
    while (old != want && (old >> 32) != t.clock) {
      const uint64_t prev = atomicCAS((unsigned long long*)(t.hkey + h), (unsigned long long)old,
                                      (unsigned long long)want);
      old = prev == old ? want : prev;
    }
    if (old == want) break;
    h = (h + 1) & t.hmask;
  }
  atomicMax((unsigned long long*)(t.hpos + h), (unsigned long long)(tag | (uint32_t)~p));
}

// True if p is the first position of the call naming row r (r >= 0 was
// inserted by k_res_mark).
__device__ __forceinline__ bool gh_is_first(const TierArgs& t, int32_t r, uint32_t p) {
  const uint64_t tag = (uint64_t)t.clock << 32;
  const uint64_t want = tag | (uint32_t)r;
  uint64_t h = gh_home(r, t.hmask);
  while (gh_load(t.hkey + h) != want) h = (h + 1) & t.hmask;
  return gh_load(t.hpos + h) == (tag | (uint32_t)~p);
}

__global__ __launch_bounds__(kMarkThreads) void k_res_mark(const TierArgs t, uint32_t T) {
  __shared__ int32_t hkey[kHashSize];
  __shared__ uint32_t hpos[kHashSize];
  const uint32_t p = blockIdx.x * kMarkThreads + threadIdx.x;
  const int32_t r = p < T ? t.row_of[p] : -1;
  const int32_t s = r >= 0 ? t.where[r] : -1;
  if (p < T) t.slot_of[p] = s;
  if (s >= 0) t.stamp[s] = t.clock;  // same value from every position naming the row
  int h;
  const bool first_here = first_of_row(r, p, hkey, hpos, &h);
  if (first_here) gh_insert(t, r, p);
}

__global__ __launch_bounds__(kMarkThreads) void k_res_first(const TierArgs t, uint32_t T) {
  __shared__ uint32_t s_cnt[3];  // hits, cache hits, prefetch used
  if (threadIdx.x < 3) s_cnt[threadIdx.x] = 0;
  const uint32_t p = blockIdx.x * kMarkThreads + threadIdx.x;
  const int32_t r = p < T ? t.row_of[p] : -1;
  const int32_t s = p < T ? t.slot_of[p] : -1;
  const bool first = r >= 0 && gh_is_first(t, r, p);
  const bool fc = first && s >= 0, fm = first && s < 0;
  bool used = false;
  if (fc && !t.prefetch && t.pref[s]) {  // a lookup uses the prefetched row
    t.pref[s] = 0;
    used = true;
  }
  __syncthreads();
  wave_tally(r >= 0, &s_cnt[0]);
  wave_tally(r >= 0 && s >= 0, &s_cnt[1]);
  wave_tally(used, &s_cnt[2]);
  uint32_t nc, nm;
  block_count(fc, &nc);
  block_count(fm, &nm);
  if (threadIdx.x == 0) {
    t.blk[blockIdx.x] = ((uint64_t)nm << 32) | nc;
    TierStats& st = t.ctl->stats;
    if (t.prefetch) {
      atomicAdd(&st.prefetch_found, (unsigned long long)s_cnt[0]);
    } else {
      atomicAdd(&st.hits, (unsigned long long)s_cnt[0]);
      atomicAdd(&st.cache_hits, (unsigned long long)s_cnt[1]);
      atomicAdd(&st.cache_misses, (unsigned long long)(s_cnt[0] - s_cnt[1]));
      atomicAdd(&st.prefetch_used, (unsigned long long)s_cnt[2]);
      atomicAdd(&st.host_bytes, (unsigned long long)(s_cnt[0] - s_cnt[1]) * t.row_bytes);
    }
  }
}

// Exclusive scan of blk[0..n) in place (packed counts: each half stays
// below 2^31, so the halves add without carries); returns the total.
__device__ uint64_t block_scan_blk(uint64_t* blk, uint32_t n) {
  __shared__ uint64_t s_w[kWaves];
  __shared__ uint64_t s_run;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  if (threadIdx.x == 0) s_run = 0;
  __syncthreads();
  for (uint32_t base = 0; base < n; base += kResolveThreads) {
    const uint32_t i = base + threadIdx.x;
    const uint64_t v = i < n ? blk[i] : 0;
    uint64_t x = v;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const uint64_t y = __shfl_up(x, d, 64);
      if (lane >= d) x += y;
    }
    if (lane == 63) s_w[wave] = x;
    __syncthreads();
    uint64_t before = s_run;
    for (int w = 0; w < wave; ++w) before += s_w[w];
    if (i < n) blk[i] = before + x - v;
    __syncthreads();
    if (threadIdx.x == kResolveThreads - 1) s_run = before + x;
    __syncthreads();
  }
  return s_run;
}

__global__ __launch_bounds__(kResolveThreads) void k_res_pop(const TierArgs t, uint32_t nblk) {
  const uint64_t tot = block_scan_blk(t.blk, nblk);
  const uint32_t ncf = (uint32_t)tot, need = (uint32_t)(tot >> 32);
  TierJob* jobs = t.jobs;
  const uint32_t got =
      need ? pop_victims_n<kGroupItems>(t, need, [&](uint32_t i, uint32_t slot, int32_t own) {
        jobs[i] = TierJob{own, (int32_t)slot};
      }) : 0;
  if (threadIdx.x == 0) {
    const unsigned long long head0 = t.ctl->head;
    t.ctl->call_head = head0;
    t.ctl->head = head0 + ncf + got;
    t.ctl->njobs = got;
    TierStats& st = t.ctl->stats;
    if (t.prefetch) {
      st.prefetch_filled += got;
      st.host_bytes += (unsigned long long)got * t.row_bytes;
    } else if (!t.fill_inline) {
      st.host_bytes += (unsigned long long)got * t.row_bytes;
    }
  }
}

__global__ __launch_bounds__(kMarkThreads) void k_res_assign(const TierArgs t, uint32_t T) {
  const uint32_t p = blockIdx.x * kMarkThreads + threadIdx.x;
  const int32_t r = p < T ? t.row_of[p] : -1;
  const int32_t s = p < T ? t.slot_of[p] : -1;
  const bool first = r >= 0 && gh_is_first(t, r, p);
  const bool fc = first && s >= 0, fm = first && s < 0;
  uint32_t nc, nm;
  const uint32_t rc = block_count(fc, &nc);
  const uint32_t rm = block_count(fm, &nm);
  const uint64_t off = t.blk[blockIdx.x];
  const uint32_t got = (uint32_t)t.ctl->njobs;
  const unsigned long long head0 = t.ctl->call_head;
  const uint32_t cbefore = (uint32_t)off + rc, mbefore = (uint32_t)(off >> 32) + rm;
  // Appended entries before this position: every cached first position,
  // and the missed first positions that got a slot (the first `got` of them).
  const uint32_t arank = cbefore + (mbefore < got ? mbefore : got);
  uint8_t ph = 3;
  int32_t slot = -1;
  if (r >= 0 && s >= 0) {
    ph = 0;
    slot = s;
    if (fc) t.ring[(head0 + arank) & t.ring_mask] = ring_entry((uint32_t)s, t.clock);
  } else if (r >= 0) {
    ph = 2;
    if (fm && mbefore < got) {
      const TierJob job = t.jobs[mbefore];
      const uint32_t v = (uint32_t)job.slot;
      if (job.row >= 0) t.where[job.row] = -1;
      t.owner[v] = r;
      t.where[r] = (int32_t)v;
      t.stamp[v] = t.clock;
      t.pref[v] = t.prefetch ? 1 : 0;
      t.jobs[mbefore] = TierJob{r, (int32_t)v};
      t.ring[(head0 + arank) & t.ring_mask] = ring_entry(v, t.clock);
      slot = (int32_t)v;
      ph = t.fill_inline ? (uint8_t)(1 | kPhaseWrite) : (uint8_t)1;
    }
  }
  if (p < T) {
    t.slot_of[p] = slot;
    t.phase[p] = ph;
  }
  if (p == 0) {
    if (t.prefetch) t.ctl->stats.prefetch_keys += T;
    else t.ctl->stats.positions += T;
  }
}

// Decode-sized lookups (T <= kSmallT): probe and residency resolution in
// one block, with the policy of k_resolve_lookup for a single group.  The
// kernel reads everything it needs first, decides in LDS, and writes last,
// so no store ever holds up a load:
//   reads: two chains side by side in every wave -- tokens -> buckets -> the
//     matched rows' `where` -> their `pref` flags for the wave's positions,
//     and the ring cursors -> one entry of the least-recent window of the
//     recency ring per thread -> that slot's stamp and owner;
//   decisions: dedupe, the set of slots this call references, victims from
//     the window (an entry is live if its stamp still matches and its slot
//     is not referenced), all in LDS;
//   writes: outputs, residency, recency appends, counters.
// If the window holds too few live entries the block falls back to
// pop_victims, after writing this call's stamps for it to see.
constexpr uint32_t kSmallT = 64;
constexpr int kSmallPer = (int)kSmallT / kWaves;  // positions per wave
constexpr int kRefHash = 128;                     // referenced-slot set

__device__ __forceinline__ uint32_t slot_hash(uint32_t s) { return (s * 2654435761u) >> 25; }

__global__ __launch_bounds__(kResolveThreads) void k_lookup_resolve_small(const TierArgs t) {
  const LookupArgs& a = t.look;
  const uint32_t T = a.T;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  __shared__ int32_t s_row[kSmallT];
  __shared__ int32_t s_where[kSmallT];
  __shared__ uint8_t s_len[kSmallT];
  __shared__ uint8_t s_pref[kSmallT];
  __shared__ int32_t hkey[kHashSize];
  __shared__ uint32_t hpos[kHashSize];
  __shared__ int32_t hslot[kHashSize];
  __shared__ uint8_t hphase[kHashSize];
  __shared__ int32_t rset[kRefHash];
  __shared__ uint32_t vict[kResolveThreads];
  __shared__ int32_t vown[kResolveThreads];
  __shared__ uint32_t s_cnt[4];  // hits, cache hits, prefetch used, host-served
  __shared__ unsigned long long s_last;
  if (threadIdx.x < kRefHash) rset[threadIdx.x] = -1;
  if (threadIdx.x < 4) s_cnt[threadIdx.x] = 0;

  // ---- reads.  Read step 1: ring cursors, counters (no other kernel
  // touches the table's state while this one runs), the tokens of the
  // wave's positions.
  const unsigned long long tail0 = t.ctl->tail, head0 = t.ctl->head;
  const TierStats st0 = t.ctl->stats;
  int32_t tw[kSmallPer][4];
#pragma unroll
  for (int k = 0; k < kSmallPer; ++k)
    dev::window_tokens(a, (uint32_t)(wave + kWaves * k), tw[k]);  // beyond T: invalid
  // Read step 2: one ring entry per thread; the first bucket of every key.
  const unsigned long long wi = tail0 + threadIdx.x;
  const bool win = wi < head0;
  const uint64_t e = win ? t.ring[wi & t.ring_mask] : 0;
  dev::Probe pr[kSmallPer];
#pragma unroll
  for (int k = 0; k < kSmallPer; ++k) pr[k] = dev::probe_begin(a, tw[k], lane);
  // Read step 3: the entry's slot state; the matches (lane k of the wave holds
  // position wave + kWaves k) and their residency.
  const uint32_t eslot = (uint32_t)(e >> 32), est = (uint32_t)e;
  const uint32_t estamp = win ? t.stamp[eslot] : 0u;
  const int32_t eowner = win ? t.owner[eslot] : -1;
  int32_t myrow = -1;
  int mylen = 0;
#pragma unroll
  for (int k = 0; k < kSmallPer; ++k) {
    int len;
    const int32_t row = dev::probe_finish(a, pr[k], lane, &len);
    if (lane == k) {
      myrow = row;
      mylen = len;
    }
  }
  const int32_t mywhere = myrow >= 0 ? t.where[myrow] : -1;
  // Read step 4: prefetched flags of the cached matches.
  const uint8_t mypref = mywhere >= 0 ? t.pref[mywhere] : (uint8_t)0;
  if (lane < kSmallPer && wave + kWaves * lane < (int)T) {
    const uint32_t q = wave + kWaves * lane;
    s_row[q] = myrow;
    s_len[q] = (uint8_t)mylen;
    s_where[q] = mywhere;
    s_pref[q] = mypref;
  }
  __syncthreads();

  // ---- decisions (LDS).  Dedupe; cached first occurrences are referenced.
  const uint32_t p = threadIdx.x;
  const bool valid = p < T;
  const int32_t r = valid ? s_row[p] : -1;
  int h;
  const bool first = first_of_row(r, p, hkey, hpos, &h);
  const int32_t s0 = first ? s_where[p] : -1;
  bool append = false;
  if (s0 >= 0) {
    append = true;
    hslot[h] = s0;
    hphase[h] = 0;
    if (s_pref[p]) atomicAdd(&s_cnt[2], 1u);
    int q = (int)slot_hash((uint32_t)s0);
    while (atomicCAS(&rset[q], -1, s0) != -1) q = (q + 1) & (kRefHash - 1);
  }
  const bool miss_first = first && s0 < 0;
  uint32_t need;
  const uint32_t mrank = block_count(miss_first, &need);  // its barrier publishes rset
  bool referenced = false;
  if (win) {
    for (int q = (int)slot_hash(eslot);; q = (q + 1) & (kRefHash - 1)) {
      const int32_t v = rset[q];
      if (v == -1) break;
      if ((uint32_t)v == eslot) {
        referenced = true;
        break;
      }
    }
  }
  const bool cur = win && est == t.clock;
  const bool live = win && !cur && estamp == est && !referenced;
  uint32_t nlive;
  const uint32_t lrank = block_count(live, &nlive);
  const uint32_t first_cur = block_first(cur);
  const bool window_ends = first_cur != 0xFFFFFFFFu || tail0 + kResolveThreads >= head0;
  const bool fast = need == 0 || nlive >= need || window_ends;
  uint32_t got = 0;
  if (fast) {
    got = nlive < need ? nlive : need;
    if (live && lrank < got) {
      vict[lrank] = eslot;
      vown[lrank] = eowner;
      if (lrank == got - 1) s_last = wi;
    }
    __syncthreads();
    if (threadIdx.x == 0 && need > 0) {
      if (got == need) t.ctl->tail = s_last + 1;
      else if (first_cur != 0xFFFFFFFFu) t.ctl->tail = tail0 + first_cur;
      else t.ctl->tail = head0;
    }
  } else {
    // The ring walk reads stamps: make this call's references visible first.
    if (s0 >= 0) t.stamp[s0] = t.clock;
    __threadfence_block();
    __syncthreads();
    got = pop_victims(t, need, vict);
  }
  bool writes = false;
  uint32_t v = 0;
  int32_t old = -1;
  if (miss_first) {
    if (mrank < got) {
      v = vict[mrank];
      old = fast ? vown[mrank] : t.owner[v];
      hslot[h] = (int32_t)v;
      hphase[h] = 1;
      append = true;
      writes = t.fill_inline != 0;
    } else {
      hslot[h] = -1;
      hphase[h] = 2;
    }
  }
  __syncthreads();

  // ---- writes.
  if (s0 >= 0) {
    t.stamp[s0] = t.clock;
    if (s_pref[p]) t.pref[s0] = 0;
  }
  if (miss_first && mrank < got) {
    if (old >= 0) t.where[old] = -1;
    t.owner[v] = r;
    t.where[r] = (int32_t)v;
    t.stamp[v] = t.clock;
    t.pref[v] = 0;
    t.jobs[mrank] = TierJob{r, (int32_t)v};
  }
  if (valid) {
    const int32_t s1 = r >= 0 ? hslot[h] : -1;
    const uint8_t ph = r >= 0 ? hphase[h] : 3;
    dev::write_result(a, p, r, s_len[p]);
    t.row_of[p] = r;
    t.slot_of[p] = s1;
    t.phase[p] = writes ? (uint8_t)(ph | kPhaseWrite) : ph;
    if (r >= 0) {
      atomicAdd(&s_cnt[0], 1u);
      if (ph == 0) atomicAdd(&s_cnt[1], 1u);
      else atomicAdd(&s_cnt[3], 1u);
    }
  }
  uint32_t napp;
  const uint32_t arank = block_count(append, &napp);
  if (append) t.ring[(head0 + arank) & t.ring_mask] = ring_entry((uint32_t)hslot[h], t.clock);
  if (threadIdx.x == 0) {
    t.ctl->head = head0 + napp;
    t.ctl->njobs = got;
    TierStats st = st0;
    st.positions += T;
    st.hits += s_cnt[0];
    st.cache_hits += s_cnt[1];
    st.cache_misses += s_cnt[0] - s_cnt[1];
    st.prefetch_used += s_cnt[2];
    st.host_bytes += (unsigned long long)((t.fill_inline ? 0u : got) + s_cnt[3]) * t.row_bytes;
    t.ctl->stats = st;
  }
}

// Priority-scored, budgeted prefetch (Eq. 17: s = p * r * c), one block,
// any number of candidates.  For candidate q with matched row r: p =
// prob[q] (the predicted token's probability; <= 0 and NaN count as 0),
// r = the matched phrase length (longer phrases are the more specific
// entries), c = 1 if the row is only in host memory and 0 if it is cached.
// A row named by several candidates keeps its highest p * len and its first
// candidate index (both kept in the call-wide row table of the scratch).
// Cached rows with a positive p * len are referenced: never victims of this
// prefetch, most recent in order of first candidate.  Rows that are not
// cached and score above zero are fetched by descending score, then first
// candidate index, until `budget` rows are fetched or no unreferenced slot
// is left; the rest are dropped.  Scores are float32 products compared as
// float32 (as bit patterns: they are never negative).
//   1. every candidate enters the row table: first index and best score;
//   2. first candidates: cached rows with a score are stamped referenced and
//      appended to the recency ring; rows to fetch go to a key list
//      (~score << 32 | first index, so ascending keys = the fetch order);
//   3. the budget-th smallest key is found by a radix select (8-bit digits
//      from the top), the keys at or below it are gathered and sorted in LDS;
//   4. victims are popped and the rows filled in that order.
constexpr int kScoredBudgetMax = 1024;

__device__ __forceinline__ uint64_t gh_insert_at(const TierArgs& t, int32_t r, uint32_t q) {
  const uint64_t tag = (uint64_t)t.clock << 32;
  const uint64_t want = tag | (uint32_t)r;
  uint64_t h = gh_home(r, t.hmask);
  for (;;) {
    uint64_t old = gh_load(t.hkey + h);
    while (old != want && (old >> 32) != t.clock) {
      const uint64_t prev = atomicCAS((unsigned long long*)(t.hkey + h), (unsigned long long)old,
                                      (unsigned long long)want);
      old = prev == old ? want : prev;
    }
    if (old == want) break;
    h = (h + 1) & t.hmask;
  }
  atomicMax((unsigned long long*)(t.hpos + h), (unsigned long long)(tag | (uint32_t)~q));
  return h;
}

__device__ __forceinline__ uint64_t gh_find(const TierArgs& t, int32_t r) {
  const uint64_t want = ((uint64_t)t.clock << 32) | (uint32_t)r;
  uint64_t h = gh_home(r, t.hmask);
  while (gh_load(t.hkey + h) != want) h = (h + 1) & t.hmask;
  return h;
}

// Returns the number of rows filled (block-uniform); the fill list is
// jobs[0 .. filled).
// LDS: the row table of calls of at most kScoredLdsMax candidates (the
// one-block prefetch) lives in LDS, with the key list; larger calls use the
// call-wide table in the scratch (fewer LDS bytes, atomics through L2).
constexpr uint32_t kScoredLdsMax = kGroup;
constexpr int kScoredLdsHash = 2 * kScoredLdsMax;

template <bool LDS>
__device__ uint32_t resolve_scored(const TierArgs& t, uint32_t N, const float* __restrict__ prob,
                                   uint32_t budget) {
  __shared__ unsigned long long sel[kScoredBudgetMax];
  __shared__ uint32_t vict[kResolveThreads];
  __shared__ uint32_t hist[256];
  __shared__ uint32_t s_found, s_nref, s_n, s_g, s_bin, s_before;
  // LDS row table: row, first candidate index (minimum), best score bits
  // (maximum); and the key list.
  __shared__ int32_t lkey[LDS ? kScoredLdsHash : 1];
  __shared__ uint32_t lpos[LDS ? kScoredLdsHash : 1];
  __shared__ uint32_t lsc[LDS ? kScoredLdsHash : 1];
  __shared__ unsigned long long lklist[LDS ? kScoredLdsMax : 1];
  const uint64_t tag = (uint64_t)t.clock << 32;
  // Rows to fetch; in the scratch version it becomes the fill list in step 4.
  uint64_t* klist = LDS ? (uint64_t*)lklist : (uint64_t*)t.jobs;
  if (threadIdx.x == 0) {
    s_found = 0;
    s_nref = 0;
    s_n = 0;
    s_g = 0;
  }
  if (LDS) {
    for (int i = threadIdx.x; i < kScoredLdsHash; i += kResolveThreads) {
      lkey[i] = -1;
      lpos[i] = 0xFFFFFFFFu;
      lsc[i] = 0;
    }
  }
  __syncthreads();
  constexpr int lshift = 32 - __builtin_ctz(kScoredLdsHash);
  auto lfind = [&](int32_t r) {
    int h = (int)(((uint32_t)r * 2654435761u) >> lshift);
    while (lkey[h] != r) h = (h + 1) & (kScoredLdsHash - 1);
    return h;
  };
  // 1. Row table: first candidate index and best score per row.
  for (uint32_t base = 0; base < N; base += kResolveThreads) {
    const uint32_t q = base + threadIdx.x;
    const int32_t r = q < N ? t.row_of[q] : -1;
    if (r >= 0) {
      const float p = prob[q];
      const float sc = (p > 0.0f ? p : 0.0f) * (float)t.phase[q];  // NaN and p <= 0 score 0
      if (LDS) {
        int h = (int)(((uint32_t)r * 2654435761u) >> lshift);
        for (;;) {
          const int old = atomicCAS(&lkey[h], -1, r);
          if (old == -1 || old == r) break;
          h = (h + 1) & (kScoredLdsHash - 1);
        }
        atomicMin(&lpos[h], q);
        atomicMax(&lsc[h], __float_as_uint(sc));
      } else {
        const uint64_t h = gh_insert_at(t, r, q);
        atomicMax((unsigned long long*)(t.hval + h),
                  (unsigned long long)(tag | __float_as_uint(sc)));
      }
    }
    wave_tally(r >= 0, &s_found);
  }
  if (!LDS) __threadfence();  // the row table's atomics have completed before any wave reads it
  __syncthreads();
  const unsigned long long head0 = t.ctl->head;
  // 2. References and the key list, in candidate order.
  for (uint32_t base = 0; base < N; base += kResolveThreads) {
    const uint32_t q = base + threadIdx.x;
    const int32_t r = q < N ? t.row_of[q] : -1;
    bool ref = false, cand = false;
    int32_t w = -1;
    uint32_t sc = 0;
    if (r >= 0) {
      bool first;
      if (LDS) {
        const int h = lfind(r);
        first = lpos[h] == q;
        sc = lsc[h];
      } else {
        const uint64_t h = gh_find(t, r);
        first = gh_load(t.hpos + h) == (tag | (uint32_t)~q);
        if (first) sc = (uint32_t)gh_load(t.hval + h);
      }
      if (first) {
        w = t.where[r];
        ref = sc != 0 && w >= 0;
        cand = sc != 0 && w < 0;
      }
    }
    if (ref) t.stamp[w] = t.clock;
    uint32_t nref, ncand;
    const uint32_t rr = block_count(ref, &nref);
    const uint32_t rc = block_count(cand, &ncand);
    if (ref) t.ring[(head0 + s_nref + rr) & t.ring_mask] = ring_entry((uint32_t)w, t.clock);
    if (cand) klist[s_n + rc] = ((uint64_t)~sc << 32) | q;
    __threadfence_block();
    __syncthreads();
    if (threadIdx.x == 0) {
      s_nref += nref;
      s_n += ncand;
    }
    __syncthreads();
  }
  const uint32_t n = s_n, nref = s_nref;
  const uint32_t want = n < budget ? n : budget;
  // 3. The want smallest keys, in ascending order, into sel.  Keys are
  // distinct (they end in the candidate index).  Up to one key per thread:
  // each thread counts the smaller keys and a key of rank below want goes
  // to sel[rank] (a few hundred broadcast reads instead of select passes
  // and a sort, each a series of barriers).  More keys: a radix select of
  // the threshold, a gather and a bitonic sort.
  if (n <= (uint32_t)kResolveThreads) {
    if (want > 0 && threadIdx.x < n) {
      const uint64_t k = klist[threadIdx.x];
      uint32_t rank = 0;
      for (uint32_t u = 0; u < n; ++u) rank += klist[u] < k ? 1u : 0u;
      if (rank < want) sel[rank] = k;
    }
    __syncthreads();
  } else {
    uint64_t prefix = 0, pmask = 0;
    if (want > 0 && want < n) {
      uint32_t rem = want;  // keys still to take at or below the prefix
      for (int shift = 56; shift >= 0; shift -= 8) {
        for (int i = threadIdx.x; i < 256; i += kResolveThreads) hist[i] = 0;
        __syncthreads();
        for (uint32_t i = threadIdx.x; i < n; i += kResolveThreads) {
          const uint64_t k = klist[i];
          if ((k & pmask) == prefix) atomicAdd(&hist[(k >> shift) & 255], 1u);
        }
        __syncthreads();
        if (threadIdx.x < 64) {
          // The bin where the running count reaches rem: lane l sums bins
          // 4l .. 4l+3, then a wave scan.
          const uint32_t c0 = hist[4 * threadIdx.x], c1 = hist[4 * threadIdx.x + 1],
                         c2 = hist[4 * threadIdx.x + 2], c3 = hist[4 * threadIdx.x + 3];
          uint32_t x = c0 + c1 + c2 + c3;
          for (int d = 1; d < 64; d <<= 1) {
            const uint32_t y = __shfl_up(x, d, 64);
            if ((int)threadIdx.x >= d) x += y;
          }
          const uint32_t before = x - (c0 + c1 + c2 + c3);
          if (before < rem && x >= rem) {
            uint32_t b = 4 * threadIdx.x, acc = before;
            const uint32_t cs[4] = {c0, c1, c2, c3};
            int j = 0;
            while (acc + cs[j] < rem) acc += cs[j++];
            s_bin = b + j;
            s_before = acc;
          }
        }
        __syncthreads();
        const uint32_t bin = s_bin;
        rem -= s_before;
        prefix |= (uint64_t)bin << shift;
        pmask |= 255ull << shift;
        const bool exact = hist[bin] == rem;  // every key of this prefix is taken
        __syncthreads();
        if (exact) break;
      }
    }
    const uint64_t thresh = want == 0 ? 0 : (want < n ? (prefix | ~pmask) : ~0ull);
    if (want > 0) {
      for (uint32_t base = 0; base < n; base += kResolveThreads) {
        const uint32_t i = base + threadIdx.x;
        const uint64_t k = i < n ? klist[i] : ~0ull;
        const bool take = i < n && k <= thresh;
        uint32_t c;
        const uint32_t rk = block_count(take, &c);
        if (take) sel[s_g + rk] = k;
        __syncthreads();
        if (threadIdx.x == 0) s_g += c;
        __syncthreads();
      }
    }
    uint32_t p2 = 1;
    while (p2 < want) p2 <<= 1;
    for (uint32_t i = want + threadIdx.x; i < p2; i += kResolveThreads) sel[i] = ~0ull;
    __syncthreads();
    // Bitonic sort, ascending: highest score first, then lowest candidate index.
    for (uint32_t size = 2; size <= p2; size <<= 1) {
      for (uint32_t stride = size >> 1; stride > 0; stride >>= 1) {
        for (uint32_t i = threadIdx.x; i < p2 / 2; i += kResolveThreads) {
          const uint32_t a = 2 * i - (i & (stride - 1));
          const uint32_t b = a + stride;
          const bool up = (a & size) == 0;
          const unsigned long long ka = sel[a], kb = sel[b];
          if ((ka > kb) == up) {
            sel[a] = kb;
            sel[b] = ka;
          }
        }
        __syncthreads();
      }
    }
  }
  // 4. Victims and fills (the key list is no longer read: jobs are rewritten).
  const uint32_t got = want ? pop_victims(t, want, vict) : 0;
  if (threadIdx.x < got) {
    const uint32_t v = vict[threadIdx.x];
    const int32_t r = t.row_of[(uint32_t)sel[threadIdx.x]];
    const int32_t old = t.owner[v];
    if (old >= 0) t.where[old] = -1;
    t.owner[v] = r;
    t.where[r] = (int32_t)v;
    t.stamp[v] = t.clock;
    t.pref[v] = 1;
    t.jobs[threadIdx.x] = TierJob{r, (int32_t)v};
    t.ring[(head0 + nref + threadIdx.x) & t.ring_mask] = ring_entry(v, t.clock);
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    t.ctl->head = head0 + nref + got;
    t.ctl->njobs = got;
    TierStats& st = t.ctl->stats;
    st.prefetch_keys += N;
    st.prefetch_found += s_found;
    st.prefetch_filled += got;
    st.prefetch_dropped += n - got;
    st.host_bytes += (unsigned long long)got * t.row_bytes;
  }
  return got;
}

__global__ __launch_bounds__(kResolveThreads) void k_resolve_prefetch_scored(
    const TierArgs t, uint32_t N, const float* __restrict__ prob, uint32_t budget) {
  (void)resolve_scored<false>(t, N, prob, budget);
}

// ---- Prefetch of up to kPrefetchFusedMax candidates in two launches: one
// block runs the probe of every candidate window and the residency
// resolution (the lookup policy for tfe_prefetch, the scored policy for
// tfe_prefetch_scored); then k_fill copies the chosen rows from pinned host
// memory into their slots over many compute units (one compute unit's
// outstanding host reads would make the copies several times slower).
constexpr uint32_t kPrefetchFusedMax = kGroup;

// Longest match of every candidate window (the row the next lookup selects
// if that candidate is the next token).  Thread items are (candidate,
// length) pairs, longest first, each probed by one thread reading whole
// buckets, so that the bucket reads of up to 1024 items are in flight at
// once.  Writes row_of[q] and phase[q] = matched length; uses slot_of as
// scratch for the N * L item results.
__device__ void prefetch_probe_block(const TierArgs& t, const int32_t* __restrict__ tail,
                                     int32_t tail_len, const int32_t* __restrict__ cand,
                                     uint32_t B, uint32_t K) {
  const LookupArgs& a = t.look;
  const uint32_t N = B * K;
  const uint32_t L = (uint32_t)(a.n_max - a.n_min + 1);
  int32_t* item_row = t.slot_of;
  for (uint32_t i = threadIdx.x; i < N * L; i += kResolveThreads) {
    const uint32_t q = i / L, l = i - q * L;
    const uint32_t b = q / K;
    int32_t tw[4];
    tw[0] = cand[q];
    for (int j = 1; j < 4; ++j)
      tw[j] = tail_len - j >= 0 ? tail[(size_t)b * tail_len + (tail_len - j)] : -1;
    uint64_t key;
    uint32_t ext;
    const bool ok = dev::window_key(a, tw, a.n_max - (int)l, &key, &ext);
    item_row[i] = ok ? dev::probe_key_thread(a, key, ext) : -1;
  }
  __syncthreads();
  for (uint32_t q = threadIdx.x; q < N; q += kResolveThreads) {
    int32_t row = -1;
    int len = 0;
    for (uint32_t l = 0; l < L; ++l) {
      const int32_t r = item_row[q * L + l];
      if (r >= 0) {
        row = r;
        len = a.n_max - (int)l;
        break;
      }
    }
    t.row_of[q] = row;
    t.phase[q] = (uint8_t)len;
  }
  __syncthreads();
}

template <bool SCORED>
__global__ __launch_bounds__(kResolveThreads) void k_prefetch_fused(
    const TierArgs t, const int32_t* __restrict__ tail, int32_t tail_len,
    const int32_t* __restrict__ cand, uint32_t B, uint32_t K, const float* __restrict__ prob,
    uint32_t budget) {
  // The probe reads only the index and the candidates: it runs before the
  // wait for the lookups that share the residency state.
  prefetch_probe_block(t, tail, tail_len, cand, B, K);
  wait_ordered_block(t);
  if (SCORED)
    (void)resolve_scored<true>(t, B * K, prob, budget);
  else
    (void)resolve_one_block(t, B * K);
}

__global__ void k_tier_wait(const TierArgs t) { wait_ordered_block(t); }

// A wave's row stored with device scope (cache policy sc1): the stores
// write through the XCD's L2, so once they have completed (wait_mem) the
// row is visible to agent-scope readers on every XCD -- without the L2
// writeback of a release fence, which cost about 7 us per block when the
// blocks of a fill issued it together.
template <int NCH>
__device__ __forceinline__ void st_dev_row(u32x4* dst, const u32x4* v, int lane) {
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc((void*)dst, (short)0, NCH * 64 * 16, 0x00020000);
#pragma unroll
  for (int k = 0; k < NCH; ++k)
    __builtin_amdgcn_raw_buffer_store_b128(v[k], rs, (k * 64 + lane) * 16, 0, 16);
}

// Host row -> cache slot copies of the current fill list, one wave per job,
// reading the pinned host rows directly over PCIe (zero-copy).
// With t.count_fill each block then counts into ctl->pf_done once its
// copies have completed (a lookup on another stream waits for it and then
// acquires).
template <int NCH>
__global__ __launch_bounds__(256) void k_fill(const TierArgs t, uint32_t max_jobs) {
  const int lane = threadIdx.x & 63;
  const uint32_t j = blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (j < max_jobs && j < t.ctl->njobs) {
    const TierJob job = t.jobs[j];
    u32x4 v[NCH];
    read_host_row<NCH, true>(t, __builtin_amdgcn_readfirstlane(job.row), v, lane);
    st_dev_row<NCH>((u32x4*)t.cache + (size_t)job.slot * (NCH * 64), v, lane);
  }
  if (!t.count_fill) return;
  wait_mem();
  __syncthreads();
  if (threadIdx.x == 0)
    __hip_atomic_fetch_add(&t.ctl->pf_done, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Probe of a tiered lookup: the resident kernel's key formation and probe,
// writing the caller's hit/slot/len and the matched row per position.
template <int WPB>
__global__ __launch_bounds__(WPB * 64) void k_tier_probe(const TierArgs t) {
  const LookupArgs& a = t.look;
  const int lane = threadIdx.x & 63;
  const uint32_t p = blockIdx.x * WPB + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (p >= a.T) return;
  int32_t tw[4];
  dev::window_tokens(a, p, tw);
  const dev::Probe pr = dev::probe_begin(a, tw, lane);
  int len;
  const int32_t row = dev::probe_finish(a, pr, lane, &len);
  if (lane == 0) {
    dev::write_result(a, p, row, len);
    t.row_of[p] = row;
  }
}

// Probe of the prefetch candidates: candidate k of row b ends the window
// (tail[b, tail_len-3 ..], cand[b, k]); its longest match is the row the
// next lookup selects if that candidate is the next token.
template <int WPB>
__global__ __launch_bounds__(WPB * 64) void k_prefetch_probe(const TierArgs t,
                                                             const int32_t* __restrict__ tail,
                                                             int32_t tail_len,
                                                             const int32_t* __restrict__ cand,
                                                             uint32_t B, uint32_t K) {
  const LookupArgs& a = t.look;
  const int lane = threadIdx.x & 63;
  const uint32_t q = blockIdx.x * WPB + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (q >= B * K) return;
  const uint32_t b = q / K;
  int32_t tw[4];
  tw[0] = cand[q];
  for (int j = 1; j < 4; ++j)
    tw[j] = tail_len - j >= 0 ? tail[(size_t)b * tail_len + (tail_len - j)] : -1;
  const dev::Probe pr = dev::probe_begin(a, tw, lane);
  int len;
  const int32_t row = dev::probe_finish(a, pr, lane, &len);
  if (lane == 0) {
    t.row_of[q] = row;
    t.phase[q] = (uint8_t)len;
  }
}

// Inject of every position: value rows come from the cache (phase 0) or
// straight from pinned host memory over PCIe (phases 1 and 2: rows that were
// not cached when the call began); phase 3 (no match) copies the hidden row
// (out of place).  With kPhaseWrite the wave also stores the row it read into
// its new cache slot.
template <int DT, int NCH, int WPB>
__global__ __launch_bounds__(WPB * 64) void k_tier_inject(const TierArgs t) {
  constexpr int ROW_VECS = NCH * 64;
  const LookupArgs& a = t.look;
  const int lane = threadIdx.x & 63;
  const uint32_t p = blockIdx.x * WPB + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (p >= a.T) return;
  const uint32_t ph_w = t.phase[p];
  const uint32_t ph = ph_w & 3u;
  u32x4 hv[NCH];
  const u32x4* hin = (const u32x4*)a.hin + (size_t)p * ROW_VECS;
#pragma unroll
  for (int k = 0; k < NCH; ++k) hv[k] = __builtin_nontemporal_load(hin + k * 64 + lane);
  u32x4* out = (u32x4*)a.hout + (size_t)p * ROW_VECS;
  if (ph == 3) {
    if (!a.inplace) {
#pragma unroll
      for (int k = 0; k < NCH; ++k) __builtin_nontemporal_store(hv[k], out + k * 64 + lane);
    }
    return;
  }
  u32x4 mv[NCH];
  if (ph != 0) {
    read_host_row<NCH, false>(t, __builtin_amdgcn_readfirstlane(t.row_of[p]), mv, lane);
  } else {
    const u32x4* mrow = (const u32x4*)t.cache + (size_t)t.slot_of[p] * ROW_VECS;
#pragma unroll
    for (int k = 0; k < NCH; ++k) mv[k] = mrow[k * 64 + lane];
  }
  if (ph_w & kPhaseWrite) {
    u32x4* dst = (u32x4*)t.cache + (size_t)t.slot_of[p] * ROW_VECS;
#pragma unroll
    for (int k = 0; k < NCH; ++k) dst[k * 64 + lane] = mv[k];
  }
  const float g = dev::gate_of<DT, NCH>(a, hv, mv);
  dev::store_injected<DT, NCH>(out, hv, mv, g, lane);
}

// Decode-sized lookups with inline fill (T <= kDecodeMaxT positions): the
// whole call in one launch of T one-wave blocks.
//   Every wave runs its position at once: key formation and probe, the
//   row's residency (where), the value row from the cache or -- when it is
//   not cached -- straight from pinned host memory, gate and injection.  A
//   row read from host memory is also written into the position's spare
//   slot: the cache has kDecodeMaxT physical slots beyond its C rows that
//   no row maps to and the recency order does not hold.  This is safe
//   before any residency decision: victims are never slots that the call
//   references, so nothing a wave reads changes during the call.
//   Each wave publishes its row and slot and counts itself in (a wave that
//   reads a cached row reads it first); the last
//   wave to arrive resolves residency for the whole call with the policy of
//   k_resolve_lookup: first positions of rows (lane q = position q), cached
//   rows referenced, victims for the missed rows from the tail of the
//   recency ring, recency appends in first-position order, counters.  A
//   filled row takes over its position's spare slot and the victim slot
//   becomes the new spare, so no row is copied.
// One launch and no cross-block waiting: a wave that is not last exits.
// What crosses blocks (row, slot) is written and read with device-scope
// stores and loads, and each wave waits for its stores to complete before
// it counts in; a device-scope fence would instead write back and
// invalidate the whole L2 in every wave.

constexpr int kWalkPer = 8;  // ring entries per lane and round of the victim walk

// The first window of the victim walk: kWalkPer x 64 ring entries from the
// tail, with their slots' stamps and owners.  Every wave of the decode
// launch reads it while its own probe is in flight (the ring, stamps and
// owners do not change until the last wave writes them), so the last wave
// starts its walk with the window in registers.
struct WalkWindow {
  unsigned long long tail, head;
  uint64_t e[kWalkPer];
  uint32_t sn[kWalkPer];
  int32_t own[kWalkPer];
};

__device__ __forceinline__ void walk_load_entries(const TierArgs& t, WalkWindow& w) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int k = 0; k < kWalkPer; ++k)
    w.e[k] = t.ring[(w.tail + (uint64_t)(k * 64 + lane)) & t.ring_mask];
}

__device__ __forceinline__ void walk_load_slots(const TierArgs& t, WalkWindow& w) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int k = 0; k < kWalkPer; ++k) {
    const bool in = w.tail + (uint64_t)(k * 64 + lane) < w.head;
    const uint32_t slot = in ? (uint32_t)(w.e[k] >> 32) : 0u;
    w.sn[k] = t.stamp[slot];
    w.own[k] = t.owner[slot];
  }
}

// The keys of a decode call's positions, in an LDS hash: a cached row's
// slot (in [0, 2^30)), or the bitwise complement of a missed row's id (in
// [-2^31 + 1, -1]: rows are below 2^31 - 1), so the two never meet; empty
// entries hold kCallEmpty, which neither can be.  At most kDecodeMaxT keys
// in kCallSet entries: every insertion finds a free or equal entry.
constexpr int kCallSet = 256;
constexpr int32_t kCallEmpty = INT32_MIN;

__device__ __forceinline__ uint32_t key_hash(uint32_t k) { return (k * 2654435761u) >> 24; }

// Whether the call references cache slot `slot`.
__device__ __forceinline__ bool call_has_slot(const int32_t* ckey, uint32_t slot) {
  for (int q = (int)key_hash(slot);; q = (q + 1) & (kCallSet - 1)) {
    const int32_t v = ckey[q];
    if (v == kCallEmpty) return false;
    if (v == (int32_t)slot) return true;
  }
}

// Published slot word of a decode position: the cache slot (< 2^30) with
// bit 30 set when the slot was filled by a prefetch and not used yet; -1
// when the row is not cached (or there is no row).
constexpr int32_t kSlotPref = 0x40000000;

template <int NCH>
__device__ void decode_resolve_last(const TierArgs& t, uint32_t T, WalkWindow& w) {
  __shared__ uint32_t vict[kDecodeMaxT];
  __shared__ int32_t vown[kDecodeMaxT];
  __shared__ int32_t ckey[kCallSet];
  __shared__ uint32_t cpos[kCallSet];
  const int lane = threadIdx.x;
  const bool valid = (uint32_t)lane < T;
  const int32_t r = valid ? ld_dev(t.row_of + lane) : -1;
  const int32_t sw = valid ? ld_dev(t.slot_of + lane) : -1;
  const int32_t sp = t.spare[lane];
  const int32_t s0 = sw >= 0 ? (sw & ~kSlotPref) : -1;
  const bool pv = sw >= 0 && (sw & kSlotPref) != 0;
#pragma unroll
  for (int i = 0; i < kCallSet / 64; ++i) {
    ckey[lane + 64 * i] = kCallEmpty;
    cpos[lane + 64 * i] = kDecodeMaxT;
  }
  __syncthreads();
  // First position of each row: the lowest lane with its key.  The cached
  // slots in the table are the ones this call references, never victims.
  int h = 0;
  if (r >= 0) {
    const int32_t key = s0 >= 0 ? s0 : ~r;
    h = (int)key_hash((uint32_t)key);
    for (;;) {
      const int32_t prev = atomicCAS(&ckey[h], kCallEmpty, key);
      if (prev == kCallEmpty || prev == key) break;
      h = (h + 1) & (kCallSet - 1);
    }
    atomicMin(&cpos[h], (uint32_t)lane);
  }
  __syncthreads();
  const bool first = r >= 0 && cpos[h] == (uint32_t)lane;
  const bool fc = first && s0 >= 0, fm = first && s0 < 0;
  const uint64_t mfm = __builtin_amdgcn_ballot_w64(fm);
  const uint32_t need = (uint32_t)__builtin_popcountll(mfm);
  const uint32_t mrank = lanes_below(mfm);
  unsigned long long tail = w.tail;
  const unsigned long long head = w.head;
  uint32_t got = 0;
  bool fresh = false;  // window w holds the entries from `tail`
  // Least recent live entries (stamp still current, not referenced by this
  // call, not this call's), kWalkPer x 64 per round; an entry of this call
  // or the head ends the walk.
  while (got < need && tail < head) {
    if (fresh) {
      w.tail = tail;
      walk_load_entries(t, w);
      walk_load_slots(t, w);
    }
    fresh = true;
    bool stop = false;
#pragma unroll
    for (int k = 0; k < kWalkPer; ++k) {
      if (stop || got == need) continue;  // wave-uniform
      const unsigned long long base = tail + (uint64_t)(k * 64);
      const bool in = base + (uint64_t)lane < head;
      const uint32_t slot = (uint32_t)(w.e[k] >> 32), st = (uint32_t)w.e[k];
      const bool cur = in && st == t.clock;
      const uint64_t mcur = __builtin_amdgcn_ballot_w64(cur);
      const uint32_t lim = mcur ? (uint32_t)__builtin_ctzll(mcur) : 64u;
      const bool live = in && !cur && w.sn[k] == st && (uint32_t)lane < lim &&
                        !call_has_slot(ckey, slot);
      const uint64_t ml = __builtin_amdgcn_ballot_w64(live);
      const uint32_t nl = (uint32_t)__builtin_popcountll(ml);
      const uint32_t rk = lanes_below(ml);
      const uint32_t take = nl < need - got ? nl : need - got;
      if (live && rk < take) {
        vict[got + rk] = slot;
        vown[got + rk] = w.own[k];
      }
      if (take == need - got && take > 0) {
        // Resume after the last victim taken.
        const uint64_t mlast = __builtin_amdgcn_ballot_w64(live && rk == take - 1);
        tail = base + (uint64_t)__builtin_ctzll(mlast) + 1;
        got = need;
        stop = true;
        continue;
      }
      got += take;
      if (mcur || base + 64 >= head) {
        tail = mcur ? base + lim : head;
        stop = true;
        continue;
      }
    }
    if (stop) break;
    tail += (uint64_t)kWalkPer * 64;
  }
  __syncthreads();  // vict, vown
  // A filled row keeps the spare slot its position's wave wrote it into; the
  // victim's row leaves the cache and the victim slot becomes that
  // position's spare.  No row data moves.
  const bool fill = fm && mrank < got;
  uint32_t slot_now = fc ? (uint32_t)s0 : 0u;
  if (fc) {
    t.stamp[s0] = t.clock;
    if (pv) t.pref[s0] = 0;
  }
  if (fill) {
    const uint32_t v = vict[mrank];
    const int32_t old = vown[mrank];
    if (old >= 0) t.where[old] = -1;
    t.owner[v] = -1;
    t.spare[lane] = (int32_t)v;
    t.owner[sp] = r;
    t.where[r] = sp;
    t.stamp[sp] = t.clock;
    t.pref[sp] = 0;
    slot_now = (uint32_t)sp;
  }
  const bool app = fc || fill;
  const uint64_t ma = __builtin_amdgcn_ballot_w64(app);
  if (app) t.ring[(head + lanes_below(ma)) & t.ring_mask] = ring_entry(slot_now, t.clock);
  const uint32_t nhit = (uint32_t)__builtin_popcountll(__builtin_amdgcn_ballot_w64(r >= 0));
  const uint32_t nch =
      (uint32_t)__builtin_popcountll(__builtin_amdgcn_ballot_w64(r >= 0 && s0 >= 0));
  const uint32_t nused = (uint32_t)__builtin_popcountll(__builtin_amdgcn_ballot_w64(fc && pv));
  if (lane == 0) {
    t.ctl->tail = tail;
    t.ctl->head = head + (uint64_t)__builtin_popcountll(ma);
    t.ctl->njobs = 0;
    TierStats& st = t.ctl->stats;
    st.positions += T;
    st.hits += nhit;
    st.cache_hits += nch;
    st.cache_misses += nhit - nch;
    st.prefetch_used += nused;
    st.host_bytes += (unsigned long long)(nhit - nch) * t.row_bytes;
    t.ctl->arrive = 0;  // the next call starts counting from zero
  }
  // Every wave of the call has read what it needed before counting in, so
  // the call is done with the shared state once the residency writes above
  // reach memory: it counts into ctl->lk_done, which a prefetch on another
  // stream waits for.
  if (t.count_lookup) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    if (lane == 0)
      __hip_atomic_fetch_add(&t.ctl->lk_done, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// Publishes this wave's row and slot word, waits for its writes, and counts
// in; true for the last wave of the call.
__device__ __forceinline__ bool decode_arrive(const TierArgs& t, uint32_t p, int32_t row,
                                              int32_t sw) {
  if (threadIdx.x == 0) {
    st_dev(t.row_of + p, row);
    st_dev(t.slot_of + p, sw);
  }
  wait_mem();
  uint32_t last = 0;
  if (threadIdx.x == 0)
    last = __hip_atomic_fetch_add(&t.ctl->arrive, 1u, __ATOMIC_RELAXED,
                                  __HIP_MEMORY_SCOPE_AGENT) == t.look.T - 1 ? 1u : 0u;
  return __builtin_amdgcn_readfirstlane(last) != 0;
}

template <int DT, int NCH>
__global__ __launch_bounds__(64) void k_tier_decode(const TierArgs t) {
  constexpr int ROW_VECS = NCH * 64;
  const LookupArgs& a = t.look;
  const int lane = threadIdx.x;
  const uint32_t p = blockIdx.x;  // grid = T <= kDecodeMaxT
  u32x4 hv[NCH];
  const u32x4* hin = (const u32x4*)a.hin + (size_t)p * ROW_VECS;
#pragma unroll
  for (int k = 0; k < NCH; ++k) hv[k] = dev::load_hidden(hin + k * 64 + lane);
  int32_t tw[4];
  dev::window_tokens(a, p, tw);
  const dev::Probe pr = dev::probe_begin(a, tw, lane);
  wait_ordered_block(t);  // a prefetch on another stream, before any residency read
  WalkWindow win;
  win.tail = t.ctl->tail;
  win.head = t.ctl->head;
  walk_load_entries(t, win);
  const int32_t sp = t.spare[p];
  int len;
  const int32_t row = dev::probe_finish(a, pr, lane, &len);
  if (lane == 0) dev::write_result(a, p, row, len);
  const int32_t w = row >= 0 ? t.where[row] : -1;
  walk_load_slots(t, win);
  u32x4* out = (u32x4*)a.hout + (size_t)p * ROW_VECS;
  if (row < 0) {
    if (decode_arrive(t, p, row, -1)) decode_resolve_last<NCH>(t, a.T, win);
    if (!a.inplace) {
#pragma unroll
      for (int k = 0; k < NCH; ++k) dev::store_out(hv[k], out + k * 64 + lane);
    }
    return;
  }
  u32x4 mv[NCH];
  if (w >= 0) {
    // Cached: the row is read before this wave counts in (with the slot's
    // prefetched flag), so once the last wave has arrived no wave of the
    // call reads the cache any more.
    const int32_t sw = t.pref[w] ? (w | kSlotPref) : w;
    const u32x4* mrow = (const u32x4*)t.cache + (size_t)w * ROW_VECS;
#pragma unroll
    for (int k = 0; k < NCH; ++k) mv[k] = mrow[k * 64 + lane];
    if (decode_arrive(t, p, row, sw)) decode_resolve_last<NCH>(t, a.T, win);
  } else {
    // Host only: the row is read once, written into this position's spare
    // slot (which no row maps to, so no wave reads it), and injected.  The
    // copy is a device-scope store that completes before the wave counts
    // in, so no line of it is left in this XCD's L2 for a later fill of the
    // same slot (after the call counts in) to be overwritten by.
    read_host_row<NCH, false>(t, __builtin_amdgcn_readfirstlane(row), mv, lane);
    st_dev_row<NCH>((u32x4*)t.cache + (size_t)sp * ROW_VECS, mv, lane);
    if (decode_arrive(t, p, row, -1)) decode_resolve_last<NCH>(t, a.T, win);
  }
  const float g = dev::gate_of<DT, NCH>(a, hv, mv);
  dev::store_injected<DT, NCH>(out, hv, mv, g, lane);
}

// Initial state: slot s < prefill holds row s; the ring lists the empty
// slots in ascending order, then the filled slots by descending row.
__global__ void k_tier_init(const TierArgs t, uint32_t C, uint32_t prefill) {
  const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= C && i < C + kDecodeMaxT) {  // spare slots: no row, not in the ring
    t.owner[i] = -1;
    t.stamp[i] = 0;
    t.pref[i] = 0;
    t.spare[i - C] = (int32_t)i;
  }
  if (i >= C) return;
  const uint32_t empty = C - prefill;
  const uint32_t slot = i < empty ? prefill + i : prefill - 1 - (i - empty);
  t.ring[i] = ring_entry(slot, 0);
  t.owner[i] = i < prefill ? (int32_t)i : -1;
  t.stamp[i] = 0;
  t.pref[i] = 0;
  if (i < prefill) t.where[i] = (int32_t)i;
  if (i == 0) {
    t.ctl->head = C;
    t.ctl->tail = 0;
    t.ctl->njobs = 0;
  }
}

// Drops dead entries: live entries move, in order, to `dst` (single block).
// With `restamp`, every live entry and its slot's stamp restart at clock 0
// (each slot has exactly one live entry, so order and liveness are kept).
__global__ __launch_bounds__(kResolveThreads) void k_ring_compact(const TierArgs t, uint64_t* dst,
                                                                  uint64_t dst_mask,
                                                                  uint32_t restamp) {
  __shared__ unsigned long long s_out;
  if (threadIdx.x == 0) s_out = 0;
  __syncthreads();
  const unsigned long long tail = t.ctl->tail, head = t.ctl->head;
  for (unsigned long long base = tail; base < head; base += kResolveThreads) {
    const unsigned long long i = base + threadIdx.x;
    const bool in = i < head;
    const uint64_t e = in ? t.ring[i & t.ring_mask] : 0;
    const bool live = in && t.stamp[(uint32_t)(e >> 32)] == (uint32_t)e;
    uint32_t n;
    const uint32_t rank = block_count(live, &n);
    if (live) {
      dst[(s_out + rank) & dst_mask] = restamp ? ring_entry((uint32_t)(e >> 32), 0u) : e;
      if (restamp) t.stamp[(uint32_t)(e >> 32)] = 0;
    }
    __syncthreads();
    if (threadIdx.x == 0) s_out += n;
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    t.ctl->tail = 0;
    t.ctl->head = s_out;
  }
}

// Residency of phrase rows: the HBM cache slot of each row (tiered tables),
// -1 where the row is only in host memory, -2 for ids outside [0, P).
__global__ void k_residency(const int32_t* __restrict__ where, int64_t P,
                            const int32_t* __restrict__ rows, int64_t n, int32_t* __restrict__ out) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int32_t r = rows[i];
  out[i] = (r < 0 || (int64_t)r >= P) ? -2 : (where ? where[r] : r);
}

template <int NCH>
hipError_t launch_fill_t(const TierArgs& t, uint32_t max_jobs, hipStream_t s) {
  if (max_jobs == 0) return hipSuccess;
  hipLaunchKernelGGL(k_fill<NCH>, dim3((max_jobs + 3) / 4), dim3(256), 0, s, t, max_jobs);
  return hipGetLastError();
}

template <int DT, int NCH>
hipError_t launch_inject_t(const TierArgs& t, hipStream_t s) {
  constexpr int WPB = 1;
  hipLaunchKernelGGL((k_tier_inject<DT, NCH, WPB>), dim3(t.look.T), dim3(64), 0, s, t);
  return hipGetLastError();
}

int chunks_of(int dtype, int dim) { return dim / (dtype == TFE_F32 ? 256 : 512); }

template <int DT, int NCH>
hipError_t launch_decode_t(const TierArgs& t, hipStream_t s) {
  hipLaunchKernelGGL((k_tier_decode<DT, NCH>), dim3(t.look.T), dim3(64), 0, s, t);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_tier_init(const TierArgs& t, uint32_t C, uint32_t prefill, hipStream_t s) {
  hipLaunchKernelGGL(k_tier_init, dim3((C + kDecodeMaxT + 255) / 256), dim3(256), 0, s, t, C,
                     prefill);
  return hipGetLastError();
}

hipError_t launch_ring_compact(const TierArgs& t, uint64_t* dst, uint64_t dst_mask,
                               bool restamp, hipStream_t s) {
  hipLaunchKernelGGL(k_ring_compact, dim3(1), dim3(kResolveThreads), 0, s, t, dst, dst_mask,
                     restamp ? 1u : 0u);
  return hipGetLastError();
}

hipError_t launch_tier_probe(const TierArgs& t, hipStream_t s) {
  if (t.look.T == 0) return hipSuccess;
  hipLaunchKernelGGL(k_tier_probe<1>, dim3(t.look.T), dim3(64), 0, s, t);
  return hipGetLastError();
}

bool lookup_resolve_fused(uint32_t T) { return T <= kSmallT; }

hipError_t launch_lookup_resolve_small(const TierArgs& t, hipStream_t s) {
  hipLaunchKernelGGL(k_lookup_resolve_small, dim3(1), dim3(kResolveThreads), 0, s, t);
  return hipGetLastError();
}

uint32_t lookup_resolve_one_block_max() { return kGroup; }

hipError_t launch_resolve_lookup(const TierArgs& t, hipStream_t s) {
  const uint32_t T = t.look.T;
  if (T <= (uint32_t)kGroup) {
    hipLaunchKernelGGL(k_resolve_lookup, dim3(1), dim3(kResolveThreads), 0, s, t, T);
    return hipGetLastError();
  }
  const uint32_t nblk = (T + kMarkThreads - 1) / kMarkThreads;
  hipLaunchKernelGGL(k_res_mark, dim3(nblk), dim3(kMarkThreads), 0, s, t, T);
  hipLaunchKernelGGL(k_res_first, dim3(nblk), dim3(kMarkThreads), 0, s, t, T);
  hipLaunchKernelGGL(k_res_pop, dim3(1), dim3(kResolveThreads), 0, s, t, nblk);
  hipLaunchKernelGGL(k_res_assign, dim3(nblk), dim3(kMarkThreads), 0, s, t, T);
  return hipGetLastError();
}

hipError_t launch_prefetch_probe(const TierArgs& t, const int32_t* tail, int32_t tail_len,
                                 const int32_t* cand, uint32_t B, uint32_t K, hipStream_t s) {
  hipLaunchKernelGGL(k_prefetch_probe<1>, dim3(B * K), dim3(64), 0, s, t, tail, tail_len, cand, B,
                     K);
  return hipGetLastError();
}

hipError_t launch_resolve_prefetch_scored(const TierArgs& t, uint32_t N, const float* prob,
                                         uint32_t budget, hipStream_t s) {
  hipLaunchKernelGGL(k_resolve_prefetch_scored, dim3(1), dim3(kResolveThreads), 0, s, t, N, prob,
                     budget);
  return hipGetLastError();
}

uint32_t scored_prefetch_budget_max() { return kScoredBudgetMax; }

uint32_t prefetch_fused_max() { return kPrefetchFusedMax; }

hipError_t launch_prefetch_fused(const TierArgs& t, const int32_t* tail, int32_t tail_len,
                                 const int32_t* cand, uint32_t B, uint32_t K, const float* prob,
                                 uint32_t budget, hipStream_t s) {
  if (B * K > kPrefetchFusedMax) return hipErrorInvalidValue;
  if (prob)
    hipLaunchKernelGGL(k_prefetch_fused<true>, dim3(1), dim3(kResolveThreads), 0, s, t, tail,
                       tail_len, cand, B, K, prob, budget);
  else
    hipLaunchKernelGGL(k_prefetch_fused<false>, dim3(1), dim3(kResolveThreads), 0, s, t, tail,
                       tail_len, cand, B, K, prob, budget);
  return hipGetLastError();
}

hipError_t launch_tier_wait(const TierArgs& t, hipStream_t s) {
  hipLaunchKernelGGL(k_tier_wait, dim3(1), dim3(64), 0, s, t);
  return hipGetLastError();
}

uint32_t fill_blocks(uint32_t max_jobs) { return (max_jobs + 3) / 4; }

hipError_t launch_residency(const int32_t* where, int64_t P, const int32_t* rows, int64_t n,
                            int32_t* out, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(k_residency, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, where, P,
                     rows, n, out);
  return hipGetLastError();
}

hipError_t launch_fill(const TierArgs& t, int dtype, int dim, uint32_t max_jobs, hipStream_t s) {
  switch (chunks_of(dtype, dim)) {
    case 1: return launch_fill_t<1>(t, max_jobs, s);
    case 2: return launch_fill_t<2>(t, max_jobs, s);
    case 4: return launch_fill_t<4>(t, max_jobs, s);
    case 8: return launch_fill_t<8>(t, max_jobs, s);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_tier_decode(const TierArgs& t, int dtype, int dim, hipStream_t s) {
  if (t.look.T == 0) return hipSuccess;
  if (t.look.T > kDecodeMaxT) return hipErrorInvalidValue;
  const int nch = chunks_of(dtype, dim);
  if (dtype == TFE_F32) {
    switch (nch) {
      case 1: return launch_decode_t<0, 1>(t, s);
      case 2: return launch_decode_t<0, 2>(t, s);
      case 4: return launch_decode_t<0, 4>(t, s);
      case 8: return launch_decode_t<0, 8>(t, s);
    }
  } else {
    switch (nch) {
      case 1: return launch_decode_t<1, 1>(t, s);
      case 2: return launch_decode_t<1, 2>(t, s);
      case 4: return launch_decode_t<1, 4>(t, s);
      case 8: return launch_decode_t<1, 8>(t, s);
    }
  }
  return hipErrorInvalidValue;
}

hipError_t launch_tier_inject(const TierArgs& t, int dtype, int dim, hipStream_t s) {
  if (t.look.T == 0) return hipSuccess;
  const int nch = chunks_of(dtype, dim);
  if (dtype == TFE_F32) {
    switch (nch) {
      case 1: return launch_inject_t<0, 1>(t, s);
      case 2: return launch_inject_t<0, 2>(t, s);
      case 4: return launch_inject_t<0, 4>(t, s);
      case 8: return launch_inject_t<0, 8>(t, s);
    }
  } else {
    switch (nch) {
      case 1: return launch_inject_t<1, 1>(t, s);
      case 2: return launch_inject_t<1, 2>(t, s);
      case 4: return launch_inject_t<1, 4>(t, s);
      case 8: return launch_inject_t<1, 8>(t, s);
    }
  }
  return hipErrorInvalidValue;
}

}  // namespace tfe
