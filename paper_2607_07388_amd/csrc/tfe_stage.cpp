// Staging of pageable host rows for tiered tables (Sec. 4.3: the value rows
// live in a hierarchy of memories, and rows that the GPU cannot read in
// place are staged into memory it can read).
//
// Host memory that can be pinned is limited per process; rows beyond the
// pinned ones stay in the caller's pageable memory.  A kernel that needs
// such a row posts a request in a queue of kStageSlots slots in coherent
// pinned memory (see StageSlot); the threads started here copy the row from
// pageable memory into the slot's staging row and publish it.  Thread i of
// n serves tickets i, i + n, i + 2n, ... in order, so a slot is never served
// before the kernel has posted it, and a kernel only posts into a slot once
// the slot's previous ticket has been read (its ack), so a staging row is
// never overwritten while it is read.
//
// The serving loop itself (stage_serve) is host-only code, tested on the CPU
// with emulated requesters.
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <string.h>

#include <new>
#include <thread>
#include <vector>

#include "../../include/tfe.h"
#include "tfe_internal.h"

namespace tfe {

struct Stager {
  StageSlot* q = nullptr;       // host address of the queue
  char* rows = nullptr;         // host address of the staging rows
  StageSlot* q_dev = nullptr;   // device addresses of both
  const void* rows_dev = nullptr;
  const char* pageable = nullptr;
  int64_t first_row = 0, n_rows = 0;
  size_t row_bytes = 0;
  volatile bool stop = false;
  std::vector<std::thread> threads;
};

tfe_status stager_start(const void* pageable, int64_t pinned_rows, int64_t n_phrases,
                        size_t row_bytes, int threads, Stager** out) {
  *out = nullptr;
  Stager* s = alloc_fails() ? nullptr : new (std::nothrow) Stager;
  if (!s) return fail(TFE_ERR_OOM, "staging state");
  s->pageable = (const char*)pageable;
  s->first_row = pinned_rows;
  s->n_rows = n_phrases - pinned_rows;
  s->row_bytes = row_bytes;
  const size_t qbytes = kStageSlots * sizeof(StageSlot);
  const size_t rbytes = kStageSlots * row_bytes;
  void* q = nullptr;
  void* rows = nullptr;
  if (pinned_malloc(&q, qbytes, hipHostMallocCoherent) != hipSuccess ||
      pinned_malloc(&rows, rbytes, hipHostMallocCoherent) != hipSuccess) {
    pinned_free(q);
    delete s;
    return fail(TFE_ERR_OOM, "staging queue (%zu bytes)", qbytes + rbytes);
  }
  memset(q, 0, qbytes);
  memset(rows, 0, rbytes);
  s->q = (StageSlot*)q;
  s->rows = (char*)rows;
  void *qd = nullptr, *rd = nullptr;
  if (hipHostGetDevicePointer(&qd, q, 0) != hipSuccess ||
      hipHostGetDevicePointer(&rd, rows, 0) != hipSuccess) {
    (void)hipGetLastError();
    pinned_free(q);
    pinned_free(rows);
    delete s;
    return fail(TFE_ERR_HIP, "staging queue device address");
  }
  s->q_dev = (StageSlot*)qd;
  s->rows_dev = rd;
  try {
    for (int i = 0; i < threads; ++i)
      s->threads.emplace_back(stage_serve, s->q, s->rows, s->pageable, s->first_row, s->n_rows,
                              s->row_bytes, (uint64_t)i, (uint64_t)threads, &s->stop);
  } catch (...) {
    stager_stop(s);
    return fail(TFE_ERR_OOM, "staging threads");
  }
  *out = s;
  return TFE_OK;
}

StageSlot* stager_queue(const Stager* s) { return s->q_dev; }
const void* stager_rows(const Stager* s) { return s->rows_dev; }

void stager_stop(Stager* s) {
  if (!s) return;
  __atomic_store_n(&s->stop, true, __ATOMIC_RELEASE);
  for (std::thread& t : s->threads) t.join();
  pinned_free(s->q);
  pinned_free(s->rows);
  delete s;
}

}  // namespace tfe
