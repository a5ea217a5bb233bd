// C ABI of libtfe: table load/free, lookup + inject, prefetch, statistics.
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <new>
#include <vector>

#include "../../include/tfe.h"
#include "tfe_internal.h"

namespace tfe {

static thread_local char g_err[512] = "";

tfe_status fail(tfe_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return st;
}

void clear_error() { g_err[0] = 0; }

static tfe_status hip_fail(hipError_t e, const char* what) {
  return fail(TFE_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

#define TFE_HIP(call, what)                                   \
  do {                                                        \
    hipError_t e_ = (call);                                   \
    if (e_ != hipSuccess) return hip_fail(e_, what);          \
  } while (0)

static size_t elem_size(int dtype) { return dtype == TFE_F32 ? 4 : 2; }

static void release(tfe_table* t) {
  if (!t) return;
  // Teardown is best effort: errors here have no one to report to.
  int cur = 0;
  (void)hipGetDevice(&cur);
  (void)hipSetDevice(t->device);
  (void)hipDeviceSynchronize();
  if (t->d_slots) (void)hipFree(t->d_slots);
  if (t->d_values) (void)hipFree(t->d_values);
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

static tfe_status load(const tfe_table_desc* d, hipStream_t stream, tfe_table** out) {
  if (!d || !out) return fail(TFE_ERR_INVALID_ARG, "null desc or out");
  *out = nullptr;
  if (d->dtype != TFE_F32 && d->dtype != TFE_BF16) return fail(TFE_ERR_INVALID_ARG, "bad dtype");
  if (!dim_supported(d->dtype, d->dim))
    return fail(TFE_ERR_UNSUPPORTED, "dim %d not supported for dtype %d", d->dim, d->dtype);
  double lf = d->max_load_factor == 0.0 ? 0.5 : d->max_load_factor;
  if (!(lf > 0.0 && lf <= 0.9)) return fail(TFE_ERR_INVALID_ARG, "max_load_factor not in (0, 0.9]");
  if (d->hbm_cache_rows < 0) return fail(TFE_ERR_INVALID_ARG, "hbm_cache_rows < 0");
  if (d->hbm_cache_rows > 0) return fail(TFE_ERR_UNSUPPORTED, "tiered tables not built yet");
  tfe_status st = validate_phrases(d->phrase_tokens, d->phrase_len, d->n_phrases, d->n_min,
                                   d->n_max, d->vocab);
  if (st != TFE_OK) return st;
  if (d->n_phrases > 0 && !d->values) return fail(TFE_ERR_INVALID_ARG, "null values");

  const int64_t cap = index_capacity(d->n_phrases, lf);
  std::vector<tfe_slot> slots;
  try {
    slots.resize((size_t)cap);
  } catch (const std::bad_alloc&) {
    return fail(TFE_ERR_OOM, "host index of %lld slots", (long long)cap);
  }
  st = build_index(d->phrase_tokens, d->phrase_len, d->n_phrases, d->n_max, slots.data(), cap);
  if (st != TFE_OK) return st;

  tfe_table* t = new (std::nothrow) tfe_table;
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

  const size_t slot_bytes = (size_t)cap * sizeof(tfe_slot);
  if (hipMalloc((void**)&t->d_slots, slot_bytes) != hipSuccess) {
    release(t);
    return fail(TFE_ERR_OOM, "device index (%zu bytes)", slot_bytes);
  }
  hipError_t e = hipMemcpyAsync(t->d_slots, slots.data(), slot_bytes, hipMemcpyHostToDevice, stream);
  if (e == hipSuccess && d->n_phrases > 0) {
    const size_t vbytes = (size_t)d->n_phrases * d->dim * elem_size(d->dtype);
    if (hipMalloc(&t->d_values, vbytes) != hipSuccess) {
      release(t);
      return fail(TFE_ERR_OOM, "device values (%zu bytes)", vbytes);
    }
    e = hipMemcpyAsync(t->d_values, d->values, vbytes,
                       d->values_on_device ? hipMemcpyDeviceToDevice : hipMemcpyHostToDevice,
                       stream);
  }
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  if (e != hipSuccess) {
    release(t);
    return hip_fail(e, "table upload");
  }
  *out = t;
  return TFE_OK;
}

static tfe_status lookup_inject(tfe_table* t, const int32_t* tokens, int32_t B, int32_t ctx,
                                int32_t S, const void* hin, void* hout, uint8_t* hit,
                                int32_t* slot, uint8_t* len, int32_t gate, float scale,
                                hipStream_t stream) {
  if (!t) return fail(TFE_ERR_INVALID_ARG, "null table");
  if (B < 0 || ctx < 0 || S < 0) return fail(TFE_ERR_INVALID_ARG, "negative B, ctx or S");
  if (gate != TFE_GATE_SIGMOID && gate != TFE_GATE_CONST) return fail(TFE_ERR_INVALID_ARG, "bad gate");
  if (!isfinite(scale)) return fail(TFE_ERR_INVALID_ARG, "scale is not finite");
  const int64_t T = (int64_t)B * S;
  if ((int64_t)ctx + S > 0x7FFFFFFFll) return fail(TFE_ERR_INVALID_ARG, "ctx + S overflows");
  if (T > 0x7FFFFFFFll) return fail(TFE_ERR_UNSUPPORTED, "B * S above 2^31 - 1 positions");
  t->stats.calls++;
  if (T == 0) return TFE_OK;
  if (!tokens || !hin || !hout || !hit || !slot)
    return fail(TFE_ERR_INVALID_ARG, "null tokens, hidden, hit_mask or slot_ids");
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
  TFE_HIP(launch_lookup_inject(a, t->dtype, t->dim, stream), "lookup_inject launch");
  t->stats.positions += (uint64_t)T;
  return TFE_OK;
}

}  // namespace tfe

extern "C" {

tfe_status tfe_table_load(const tfe_table_desc* desc, void* stream, tfe_table** out) {
  tfe::clear_error();
  return tfe::load(desc, (hipStream_t)stream, out);
}

tfe_status tfe_table_free(tfe_table* table) {
  tfe::clear_error();
  tfe::release(table);
  return TFE_OK;
}

tfe_status tfe_lookup_inject(tfe_table* table, const int32_t* tokens, int32_t B, int32_t ctx,
                             int32_t S, const void* hidden_in, void* hidden_out,
                             uint8_t* hit_mask, int32_t* slot_ids, uint8_t* match_len,
                             int32_t gate, float scale, void* stream) {
  tfe::clear_error();
  return tfe::lookup_inject(table, tokens, B, ctx, S, hidden_in, hidden_out, hit_mask, slot_ids,
                            match_len, gate, scale, (hipStream_t)stream);
}

tfe_status tfe_prefetch(tfe_table* table, const int32_t* tail, int32_t tail_len,
                        const int32_t* candidates, int32_t B, int32_t K, void* side_stream) {
  tfe::clear_error();
  (void)side_stream;
  if (!table) return tfe::fail(TFE_ERR_INVALID_ARG, "null table");
  if (tail_len < 0 || B < 0 || K < 0) return tfe::fail(TFE_ERR_INVALID_ARG, "negative size");
  if ((int64_t)B * K > 0 && (!candidates || (tail_len > 0 && !tail)))
    return tfe::fail(TFE_ERR_INVALID_ARG, "null tail or candidates");
  return TFE_OK;  // resident tables have nothing to prefetch
}

tfe_status tfe_get_stats(tfe_table* table, tfe_stats* out) {
  tfe::clear_error();
  if (!table || !out) return tfe::fail(TFE_ERR_INVALID_ARG, "null table or out");
  *out = table->stats;
  return TFE_OK;
}

tfe_status tfe_reset_stats(tfe_table* table) {
  tfe::clear_error();
  if (!table) return tfe::fail(TFE_ERR_INVALID_ARG, "null table");
  table->stats = tfe_stats{};
  return TFE_OK;
}

const char* tfe_last_error(void) { return tfe::g_err; }

}  // extern "C"
