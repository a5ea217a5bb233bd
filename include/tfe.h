/*
 * tfe.h -- C ABI of the TF-Engram phrase-memory lookup + inject library for
 * AMD MI355X (gfx950).
 *
 * The operation (paper: "TF-Engram: A Train-Free Engram with SSD-Backed
 * Memory for Large Language Models"):
 *   - the memory is a key -> value table whose keys are token n-grams
 *     (phrases) and whose values are D-wide vectors in the hidden space
 *     (Sec. 2.2, Eq. 2); each phrase has its own entry, so two phrases never
 *     share a slot (Sec. 1, Sec. 4.1, Sec. 4.2);
 *   - at every position t the n-grams that end at t, n = n_min..n_max, are
 *     matched exactly against the table (Eq. 3, first index level of Eq. 10)
 *     and the longest match is selected (Sec. 4.2);
 *   - the selected value row m is injected as h' = h + g * m (Eq. 5);
 *   - tables larger than device memory live in pinned host memory behind an
 *     HBM cache tier (Sec. 4.3, Eq. 12, lookup through the hierarchy), which
 *     is filled ahead of use from predicted next-token candidates (Sec. 4.4,
 *     Eq. 14-16).
 *
 * Conventions shared by every call:
 *   - "DEVICE" pointers are HIP device memory of the device that was current
 *     when the table was loaded; "HOST" pointers are ordinary host memory.
 *   - Streams are hipStream_t handles passed as void* (NULL = the default
 *     stream).  Device work is enqueued asynchronously; results are valid once
 *     the stream has reached the enqueued work.
 *   - Argument errors are detected on the host before anything is enqueued and
 *     return a negative status; tfe_last_error() then describes the problem.
 *     A failed HIP call returns TFE_ERR_HIP.  No C++ exception crosses the ABI.
 *   - A failed allocation returns TFE_ERR_OOM and leaks nothing: a failed
 *     load or head creation returns no handle and holds no memory; a lookup
 *     or prefetch that fails leaves the table usable, and its results and
 *     statistics as if the call had not been made (a scratch buffer grown
 *     before the failure stays with the table, as a successful call's
 *     would).  For tests of these paths, TFE_FAIL_ALLOC=k in the environment
 *     makes the k-th device, pinned-host or host allocation of every library
 *     call fail (the count restarts at each call).
 *   - A table handle is not thread-safe: calls on one handle must be issued
 *     from one host thread at a time.
 *   - HIP graph capture: lookups on resident tables (tfe_lookup_inject,
 *     tfe_lookup_inject_multi) and tfe_head_topk enqueue kernels only and may
 *     be captured.  Lookups on tiered tables, tfe_prefetch,
 *     tfe_prefetch_scored and tfe_ngram_top keep per-call host state or
 *     synchronise; on a capturing stream they return TFE_ERR_UNSUPPORTED
 *     without enqueuing anything.
 */
#ifndef TFE_H_
#define TFE_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct tfe_table tfe_table; /* opaque; owned by the library */

typedef enum {
  TFE_OK = 0,
  TFE_ERR_INVALID_ARG = -1,   /* bad size, pointer, length range or token */
  TFE_ERR_DUPLICATE_KEY = -2, /* the same phrase appears twice */
  TFE_ERR_OOM = -3,           /* device or pinned host allocation failed */
  TFE_ERR_HIP = -4,           /* a HIP runtime call or kernel launch failed */
  TFE_ERR_UNSUPPORTED = -5    /* valid request outside what is implemented */
} tfe_status;

typedef enum { TFE_F32 = 0, TFE_BF16 = 1 } tfe_dtype;

/* Gate of Eq. 5.  The paper allows a scalar, a vector or a function of h and
 * m; the method trains nothing, so the library offers two parameter-free
 * gates:
 *   TFE_GATE_SIGMOID: g = scale * sigmoid(<h / rms(h), m / rms(m)> / sqrt(D)),
 *                     rms(x) = sqrt(mean(x^2) + 1e-6), i.e. scale times the
 *                     logistic function of sqrt(D) * cos(h, m);
 *   TFE_GATE_CONST:   g = scale.
 * `scale` is the memory-injection scale of the evaluation (Sec. 5.1). */
typedef enum { TFE_GATE_SIGMOID = 0, TFE_GATE_CONST = 1 } tfe_gate;

/* Weights of the multi-match aggregation m = sum_i alpha_i v_i (Eq. 4,
 * Eq. 11; the paper lets alpha depend on phrase length, frequency or
 * confidence).  Over the phrases retained at one position:
 *   TFE_WEIGHT_LENGTH:  alpha_i = n_i / sum_k n_k  (n = phrase length);
 *   TFE_WEIGHT_UNIFORM: alpha_i = 1 / (number retained).
 * Both add up to 1, so one retained phrase injects its own row. */
typedef enum { TFE_WEIGHT_LENGTH = 0, TFE_WEIGHT_UNIFORM = 1 } tfe_weighting;

/* Tiered tables: how a row that a lookup finds only in host memory reaches
 * the cache slot it is given (staging into the faster tier, Sec. 4.3).
 * Either way the lookup injects the row read straight from host memory and
 * never waits for the copy.
 *   TFE_FILL_INLINE:      the injection kernel that reads the row also writes
 *                         it into the slot: one host read per missed row and
 *                         no cross-stream events;
 *   TFE_FILL_SIDE_STREAM: a copy kernel on the table's side stream, overlapped
 *                         with the injection, reads the row from host memory a
 *                         second time; the next call waits for it. */
typedef enum { TFE_FILL_INLINE = 0, TFE_FILL_SIDE_STREAM = 1 } tfe_fill_mode;

typedef struct {
  /* Phrases (Sec. 4.2): phrase i is phrase_tokens[i*n_max .. i*n_max+len-1],
   * oldest token first, len = phrase_len[i]; unused columns are ignored.
   * HOST memory, read during tfe_table_load only. */
  int64_t n_phrases;            /* P >= 0; P = 0 gives a table that never matches */
  int32_t n_min, n_max;         /* 2 <= n_min <= n_max <= 4 */
  int32_t vocab;                /* token ids are valid in [0, vocab), vocab <= 2^18 */
  const int32_t *phrase_tokens; /* HOST [P x n_max] */
  const uint8_t *phrase_len;    /* HOST [P], each in [n_min, n_max] */
  /* Value rows (Eq. 2): row i belongs to phrase i.  [P x dim], row-major. */
  const void *values;
  int32_t dim;                  /* D: bf16 512/1024/2048/4096, f32 256/512/1024/2048 */
  int32_t dtype;                /* tfe_dtype of values and of hidden states */
  int32_t values_on_device;     /* 1: `values` is DEVICE memory (copied); 0: HOST */
  double max_load_factor;       /* index occupancy bound in (0, 0.9]; 0 means 0.5 */
  /* Tiered mode (Sec. 4.3): hbm_cache_rows > 0 keeps the value rows in pinned
   * host memory and serves them through an HBM cache of that many rows with
   * least-recently-used replacement. */
  int64_t hbm_cache_rows;       /* 0: every value row is resident in HBM */
  int32_t adopt_host_values;    /* tiered: 1 = use the caller's `values` in place; it
                                   must come from hipHostMalloc and outlive the table */
  int64_t prefill_rows;         /* tiered: rows [0, prefill_rows) start cached */
  int32_t miss_fill;            /* tiered: tfe_fill_mode (0 = inline); must be 0 or 1 */
  /* Tiered, when not every row can be pinned (the pinnable host memory of a
   * process is limited): with 0 < pinned_rows < n_phrases, `values` holds
   * rows [0, pinned_rows) only (pinned as above), and rows [pinned_rows, P)
   * stay in the caller's pageable host memory `pageable_values`
   * (HOST [(P - pinned_rows) x dim], read in place; it must outlive the
   * table and not change).  A kernel that needs one of those rows has a
   * host thread of the table copy it into pinned staging memory first (the
   * staging of rows into GPU-readable memory of Sec. 4.3); results are the
   * same, only slower for those rows (a few microseconds each).  Order the
   * rows by expected use (e.g. phrase frequency) so the pinned ones are the
   * hot ones.  The table's host threads (4) need CPU time while kernels
   * wait for them: thread pools that spin while idle (OpenMP's default wait
   * policy; OMP_WAIT_POLICY=PASSIVE avoids it) delay them by milliseconds.
   * pinned_rows = 0 (or P): every row is pinned; pageable_values is ignored. */
  int64_t pinned_rows;
  const void *pageable_values;
} tfe_table_desc;

typedef struct {
  uint64_t calls;            /* tfe_lookup_inject(_multi) calls that returned TFE_OK */
  uint64_t positions;        /* injected positions looked up */
  uint64_t hits;             /* positions with a match (multi-match: any length) */
  uint64_t cache_hits;       /* tiered: matched rows found in the HBM cache */
  uint64_t cache_misses;     /* tiered: matched rows fetched from host memory */
  uint64_t prefetch_keys;    /* tiered: candidate phrases probed by tfe_prefetch */
  uint64_t prefetch_found;   /* tiered: candidate phrases present in the table */
  uint64_t prefetch_filled;  /* tiered: rows copied host -> HBM by tfe_prefetch */
  uint64_t prefetch_used;    /* tiered: prefetched rows later hit by a lookup */
  uint64_t host_bytes;       /* tiered: bytes read from host memory (both paths) */
  uint64_t prefetch_dropped; /* tiered: candidate rows worth fetching but over budget */
} tfe_stats;

/* Builds the exact-match phrase index and places the value rows.
 * Paper: Eq. 2 (table), Eq. 10 (token n-gram -> phrase id -> memory address),
 * Sec. 4.3 and Eq. 12 (tiers).
 * Rejects (before any device work) phrases whose length is outside
 * [n_min, n_max], tokens outside [0, vocab) and repeated phrases
 * (TFE_ERR_DUPLICATE_KEY).  The library copies the phrases, and copies the
 * values unless adopt_host_values is set.  `stream` orders the uploads; the
 * call returns after they completed.  On success *out owns all device and
 * pinned memory of the table until tfe_table_free. */
tfe_status tfe_table_load(const tfe_table_desc *desc, void *stream, tfe_table **out);

/* Releases a table (waits for its pending work made outside stream capture
 * first).  A captured graph that holds lookups of the table must have
 * finished running, and must not run again.  NULL is accepted. */
tfe_status tfe_table_free(tfe_table *table);

/* Lookup + inject for B rows of ctx + S tokens.
 * Paper: Eq. 3 (lookup from recent tokens), Sec. 4.2 (longest match),
 * Eq. 5 (gated residual injection), Sec. 4.3 (lookup through the hierarchy).
 *   tokens     DEVICE int32 [B x (ctx + S)], oldest first.  The first ctx
 *              columns of a row are history: they take part in the windows
 *              of later columns but are not injected.  Position (b, s) is
 *              column ctx + s of row b; its n-gram is columns
 *              ctx+s-n+1 .. ctx+s of the same row and exists only if it starts
 *              at column >= 0 and all its tokens are in [0, vocab).
 *   hidden_in  DEVICE [B*S x dim] of the table's dtype, row p = b*S + s.
 *   hidden_out DEVICE [B*S x dim]; may equal hidden_in (in place: rows
 *              without a match are then not written); partial overlap is
 *              undefined.
 *   hit_mask   DEVICE uint8 [B*S]: 1 where a phrase matched.
 *   slot_ids   DEVICE int32 [B*S]: the matched phrase's row id (its index in
 *              the loaded phrase list), -1 where nothing matched.
 *   match_len  DEVICE uint8 [B*S] or NULL: matched n, 0 where nothing matched.
 *   gate, scale: see tfe_gate.
 * Tiered tables read the rows that are not cached straight from pinned host
 * memory (zero-copy over PCIe) and insert them into the HBM cache for later
 * calls, from the copy the inject read (TFE_FILL_INLINE) or with a second
 * read on an internal side stream (TFE_FILL_SIDE_STREAM); results do not
 * depend on the cache state. */
tfe_status tfe_lookup_inject(tfe_table *table, const int32_t *tokens, int32_t B, int32_t ctx,
                             int32_t S, const void *hidden_in, void *hidden_out,
                             uint8_t *hit_mask, int32_t *slot_ids, uint8_t *match_len,
                             int32_t gate, float scale, void *stream);

/* Multi-match lookup + inject (resident tables).
 * Paper: Eq. 4 and Eq. 11 (every matched phrase retained, memory vectors
 * aggregated with weights alpha_i), Eq. 3, Eq. 5.
 * Same tokens, windows, hidden_in / hidden_out, gate and scale as
 * tfe_lookup_inject; every n-gram ending at the position that is in the
 * table is retained (at most one per length) and m = sum_i alpha_i v_i with
 * the weights of `weighting` (tfe_weighting) replaces the single row.  The
 * aggregate is kept in float32 and rounded only in h'.
 *   match_mask DEVICE uint8 [B*S]: bit j set where the phrase of length
 *              n_min + j matched (0: no match, the row is left unchanged).
 *   slot_ids   DEVICE int32 [B*S x L], L = n_max - n_min + 1: column j is
 *              the row id of the matched phrase of length n_min + j, -1 if
 *              none.
 * Returns TFE_ERR_UNSUPPORTED for tiered tables (hbm_cache_rows > 0). */
tfe_status tfe_lookup_inject_multi(tfe_table *table, const int32_t *tokens, int32_t B,
                                   int32_t ctx, int32_t S, const void *hidden_in,
                                   void *hidden_out, uint8_t *match_mask, int32_t *slot_ids,
                                   int32_t weighting, int32_t gate, float scale, void *stream);

/* Prefetch for the next step (tiered tables; a no-op on resident tables).
 * Paper: Eq. 14 (top-K next-token candidates), Eq. 15 (candidate phrases via
 * the token-to-phrase index), Eq. 16 (fetch overlapped with the remaining
 * layers), Sec. 4.3 (insert into the faster tier).
 *   tail        DEVICE int32 [B x tail_len]: the last tail_len tokens of each
 *               row, oldest first (tail_len >= n_max - 1 uses every length).
 *   candidates  DEVICE int32 [B x K]: predicted next tokens of each row.
 * For every row b and candidate c the phrases ending at c, i.e. the n-grams
 * (tail[b, tail_len-n+1 ..], c) for n = n_min..n_max, are looked up; the
 * longest one present in the table (the phrase the next lookup selects if c
 * is the next token) is that candidate's row.  The candidates' rows are
 * referenced as a lookup references its positions' rows: cached ones are
 * never evicted by this prefetch and become most recent; the others are
 * copied into least-recently-used unreferenced slots (in candidate order,
 * while such slots are left) and become most recent too.
 * The work runs on `side_stream` after the table's previous lookup; the
 * next tfe_lookup_inject waits for it. */
tfe_status tfe_prefetch(tfe_table *table, const int32_t *tail, int32_t tail_len,
                        const int32_t *candidates, int32_t B, int32_t K, void *side_stream);

/* Priority-scored, budgeted prefetch (tiered tables; a no-op on resident
 * tables).  Paper: Eq. 17 (s_i = p_i * r_i * c_i; high-priority candidates
 * first, low-priority ones dropped when the I/O budget is exhausted) and the
 * tunable top-K budget and queue size (Sec. 4.4).
 * Same windows as tfe_prefetch; additionally
 *   cand_prob   DEVICE float [B x K]: p_i, the predicted probability of each
 *               candidate token (values <= 0 or NaN count as 0);
 *   budget      at most this many rows are fetched (<= 1024).
 * Each candidate's longest match r gets s = p * len(r) * c, with c = 1 when
 * the row is only in host memory and 0 when it is cached (r_i reads as the
 * phrase length: longer phrases are the more specific entries).  A row named
 * by several candidates keeps its highest score.  Cached rows with a
 * positive p * len are referenced (not evicted by this prefetch; most
 * recent, by first candidate).  Rows with a positive score are fetched by
 * descending score (ties: lowest candidate index) until the budget or the
 * unreferenced cache slots run out; the rest count as dropped.  Any B * K
 * (scratch of about 40 bytes per candidate stays with the table). */
tfe_status tfe_prefetch_scored(tfe_table *table, const int32_t *tail, int32_t tail_len,
                               const int32_t *candidates, const float *cand_prob, int32_t B,
                               int32_t K, int32_t budget, void *side_stream);

/* ---- Early-exit prefetch head ---------------------------------------------
 * Paper: Eq. 13 (approximate next-token distribution softmax(W_pref h) from
 * the hidden state of an intermediate layer), Eq. 14 (its top-K tokens), and
 * Sec. 4.4 (the candidates drive the prefetch: pass top_ids and top_prob to
 * tfe_prefetch_scored as candidates and cand_prob). */
typedef struct tfe_head tfe_head; /* opaque; owned by the library */

/* Prepares a head for the projection w_pref: DEVICE bf16 [vocab x dim],
 * row-major, 16-byte aligned, on the current device.  The head keeps the
 * pointer (no copy): w_pref must stay valid and unchanged until
 * tfe_head_free.  dim is 256, 512 or 1024; 1 <= vocab <= 2^18;
 * 1 <= max_k <= min(256, vocab); 1 <= max_batch <= 65535 sizes the scratch
 * (max_batch x vocab float32 logits plus candidate lists, and the one-launch
 * path's per-block maxima and candidate segments: 64 rows x compute units x
 * (16 x ceil(vocab / (16 x compute units)) + 1) keys, rounded up to 16,
 * about 80 MB for the 151936-token vocabulary on 256 compute units). */
tfe_status tfe_head_create(const void *w_pref, int32_t vocab, int32_t dim, int32_t max_batch,
                           int32_t max_k, tfe_head **out);

/* For each of the B rows of `hidden` (DEVICE bf16 [B x dim], 16-byte
 * aligned): top_ids[b*K + i] (DEVICE int32) is the token of i-th largest
 * probability under softmax(W_pref h_b) (ties in logit go to the lower id)
 * and top_prob[b*K + i] (DEVICE float32) its probability.  Logits and the
 * softmax are computed in float32 (bf16 products, float32 accumulation).
 * 0 <= B <= max_batch, 0 <= K <= max_k; stream-ordered on `stream`.  Calls
 * on one head share its scratch: they must be ordered (same stream, or
 * synchronised).
 * Calls of at most 64 rows with K at most the number of compute units (a
 * power of two up to 256; at most 48 16-token tiles per compute unit)
 * take a one-launch path, also under stream capture: one block per
 * compute unit keeps its logits in registers, and two device-wide barriers
 * inside the launch replace the write of the logits.  Its blocks must all
 * be resident at once: the library runs the one-launch calls of all heads
 * on a device one after another (each waits on the device for the previous
 * one, whatever its stream; a captured call is ordered only by its graph
 * and the stream the graph is launched on, so two such calls must not sit
 * on parallel branches, nor run beside an eager one-launch call of another
 * head on another stream), and such
 * a call must not overlap on the device with other work that holds compute
 * units while waiting for it.  Its waits are bounded
 * (about a second); if one runs out,
 * that call's top_ids are all -1 and its top_prob 0.  Other calls take two
 * launches (logits, then the per-row selection), which have no such
 * requirement. */
tfe_status tfe_head_topk(tfe_head *head, const void *hidden, int32_t B, int32_t K,
                         int32_t *top_ids, float *top_prob, void *stream);

/* *call = the number, counted from 1 over the head's one-launch calls, of
 * the latest one-launch call whose barrier waits gave up (its top_ids all
 * -1 and its top_prob 0), or 0 if none has.  Waits for the head's last call
 * made outside stream capture first; calls replayed from a graph count like
 * the others.  For callers that cannot read every call's ids back. */
tfe_status tfe_head_last_fault(tfe_head *head, int64_t *call);

/* Releases a head (waits for its last call made outside stream capture
 * first).  A captured graph that holds calls of the head must have finished
 * running, and must not run again.  NULL is accepted. */
tfe_status tfe_head_free(tfe_head *head);

/* tfe_head_topk without a head and without any allocation, for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc).  Same arguments and results as
 * tfe_head_create(w_pref, vocab, dim, B, K) + tfe_head_topk(...), always
 * through the two-launch kernels (the same ids as the one-launch path, and
 * probabilities within float32 rounding of its):
 *   w_pref  DEVICE bf16 [vocab x dim], 16-byte aligned, on the current device;
 *   hidden  DEVICE bf16 [B x dim], 16-byte aligned;
 *   top_ids DEVICE int32 [B x K], top_prob DEVICE float32 [B x K].
 * Limits: 0 <= B <= 64, 1 <= vocab <= 2^18, 0 <= K <= min(256, vocab), dim
 * 256, 512 or 1024; larger sizes return TFE_ERR_INVALID_ARG.  The scratch
 * (logits, tile statistics and the logits blocks' maxima: 76.5 MiB) is a
 * static device array that every GPU the library runs on holds until the
 * process ends; the call allocates nothing.  A device with more than 1024
 * compute units is refused (TFE_ERR_UNSUPPORTED).  Every call on one GPU shares that GPU's scratch: calls that
 * overlap on one GPU (different streams, or host threads) race and must be
 * ordered by the caller. */
tfe_status tfe_head_topk_noalloc(const void *w_pref, int32_t vocab, int32_t dim,
                                 const void *hidden, int32_t B, int32_t K, int32_t *top_ids,
                                 float *top_prob, void *stream);

/* ---- Offline phrase-table construction -----------------------------------
 * Paper: Sec. 4.2 (candidate phrases mined from a corpus and selected by
 * frequency; n-gram extraction is the dominant construction cost reported in
 * the evaluation).
 * Counts the distinct n-grams of a token stream and returns the most
 * frequent ones: every window tokens[i .. i+n-1] whose tokens all lie in
 * [0, vocab) is one occurrence of its tuple (tokens outside the range, e.g.
 * -1 document separators, break windows); distinct tuples are ranked by
 * count, most frequent first, equal counts by the tuple in lexicographic
 * order (oldest token first); ranks [skip, skip + top) are written.
 *   tokens      DEVICE int32 [n_tokens], n_tokens <= 2^28
 *   vocab       1 <= vocab <= 2^18;  n: 1 <= n <= 4
 *   out_tuples  DEVICE int32 [top x n], oldest token first
 *   out_counts  DEVICE int64 [top]
 *   written     HOST: number of ranks written (fewer than top when the
 *               stream has fewer than skip + top distinct tuples)
 * Synchronous: returns once the outputs are complete.  Its scratch (device
 * memory of the current device: about 20 bytes per token, 40 for 4-grams)
 * stays with the library after the call and is reused by later calls of a
 * similar size, until tfe_ngram_release; a call that finds no fitting idle
 * buffer first returns the idle ones.  Safe to call from several host
 * threads (each call takes buffers of its own). */
tfe_status tfe_ngram_top(const int32_t *tokens, int64_t n_tokens, int32_t vocab, int32_t n,
                         int64_t skip, int64_t top, int32_t *out_tuples, int64_t *out_counts,
                         int64_t *written, void *stream);

/* Returns the idle scratch that tfe_ngram_top keeps for reuse (all devices)
 * to the device allocator.  Buffers of calls still running are kept. */
tfe_status tfe_ngram_release(void);

/* Copies the table's counters.  Waits on the host for the work the table
 * has enqueued (its last lookup's stream up to now, a pending prefetch, the
 * table's internal stream) and for nothing else: other streams keep running.
 * The stream of the last lookup must still exist.  `calls` and `positions`
 * count API calls; a lookup captured into a HIP graph counts its matched
 * positions in `hits` at every replay (once the replay's stream has been
 * synchronised by the caller), its call and positions once. */
tfe_status tfe_get_stats(const tfe_table *table, tfe_stats *out);

/* Resets the table's counters to zero, after the table's pending work (the
 * same wait as tfe_get_stats). */
tfe_status tfe_reset_stats(tfe_table *table);

/* Residency of phrase rows: where each phrase's memory vector lives (the
 * second index level of Eq. 10, phrase id -> storage tier and offset, and the
 * tiers of Eq. 12).
 *   rows  DEVICE int32 [n]: phrase row ids.
 *   out   DEVICE int32 [n]: tiered tables: the HBM cache slot holding the
 *         row, or -1 where it is only in host memory; resident tables: the
 *         row itself (every row is in HBM at its own index); -2 for ids
 *         outside [0, n_phrases).
 * Stream-ordered on `stream` after the table's last lookup and a pending
 * prefetch; changes nothing. */
tfe_status tfe_residency(const tfe_table *table, const int32_t *rows, int64_t n, int32_t *out,
                         void *stream);

/* Message describing the last error returned on this host thread ("" if none). */
const char *tfe_last_error(void);

/* Device and pinned host bytes the library holds right now, over every
 * table, head and construction buffer of the process (either pointer may be
 * NULL, not both).  Returns to its earlier value once what was loaded or
 * created since is freed (and tfe_ngram_release has run).  No GPU needed. */
tfe_status tfe_memory_held(int64_t *device_bytes, int64_t *pinned_bytes);

/* ---- Host-only index utilities (no GPU needed) ----------------------------
 * The index is an open-addressing table of 16-byte slots grouped in buckets
 * of 8 (128 bytes): {uint64 key, uint32 key_ext, int32 row}.  A phrase of n
 * tokens x0..x{n-1} (oldest first) has key = n << 61 | x{n-3} << 36 |
 * x{n-2} << 18 | x{n-1} (absent tokens are 0) and key_ext = x0 when n = 4,
 * else 0.  Its home bucket is murmur3-fmix64(key ^ key_ext * 0x9E3779B97F4A7C15)
 * mod (capacity / 8); a phrase lives in the first bucket at or after its home
 * bucket (cyclically) that had a free slot when it was inserted; an empty slot
 * has key = ~0.  Capacity = smallest power of two >= max(8, P / load factor). */

/* Number of slots for n_phrases phrases at the given load factor (0 = 0.5). */
int64_t tfe_index_capacity(int64_t n_phrases, double max_load_factor);

/* Builds the index into caller memory `slots` of 16 * capacity bytes (HOST).
 * Same validation as tfe_table_load. */
tfe_status tfe_index_build_host(const int32_t *phrase_tokens, const uint8_t *phrase_len,
                                int64_t n_phrases, int32_t n_min, int32_t n_max,
                                int32_t vocab, void *slots, int64_t capacity);

/* Looks one phrase up in a host-built index.  *row = its row or -1;
 * *buckets_read = buckets inspected (>= 1); *home = its home bucket. */
tfe_status tfe_index_probe_host(const void *slots, int64_t capacity, const int32_t *tokens,
                                int32_t n, int32_t *row, int32_t *buckets_read, int64_t *home);

#ifdef __cplusplus
}
#endif

#endif /* TFE_H_ */
