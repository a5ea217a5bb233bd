"""Reference model of the HBM cache tier's replacement policy.

TEST INFRASTRUCTURE ONLY (see the package docstring).  A plain Python model
of the residency bookkeeping that the tiered table keeps on the device, used
to check the device's cache statistics exactly.  It follows the paper's
lookup through the hierarchy (Sec. 4.3: check the GPU cache, else stage the
entry from host memory and insert it into the faster tier) with recency as
the cache-ranking signal (Sec. 4.3 lists recency among the ranking inputs)
and the prefetch of candidate phrases (Eq. 15) into the cache.

Policy (the precise reading; a call is one lookup or one prefetch):
* The cache has C slots.  At load, slot s holds row s for s < prefill; the
  recency order from least to most recent is: empty slots by ascending slot,
  then filled slots by descending row (the least frequent row goes first).
* Lookup: the distinct matched rows of the call are taken in order of their
  first position.  First, every such row that is cached marks its slot
  referenced -- whichever position of the call names it.  Then each row that
  is not cached, in that order, takes the least recent slot that is not
  referenced in this call (its old row leaves the cache, and the slot counts
  as referenced from then on); a row that finds no such slot is read from
  host memory without being cached.  Finally every referenced slot becomes
  most recent, in order of the first position that named its row.  So a
  victim is never a slot that any position of the same call uses, however
  long the call (nothing here depends on how an implementation splits a
  call into blocks).
* Prefetch: the candidates' matched rows are referenced exactly like a
  lookup's rows (candidate order stands for position order): cached rows
  mark their slots referenced first, so a prefetch never evicts a row it
  names itself (the paper ranks cache entries by prefetch confidence among
  other signals, Sec. 4.3); then each distinct row that is not cached takes
  the least recent slot that is not referenced (none left: it stays in host
  memory) and is marked prefetched; finally every referenced slot becomes
  most recent in order of first candidate.  Nothing is counted as a hit.
* Scored prefetch (Eq. 17): a candidate's score is p * len as if its row
  were not cached; a row keeps its best score and its first candidate.
  Cached rows with a positive score are referenced (most recent, in order
  of first candidate); the rows that are not cached and score above zero
  are filled by descending score, then first candidate, into least recent
  unreferenced slots, up to the budget; they become most recent after the
  referenced rows, in fill order.
* Statistics: hits = matched positions; cache_hits = matched positions whose
  row was cached when the call began (cache_misses = the rest);
  prefetch_used counts a prefetched slot the first time a lookup finds it
  cached.  A position is served from host memory when its row was not cached
  when the call began (it was filled by this call or found no slot);
  host_bytes = row bytes x positions served from host, plus row bytes x rows
  filled when the fill is a separate copy that reads the row from host
  memory again (fill_rereads=True; the library's side-stream fill).  Rows
  filled by a prefetch always count once.
"""
import collections


class LruModel:
    def __init__(self, cache_rows, prefill_rows, row_bytes, fill_rereads=False):
        self.C = cache_rows
        self.row_bytes = row_bytes
        self.fill_rereads = fill_rereads
        self.slot_row = [-1] * cache_rows
        self.where = {}
        # Recency order: OrderedDict of slot -> None, least recent first.
        self.order = collections.OrderedDict()
        for s in range(prefill_rows, cache_rows):
            self.order[s] = None
        for s in range(prefill_rows - 1, -1, -1):
            self.order[s] = None
        for s in range(prefill_rows):
            self.slot_row[s] = s
            self.where[s] = s
        self.prefetched = set()
        self.stats = collections.Counter()

    def _victim(self, referenced):
        for s in self.order:
            if s not in referenced:
                return s
        return None

    def _fill(self, row, slot):
        old = self.slot_row[slot]
        if old >= 0:
            del self.where[old]
        self.slot_row[slot] = row
        self.where[row] = slot

    def _resolve(self, rows, pref_fill):
        """The referencing step shared by lookups and prefetches: returns the
        per-row status (('cache', slot), ('fill', slot) or ('host', None))
        and the number of rows filled."""
        first_pos = {}
        for r in rows:
            if r >= 0 and r not in first_pos:
                first_pos[r] = len(first_pos)
        # Every cached row of the call is referenced before any victim is
        # chosen.
        status = {}
        referenced = set()
        newly = []
        for r in first_pos:
            if r in self.where:
                s = self.where[r]
                referenced.add(s)
                status[r] = ("cache", s)
                newly.append((first_pos[r], s))
        filled = 0
        for r in first_pos:
            if r in status:
                continue
            v = self._victim(referenced)
            if v is None:
                status[r] = ("host", None)
                continue
            self._fill(r, v)
            if pref_fill:
                self.prefetched.add(v)
            else:
                self.prefetched.discard(v)
            referenced.add(v)
            filled += 1
            newly.append((first_pos[r], v))
            status[r] = ("fill", v)
        for _, s in sorted(newly):
            self.order.move_to_end(s)
        return status, filled

    def lookup(self, rows):
        """rows: matched row per position (-1 = no match).  Returns the list of
        per-position sources: ('cache', slot), ('fill', slot), ('host', None)
        or None for a miss."""
        status, filled = self._resolve(rows, pref_fill=False)
        out = []
        for r in rows:
            if r < 0:
                out.append(None)
                continue
            self.stats["hits"] += 1
            kind, s = status[r]
            out.append((kind, s))
            if kind == "cache":
                self.stats["cache_hits"] += 1
                if s in self.prefetched:
                    self.prefetched.discard(s)
                    self.stats["prefetch_used"] += 1
            else:
                self.stats["cache_misses"] += 1
                self.stats["host_bytes"] += self.row_bytes
        if self.fill_rereads:
            self.stats["host_bytes"] += self.row_bytes * filled
        self.stats["positions"] += len(rows)
        return out

    def prefetch(self, cand_rows):
        """cand_rows: matched row per candidate (-1 = none), candidate order."""
        self.stats["prefetch_keys"] += len(cand_rows)
        self.stats["prefetch_found"] += sum(1 for r in cand_rows if r >= 0)
        _, filled = self._resolve(cand_rows, pref_fill=True)
        self.stats["prefetch_filled"] += filled
        self.stats["host_bytes"] += self.row_bytes * filled

    def prefetch_scored(self, cand_rows, cand_lens, cand_probs, budget):
        """Priority-scored, budgeted prefetch (Eq. 17, s = p * r * c): each
        candidate's matched row scores float32(p) * float32(len) (p <= 0 or
        NaN: 0); a row keeps its best score and its first candidate index.
        Cached rows with a positive score are referenced (c = 0: nothing to
        fetch, but not evictable by this prefetch) and become most recent in
        order of first candidate; the rows that are not cached (c = 1) and
        score above zero are filled by descending score, then candidate
        index, up to `budget` fills or until no unreferenced slot is left
        (the others count as dropped); filled slots become most recent in
        fill order, after the referenced ones."""
        import numpy as np
        self.stats["prefetch_keys"] += len(cand_rows)
        self.stats["prefetch_found"] += sum(1 for r in cand_rows if r >= 0)
        best = {}
        for q, r in enumerate(cand_rows):
            if r < 0:
                continue
            p = np.float32(cand_probs[q])
            p = p if p > 0 else np.float32(0)
            s = np.float32(p * np.float32(cand_lens[q]))
            if r not in best:
                best[r] = [s, q]
            elif s > best[r][0]:
                best[r][0] = s
        refs = sorted((q, r) for r, (s, q) in best.items() if s > 0 and r in self.where)
        referenced = set()
        for _, r in refs:
            referenced.add(self.where[r])
        for _, r in refs:
            self.order.move_to_end(self.where[r])
        entries = [(r, s, q) for r, (s, q) in best.items() if s > 0 and r not in self.where]
        entries.sort(key=lambda e: (-float(e[1]), e[2]))
        fills = 0
        for r, _, _ in entries[:budget]:
            v = self._victim(referenced)
            if v is None:
                break
            self._fill(r, v)
            referenced.add(v)
            self.order.move_to_end(v)
            self.prefetched.add(v)
            fills += 1
        self.stats["prefetch_filled"] += fills
        self.stats["prefetch_dropped"] += len(entries) - fills
        self.stats["host_bytes"] += self.row_bytes * fills

    def resident(self):
        return dict(self.where)
