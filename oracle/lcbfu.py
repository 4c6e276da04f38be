"""Cache maintenance under the LCBFU policy, and hole-aware state choice
(test infrastructure only).

Follows Sec. 5.4 (cache maintenance): every cached intermediate state i
carries the score f_i * K_i (its access count times the denoising step it
was saved after); once the storage limit is reached, the states with the
lowest scores are evicted, |K-set| of them before the |K-set| states of a new
prompt are stored.  Evictions leave holes; a request whose chosen K has been
evicted uses the state with the largest K' <= K that is still present; a
prompt whose states are all gone is dropped from the vector DB.

Plain lists and dicts; each eviction takes the minimum over every live state
afresh (no heap), so the result can be checked by eye.

Readings where the paper is silent (each applies to both sides):
  * f_i starts at 1 when a state is stored (its own generation is its first
    use), and grows by 1 each time a request is served from it;
  * equal scores go to the state stored first (a global sequence number
    assigned in insertion order, slot by slot);
  * a batch of m new prompts evicts, before any of them is stored, the
    fewest states that make the m * |K-set| new ones fit under the limit
    (exactly |K-set| per prompt once the cache is full);
  * freed pool slots and entry ids are reused lowest first;
  * a dropped prompt's vector-DB row is refilled from the end: the live rows
    at positions >= the new row count, in ascending order, move into the
    vacated positions below it, in ascending order;
  * new prompts' rows are appended in request order after that compaction.
"""


class LCBFU:
    def __init__(self, slot_k, state_capacity, entry_capacity):
        slot_k = [int(k) for k in slot_k]
        if not slot_k or len(set(slot_k)) != len(slot_k) or min(slot_k) < 1:
            raise ValueError("slot K values must be distinct and positive")
        self.slot_k = slot_k
        self.S = len(slot_k)
        self.cap = int(state_capacity)
        self.ecap = int(entry_capacity)
        if self.cap < 1 or self.ecap < self.cap:
            # every live prompt keeps at least one state, so this bounds live prompts
            raise ValueError("entry capacity must be at least the state limit")
        self.states = {}        # (entry, slot) -> {"pool", "f", "seq"}
        self.rows = []          # vector-DB row -> entry id
        self.free_pool = set(range(self.cap))
        self.free_entries = set(range(self.ecap))
        self.seq = 0
        self.evicted = 0
        self.dropped = 0

    # --- scoring (Sec. 5.4: f_i * K_i) ---
    def score(self, key):
        st = self.states[key]
        return st["f"] * self.slot_k[key[1]]

    def state_pool(self, entry, slot):
        st = self.states.get((entry, slot))
        return -1 if st is None else st["pool"]

    def table(self):
        """entry -> list of pool indices per slot (-1 = hole), live entries only."""
        out = {}
        for e in self.rows:
            out[e] = [self.state_pool(e, s) for s in range(self.S)]
        return out

    # --- hole handling (Sec. 5.4) ---
    def choose_k(self, row, k):
        """K' actually served for a lookup result (row, K): the largest stored
        K' <= K of that row's prompt, else 0 (full generation)."""
        if row < 0 or k <= 0:
            return 0
        e = self.rows[row]
        best = 0
        for s in range(self.S):
            if self.slot_k[s] <= k and (e, s) in self.states and self.slot_k[s] > best:
                best = self.slot_k[s]
        return best

    def access(self, rows, ks):
        """One served request per (row, K'), K' > 0: its state's count grows by one."""
        for row, k in zip(rows, ks):
            if k <= 0:
                continue
            e = self.rows[row]
            s = self.slot_k.index(k)
            self.states[(e, s)]["f"] += 1

    # --- insertion with eviction (Sec. 5.4) ---
    def insert(self, m):
        """Store m new prompts (all |K-set| states each).  Returns a dict with
        the new entry ids, their pool indices [m][S], the row moves of the
        compaction (src, dst), and the row count kept before the new rows."""
        if m < 1 or m * self.S > self.cap:
            raise ValueError("batch does not fit the state limit")
        need = len(self.states) + m * self.S - self.cap
        touched = set()
        dead = []
        for _ in range(max(0, need)):
            victim = min(self.states, key=lambda key: (self.score(key), self.states[key]["seq"]))
            self.free_pool.add(self.states.pop(victim)["pool"])
            self.evicted += 1
            e = victim[0]
            touched.add(e)
            if not any((e, s) in self.states for s in range(self.S)):
                dead.append(e)
        # drop prompts with no state left: compaction of the vector-DB rows
        dead_rows = sorted(self.rows.index(e) for e in dead)
        kept = len(self.rows) - len(dead_rows)
        holes = [r for r in dead_rows if r < kept]
        movers = [r for r in range(kept, len(self.rows)) if r not in dead_rows]
        assert len(holes) == len(movers)
        moves = list(zip(movers, holes))
        for src, dst in moves:
            self.rows[dst] = self.rows[src]
        del self.rows[kept:]
        for e in dead:
            self.free_entries.add(e)
        self.dropped += len(dead)
        assert len(self.rows) + m <= self.ecap
        entries, pools = [], []
        for _ in range(m):
            e = min(self.free_entries)
            self.free_entries.remove(e)
            row_pools = []
            for s in range(self.S):
                p = min(self.free_pool)
                self.free_pool.remove(p)
                self.states[(e, s)] = {"pool": p, "f": 1, "seq": self.seq}
                self.seq += 1
                row_pools.append(p)
            self.rows.append(e)
            entries.append(e)
            pools.append(row_pools)
        touched.update(entries)
        return {"entries": entries, "pools": pools, "moves": moves, "kept": kept,
                "touched": sorted(touched)}
