"""Reference model of the pool index -- TEST INFRASTRUCTURE ONLY (oracle).

Only tests/ and the benchmark's CPU-baseline leg use it.  It shares no code with the
library: keys here are the exact (salt, token prefix) tuples, never hashes.

What it models (the paper's shared tier, Table 1 and Sec. 3.1-3.2):
  * the tier is a fixed budget of chunk slots with LRU eviction;
  * a chunk is identified by the whole token prefix it completes plus a cache salt (a new
    salt forces zero hits, Sec. 3.2); only whole chunks are keyed, so hits are counted in
    whole chunks (25,088 = 16 x 1,568 and 127,008 = 81 x 1,568 hit tokens, Sec. 3.1-3.2);
  * under aligned recovery a hit needs the recurrent snapshot at its boundary (Sec. 2.2,
    the rule of recovery.py).

Rules where the paper is silent (one reading, stated so the library can be held to it):
  * a new entry takes the lowest-numbered free slot; with none free it evicts the least
    recently used committed entry that is not pinned (its snapshot goes with it);
  * an operation on a prefix touches its chunks from last to first, so a prefix's head is
    more recent than its tail and eviction trims prefixes from the end;
  * a store is two-phase: reserve (entries pending: invisible to lookups, never evicted)
    then commit once the host has seen the store complete (Sec. 3.2's host-side
    completion), or abort.  Reserve pins every entry it returns.  Only the caller that
    created a pending entry (is_new) publishes or aborts it; other holders only unpin.
    An aborted entry loses its key at once and frees its slot when its last pin goes;
  * snapshots have their own slot budget and LRU; evicting a snapshot keeps its chunk;
    a snapshot is evictable only while its chunk entry is committed and unpinned.
"""
from __future__ import annotations

from collections import Counter, OrderedDict

from oracle.recovery import KV, STATE, restorable_chunks

EBUSY = -6
EINVAL = -1


class PoolIndexModel:
    def __init__(self, chunk_tokens: int, num_slots: int, num_state_slots: int = 0):
        self.C = chunk_tokens
        self.num_slots = num_slots
        self.num_state_slots = num_state_slots
        self.by_key = {}                 # key -> slot
        self.slot = {}                   # slot -> dict(key, pending, pins, state, state_pending)
        self.lru = OrderedDict()         # committed slots, least recent first
        self.state_owner = {}            # state slot -> chunk slot
        self.state_lru = OrderedDict()   # committed state slots, least recent first
        self.evictions = 0
        self.state_evictions = 0

    # -- keys -------------------------------------------------------------------------
    def keys(self, salt, tokens, n_tokens):
        tokens = list(tokens[:n_tokens])
        return [(salt, tuple(tokens[:(i + 1) * self.C])) for i in range(n_tokens // self.C)]

    # -- helpers ----------------------------------------------------------------------
    def _touch(self, s):
        if s in self.lru:
            self.lru.move_to_end(s)

    def _touch_prefix(self, slots):
        for s in reversed(slots):
            self._touch(s)

    def _free_state_of(self, s):
        e = self.slot[s]
        if e["state"] is not None:
            ss = e["state"]
            del self.state_owner[ss]
            self.state_lru.pop(ss, None)
            e["state"] = None
            e["state_pending"] = False

    def _drop(self, s):
        e = self.slot[s]
        self._free_state_of(s)
        if self.by_key.get(e["key"]) == s:
            del self.by_key[e["key"]]
        self.lru.pop(s, None)
        del self.slot[s]

    def _evict_one(self):
        for s in self.lru:
            if self.slot[s]["pins"] == 0:
                self._drop(s)
                self.evictions += 1
                return True
        return False

    def _alloc(self):
        free = [s for s in range(self.num_slots) if s not in self.slot]
        if not free:
            if not self._evict_one():
                return None
            free = [s for s in range(self.num_slots) if s not in self.slot]
        return min(free)

    def _alloc_state(self):
        free = [s for s in range(self.num_state_slots) if s not in self.state_owner]
        if free:
            return min(free)
        for ss in self.state_lru:
            owner = self.state_owner[ss]
            if self.slot[owner]["pins"] == 0 and not self.slot[owner]["pending"]:
                self._free_state_of(owner)
                self.state_evictions += 1
                return ss
        return None

    # -- operations -------------------------------------------------------------------
    def lookup(self, salt, tokens, n_tokens, require_state=False, pin=False):
        """(kv_chunks, hit_chunks, slots of the hit chunks, state slot at the hit boundary or -1)."""
        slots = []
        for key in self.keys(salt, tokens, n_tokens):
            s = self.by_key.get(key)
            if s is None or self.slot[s]["pending"]:
                break
            slots.append(s)
        flags = [KV | (STATE if self.slot[s]["state"] is not None and not self.slot[s]["state_pending"] else 0)
                 for s in slots]
        hit = restorable_chunks(flags, require_state)
        state_slot = -1
        if hit and flags[hit - 1] & STATE:
            state_slot = self.slot[slots[hit - 1]]["state"]
            self.state_lru.move_to_end(state_slot)
        self._touch_prefix(slots[:hit])
        if pin:
            for s in slots[:hit]:
                self.slot[s]["pins"] += 1
        return len(slots), hit, slots[:hit], state_slot

    def unpin(self, slots):
        for s, times in Counter(slots).items():
            if s not in self.slot or self.slot[s]["pins"] < times:
                return EINVAL
        for s in slots:
            self._release(s)
        return 0

    def _release(self, s):
        e = self.slot[s]
        e["pins"] -= 1
        if e["aborted"] and e["pins"] == 0:
            self._drop(s)

    def reserve(self, salt, tokens, n_tokens):
        """(status, slots of every whole chunk, is_new flags).  All returned entries are pinned."""
        slots, new = [], []
        for key in self.keys(salt, tokens, n_tokens):
            s = self.by_key.get(key)
            if s is not None:
                self.slot[s]["pins"] += 1
                slots.append(s)
                new.append(0)
                continue
            s = self._alloc()
            if s is None:
                for t, is_new in zip(slots, new):  # undo this call (evictions stand)
                    if is_new:
                        self._drop(t)
                    else:
                        self._release(t)
                return EBUSY, [], []
            self.slot[s] = dict(key=key, pending=True, aborted=False, pins=1, state=None, state_pending=False)
            self.by_key[key] = s
            slots.append(s)
            new.append(1)
        return 0, slots, new

    def commit(self, slots, new, ok=True):
        """Publish (ok) or abort the entries this caller created (new[i] = 1, as reserve returned),
        and release the pins of all of them."""
        if len(slots) != len(new) or len(set(slots)) != len(slots):
            return EINVAL
        for s, is_new in zip(slots, new):
            if s not in self.slot or self.slot[s]["pins"] == 0 or (is_new and not self.slot[s]["pending"]):
                return EINVAL
            if is_new and self.slot[s]["aborted"]:
                return EINVAL
        for s, is_new in zip(slots, new):
            e = self.slot[s]
            if is_new:
                if ok:
                    e["pending"] = False
                    self.lru[s] = None
                else:
                    e["aborted"] = True
                    self._free_state_of(s)
                    del self.by_key[e["key"]]
            self._release(s)
        self._touch_prefix([s for s in slots if s in self.slot and not self.slot[s]["pending"]])
        return 0

    def reserve_state(self, s):
        """(status, state slot, is_new) for the snapshot at the boundary after the chunk in slot s."""
        if s not in self.slot or self.slot[s]["pins"] == 0 or self.slot[s]["aborted"]:
            return EINVAL, -1, 0
        e = self.slot[s]
        if e["state"] is not None:
            return 0, e["state"], 0
        ss = self._alloc_state()
        if ss is None:
            return EBUSY, -1, 0
        e["state"], e["state_pending"] = ss, True
        self.state_owner[ss] = s
        return 0, ss, 1

    def commit_state(self, s, ok=True):
        if s not in self.slot or self.slot[s]["state"] is None or not self.slot[s]["state_pending"]:
            return EINVAL
        e = self.slot[s]
        if ok:
            e["state_pending"] = False
            self.state_lru[e["state"]] = None
        else:
            ss = e["state"]
            del self.state_owner[ss]
            e["state"], e["state_pending"] = None, False
        return 0

    def stats(self):
        return dict(entries=sum(1 for e in self.slot.values() if not e["pending"]),
                    pending=sum(1 for e in self.slot.values() if e["pending"] and not e["aborted"]),
                    free_slots=self.num_slots - len(self.slot),
                    state_entries=len(self.state_lru),
                    free_state_slots=self.num_state_slots - len(self.state_owner),
                    evictions=self.evictions, state_evictions=self.state_evictions)
