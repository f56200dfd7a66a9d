"""Pins for the pool-index reference model (CPU only): textbook LRU behaviour, the paper's
whole-chunk hit counts and salt control, aligned recovery, two-phase stores and invariants."""
import numpy as np

from oracle.pool_index import EBUSY, PoolIndexModel
from oracle.recovery import KV, STATE, restorable_chunks


def _store(m, salt, toks, n=None):
    n = len(toks) if n is None else n
    st, slots, new = m.reserve(salt, toks, n)
    assert st == 0
    assert m.commit(slots, new, True) == 0
    return slots


def test_textbook_lru_eviction():
    """Capacity 3, one chunk per prompt: store A, B, C; use A; store D -> B (least recently used) goes."""
    m = PoolIndexModel(chunk_tokens=4, num_slots=3)
    A, B, C, D = ([k] * 4 for k in range(1, 5))
    for p in (A, B, C):
        _store(m, 0, p)
    assert m.lookup(0, A, 4)[1] == 1
    _store(m, 0, D)
    assert [m.lookup(0, p, 4)[1] for p in (A, B, C, D)] == [1, 0, 1, 1]
    assert m.stats()["evictions"] == 1


def test_paper_whole_chunk_hits_and_salt():
    """Sec. 3.1-3.2: hits are whole 1,568-token chunks (25,088 = 16 chunks, 127,008 = 81), and a
    new cache salt forces zero hits on identical tokens."""
    C = 1568
    m = PoolIndexModel(C, num_slots=200)
    rng = np.random.default_rng(5)
    prompt = rng.integers(0, 150000, size=127008 + 700).tolist()
    _store(m, 11, prompt)
    kv, hit, slots, _ = m.lookup(11, prompt, len(prompt))
    assert hit * C == 127008 and kv == 81 and len(set(slots)) == 81
    assert m.lookup(11, prompt, 25088 + 1000)[1] * C == 25088
    assert m.lookup(12, prompt, len(prompt))[1] == 0


def test_prefix_property():
    m = PoolIndexModel(8, 64)
    rng = np.random.default_rng(1)
    a = rng.integers(0, 1000, size=8 * 12).tolist()
    b = list(a)
    b[8 * 10 + 3] += 1  # differs inside chunk 10
    _store(m, 0, a)
    assert m.lookup(0, b, len(b))[1] == 10
    b2 = list(a)
    b2[0] += 1
    assert m.lookup(0, b2, len(b2))[1] == 0


def test_aligned_recovery_follows_the_rule():
    m = PoolIndexModel(4, 16, num_state_slots=4)
    toks = list(range(24))
    slots = m.reserve(0, toks, 24)[1]
    for i in (1, 3):
        st, ss, new = m.reserve_state(slots[i])
        assert st == 0 and new == 1
        assert m.commit_state(slots[i]) == 0
    m.commit(slots, [1] * 6, True)
    flags = [KV | (STATE if i in (1, 3) else 0) for i in range(6)]
    kv, hit, got, ss = m.lookup(0, toks, 24, require_state=True)
    assert (kv, hit) == (6, restorable_chunks(flags, True)) == (6, 4)
    assert ss == m.slot[slots[3]]["state"]
    assert m.lookup(0, toks, 24)[1] == 6


def test_two_phase_store():
    m = PoolIndexModel(4, 8)
    toks = list(range(8))
    st, slots, new = m.reserve(0, toks, 8)
    assert st == 0 and new == [1, 1]
    assert m.lookup(0, toks, 8)[1] == 0                    # pending: invisible
    st2, slots2, new2 = m.reserve(0, toks, 8)              # a second replica reserves the same prefix
    assert slots2 == slots and new2 == [0, 0]
    assert m.commit(slots2, new2, True) == 0               # a non-creator's commit publishes nothing
    assert m.lookup(0, toks, 8)[1] == 0
    assert m.commit(slots, new, False) == 0                # the creator aborts
    assert m.lookup(0, toks, 8)[1] == 0 and m.stats()["free_slots"] == 8
    _store(m, 0, toks)
    assert m.lookup(0, toks, 8)[1] == 2


def test_eviction_trims_prefix_tails_first():
    m = PoolIndexModel(2, 4)
    a = list(range(8))                 # 4 chunks
    _store(m, 0, a)
    _store(m, 0, [100, 101, 102, 103])  # 2 chunks: evicts a's chunks 3 and 2
    assert m.lookup(0, a, 8)[1] == 2
    assert m.stats()["evictions"] == 2


def test_pinned_entries_are_never_evicted():
    m = PoolIndexModel(2, 3)
    a = list(range(6))
    _store(m, 0, a)
    kv, hit, slots, _ = m.lookup(0, a, 6, pin=True)
    assert hit == 3
    st, s2, n2 = m.reserve(0, [9, 9, 9, 9], 4)
    assert st == EBUSY and m.stats()["free_slots"] == 0 and m.stats()["pending"] == 0
    assert m.unpin(slots) == 0
    st, s2, n2 = m.reserve(0, [9, 9, 9, 9], 4)
    assert st == 0 and n2 == [1, 1]


def _invariants(m):
    for key, s in m.by_key.items():
        assert m.slot[s]["key"] == key and not m.slot[s]["aborted"]
    assert set(m.lru) == {s for s, e in m.slot.items() if not e["pending"]}
    for ss, owner in m.state_owner.items():
        assert m.slot[owner]["state"] == ss
    assert set(m.state_lru) <= set(m.state_owner)
    for s, e in m.slot.items():
        assert 0 <= s < m.num_slots and e["pins"] >= 0
        if e["state"] is not None:
            assert m.state_owner[e["state"]] == s
            assert (e["state"] in m.state_lru) == (not e["state_pending"])


def test_random_sequences_keep_invariants():
    rng = np.random.default_rng(3)
    m = PoolIndexModel(4, 12, num_state_slots=3)
    prompts = [rng.integers(0, 3, size=int(rng.integers(4, 24))).tolist() for _ in range(10)]
    held = []
    for _ in range(3000):
        op = rng.integers(0, 5)
        p = prompts[rng.integers(0, len(prompts))]
        if op == 0:
            st, slots, new = m.reserve(0, p, len(p))
            if st == 0:
                if slots and rng.integers(0, 2):
                    r, ss, nw = m.reserve_state(slots[-1])
                    if r == 0 and nw:
                        m.commit_state(slots[-1], bool(rng.integers(0, 4)))
                held.append((slots, new, bool(rng.integers(0, 5))))
        elif op == 1 and held:
            slots, new, ok = held.pop(int(rng.integers(0, len(held))))
            assert m.commit(slots, new, ok) == 0
        elif op == 2:
            kv, hit, slots, ss = m.lookup(0, p, len(p), require_state=bool(rng.integers(0, 2)), pin=True)
            assert hit <= kv and (ss == -1 or ss in m.state_owner)
            assert m.unpin(slots) == 0
        _invariants(m)
    for slots, new, ok in held:
        assert m.commit(slots, new, ok) == 0
    _invariants(m)
    assert all(e["pins"] == 0 for e in m.slot.values())


def test_new_entries_take_the_lowest_free_slot():
    m = PoolIndexModel(2, 6)
    a = _store(m, 0, [1, 1, 2, 2, 3, 3])          # 3 chunks -> slots 0, 1, 2
    assert a == [0, 1, 2]
    st, slots, new = m.reserve(0, [7, 7, 8, 8], 4)  # 2 chunks -> 3, 4; then abort them
    assert slots == [3, 4]
    m.commit(slots, new, False)
    b = _store(m, 0, [9, 9], 2)                    # the freed slot 3 is the lowest again
    assert b == [3]


def test_unpin_releases_one_pin_per_occurrence():
    """A pin is a count of holders (Sec. 3.2: slots a load still reads are not reused before the host
    has seen that load complete), so it never goes below zero.  Two pinned lookups of one prefix hold
    two pins; one unpin naming the slot twice releases both.  Naming it three times releases more than
    are held: an error that releases nothing, and the entry stays protected from eviction."""
    from oracle.pool_index import EINVAL
    m = PoolIndexModel(2, 2)
    a = [1, 1]
    _store(m, 0, a)
    s = m.lookup(0, a, 2, pin=True)[2][0]
    assert m.lookup(0, a, 2, pin=True)[2] == [s]
    assert m.unpin([s, s, s]) == EINVAL
    assert m.slot[s]["pins"] == 2
    st, _, _ = m.reserve(0, [5, 5, 6, 6], 4)      # needs both slots; the pinned one cannot be evicted
    assert st == EBUSY and m.lookup(0, a, 2)[1] == 1
    assert m.unpin([s, s]) == 0 and m.slot[s]["pins"] == 0
    st, slots, new = m.reserve(0, [5, 5, 6, 6], 4)
    assert st == 0 and new == [1, 1] and m.stats()["evictions"] == 1


def test_commit_names_each_reserved_slot_once():
    """A commit hands back what one reserve returned: one slot per whole chunk, all distinct (each
    chunk completes a different prefix, so has its own key).  A commit naming a slot twice would
    release a pin its caller does not hold (here the second replica's): an error that publishes and
    releases nothing."""
    from oracle.pool_index import EINVAL
    m = PoolIndexModel(2, 4)
    toks = [1, 1, 2, 2]
    st, slots, new = m.reserve(0, toks, 4)
    st2, slots2, new2 = m.reserve(0, toks, 4)      # a second replica holds the same entries
    assert st == st2 == 0 and slots2 == slots and new2 == [0, 0]
    assert m.commit(slots + [slots[0]], new + [new[0]], True) == EINVAL
    assert m.lookup(0, toks, 4)[1] == 0 and m.stats()["pending"] == 2
    assert [m.slot[s]["pins"] for s in slots] == [2, 2]
    assert m.commit(slots, new, True) == 0
    assert m.lookup(0, toks, 4)[1] == 2
    assert [m.slot[s]["pins"] for s in slots] == [1, 1]   # the second replica's pins stand
    assert m.commit(slots2, new2, True) == 0
    assert [m.slot[s]["pins"] for s in slots] == [0, 0]


def _store_with_snapshot(m, salt, toks, at):
    """Store a prefix and the snapshot at the boundary after chunk `at` (both committed)."""
    st, slots, new = m.reserve(salt, toks, len(toks))
    assert st == 0
    st, ss, is_new = m.reserve_state(slots[at])
    assert st == 0 and is_new == 1
    assert m.commit_state(slots[at]) == 0
    assert m.commit(slots, new, True) == 0
    return slots, ss


def test_pending_snapshot_is_invisible():
    """Sec. 3.2 (the host must see a store complete before anything reads it), applied to the
    boundary snapshot: a reserved snapshot does not make a prefix restorable until it is committed."""
    m = PoolIndexModel(4, 8, num_state_slots=2)
    toks = list(range(8))
    _store(m, 0, toks)
    slots = m.lookup(0, toks, 8, pin=True)[2]
    st, ss, is_new = m.reserve_state(slots[1])
    assert st == 0 and is_new == 1
    assert m.lookup(0, toks, 8, require_state=True)[1] == 0   # the snapshot is still pending
    assert m.lookup(0, toks, 8)[1] == 2                        # the chunks alone are a hit
    assert m.commit_state(slots[1]) == 0
    kv, hit, _, got = m.lookup(0, toks, 8, require_state=True)
    assert hit == 2 and got == ss
    assert m.unpin(slots) == 0


def test_aborted_store_frees_its_snapshot_and_takes_no_new_one():
    """An aborted store publishes nothing (Sec. 3.2): its snapshot slot is freed with it, and an
    aborted entry that another holder still pins cannot take a snapshot."""
    m = PoolIndexModel(4, 8, num_state_slots=2)
    toks = list(range(8))
    st, slots, new = m.reserve(0, toks, 8)
    assert m.reserve_state(slots[1])[0] == 0
    assert m.stats()["free_state_slots"] == 1
    st2, slots2, new2 = m.reserve(0, toks, 8)                  # a second replica holds the same entries
    assert slots2 == slots and new2 == [0, 0]
    assert m.commit(slots, new, False) == 0                   # the creator aborts
    assert m.stats()["free_state_slots"] == 2
    assert m.reserve_state(slots[1])[0] != 0                  # aborted, though still pinned
    assert m.commit(slots2, new2, True) == 0                  # the other holder lets go
    assert m.stats()["free_slots"] == 8 and m.lookup(0, toks, 8)[1] == 0


def test_snapshot_lru_skips_pinned_owners_and_keeps_the_chunks():
    """Snapshot slots have their own LRU (reading of Table 1's LRU for the snapshot budget): a hit
    refreshes its snapshot, the least recently used snapshot of an unpinned entry is evicted first,
    and evicting a snapshot keeps its chunk entry (still a hit without aligned recovery)."""
    m = PoolIndexModel(2, 16, num_state_slots=2)
    P1, P2, P3, P4 = ([k] * 2 for k in range(1, 5))
    _store_with_snapshot(m, 0, P1, 0)
    _store_with_snapshot(m, 0, P2, 0)
    assert m.lookup(0, P1, 2, require_state=True)[1] == 1     # refreshes P1's snapshot
    _store_with_snapshot(m, 0, P3, 0)                          # evicts P2's snapshot, not P1's
    assert m.lookup(0, P2, 2, require_state=True)[1] == 0
    assert m.lookup(0, P2, 2)[1] == 1
    assert m.stats()["state_evictions"] == 1
    held = m.lookup(0, P1, 2, pin=True)[2]                    # P1 pinned ...
    assert m.lookup(0, P3, 2)[1] == 1                          # ... and now its snapshot is the older one
    _store_with_snapshot(m, 0, P4, 0)                          # must evict P3's snapshot: P1's owner is pinned
    assert m.lookup(0, P1, 2, require_state=True)[1] == 1
    assert m.lookup(0, P3, 2, require_state=True)[1] == 0
    assert m.unpin(held) == 0


def test_lookup_refreshes_only_the_chunks_it_hits():
    """LRU use is what a hit restores: with aligned recovery the hit stops at the last snapshot, and
    the chunks past it are not refreshed, so they are evicted before another prompt's chunk."""
    m = PoolIndexModel(2, 4, num_state_slots=1)
    X = list(range(6))                                        # 3 chunks, snapshot after chunk 0
    _store_with_snapshot(m, 0, X, 0)
    Y = [50, 51]
    _store(m, 0, Y)
    assert m.lookup(0, X, 6, require_state=True)[1] == 1      # touches X's chunk 0 only
    _store(m, 0, [60, 61])                                    # one eviction: X's chunk 2, the oldest
    assert m.lookup(0, Y, 2)[1] == 1
    assert m.lookup(0, X, 6)[1] == 2
