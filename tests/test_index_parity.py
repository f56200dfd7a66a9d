"""The library's pool index (C++, hashed keys) against the oracle's exact-key model, on the CPU.

Every operation of seeded random sequences -- prompts sharing prefixes, two salts, reserves by
two replicas of one prefix, aborts, snapshots, pinned lookups, slot budgets small enough to
force evictions and KV_EBUSY -- must give identical statuses, slots, flags and hit counts,
and identical statistics after every step (bit-exact: this is integer and index work).
"""
import numpy as np
import pytest

from oracle.pool_index import PoolIndexModel
from paper_2609_15021_amd import kvx


def _prompts(rng, C, count, vocab=4):
    base = rng.integers(0, vocab, size=12 * C).tolist()
    out = []
    for _ in range(count):
        keep = int(rng.integers(0, 10)) * C + int(rng.integers(0, C))
        tail = rng.integers(0, vocab, size=int(rng.integers(0, 5 * C))).tolist()
        out.append(base[:keep] + tail)
    return out


def _call(fn, *a, **k):
    try:
        return 0, fn(*a, **k)
    except kvx.KvError as e:
        return e.status, None


@pytest.mark.parametrize("seed,C,num_slots,num_state", [(1, 4, 10, 3), (2, 3, 25, 0), (3, 8, 40, 6),
                                                        (4, 1, 6, 2), (5, 16, 40, 12)])
def test_index_matches_model(seed, C, num_slots, num_state):
    rng = np.random.default_rng(seed)
    prompts = _prompts(rng, C, 14)
    m = PoolIndexModel(C, num_slots, num_state)
    x = kvx.kv_index_create(C, num_slots, num_state)
    held = []       # reservations not yet committed: (slots, new)
    pinned = []     # pinned lookups not yet released
    counts = dict(reserve=0, busy=0, hits=0, state_hits=0)
    for step in range(4000):
        op = int(rng.integers(0, 6))
        p = prompts[int(rng.integers(0, len(prompts)))]
        salt = int(rng.integers(0, 2))
        if op in (0, 1):
            st_m, slots_m, new_m = m.reserve(salt, p, len(p))
            st_x, r = _call(kvx.kv_index_reserve, x, salt, p)
            assert st_m == st_x, (step, st_m, st_x)
            if st_x == 0:
                assert r[0].tolist() == slots_m and r[1].tolist() == new_m, step
                counts["reserve"] += 1
                if slots_m and num_state and rng.integers(0, 2):
                    s = slots_m[int(rng.integers(0, len(slots_m)))]
                    a = m.reserve_state(s)
                    stx, b = _call(kvx.kv_index_reserve_state, x, s)
                    assert a[0] == stx and (stx != 0 or (b[0], b[1]) == (a[1], a[2])), (step, a, stx, b)
                    if stx == 0 and a[2]:
                        ok = bool(rng.integers(0, 4))
                        assert m.commit_state(s, ok) == 0
                        kvx.kv_index_commit_state(x, s, ok)
                held.append((slots_m, new_m))
            else:
                counts["busy"] += 1
        elif op == 2 and held:
            slots, new = held.pop(int(rng.integers(0, len(held))))
            ok = bool(rng.integers(0, 6))
            assert m.commit(slots, new, ok) == 0
            kvx.kv_index_commit(x, slots, new, ok)
        elif op in (3, 4):
            req, pin = bool(rng.integers(0, 2)), bool(rng.integers(0, 2))
            kv, hit, slots, ss = m.lookup(salt, p, len(p), require_state=req, pin=pin)
            r = kvx.kv_index_lookup(x, salt, p, require_state=req, pin=pin)
            assert (r["kv_chunks"], r["hit_chunks"], r["hit_tokens"], r["state_slot"]) == (kv, hit, hit * C, ss), step
            assert r["slots"].tolist() == slots
            counts["hits"] += hit
            counts["state_hits"] += ss >= 0
            if pin:
                pinned.append(slots)
        elif op == 5 and pinned:
            slots = pinned.pop(int(rng.integers(0, len(pinned))))
            assert m.unpin(slots) == 0
            kvx.kv_index_unpin(x, slots)
        assert kvx.kv_index_get_stats(x) == m.stats(), step
    for slots, new in held:
        m.commit(slots, new, True)
        kvx.kv_index_commit(x, slots, new, True)
    for slots in pinned:
        m.unpin(slots)
        kvx.kv_index_unpin(x, slots)
    assert kvx.kv_index_get_stats(x) == m.stats()
    # The sequence exercised the interesting paths.
    assert counts["reserve"] > 100 and counts["hits"] > 100
    assert m.stats()["evictions"] > 0
    if num_state:
        assert counts["state_hits"] > 0
    kvx.kv_index_destroy(x)


def test_paper_whole_chunk_hits_and_new_salt():
    """Sec. 3.1-3.2: a 127,008 + 700-token prompt hits 81 whole 1,568-token chunks (127,008
    tokens); its 26,088-token prefix hits 16 (25,088 tokens); a new cache salt hits nothing."""
    C = 1568
    x = kvx.kv_index_create(C, 4096)
    prompt = np.random.default_rng(8).integers(0, 151000, size=127008 + 700).astype(np.int32)
    slots, new = kvx.kv_index_reserve(x, 7, prompt)
    assert slots.size == 81 and new.all()
    kvx.kv_index_commit(x, slots, new)
    assert kvx.kv_index_lookup(x, 7, prompt)["hit_tokens"] == 127008
    assert kvx.kv_index_lookup(x, 7, prompt[:25088 + 1000])["hit_tokens"] == 25088
    assert kvx.kv_index_lookup(x, 8, prompt)["hit_tokens"] == 0


def test_keys_name_the_whole_prefix():
    C = 16
    x = kvx.kv_index_create(C, 8)
    rng = np.random.default_rng(4)
    a = rng.integers(0, 50000, size=10 * C).astype(np.int32)
    ka = kvx.kv_index_keys(x, 1, a)
    assert ka.shape == (10, 2) and len({tuple(k) for k in ka}) == 10
    b = a.copy()
    b[5 * C + 3] ^= 1
    kb = kvx.kv_index_keys(x, 1, b)
    assert (ka[:5] == kb[:5]).all() and not (ka[5:] == kb[5:]).all(axis=1).any()
    assert not (kvx.kv_index_keys(x, 2, a) == ka).all(axis=1).any()           # salt
    y = kvx.kv_index_create(8, 8)
    assert not (kvx.kv_index_keys(y, 1, a)[1::2] == ka).all(axis=1).any()      # chunk length
    assert kvx.kv_index_keys(x, 1, a[:C - 1]).shape == (0, 2)                # no whole chunk


def test_index_argument_errors():
    with pytest.raises(kvx.KvError):
        kvx.kv_index_create(0, 4)
    x = kvx.kv_index_create(4, 2)
    slots, new = kvx.kv_index_reserve(x, 0, list(range(8)))
    with pytest.raises(kvx.KvError):
        kvx.kv_index_commit(x, [slots[0], slots[0]], [1, 1])                 # a slot twice
    with pytest.raises(kvx.KvError):
        kvx.kv_index_unpin(x, [slots[0], slots[0]])                          # pinned once
    with pytest.raises(kvx.KvError) as e:
        kvx.kv_index_reserve(x, 0, list(range(100, 108)))                    # both slots pending
    assert e.value.status == kvx.KV_EBUSY
    kvx.kv_index_commit(x, slots, new)
    with pytest.raises(kvx.KvError):
        kvx.kv_index_commit(x, slots, new)                                   # no longer pinned
    with pytest.raises(kvx.KvError):
        kvx.kv_index_reserve_state(x, int(slots[0]))                         # not pinned


def test_index_under_concurrent_threads():
    """Four threads store and look up their own prompts on one index at the same time (the calls
    release the GIL): every thread's final lookups hit its whole prompt and no pin is left."""
    import threading
    C, per = 8, 6
    x = kvx.kv_index_create(C, 4 * per)
    rng = np.random.default_rng(17)
    prompts = [rng.integers(0, 50000, size=per * C).astype(np.int32) for _ in range(4)]
    errors = []

    def worker(k):
        try:
            for _ in range(300):
                slots, new = kvx.kv_index_reserve(x, k, prompts[k])
                kvx.kv_index_commit(x, slots, new, True)
                r = kvx.kv_index_lookup(x, k, prompts[k], pin=True)
                kvx.kv_index_unpin(x, r["slots"])
                if r["hit_chunks"] != per:
                    errors.append((k, r["hit_chunks"]))
        except Exception as e:  # surfaced below
            errors.append(repr(e))

    threads = [threading.Thread(target=worker, args=(k,)) for k in range(4)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors[:5]
    st = kvx.kv_index_get_stats(x)
    assert st["entries"] == 4 * per and st["pending"] == 0 and st["evictions"] == 0
    for k in range(4):
        assert kvx.kv_index_lookup(x, k, prompts[k])["hit_chunks"] == per
    kvx.kv_index_destroy(x)
