"""Pins for the oracle's aligned-recovery rule (CPU only)."""
import itertools

from oracle.recovery import KV, STATE, restorable_chunks


def test_attention_hit_alone_is_not_a_hybrid_hit():
    # Sec. 2.2: K/V pages without the boundary snapshot do not recover the hybrid state.
    assert restorable_chunks([KV, KV, KV], require_state=True) == 0
    assert restorable_chunks([KV, KV, KV], require_state=False) == 3


def test_recovery_stops_at_the_last_boundary_with_a_snapshot():
    f = [KV | STATE, KV, KV | STATE, KV, KV]
    assert restorable_chunks(f, True) == 3
    assert restorable_chunks(f, False) == 5


def test_missing_kv_breaks_the_prefix_even_with_later_snapshots():
    f = [KV | STATE, STATE, KV | STATE]
    assert restorable_chunks(f, True) == 1
    assert restorable_chunks(f, False) == 1
    assert restorable_chunks([], True) == 0


def test_paper_whole_chunk_hits():
    # Sec. 3.1/3.2: 25,088 and 127,008 externally hit tokens are 16 and 81 whole 1,568-token chunks.
    for tokens, chunks in ((25088, 16), (127008, 81)):
        n_full = tokens // 1568
        assert n_full == chunks and n_full * 1568 == tokens
        assert restorable_chunks([KV | STATE] * n_full, True) * 1568 == tokens


def test_brute_force_against_definition_by_enumeration():
    """Every flag sequence of length <= 5: the result is the longest prefix that qualifies."""
    for length in range(6):
        for flags in itertools.product([0, KV, STATE, KV | STATE], repeat=length):
            for req in (False, True):
                ok = [k for k in range(length + 1)
                      if k == 0 or (all(f & KV for f in flags[:k]) and (not req or flags[k - 1] & STATE))]
                assert restorable_chunks(list(flags), req) == max(ok)
