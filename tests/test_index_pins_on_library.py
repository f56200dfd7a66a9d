"""The library's pool index held to the model's own pins (CPU only; the index makes no GPU call).

The index parity test compares the library with the oracle's model over random operation
sequences.  Here the scripted pins of the model (textbook LRU, the paper's whole-chunk hits and
salt control, two-phase stores, pinning, the snapshot rules) run unchanged against the library
through an adapter with the model's interface, so the library is checked against what the paper
and its readings fix, not only against the model.  Pins that inspect the model's internal tables
(aligned recovery's slot records, the invariants, pin counts) are left out; the library's repeated-
slot errors are checked in the index parity tests.
"""
import numpy as np
import pytest

import tests.test_oracle_pool_index as pins
from oracle.pool_index import EBUSY, EINVAL
from paper_2609_15021_amd import kvx

_STATUS = {kvx.KV_EBUSY: EBUSY, kvx.KV_EINVAL: EINVAL}


class LibraryIndex:
    """kv_index_* behind the model's method names and return shapes."""

    def __init__(self, chunk_tokens, num_slots, num_state_slots=0):
        self.x = kvx.kv_index_create(chunk_tokens, num_slots, num_state_slots)

    @staticmethod
    def _status(e):
        return _STATUS.get(e.status, e.status)

    @staticmethod
    def _tokens(tokens, n):
        return np.asarray(list(tokens)[:n], dtype=np.int32)

    def reserve(self, salt, tokens, n_tokens):
        try:
            slots, new = kvx.kv_index_reserve(self.x, salt, self._tokens(tokens, n_tokens))
        except kvx.KvError as e:
            return self._status(e), [], []
        return 0, slots.tolist(), new.tolist()

    def commit(self, slots, new, ok=True):
        try:
            kvx.kv_index_commit(self.x, slots, new, ok)
        except kvx.KvError as e:
            return self._status(e)
        return 0

    def lookup(self, salt, tokens, n_tokens, require_state=False, pin=False):
        r = kvx.kv_index_lookup(self.x, salt, self._tokens(tokens, n_tokens), require_state=require_state, pin=pin)
        return r["kv_chunks"], r["hit_chunks"], r["slots"].tolist(), r["state_slot"]

    def unpin(self, slots):
        try:
            kvx.kv_index_unpin(self.x, slots)
        except kvx.KvError as e:
            return self._status(e)
        return 0

    def reserve_state(self, s):
        try:
            ss, new = kvx.kv_index_reserve_state(self.x, int(s))
        except kvx.KvError as e:
            return self._status(e), -1, 0
        return 0, ss, new

    def commit_state(self, s, ok=True):
        try:
            kvx.kv_index_commit_state(self.x, int(s), ok)
        except kvx.KvError as e:
            return self._status(e)
        return 0

    def stats(self):
        return kvx.kv_index_get_stats(self.x)


PINS = ["test_textbook_lru_eviction", "test_paper_whole_chunk_hits_and_salt", "test_prefix_property",
        "test_two_phase_store", "test_eviction_trims_prefix_tails_first", "test_pinned_entries_are_never_evicted",
        "test_new_entries_take_the_lowest_free_slot", "test_pending_snapshot_is_invisible",
        "test_aborted_store_frees_its_snapshot_and_takes_no_new_one",
        "test_snapshot_lru_skips_pinned_owners_and_keeps_the_chunks", "test_lookup_refreshes_only_the_chunks_it_hits"]


@pytest.mark.parametrize("name", PINS)
def test_library_passes_model_pin(name, monkeypatch):
    monkeypatch.setattr(pins, "PoolIndexModel", LibraryIndex)
    getattr(pins, name)()
