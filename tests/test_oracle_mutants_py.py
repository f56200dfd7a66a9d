"""Pin strength for the oracle's Python models (aligned recovery, pool index): plausible mistakes
planted in a copy of the oracle package must fail the pins.  CPU only."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

MUTANTS = {
    "recovery.py": {
        "snapshot_of_first_chunk": ("not (flags[k - 1] & STATE)", "not (flags[0] & STATE)"),
        "gaps_allowed": ("if not all(f & KV for f in flags[:k]):", "if False:"),
    },
    "pool_index.py": {
        "touch_head_first": ("for s in reversed(slots):", "for s in slots:"),
        "highest_free_slot": ("        return min(free)\n\n    def _alloc_state", "        return max(free)\n\n    def _alloc_state"),
        "evict_pinned": ('            if self.slot[s]["pins"] == 0:\n                self._drop(s)',
                         '            if True:\n                self._drop(s)'),
        "pending_visible": ('if s is None or self.slot[s]["pending"]:', "if s is None:"),
        "salt_ignored": ("return [(salt, tuple(", "return [(0, tuple("),
        "non_creator_publishes": ("            if is_new:\n                if ok:", "            if True:\n                if ok:"),
        "unpin_on_lookup_missing": ('                self.slot[s]["pins"] += 1\n        return len(slots)',
                                    '                pass\n        return len(slots)'),
        "unpin_checks_each_occurrence_alone": (
            'for s, times in Counter(slots).items():\n            if s not in self.slot or self.slot[s]["pins"] < times:',
            'for s in slots:\n            if s not in self.slot or self.slot[s]["pins"] == 0:'),
        "commit_allows_repeated_slots": ("if len(slots) != len(new) or len(set(slots)) != len(slots):",
                                         "if len(slots) != len(new):"),
        "lookup_refreshes_past_the_hit": ("        self._touch_prefix(slots[:hit])", "        self._touch_prefix(slots)"),
        "pending_snapshot_visible": (
            'if self.slot[s]["state"] is not None and not self.slot[s]["state_pending"] else 0',
            'if self.slot[s]["state"] is not None else 0'),
        "abort_keeps_snapshot": ('                    e["aborted"] = True\n                    self._free_state_of(s)',
                                 '                    e["aborted"] = True'),
        "snapshot_evicted_under_pinned_owner": (
            'if self.slot[owner]["pins"] == 0 and not self.slot[owner]["pending"]:',
            'if not self.slot[owner]["pending"]:'),
        "snapshot_lru_not_refreshed_by_hits": ("            self.state_lru.move_to_end(state_slot)\n", ""),
        "snapshot_reserved_on_aborted_entry": (
            'self.slot[s]["pins"] == 0 or self.slot[s]["aborted"]:\n            return EINVAL, -1, 0',
            'self.slot[s]["pins"] == 0:\n            return EINVAL, -1, 0'),
        "snapshot_abort_keeps_its_slot": (
            '            ss = e["state"]\n            del self.state_owner[ss]\n            e["state"], e["state_pending"] = None, False',
            '            ss = e["state"]\n            e["state"], e["state_pending"] = None, False'),
    },
}

CASES = [(f, name) for f, muts in MUTANTS.items() for name in sorted(muts)]


@pytest.mark.parametrize("fname,name", CASES, ids=[f"{f}:{n}" for f, n in CASES])
def test_pins_catch_python_mutant(fname, name, tmp_path):
    old, new = MUTANTS[fname][name]
    pkg = tmp_path / "oracle"
    shutil.copytree(os.path.join(ROOT, "oracle"), pkg, ignore=shutil.ignore_patterns("__pycache__"))
    src = (pkg / fname).read_text()
    assert src.count(old) == 1, f"mutation anchor for {name} must occur exactly once in {fname}"
    (pkg / fname).write_text(src.replace(old, new))
    env = dict(os.environ, PYTHONPATH=str(tmp_path) + os.pathsep + ROOT,
               KVX_ORACLE_LIB=os.path.join(ROOT, "oracle", "libkvx_oracle.so"))
    probe = subprocess.run([sys.executable, "-c", "import oracle, sys; print(oracle.__file__)"], cwd=str(tmp_path),
                           env=env, capture_output=True, text=True)
    assert probe.stdout.strip().startswith(str(pkg)), probe.stdout + probe.stderr
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", "--rootdir",
                        str(tmp_path), os.path.join(ROOT, "tests", "test_oracle_recovery.py"),
                        os.path.join(ROOT, "tests", "test_oracle_pool_index.py")],
                       cwd=str(tmp_path), env=env, capture_output=True, text=True, timeout=300)
    assert r.returncode != 0, f"mutant {name} of {fname} survived the pins:\n{r.stdout[-2000:]}"
