"""Pin strength: plausible mistakes planted in a copy of the oracle must fail the pins.

Each mutant is a textual edit of ``oracle/kvx_oracle.c`` compiled with gcc into
a temporary library; the pin suite then runs against it in a subprocess and
must fail.  Runs on the CPU only (the mistakes are planted in the oracle, never
in GPU code).
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "kvx_oracle.c")

MUTANTS = {
    "kv_order_swapped": ("((kv * H + h) * BS + s) * row_bytes", "(((1 - kv) * H + h) * BS + s) * row_bytes"),
    "plane_stride_C_for_partial": ("chunk_row_offset(lay, r, l, kv, u, h)",
                                   "chunk_row_offset(lay, lay->chunk_tokens, l, kv, u, h)"),
    "kv_dropped_in_chunk": ("(((l * 2 + kv) * r + u) * H + h)", "(((l * 2) * r + u) * H + h)"),
    "chunk_planes_head_major": ("(((l * 2 + kv) * r + u) * H + h)", "(((l * 2 + kv) * H + h) * r + u)"),
    "slot_off_by_one": ("int64_t s = t % BS;", "int64_t s = (t + 1) % BS;"),
    "chunk_offset_forgotten": ("job->block_table[t / BS]", "job->block_table[u / BS]"),
    "unpack_copies_wrong_way": ("memcpy(cache_row, chunk_row, (size_t)row_bytes);",
                                "memcpy(chunk_row, cache_row, (size_t)row_bytes);"),
    "divisibility_check_dropped": ("if (lay->chunk_tokens % lay->block_size != 0)", "if (0)"),
    "head_and_slot_swapped": ("return b * block_stride + ((kv * H + h) * BS + s) * row_bytes;",
                              "return b * block_stride + ((kv * BS + s) * H + h) * row_bytes;"),
    "nhd_read_as_hnd": ("return b * block_stride + ((kv * BS + s) * H + h) * row_bytes;",
                        "return b * block_stride + ((kv * H + h) * BS + s) * row_bytes;"),
    "nhd_block_stride_ignored": ("return b * block_stride + ((kv * BS + s) * H + h) * row_bytes;",
                                 "return b * (2 * H * BS * row_bytes) + ((kv * BS + s) * H + h) * row_bytes;"),
    "duplicate_store_slots_accepted": ("    if (for_pack) {\n        /* Two chunks", "    if (0) {\n        /* Two chunks"),
    "chunk_ids_ignored": ("uint8_t *slot = job->pool + job->chunk_ids[i] * slot_bytes;",
                          "uint8_t *slot = job->pool + i * slot_bytes;"),
    "last_block_id_unchecked": ("for (int64_t k = 0; k < n_blocks_used; ++k)",
                                "for (int64_t k = 0; k + 1 < n_blocks_used; ++k)"),
    "cache_without_blocks_accepted": ("if (n_tokens < 0 || num_blocks <= 0 || num_slots < 0)",
                                      "if (n_tokens < 0 || num_blocks < 0 || num_slots < 0)"),
    "partial_chunk_last_token_dropped": ("for (int64_t u = 0; u < r; ++u) {", "for (int64_t u = 0; u + 1 < r; ++u) {"),
    "slot_one_token_too_long": ("return (int64_t)lay->chunk_tokens * token_bytes;",
                                "return (int64_t)(lay->chunk_tokens + 1) * token_bytes;"),
    "state_load_slot_range_unchecked": (
        "        if (slot_ids[k] < 0 || slot_ids[k] >= num_state_slots)\n            return ORACLE_EINVAL;",
        "        if (for_pack && (slot_ids[k] < 0 || slot_ids[k] >= num_state_slots))\n            return ORACLE_EINVAL;"),
    "state_null_layer_unchecked": ("    for (int64_t g = 0; g < num_layers; ++g)\n        if (!state_layers[g])\n            return ORACLE_EINVAL;", ""),
    "state_layer_offset_dropped": ("uint8_t *packed = slot + g * page_bytes;", "uint8_t *packed = slot;"),
    "state_page_stride_ignored": ("state_layers[g] + pages[k] * page_stride;",
                                  "state_layers[g] + pages[k] * page_bytes;"),
    "state_slot_stride_one_page": ("state_pool + slot_ids[k] * snapshot_bytes;",
                                   "state_pool + slot_ids[k] * page_bytes;"),
    "state_unpack_wrong_way": ("memcpy(page, packed, (size_t)page_bytes);",
                               "memcpy(packed, page, (size_t)page_bytes);"),
    "state_duplicate_check_one_side": ("const int64_t *written = for_pack ? slot_ids : pages;",
                                       "const int64_t *written = slot_ids;"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation anchor for {name} must occur exactly once in the oracle source"
    mutated = tmp_path / "mut.c"
    mutated.write_text(src.replace(old, new))
    lib = tmp_path / "libmut.so"
    subprocess.run(["gcc", "-std=c11", "-O1", "-fPIC", "-shared", "-I", os.path.join(ROOT, "oracle"),
                    "-o", str(lib), str(mutated), "-lpthread"], check=True)
    env = dict(os.environ, KVX_ORACLE_LIB=str(lib))
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_pins.py"),
                        os.path.join(ROOT, "tests", "test_oracle_nhd.py"),
                        os.path.join(ROOT, "tests", "test_oracle_state.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, f"mutant {name} survived the oracle pins:\n{r.stdout[-2000:]}"
