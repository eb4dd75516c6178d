"""Plants one plausible mistake at a time in a copy of the oracle's C source
(on the CPU, in a temporary directory) and checks that the pins catch it.
This shows the pins are sensitive to dropped terms, wrong rotations, swapped
operands and wrong indices, not just that the oracle agrees with itself."""
import importlib.util
import os
import subprocess

import pytest

import tests.test_oracle_bank as B
import tests.test_oracle_contract as C
import tests.test_oracle_hash as H
import tests.test_oracle_ring_classify as R

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "pcs_oracle.c")

MUTATIONS = {
    "round_rotation": ("acc = rotl64(acc, 31);", "acc = rotl64(acc, 30);"),
    "merge_drops_prime4": ("acc = acc * PRIME64_1 + PRIME64_4;\n    return acc;", "acc = acc * PRIME64_1;\n    return acc;"),
    "length_not_added": ("acc = acc + len;", "acc = acc + 0;"),
    "byte_tail_prime": ("((uint64_t)p[pos] * PRIME64_5)", "((uint64_t)p[pos] * PRIME64_1)"),
    "avalanche_shift": ("acc = acc ^ (acc >> 29);", "acc = acc ^ (acc >> 28);"),
    "big_endian_read": ("for (int i = 7; i >= 0; --i) v = (v << 8) | p[i];", "for (int i = 0; i < 8; ++i) v = (v << 8) | p[i];"),
    "merkle_swapped": ("orc_node_hash(work[j], work[j + 1])", "orc_node_hash(work[j + 1], work[j])"),
    "merkle_duplicates_odd": ("if (m % 2 == 1) work[next++] = work[m - 1];", "if (m % 2 == 1) { work[next] = orc_node_hash(work[m - 1], work[m - 1]); next++; }"),
    "chunk_padding": ("uint64_t len = nbytes - start < ORC_CHUNK ? nbytes - start : ORC_CHUNK;", "uint64_t len = ORC_CHUNK; (void)nbytes;"),
    "ring_off_by_one": ("uint64_t phys = (head + t) % capacity;\n            memcpy(out", "uint64_t phys = (head + t + 1) % capacity;\n            memcpy(out"),
    "bitmap_msb_first": ("1ULL << (i % 64)", "1ULL << (63 - i % 64)"),
    "classify_ignores_last_replay": ("for (uint32_t k = 1; k < K; ++k)", "for (uint32_t k = 1; k + 1 < K; ++k)"),
    "dirty_parent_index": ("(hashes[base + i] != parent_hashes[pbase + i])", "(hashes[base + i] != parent_hashes[base + i])"),
    "payload_unaligned": ("off += orc_chunk_count(nbytes[b]) * ORC_CHUNK;", "off += nbytes[b];"),
    "shrink_positive_zero_first": ("if (sa != sb) return sa;", "if (sa != sb) return sb;"),
    "shrink_nan_first": ("        return nb;  /* a is a number, b is NaN */", "        return na;"),
    "shrink_ties_higher_index": ("    return ia < ib;\n}\n\nstatic const float", "    return ia > ib;\n}\n\nstatic const float"),
    "shrink_rank_order_kept": ("    qsort(kept, keep, sizeof(uint32_t), cmp_index);\n", ""),
    "shrink_higher_is_better": ("    if (a < b) return 1;\n    if (a > b) return 0;", "    if (a > b) return 1;\n    if (a < b) return 0;"),
}

PINS = [
    H.test_xxh64_empty,
    lambda o: H.test_xxh64_all_short_lengths(o, 0),
    H.test_xxh64_chunk_boundaries_and_random,
    lambda o: H.test_chunk_hashes_are_xxh64_of_slices(o, 4097),
    H.test_merkle_small_closed_forms,
    H.test_merkle_matches_recursive_split,
    lambda o: R.test_ring_window_matches_numpy(o, 3, 10, 32, 7, 9, 48),
    R.test_classify_bitmap_layout,
    R.test_classify_matches_byte_comparison,
    C.test_full_round_trip_and_layout,
    C.test_incremental_dirty_set_is_byte_difference,
    B.test_select_against_python_sort,
    B.test_special_cases,
]


def load_variant(tmp_path, name, old, new):
    src = open(SRC).read()
    assert src.count(old) == 1, name
    d = tmp_path / name
    d.mkdir()
    (d / "pcs_oracle.c").write_text(src.replace(old, new))
    subprocess.run(["gcc", "-O1", "-fPIC", "-shared", "-o", str(d / "liboracle.so"), str(d / "pcs_oracle.c")],
                   check=True)
    spec = importlib.util.spec_from_file_location("oracle_" + name, os.path.join(ROOT, "oracle", "__init__.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    mod._SRC = str(d / "pcs_oracle.c")
    mod._LIB_PATH = str(d / "liboracle.so")
    return mod


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_is_caught(tmp_path, name):
    old, new = MUTATIONS[name]
    mod = load_variant(tmp_path, name, old, new)
    caught = []
    for pin in PINS:
        try:
            pin(mod)
        except AssertionError:
            caught.append(pin)
    assert caught, "no pin caught the planted mistake %r" % name
