"""Planted mistakes in the oracle must each fail at least one pin.

Every mutant is oracle.c with one plausible slip (a constant, a shift, the
word index, byte order, the partial-block rule, the layout, padding, the
verify index ...), compiled with gcc into a temporary library on the CPU.
"""
import os
import shutil
import subprocess
import tempfile

import pytest

import oracle
from oracle_pins import ALL_PINS

MUTANTS = [
    ("shift30", "z ^= z >> 30;", "z ^= z >> 29;"),
    ("c1_digit", "0xBF58476D1CE4E5B9ull", "0xBF58476D1CE4E5B1ull"),
    ("c2_digit", "0x94D049BB133111EBull", "0x94D049BB133111EDull"),
    ("g_digit", "0x9E3779B97F4A7C15ull", "0x9E3779B97F4A7C17ull"),
    ("drop_last_xorshift", "    z ^= z >> 31;\n", ""),
    ("index_block_relative", "((j0 + q) * ORACLE_G)", "(q * ORACLE_G)"),
    ("index_dropped", "oracle_word(blk, len, q) ^ ((j0 + q) * ORACLE_G)", "oracle_word(blk, len, q)"),
    ("index_plus_one", "((j0 + q) * ORACLE_G)", "((j0 + q + 1) * ORACLE_G)"),
    ("index_bytes_not_words", "ORACLE_BLOCK * b / 8) : 0;\n}\n\n/* Same", "ORACLE_BLOCK * b) : 0;\n}\n\n/* Same"),
    ("big_endian_word", "w |= byte << (8 * k);", "w |= byte << (8 * (7 - k));"),
    ("pad_with_ones", "pos < n ? x[pos] : 0;", "pos < n ? x[pos] : 0xFF;"),
    ("hash_pad_words", "q < ceil_div(len, 8); ++q", "q < ceil_div(len, 8) + (len < ORACLE_BLOCK); ++q"),
    ("block_8k", '#include "oracle.h"\n', '#include "oracle.h"\n#undef ORACLE_BLOCK\n#define ORACLE_BLOCK 8192u\n'),
    ("last_word_truncated", "return n - lo < ORACLE_BLOCK ? n - lo : ORACLE_BLOCK;",
     "return n - lo < ORACLE_BLOCK ? (n - lo) / 8 * 8 : ORACLE_BLOCK;"),
    ("tensor_add", "        t ^= hb;", "        t += hb;"),
    ("layout_unaligned", "        off += ceil_div(nbytes[i], ORACLE_BLOCK) * ORACLE_BLOCK;\n        blk +=",
     "        off += nbytes[i];\n        blk +="),
    ("pack_no_zero_pad", "        memset(image + off + nbytes[i], 0, slot - nbytes[i]);\n", ""),
    ("unpack_whole_slot", "        if (nbytes[i]) memcpy(dst[i], image + off, nbytes[i]);",
     "        if (nbytes[i]) memcpy(dst[i], image + off, nbytes[i] + (nbytes[i] % 8 ? 1 : 0));"),
    ("verify_index_off_by_one", "mismatch_list[found] = blk + b;", "mismatch_list[found] = blk + b + 1;"),
    ("verify_skips_last_block", "        for (uint64_t b = 0; b < nblk; ++b) {\n            if (oracle_block_hash",
     "        for (uint64_t b = 0; b + 1 < nblk; ++b) {\n            if (oracle_block_hash"),
]


@pytest.fixture(scope="module")
def workdir():
    d = tempfile.mkdtemp(prefix="oracle_mut_")
    yield d
    shutil.rmtree(d, ignore_errors=True)


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(workdir, name, old, new):
    src = open(oracle.SOURCE).read()
    assert src.count(old) >= 1, f"mutation site for {name} not found in oracle.c"
    mutated = src.replace(old, new, 1)
    path_c = os.path.join(workdir, f"{name}.c")
    with open(path_c, "w") as f:
        f.write(mutated)
    path_so = os.path.join(workdir, f"lib{name}.so")
    subprocess.run(["gcc", "-O2", "-fPIC", "-shared", "-I", oracle.HERE, path_c, "-o", path_so], check=True)
    o = oracle.Oracle(path_so)
    failed = []
    for pin in ALL_PINS:
        try:
            pin(o)
        except AssertionError:
            failed.append(pin.__name__)
            break
    assert failed, f"no pin caught mutant {name}"
