"""Pins of the oracle's 2-bit code storage (orc_pack_codes / orc_unpack_codes)
to the byte layout that include/fgq.h documents (Sec. 3.2: ternary weights
stored in 2 bits), by hand-worked bytes in tests/golden/code_bytes.txt.

A round trip alone cannot pin the layout (a consistent swap of the +1/-1
codes, or of the order inside a byte, in both functions would survive it);
the hand-written bytes do.
"""
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "code_bytes.txt")


def golden_rows():
    cases = []
    for line in open(GOLDEN):
        if line.startswith("#") or not line.strip():
            continue
        K, ts, bs = (p.strip() for p in line.split("|"))
        t = np.array([[int(v) for v in r.split()] for r in ts.split(";")], np.int8)
        b = np.array([[int(v, 16) for v in r.split()] for r in bs.split(";")], np.uint8)
        assert t.shape[1] == int(K) and b.shape[1] == (int(K) + 3) // 4
        cases.append((int(K), t, b))
    return cases


CASES = golden_rows()


def test_golden_file_covers_the_layout():
    # every code value, every position in a byte, row tails and several rows
    assert len(CASES) >= 10
    ks = {K % 4 for K, _, _ in CASES}
    assert ks == {0, 1, 2, 3}
    assert any(t.shape[0] > 1 for _, t, _ in CASES)


@pytest.mark.parametrize("K,t,b", CASES, ids=[f"K{c[0]}_{i}" for i, c in enumerate(CASES)])
def test_pack_matches_hand_worked_bytes(K, t, b):
    assert np.array_equal(oracle.pack_codes(t), b)


@pytest.mark.parametrize("K,t,b", CASES, ids=[f"K{c[0]}_{i}" for i, c in enumerate(CASES)])
def test_unpack_matches_hand_worked_bytes(K, t, b):
    assert np.array_equal(oracle.unpack_codes(b, K), t)


def test_code_10_is_never_written_and_reads_as_zero():
    rng = np.random.default_rng(7)
    t = rng.integers(-1, 2, size=(5, 37)).astype(np.int8)
    c = oracle.pack_codes(t)
    pairs = np.stack([(c >> (2 * i)) & 3 for i in range(4)], axis=-1)
    assert not np.any(pairs == 2)
    # a 10 in storage decodes to 0 (the layout reserves it)
    assert np.array_equal(oracle.unpack_codes(np.array([[0b10]], np.uint8), 1), np.zeros((1, 1), np.int8))
