"""Pins for the oracle's suffix array and its linear-time checker
(suffix order of Section III-A)."""
import numpy as np
import pytest

import brute
import oracle
import synth


@pytest.mark.parametrize("vocab", [2, 3, 4, 16, 32256])
@pytest.mark.parametrize("seed", range(6))
def test_sa_matches_sorted_suffix_lists(vocab, seed):
    n = 1 + (seed * 37 + vocab) % 400
    t = synth.random_text(seed * 1000 + vocab, n, vocab, sep_prob=0.05)
    assert oracle.suffix_array(t).tolist() == brute.suffix_array(t)


def test_sa_special_cases():
    for n in (1, 2, 7, 100):
        eq = np.full(n, 9, np.uint16)
        assert oracle.suffix_array(eq).tolist() == list(range(n - 1, -1, -1))
        inc = np.arange(1, n + 1, dtype=np.uint16)
        assert oracle.suffix_array(inc).tolist() == list(range(n))
        dec = np.arange(n, 0, -1).astype(np.uint16)
        assert oracle.suffix_array(dec).tolist() == list(range(n - 1, -1, -1))
    assert oracle.suffix_array(np.zeros(0, np.uint16)).tolist() == []
    # separator 0 sorts below every token; a suffix that ends sorts below all
    assert oracle.suffix_array(np.array([0, 0, 0], np.uint16)).tolist() == [2, 1, 0]
    assert oracle.suffix_array(np.array([65535, 0, 65535], np.uint16)).tolist() == [1, 2, 0]


def test_sa_example_a(golden):
    g = golden("example_a.json")
    assert oracle.suffix_array(g["text"]).tolist() == g["sa"]
    gb = golden("example_b.json")
    assert oracle.suffix_array(gb["project"]).tolist() == gb["project_sa"]


def test_suffix_cmp_prefix_rule():
    t = np.array([4, 4, 4], np.uint16)
    assert oracle.suffix_cmp(t, 2, 1) == -1   # [4] is a prefix of [4 4]
    assert oracle.suffix_cmp(t, 0, 1) == 1
    assert oracle.suffix_cmp(t, 1, 1) == 0


@pytest.mark.parametrize("vocab", [2, 4, 32256])
def test_checker_accepts_and_rejects(vocab):
    t = synth.random_text(77 + vocab, 120, vocab, sep_prob=0.03)
    sa = oracle.suffix_array(t)
    assert oracle.check_sa(t, sa) == (0, 0)
    # every swap of two entries breaks it
    for a in range(0, len(sa), 7):
        for b in range(a + 1, len(sa), 11):
            bad = sa.copy()
            bad[a], bad[b] = bad[b], bad[a]
            code, _ = oracle.check_sa(t, bad)
            assert code == 2
    dup = sa.copy()
    dup[5] = dup[6]
    assert oracle.check_sa(t, dup)[0] == 1
    oob = sa.copy()
    oob[0] = len(t)
    assert oracle.check_sa(t, oob)[0] == 1


def test_checker_on_store_slice():
    s = synth.store(1, "single")[:20000]
    sa = oracle.suffix_array(s)
    assert oracle.check_sa(s, sa)[0] == 0
