"""Host-side logic of the tests' host-driven replay, checked on the CPU
against the oracle's independent implementation."""
import random

import oracle
from host_replay import _Sequences


def test_replay_cache_text_matches_oracle_cache():
    """The host-driven replay's CACHE bookkeeping (a flat text with separators and
    oldest-first eviction) gives the oracle CACHE's text after every add."""
    rng = random.Random(5)
    for _ in range(300):
        cap = rng.randint(1, 60)
        a, b = oracle.Cache(cap), _Sequences(cap)
        for _ in range(rng.randint(1, 40)):
            seq = [rng.randint(1, 9) for _ in range(rng.randint(0, 70))]
            a.add(seq)
            b.add(seq)
            assert a.text().tolist() == b.text()
            assert a.size == len(b.lens)
