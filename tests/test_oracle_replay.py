"""Pins for the oracle's decode-trace replay: position bookkeeping, accepted
length bounds, the LRU's hit count against an independent list-based LRU,
and cache transparency (a cache never changes what is accepted)."""
import numpy as np

import oracle
import synth


def _setup():
    store = synth.store(3, "project")[:300_000]
    truth = synth.truth(n_seq=5, length=260)
    return [store], truth


def _lru_hits(keys, size):
    """Hits of a least-recently-used cache of `size` keys, list based."""
    cache, hits = [], 0
    for k in keys:
        if k in cache:
            hits += 1
            cache.remove(k)
        elif len(cache) == size:
            cache.pop(0)
        cache.append(k)
    return hits


def test_replay_bookkeeping_and_lru():
    texts, truth = _setup()
    m = 6
    for lru in (1, 4, 32):
        r = oracle.replay(texts, truth, m=m, k=300, c=16, alpha=(1,), lru=lru, max_steps=400)
        acc = r["accept"]
        assert acc.shape[1] == truth.shape[0]
        for b in range(truth.shape[0]):
            live = acc[:, b][acc[:, b] >= 0]
            assert ((live >= 1) & (live <= m + 1)).all()
            assert r["pos"][b] == 16 + live.sum()
            assert r["pos"][b] >= truth.shape[1]            # every stream ran to its end
            assert r["pos"][b] - live[-1] < truth.shape[1]  # and stopped right after
            # the keys the stream looked up, from its recorded positions
            p = 16
            keys = []
            for a in live:
                keys.append(truth[b, p - 16:p].tobytes())
                p += int(a)
            assert r["lookups"][b] == len(keys)
            assert r["hits"][b] == _lru_hits(keys, lru)
        if lru == 1:
            base = acc
        else:
            assert (acc == base).all()  # caching never changes what is accepted
    # streams drawn from the store's own pool are mostly predictable
    assert r["acc_len"] > 2.0


def test_replay_periodic_stream_lru_counts():
    """A store that never matches the stream gives a bare root every step, so
    the stream advances one token per step and its contexts cycle with the
    stream's period: 20 distinct keys.  An LRU holding all of them misses
    only on the first cycle; a smaller one thrashes and never hits."""
    store = np.full(5000, 7, np.uint16)
    period = (np.arange(20) * 13 % 97 + 100).astype(np.uint16)
    t = np.tile(period, 12)[None, :]  # 240 tokens
    lookups = t.shape[1] - 16
    r = oracle.replay([store], t, m=4, k=50, c=8, alpha=(1,), lru=32, max_steps=1000)
    assert (r["accept"][:, 0] == 1).all() and r["lookups"][0] == lookups
    assert r["hits"][0] == lookups - 20
    r = oracle.replay([store], t, m=4, k=50, c=8, alpha=(1,), lru=10, max_steps=1000)
    assert r["hits"][0] == 0
    assert r["acc_len"] == 1.0
