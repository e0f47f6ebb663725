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


# ------------------------------------------------------------------ CACHE ---

def _brute_cache_replay(texts, truth, n_max, n_min, k, m, c, alpha, ctx_len, cache_l, every, cap, max_steps,
                        missing=False, skip_tok=None, skip_p=0.5, draws=None):
    """Alg. 1 (the CACHE branch, the missing table and the skip gate) and
    the CACHE updates of Section IV-B, restated with the brute-force
    retrieval, trie and acceptance (no LRU: it never changes what is
    accepted)."""
    import brute

    nseq, tlen = truth.shape
    pos = [ctx_len] * nseq
    seqs = [[] for _ in range(nseq)]
    done = [0] * nseq
    served = [0] * nseq
    mtab = [set() for _ in range(nseq)]
    skips = [0, 0]

    def text(b):
        out = []
        for i, x in enumerate(seqs[b]):
            out += ([0] if i else []) + x
        return out

    def add(b, seq):
        seq = [int(x) for x in seq][-cap:]
        if seq:
            seqs[b].append(seq)
            while sum(len(x) for x in seqs[b]) + len(seqs[b]) - 1 > cap:
                seqs[b].pop(0)

    steps = []
    for step in range(max_steps):
        act = [b for b in range(nseq) if pos[b] < tlen]
        if not act:
            break
        row = [-1] * nseq
        for b in act:
            p = pos[b]
            ctx = [int(x) for x in truth[b, p - ctx_len:p]]
            r, al = None, tuple(alpha)
            if len(seqs[b]) >= cache_l:
                rc = brute.retrieve([text(b)], ctx, n_max, n_min, k, m)
                if sum(rc["taken"]) > 0:
                    r, al = rc, (1,)
                    served[b] += 1
            if r is None:
                if missing and tuple(ctx) in mtab[b]:
                    r = dict(taken=[0], slots=[])
                    skips[0] += 1
                elif skip_tok is not None and ctx[-1] == skip_tok and draws[step][b] >= skip_p * 2 ** 31:
                    r = dict(taken=[0], slots=[])
                    skips[1] += 1
                else:
                    r = brute.retrieve(texts, ctx, n_max, n_min, k, m)
                    if missing and sum(r["taken"]) == 0:
                        mtab[b].add(tuple(ctx))
            conts = [(s, cont) for s, _, cont in r["slots"]]
            t = brute.draft_tree(conts, al, c, ctx[-1])
            target = [int(truth[b, p + d]) if p + d < tlen else -1 for (_, _, _, d) in t["rows"]]
            acc, _, u = brute.accept(t["rows"], target)
            depth = t["rows"][u][3]
            if sum(r["taken"]) > 0 and depth >= 1:
                add(b, ctx + [int(x) for x in truth[b, p:p + depth]])
            row[b] = acc
            pos[b] += acc
            while ctx_len + every * (done[b] + 1) <= min(pos[b], tlen):
                lo = ctx_len + every * done[b]
                add(b, truth[b, lo:lo + every])
                done[b] += 1
        steps.append(row)
    return np.array(steps), np.array(pos), np.array(served), skips


def test_cache_text_and_eviction():
    c = oracle.Cache(cap=10)
    assert c.size == 0 and len(c.text()) == 0
    c.add([1, 2, 3])
    c.add([4, 5])
    assert c.text().tolist() == [1, 2, 3, 0, 4, 5] and c.size == 2
    c.add([6, 7, 8])  # 10 tokens with separators: fits exactly
    assert c.text().tolist() == [1, 2, 3, 0, 4, 5, 0, 6, 7, 8]
    c.add([9])  # 12 > 10: the oldest sequence goes
    assert c.text().tolist() == [4, 5, 0, 6, 7, 8, 0, 9] and c.size == 3
    c.add(list(range(1, 15)))  # longer than the cap alone: its last 10 tokens, everything else dropped
    assert c.text().tolist() == list(range(5, 15)) and c.size == 1
    c.add([])
    assert c.size == 1


def test_cache_replay_matches_brute_force():
    """Tiny vocabularies make long repeats, so the CACHE activates, serves
    steps, fills past its cap and evicts; every accepted length, final
    position and cache-served count must equal an independent restatement."""
    for seed, (vocab, cache_l, every, cap) in enumerate([(5, 2, 7, 60), (7, 1, 5, 40), (4, 3, 9, 200)]):
        store = synth.random_text(300 + seed, 250, vocab, 0.03)
        truth = np.stack([synth.random_text(400 + 10 * seed + i, 90, vocab) for i in range(3)])
        kw = dict(n_max=6, n_min=2, k=20, m=4, c=8, alpha=(1,))
        r = oracle.replay([store], truth, lru=4, ctx_len=6, max_steps=200, cache_l=cache_l, cache_every=every,
                          cache_cap=cap, **kw)
        acc, pos, served, _ = _brute_cache_replay([store], truth, ctx_len=6, cache_l=cache_l, every=every, cap=cap,
                                                  max_steps=200, **kw)
        assert (r["accept"] == acc).all(), seed
        assert (r["pos"] == pos).all() and (r["cache_served"] == served).all()
        assert served.sum() > 0  # the cache branch was exercised


def test_cache_inactive_is_plain_replay():
    texts, truth = _setup()
    kw = dict(m=6, k=300, c=16, alpha=(1,), lru=4, max_steps=120)
    base = oracle.replay(texts, truth, **kw)
    never = oracle.replay(texts, truth, cache_l=10 ** 9, **kw)
    for f in ("accept", "hits", "lookups", "pos"):
        assert (base[f] == never[f]).all(), f
    assert (never["cache_served"] == 0).all()



# ---------------------------------------------- missing table, skip gate ---

def _draws(n_steps: int, n_seq: int, seed: int = 9) -> np.ndarray:
    return np.stack([synth.uniform(seed, 30, step, n_seq, 0, 2 ** 31 - 1) for step in range(n_steps)])


def test_missing_table_closed_form():
    """A store that never matches a periodic stream: each of the 20
    contexts is retrieved once, fails, enters M, and is never retrieved
    again."""
    store = np.full(5000, 7, np.uint16)
    period = (np.arange(20) * 13 % 97 + 100).astype(np.uint16)
    t = np.tile(period, 12)[None, :]
    steps = t.shape[1] - 16
    r = oracle.replay([store], t, m=4, k=50, c=8, alpha=(1,), lru=32, max_steps=1000, missing=True)
    assert (r["accept"][:, 0] == 1).all()
    assert r["lookups"][0] == 20 and r["missing_skips"][0] == steps - 20 and r["gate_skips"][0] == 0


def test_skip_gate_closed_form():
    """p = 0 skips every context ending with the skip token, p = 1 none; with
    a store that never matches every step advances one token, so the
    skipped count is the number of such contexts."""
    store = np.full(5000, 7, np.uint16)
    period = (np.arange(20) * 13 % 97 + 100).astype(np.uint16)
    t = np.tile(period, 12)[None, :]
    tok = int(period[5])
    draws = _draws(300, 1)
    want = int(sum(1 for p in range(16, t.shape[1]) if t[0, p - 1] == tok))
    kw = dict(m=4, k=50, c=8, alpha=(1,), lru=32, max_steps=1000, skip_tok=tok, skip_draws=draws)
    r0 = oracle.replay([store], t, skip_p=0.0, **kw)
    r1 = oracle.replay([store], t, skip_p=1.0, **kw)
    assert r0["gate_skips"][0] == want and r1["gate_skips"][0] == 0
    assert r0["lookups"][0] == t.shape[1] - 16 - want and r1["lookups"][0] == t.shape[1] - 16


def test_control_replay_matches_brute_force():
    """CACHE, missing table and skip gate together against the independent
    restatement: every accepted length, position, CACHE-served count and
    skip count equal."""
    tot = np.zeros(3, np.int64)
    for seed, (vocab, cache_l, every, cap, period) in enumerate([(5, 3, 7, 80, 0), (8, 2, 5, 120, 0),
                                                                 (40, 6, 9, 100, 23), (30, 50, 20, 400, 17)]):
        store = synth.random_text(600 + seed, 200, vocab, 0.05)
        if period:  # recurring contexts that the store rarely matches: the missing table's case
            truth = np.stack([np.resize(synth.random_text(700 + 10 * seed + i, period, vocab), 100)
                              for i in range(3)])
        else:
            truth = np.stack([synth.random_text(700 + 10 * seed + i, 100, vocab) for i in range(3)])
        draws = _draws(250, 3, seed=20 + seed)
        tok = int(truth[0, 3])
        kw = dict(n_max=6, n_min=2, k=20, m=4, c=8, alpha=(1,))
        r = oracle.replay([store], truth, lru=4, ctx_len=6, max_steps=250, cache_l=cache_l, cache_every=every,
                          cache_cap=cap, missing=True, skip_tok=tok, skip_p=0.5, skip_draws=draws, **kw)
        acc, pos, served, skips = _brute_cache_replay([store], truth, ctx_len=6, cache_l=cache_l, every=every,
                                                      cap=cap, max_steps=250, missing=True, skip_tok=tok,
                                                      skip_p=0.5, draws=draws, **kw)
        assert (r["accept"] == acc).all(), seed
        assert (r["pos"] == pos).all() and (r["cache_served"] == served).all()
        assert r["missing_skips"].sum() == skips[0] and r["gate_skips"].sum() == skips[1]
        tot += [served.sum(), skips[0], skips[1]]
    assert (tot > 0).all()  # every branch of Alg. 1 was exercised
