"""Pins for the oracle's retrieval: brute-force substring scans per n
(Section III-A), the two-store priority budget (Section IV-A, Section IV-C),
the strided sample's closed form and the hand-worked examples."""
import numpy as np
import pytest

import brute
import oracle
import synth


def _ctx_from(text, rng, L=16, fresh_prob=0.3, vocab=4):
    """A context row: a window of `text` (so long matches exist) or random."""
    if rng.random() < fresh_prob or len(text) < L:
        return rng.integers(1, vocab, size=L).astype(np.uint16)
    j = int(rng.integers(0, len(text) - L + 1))
    return np.asarray(text[j:j + L], np.uint16)


def _compare(texts, ctx, n_max, n_min, k, m):
    for batched in (False, True):
        _compare_one(oracle.retrieve(texts, ctx, n_max=n_max, n_min=n_min, k=k, m=m, batched=batched),
                     texts, ctx, n_max, n_min, k, m)


def _compare_one(got, texts, ctx, n_max, n_min, k, m):
    for b in range(ctx.shape[0]):
        want = brute.retrieve(texts, ctx[b], n_max, n_min, k, m)
        for f in ("match_n", "range_lo", "range_cnt", "taken"):
            assert got[f][b].tolist() == want[f], (f, b)
        used = len(want["slots"])
        for i, (s, start, cont) in enumerate(want["slots"]):
            assert got["cont_src"][b, i] == s
            assert got["cont_pos"][b, i] == start
            assert got["cont_len"][b, i] == len(cont)
            assert got["cont_tok"][b, i, :len(cont)].tolist() == cont
            assert not got["cont_tok"][b, i, len(cont):].any()
        assert (got["cont_pos"][b, used:] == 0xFFFFFFFF).all()
        assert (got["cont_src"][b, used:] == 0xFF).all()
        assert not got["cont_len"][b, used:].any()
        assert not got["cont_tok"][b, used:].any()


@pytest.mark.parametrize("vocab", [2, 3, 5, 40])
@pytest.mark.parametrize("seed", range(4))
def test_single_store_vs_brute(vocab, seed):
    rng = np.random.default_rng(seed * 100 + vocab)
    t = synth.random_text(seed + 31 * vocab, 150 + 30 * seed, vocab, sep_prob=0.04)
    ctx = np.stack([_ctx_from(t, rng, L=8, vocab=vocab) for _ in range(6)])
    for k in (1, 3, 7, 50):
        _compare([t], ctx, n_max=6, n_min=2, k=k, m=4)


@pytest.mark.parametrize("seed", range(4))
def test_two_stores_vs_brute(seed):
    rng = np.random.default_rng(seed)
    tp = synth.random_text(500 + seed, 90, 4, sep_prob=0.05)
    tg = synth.random_text(900 + seed, 220, 4, sep_prob=0.05)
    rows = []
    for _ in range(8):
        rows.append(_ctx_from(tp if rng.random() < 0.5 else tg, rng, L=10))
    ctx = np.stack(rows)
    for k in (2, 5, 9, 100):
        _compare([tp, tg], ctx, n_max=8, n_min=2, k=k, m=3)


def test_limits_and_degenerate_cases():
    t = np.array([1, 2, 3, 1, 2, 3, 0, 1, 2], np.uint16)
    # separator inside the context caps the usable suffix
    ctx = np.array([[3, 3, 0, 1, 2]], np.uint16)
    _compare([t], ctx, 16, 2, 4, 3)
    r = oracle.retrieve([t], ctx, n_max=16, n_min=2, k=4, m=3)
    assert r["match_n"][0, 0] == 2
    # context ending in 0: nothing is usable
    r = oracle.retrieve([t], np.array([[1, 2, 0]], np.uint16), n_max=16, n_min=2, k=4, m=3)
    assert r["match_n"][0, 0] == 0 and r["taken"][0, 0] == 0 and r["range_lo"][0, 0] == 0
    # L below n_min
    r = oracle.retrieve([t], np.array([[2]], np.uint16), n_max=16, n_min=2, k=4, m=3)
    assert r["match_n"][0, 0] == 0
    # n_min = 1 allows single-token matches
    r = oracle.retrieve([t], np.array([[9, 3]], np.uint16), n_max=16, n_min=1, k=4, m=3)
    assert r["match_n"][0, 0] == 1 and r["range_cnt"][0, 0] == 2
    # empty store
    r = oracle.retrieve([np.zeros(0, np.uint16)], np.array([[1, 2]], np.uint16), n_max=4, n_min=2, k=3, m=2)
    assert r["match_n"][0, 0] == 0 and (r["cont_pos"][0] == 0xFFFFFFFF).all()
    # continuation cut at the end of the text and at m
    _compare([t], np.array([[5, 1, 2]], np.uint16), 3, 2, 4, 1)
    _compare([t], np.array([[5, 2, 3]], np.uint16), 3, 2, 4, 7)


def test_maximality_and_count_budget():
    """match_n is maximal; taken in {cnt-1, cnt, cnt+1} budgets."""
    t = synth.random_text(7, 300, 3, sep_prob=0.02)
    rng = np.random.default_rng(3)
    ctx = np.stack([_ctx_from(t, rng, L=12, vocab=3) for _ in range(10)])
    base = oracle.retrieve([t], ctx, n_max=12, n_min=2, k=10_000, m=4)
    tl = t.tolist()
    for b in range(ctx.shape[0]):
        n = int(base["match_n"][b, 0])
        hi = brute.query_limit(ctx[b], 12)
        row = ctx[b].tolist()
        for n2 in range(n + 1, hi + 1):
            q = row[len(row) - n2:]
            assert all(tl[j:j + n2] != q for j in range(len(tl) - n2 + 1))
        cnt = int(base["range_cnt"][b, 0])
        for k in {max(cnt - 1, 1), cnt, cnt + 1}:
            if cnt == 0:
                continue
            r = oracle.retrieve([t], ctx[b:b + 1], n_max=12, n_min=2, k=k, m=4)
            assert r["taken"][0, 0] == min(k, cnt)


def test_strided_sample_closed_form():
    """Kept SA offsets are floor(i*cnt/b); every run of equal continuation
    prefixes keeps its share of the budget to within one."""
    t = synth.store(1, "single")[:60_000]
    sa = oracle.suffix_array(t)
    # the most frequent separator-free bigram of the slice
    pairs = t[:-1].astype(np.uint32) * 65536 + t[1:]
    pairs = pairs[(t[:-1] != 0) & (t[1:] != 0)]
    vals, counts = np.unique(pairs, return_counts=True)
    top = int(vals[np.argmax(counts)])
    ctx = np.array([[top >> 16, top & 0xFFFF]], np.uint16)
    full = oracle.retrieve([t], ctx, n_max=2, n_min=2, k=100_000, m=3)
    cnt = int(full["range_cnt"][0, 0])
    assert cnt > 8
    lo = int(full["range_lo"][0, 0])
    for b in (1, 2, 3, cnt // 2, cnt - 1):
        r = oracle.retrieve([t], ctx, n_max=2, n_min=2, k=b, m=3)
        want = [int(sa[lo + (i * cnt) // b]) + 2 for i in range(b)]
        assert r["cont_pos"][0, :b].tolist() == want
        firsts = full["cont_tok"][0, :cnt, 0]
        kept = r["cont_tok"][0, :b, 0]
        for tok in set(firsts.tolist()):
            share = (firsts == tok).sum() * b / cnt
            assert abs((kept == tok).sum() - share) <= 1.0 + 1e-9


def test_example_a(golden):
    g = golden("example_a.json")
    t = np.array(g["text"], np.uint16)
    ctx = np.array([g["ctx"]], np.uint16)
    p = g["params"]
    for k, key, batched in ((2, "retrieve_k2", False), (3, "retrieve_k3", False), (2, "retrieve_k2", True),
                            (3, "retrieve_k3", True)):
        r = oracle.retrieve([t], ctx, n_max=p["n_max"], n_min=p["n_min"], k=k, m=p["m"], batched=batched)
        w = g[key]
        assert r["match_n"][0, 0] == w["match_n"]
        assert r["range_lo"][0, 0] == w["range_lo"]
        assert r["range_cnt"][0, 0] == w["range_cnt"]
        assert r["taken"][0, 0] == w["taken"]
        assert r["cont_pos"][0].tolist() == w["cont_pos"]
        assert r["cont_len"][0].tolist() == w["cont_len"]
        assert r["cont_tok"][0].tolist() == w["cont_tok"]


def test_example_b(golden):
    g = golden("example_b.json")
    p = g["params"]
    for batched in (False, True):
        r = oracle.retrieve([np.array(g["project"], np.uint16), np.array(g["general"], np.uint16)],
                            np.array([g["ctx"]], np.uint16), n_max=p["n_max"], n_min=p["n_min"], k=p["k"], m=p["m"],
                            batched=batched)
        for f, v in g["retrieve"].items():
            assert r[f][0].tolist() == v, f


def _same(a: dict, b: dict) -> None:
    for f in a:
        assert a[f].shape == b[f].shape and (a[f] == b[f]).all(), f


@pytest.mark.parametrize("seed", range(6))
def test_batched_equals_definition(seed):
    """The batch-shared scans give the per-query definition's answer on
    every field, padding included: one to four stores (one empty), small
    vocabularies (long repeats, many queries sharing a last or first
    token), contexts with separators, of length 1..16, n_min 1..3 and
    budgets below, at and above the counts."""
    rng = np.random.default_rng(700 + seed)
    vocab = [2, 3, 5, 16, 300, 32256][seed]
    S = 1 + seed % 4
    texts = [synth.random_text(40 * seed + s, int(rng.integers(0, 3000)) if s != 1 else 0, vocab,
                               sep_prob=0.02 * (s % 2)) for s in range(S)]
    for L, n_min in ((16, 2), (5, 1), (1, 1), (3, 3)):
        rows = []
        for _ in range(40):
            src = texts[int(rng.integers(0, S))]
            rows.append(_ctx_from(src, rng, L=L, fresh_prob=0.3, vocab=vocab))
        ctx = np.stack(rows)
        if L > 1:
            ctx[::7, -2] = 0
        ctx[::11, -1] = 0
        for k, m in ((1, 1), (7, 3), (64, 10), (5000, 16)):
            want = oracle.retrieve(texts, ctx, n_max=min(16, max(L, n_min)), n_min=n_min, k=k, m=m)
            got = oracle.retrieve(texts, ctx, n_max=min(16, max(L, n_min)), n_min=n_min, k=k, m=m, batched=True)
            _same(want, got)


def test_batched_equals_definition_on_workload():
    """The 1M-token store and its 64 queries, and the 2M project store with
    the first 96 queries of the two-store batch: both forms agree."""
    t = synth.store(1, "single")
    ctx = synth.queries(1)
    _same(oracle.retrieve([t], ctx), oracle.retrieve([t], ctx, batched=True))
    tp = synth.store(2, "project")
    ctx = synth.queries(2, count=96)
    _same(oracle.retrieve([tp, t], ctx), oracle.retrieve([tp, t], ctx, batched=True))
