"""GPU parity: every output of the HIP path, called through the C ABI, equals
the oracle's bit for bit on the same seeded inputs.

Sizes: tiny adversarial texts (small vocabularies force long repeats and
ties) spanning several 4096-suffix sort tiles with ragged tails; the 1M-token
single store of the first workload in full; the 2M + 100M two-store workload
in full; the 10M + 1B headline workload in the batch shape the benchmark
launches, every query of it (the oracle's batched form makes one pass over
each store for the batch), with the suffix arrays by the linear-time
checker; and the decode-trace replay on those stores, 128 streams for 32
steps against the oracle run live and for the full 512 steps against the
oracle's stored trace.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_pipeline import (compare_retrieve, compare_tree, dev, gpu_pipeline, gpu_store, host,
                          oracle_pipeline, say, targets_from_truth)

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - CPU container
    pytest.skip("no GPU", allow_module_level=True)

import paper_2502_17139_amd as fc  # noqa: E402
from host_replay import GpuReplay  # noqa: E402

P = dict(synth.PARAMS)


def _targets(tree: dict, seed: int, row_ids=None) -> np.ndarray:
    """Seeded targets that follow the tree most of the time; computed from
    one side's own tree output.  row_ids name each row's query in the full
    batch, so a sampled subset draws the same targets as the full batch."""
    B, R = tree["node_tok"].shape
    out = np.full((B, R), -1, np.int32)
    for b in range(B):
        n = int(tree["num_nodes"][b])
        par = tree["parent"][b]
        qid = b if row_ids is None else int(row_ids[b])
        for i in range(max(n, 0)):
            rng = np.random.default_rng([seed, qid, i])
            kids = [v for v in range(1, n) if par[v] == i]
            if kids and rng.random() < 0.75:
                out[b, i] = int(tree["node_tok"][b, kids[int(rng.integers(len(kids)))]])
            else:
                out[b, i] = int(rng.integers(-1, 40000))
    return out


def _check_accept(g: dict, o: dict, m: int, seed: int = 0, rows=None):
    tg = _targets({f: g[f] for f in ("node_tok", "parent", "num_nodes")}, seed)
    to = _targets({f: o[f] for f in ("node_tok", "parent", "num_nodes")}, seed)
    ga = fc.fc_verify_accept(g["_tree_dev"], dev(tg), m=m)
    torch.cuda.synchronize()
    oa = oracle.verify_accept(o, to, m=m)
    rows = range(len(oa["accept_len"])) if rows is None else rows
    for i, b in enumerate(rows):
        for f in ("accept_len", "accept_tok", "last_node"):
            assert (host(ga[f])[b] == oa[f][i]).all(), (f, b)


# ------------------------------------------------------------ suffix arrays --

def _sa_case(t: np.ndarray):
    g = host(fc.fc_datastore_build(dev(t)))
    torch.cuda.synchronize()
    o = oracle.suffix_array(t)
    assert (g == o).all()


@pytest.mark.parametrize("vocab", [2, 3, 4, 16, 32256])
def test_sa_small_texts(vocab):
    for seed, n in enumerate([1, 2, 3, 7, 64, 4095, 4096, 4097, 9000, 20011]):
        say(f"sa vocab={vocab} n={n}")
        _sa_case(synth.random_text(1000 * vocab + seed, n, vocab, sep_prob=0.03 if seed % 2 else 0.0))


def test_sa_degenerate_texts():
    for n in (1, 5, 4096, 12345):
        say(f"sa degenerate n={n}")
        _sa_case(np.full(n, 7, np.uint16))                       # all equal: n rounds of doubling
        _sa_case(np.zeros(n, np.uint16))                         # all separators
        _sa_case(np.arange(1, n + 1, dtype=np.uint16))           # increasing
        _sa_case(np.full(n, 65535, np.uint16))                   # largest token
    _sa_case((np.arange(30000) % 2).astype(np.uint16))           # period 2
    _sa_case(np.tile(np.array([5, 9, 5, 9, 1], np.uint16), 3000))


def test_sa_first_workload():
    t = synth.store(1, "single")
    _sa_case(t)


def test_sa_two_store_workload():
    _sa_case(synth.store(2, "project"))
    g = synth.store(2, "general")
    sa = host(fc.fc_datastore_build(dev(g)))
    torch.cuda.synchronize()
    assert oracle.check_sa(g, sa) == (0, 0)


def test_sa_large_texts_rank_pairs():
    """Stores of 64M suffixes or more take their ranks through sorted
    (suffix, rank) pairs instead of random writes: just past that size, with
    a ragged last tile, a near-periodic text (about 25 doubling rounds,
    nearly every rank rewritten in each) and a 4-token random text, each
    checked by the linear-time checker."""
    n = (1 << 26) + 4097
    periodic = np.tile(np.array([5, 9, 5, 9, 1], np.uint16), n // 5 + 1)[:n].copy()
    periodic[n // 3] = 7  # one break, so two long runs of the period
    for name, t, min_rounds in (("near-periodic", periodic, 20), ("vocab 4", synth.random_text(4242, n, 4), 3)):
        say(f"sa rank pairs: {name} n={n}")
        sa, stats = fc.fc_datastore_build_stats(dev(t))
        torch.cuda.synchronize()
        assert stats["rounds"] >= min_rounds, (name, stats["rounds"])
        assert oracle.check_sa(t, host(sa)) == (0, 0), name


def _batched_case(tok: np.ndarray, off: np.ndarray, full: bool = True):
    """Batched build: store r's slice of the output is the suffix array of
    store r alone (oracle comparison sort, or the linear-time checker)."""
    g = host(fc.fc_datastore_build_batched(dev(tok), off))
    torch.cuda.synchronize()
    for r in range(len(off) - 1):
        a, b = int(off[r]), int(off[r + 1])
        if full:
            assert (g[a:b] == oracle.suffix_array(tok[a:b])).all(), (r, a, b)
        else:
            assert oracle.check_sa(tok[a:b], g[a:b]) == (0, 0), (r, a, b)


def _concat(parts):
    off = np.zeros(len(parts) + 1, np.uint64)
    off[1:] = np.cumsum([len(x) for x in parts])
    return np.concatenate([np.asarray(x, np.uint16) for x in parts]), off


@pytest.mark.parametrize("vocab", [2, 4, 32256])
def test_sa_batched_ragged_stores(vocab):
    lens = [0, 1, 2, 3, 0, 7, 64, 4095, 4096, 4097, 0, 9000, 5]
    say(f"sa batched vocab={vocab} lens={lens}")
    _batched_case(*_concat([synth.random_text(5000 * vocab + i, n, vocab, sep_prob=0.03 if i % 2 else 0.0)
                            for i, n in enumerate(lens)]))


def test_sa_batched_stores_do_not_see_each_other():
    # equal stores back to back: a suffix that ran on into the next store
    # would sort differently from the same suffix of a store built alone
    for t in (np.full(1000, 7, np.uint16), synth.random_text(3, 2500, 2), np.zeros(300, np.uint16),
              (np.arange(3000) % 3).astype(np.uint16)):
        say(f"sa batched repeated n={len(t)}")
        _batched_case(*_concat([t] * 5))
        _batched_case(*_concat([t, t[: len(t) // 2], t, t[:1]]))


def test_sa_batched_single_store_equals_plain_build():
    t = synth.random_text(77, 20011, 4, sep_prob=0.01)
    g = host(fc.fc_datastore_build_batched(dev(t), np.array([0, len(t)], np.uint64)))
    torch.cuda.synchronize()
    assert (g == host(fc.fc_datastore_build(dev(t)))).all()
    assert (g == oracle.suffix_array(t)).all()


def test_sa_batched_many_tiny_stores():
    lens = synth.uniform(9, 30, 0, 3000, 0, 50)
    say(f"sa batched {len(lens)} tiny stores")
    _batched_case(*_concat([synth.random_text(90_000 + i, int(n), 4) for i, n in enumerate(lens)]))
    _batched_case(np.zeros(0, np.uint16), np.zeros(4, np.uint64))   # only empty stores


def test_sa_batched_repository_set():
    tok, off = synth.repos(11, 48, 2, 400)
    say(f"sa batched repositories n={len(tok)}")
    _batched_case(tok, off)
    tok, off = synth.repos(12, 64, 60, 2000)   # the benchmark's repository set
    say(f"sa batched benchmark repositories n={len(tok)}")
    _batched_case(tok, off, full=False)


def _inverse(sa: np.ndarray) -> np.ndarray:
    inv = np.empty(len(sa), np.uint32)
    inv[sa.astype(np.int64)] = np.arange(len(sa), dtype=np.uint32)
    return inv


def _extend_case(new: np.ndarray, old: np.ndarray, full: bool = True):
    """Extension: the new files in front of an old store, from the old
    store's suffix array (with and without its inverse); must equal the
    suffix array of the whole text, and isa_out its inverse."""
    t = np.concatenate([np.asarray(new, np.uint16), np.asarray(old, np.uint16)])
    o_sa = oracle.suffix_array(old) if full else host(fc.fc_datastore_build(dev(old)))
    want = oracle.suffix_array(t) if full else None
    for give_isa in (False, True):
        isa_out = torch.empty(len(t), dtype=torch.uint32, device="cuda")
        g = host(fc.fc_datastore_extend(dev(t), len(new), dev(o_sa), old_isa=dev(_inverse(o_sa)) if give_isa else None,
                                        isa_out=isa_out))
        torch.cuda.synchronize()
        if full:
            assert (g == want).all(), (len(new), len(old), give_isa)
        else:
            assert oracle.check_sa(t, g) == (0, 0), (len(new), len(old), give_isa)
        assert (host(isa_out) == _inverse(g)).all(), (len(new), len(old), give_isa)


@pytest.mark.parametrize("vocab", [2, 4, 32256])
def test_sa_extend_small_texts(vocab):
    for seed, (n_new, n_old) in enumerate([(0, 5), (5, 0), (1, 1), (1, 4096), (4097, 1), (3, 9000), (9000, 3),
                                           (4095, 4097), (20011, 7000), (64, 64)]):
        say(f"sa extend vocab={vocab} new={n_new} old={n_old}")
        new = synth.random_text(7000 * vocab + seed, n_new, vocab, sep_prob=0.03 if seed % 2 else 0.0)
        old = synth.random_text(8000 * vocab + seed, n_old, vocab, sep_prob=0.03 if seed % 2 else 0.0)
        _extend_case(new, old)


def test_sa_extend_degenerate_texts():
    for n_new, n_old in ((1, 5000), (5000, 1), (3000, 3000)):
        say(f"sa extend degenerate new={n_new} old={n_old}")
        _extend_case(np.full(n_new, 7, np.uint16), np.full(n_old, 7, np.uint16))   # one long run
        _extend_case(np.zeros(n_new, np.uint16), np.zeros(n_old, np.uint16))
        _extend_case(np.full(n_new, 65535, np.uint16), np.full(n_old, 1, np.uint16))
    old = synth.random_text(31, 6000, 3)
    _extend_case(np.concatenate([old, [0]]), old)                                  # new files repeat the old store
    _extend_case(np.concatenate([old[:2500], [0], old[:2500], [0]]), old)
    _extend_case((np.arange(5000) % 2).astype(np.uint16), (np.arange(7000) % 2).astype(np.uint16))


def test_sa_extend_twice_with_kept_inverse():
    # a store grows twice; the second extension takes the first's inverse
    a, b, c = (synth.random_text(600 + i, n, 5, sep_prob=0.02) for i, n in enumerate((3000, 5000, 8000)))
    t1 = np.concatenate([b, c])
    isa1 = torch.empty(len(t1), dtype=torch.uint32, device="cuda")
    sa1 = fc.fc_datastore_extend(dev(t1), len(b), dev(oracle.suffix_array(c)), isa_out=isa1)
    t2 = np.concatenate([a, t1])
    sa2 = fc.fc_datastore_extend(dev(t2), len(a), sa1, old_isa=isa1)
    torch.cuda.synchronize()
    assert (host(sa2) == oracle.suffix_array(t2)).all()


def test_sa_extend_repository_files():
    # a repository's new files (own seed, shared templates) in front of the
    # 1M-token single store, and in front of the 2M project store
    for cfg, role in ((1, "single"), (2, "project")):
        old = synth.store(cfg, role)
        tok, off = synth.repos(40 + cfg, 1, 20, 200)
        new = np.concatenate([tok, [0]]).astype(np.uint16)
        say(f"sa extend {role} by {len(new)} tokens")
        _extend_case(new, old, full=False)
        t = np.concatenate([new, old])
        ext = host(fc.fc_datastore_extend(dev(t), len(new), fc.fc_datastore_build(dev(old))))
        torch.cuda.synchronize()
        assert (ext == host(fc.fc_datastore_build(dev(t)))).all()


def test_bucket_table():
    for t in (synth.random_text(5, 5000, 300, 0.02), synth.store(1, "single"), np.zeros(0, np.uint16)):
        st = gpu_store(t) if len(t) else None
        if st is None:
            b = host(fc.fc_store_prepare(dev(np.zeros(1, np.uint16))[:0], dev(np.zeros(1, np.uint32))[:0]))
            assert (b == 0).all()
            continue
        b = host(st.bucket).astype(np.int64)
        counts = np.bincount(t.astype(np.int64), minlength=65536)
        want = np.concatenate([[0], np.cumsum(counts)])
        assert (b == want).all()


def _pair_table_expected(t: np.ndarray, V: int) -> np.ndarray:
    """Number of suffixes whose first two tokens sort below each (t0, u),
    by counting 2-prefix keys of every suffix (u = 0: suffix of length 1)."""
    n = len(t)
    t0 = t.astype(np.int64)
    u = np.zeros(n, np.int64)
    u[:-1] = t0[1:] + 1
    keys = t0 * (V + 1) + u
    counts = np.bincount(keys, minlength=V * (V + 1))
    return np.concatenate([[0], np.cumsum(counts)])


def test_pair_table():
    for seed, (n, V) in enumerate([(1, 3), (2, 3), (500, 5), (5000, 40), (70000, 300)]):
        t = synth.random_text(50 + seed, n, V, 0.05)
        say(f"pair table n={n} V={V}")
        st = gpu_store(t, pair_vocab=V)
        torch.cuda.synchronize()
        assert (host(st.pair).astype(np.int64) == _pair_table_expected(t, V)).all()
    # a larger vocabulary than needed is fine; a smaller one is rejected
    t = synth.random_text(9, 3000, 50, 0.05)
    st = gpu_store(t, pair_vocab=64)
    assert (host(st.pair).astype(np.int64) == _pair_table_expected(t, 64)).all()
    with pytest.raises(fc.FcError, match="INVALID"):
        fc.fc_store_prepare_pairs(st.tokens, st.sa, 49)


def test_records():
    """Record i = {sa[i], T[sa[i]+2 .. sa[i]+32)} with 0 past the end."""
    for seed, n in enumerate((1, 2, 17, 3000, 70001)):
        t = synth.random_text(70 + seed, n, 500, 0.05)
        say(f"records n={n}")
        st = fc.Store(dev(t), pair_vocab=500, records=True)
        torch.cuda.synchronize()
        sa = host(st.sa).astype(np.int64)
        rec = host(st.rec).view(np.uint32).reshape(n, 16)
        assert (rec[:, 0] == sa).all()
        padded = np.concatenate([t.astype(np.uint32), np.zeros(32, np.uint32)])
        idx = sa[:, None] + 2 + np.arange(30)[None, :]
        want = padded[idx]
        got = np.stack([rec[:, 1:] & 0xFFFF, rec[:, 1:] >> 16], axis=2).reshape(n, 30)
        assert (got == want).all()


# --------------------------------------------------------------- retrieval --

def test_first_workload_full_batch():
    t = synth.store(1, "single")
    ctx = synth.queries(1)
    st = gpu_store(t)
    st_pairs = fc.Store(st.tokens, st.sa, st.bucket, pair_vocab=synth.VOCAB)
    st_rec = fc.Store(st.tokens, st.sa, st.bucket, pair_vocab=synth.VOCAB, records=True)
    st_rec_only = fc.Store(st.tokens, st.sa, st.bucket, pair_vocab=synth.VOCAB, records=True, top=False)
    variants = {P["k"]: st_rec, 1000: st_pairs, 1200: st_rec, 257: st_rec_only}
    for (k, m, c) in ((P["k"], P["m"], P["c"]), (1000, 10, 64), (257, 3, 5), (1200, 13, 40), (1, 1, 1)):
        say(f"workload 1: k={k} m={m} c={c}")
        p = dict(P, k=k, m=m)
        g = gpu_pipeline([variants.get(k, st)], ctx, p, (1,), c)
        o = oracle_pipeline([t], ctx, p, (1,), c)
        compare_retrieve(g, o)
        compare_tree(g, o)
        _check_accept(g, o, m)


def test_two_store_workload_full_batch():
    tp, tg = synth.store(2, "project"), synth.store(2, "general")
    ctx = synth.queries(2)
    stores = [gpu_store(tp, synth.VOCAB, records=True), gpu_store(tg, synth.VOCAB, records=True)]
    say("workload 2: gpu")
    g = gpu_pipeline(stores, ctx, P, (1, 1), P["c"])
    say("workload 2: oracle")
    o = oracle_pipeline([tp, tg], ctx, P, (1, 1), P["c"])
    compare_retrieve(g, o)
    compare_tree(g, o)
    _check_accept(g, o, P["m"])
    # two-token tables without records
    plain = [fc.Store(x.tokens, x.sa, x.bucket, pair_vocab=synth.VOCAB) for x in stores]
    g = gpu_pipeline(plain, ctx[:128], P, (1, 1), P["c"])
    compare_retrieve(g, {f: v[:128] for f, v in o.items()})
    # unequal store weights, first-token tables only
    stores = [fc.Store(x.tokens, x.sa, x.bucket) for x in stores]
    g = gpu_pipeline(stores, ctx[:64], P, (3, 1), 32)
    o = oracle_pipeline([tp, tg], ctx[:64], P, (3, 1), 32)
    compare_tree(g, o)


@pytest.fixture(scope="module")
def headline():
    """The 10M-token project store and the 1B-token general store, on the GPU
    with two-token tables and records (as the benchmark runs them)."""
    say("headline: generating stores")
    tp, tg = synth.store(3, "project"), synth.store(3, "general")
    say("headline: building suffix arrays")
    stores = [gpu_store(tp, synth.VOCAB, records=True), gpu_store(tg, synth.VOCAB, records=True)]
    torch.cuda.synchronize()
    yield tp, tg, stores
    del stores
    synth.drop_cache()
    torch.cuda.empty_cache()


def test_headline_workload_full_batch(headline):
    """10M + 1B stores: the whole 1,024-query batch in the launch shape the
    benchmark times, every query compared with the oracle (its batched form,
    one pass over each store for the batch); suffix arrays by the
    linear-time checker."""
    tp, tg, stores = headline
    ctx = synth.queries(3)
    say("headline: checking suffix arrays")
    for t, st in zip((tp, tg), stores):
        assert oracle.check_sa(t, host(st.sa)) == (0, 0)
    say("headline: gpu pipeline")
    g = gpu_pipeline(stores, ctx, P, (1, 1), P["c"])
    say("headline: oracle on all 1024 queries")
    r = oracle.retrieve([tp, tg], ctx, n_max=P["n_max"], n_min=P["n_min"], k=P["k"], m=P["m"], batched=True)
    o = dict(r)
    o.update(oracle.build_tree(r["taken"], r["cont_len"], r["cont_tok"], ctx, c=P["c"], alpha=(1, 1)))
    say("headline: comparing")
    compare_retrieve(g, o)
    compare_tree(g, o)
    assert int(o["taken"].sum()) > 800_000  # the batch keeps ~900k slots: the heavy paths run
    _check_accept(g, o, P["m"], seed=3)


def test_headline_replay_live(headline):
    """Decode-trace replay on the 10M + 1B stores, all 128 streams, the
    first 32 steps: the device engine against the oracle run now (every
    accepted length, LRU hit and lookup, and position)."""
    tp, tg, stores = headline
    truth = synth.truth()
    say("headline replay: engine, 128 streams x 32 steps")
    eng = fc.ReplayEngine(stores, dev(truth), max_steps=512, **P)
    g = eng.run(limit=32)
    say("headline replay: oracle")
    o = oracle.replay([tp, tg], truth, **P, max_steps=32)
    assert g["steps"] == o["steps"] == 32
    for f in ("accept", "hits", "lookups", "pos"):
        assert (g[f] == o[f]).all(), f


def test_headline_replay_golden(headline, golden):
    """The full replay shape, 128 streams x 512 steps on the 10M + 1B
    stores: the device engine against the oracle's trace stored in
    tests/golden (written by make_replay_golden.py, which calls only the
    oracle and the generator), after checking the inputs' SHA-256."""
    import hashlib
    tp, tg, stores = headline
    truth = synth.truth()
    gold = golden("replay_10M_1B_128x512.json")
    sha = lambda a: hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()  # noqa: E731
    assert gold["sha256"] == {"project": sha(tp), "general": sha(tg), "truth": sha(truth)}
    assert gold["params"] == {kk: (list(v) if isinstance(v, tuple) else v) for kk, v in P.items()}
    say("headline replay: engine, 128 streams x 512 steps")
    eng = fc.ReplayEngine(stores, dev(truth), max_steps=512, lru=gold["lru"], **P)
    g = eng.run(limit=gold["max_steps"])
    digits = "0123456789abcdefghijklmnopqrstuvwxyz"
    acc = np.array([[-1 if ch == "." else digits.index(ch) for ch in col] for col in gold["accept"]]).T
    assert g["steps"] == gold["steps"] and g["accept"].shape == acc.shape
    assert (g["accept"] == acc).all()
    for f in ("hits", "lookups", "pos"):
        assert g[f].tolist() == gold[f], f
    assert abs(g["acc_len"] - gold["acc_len"]) < 1e-12


# ------------------------------------------------------------------ replay --

@pytest.mark.parametrize("native", [True, False], ids=["engine", "driver"])
def test_replay_matches_oracle(native):
    """Decode-trace replay, by the device engine and by the host-driven
    loop: 16 streams from the project pool, 10M-token project store +
    1M-token store, first 60 steps; every accepted length, cache hit and
    final position equal."""
    tp, t1 = synth.store(3, "project"), synth.store(1, "single")
    truth = synth.truth(n_seq=16, length=600)
    stores = [gpu_store(tp, synth.VOCAB), gpu_store(t1)]
    say(f"replay: gpu native={native}")
    g = GpuReplay(stores, truth, **P).run(max_steps=60, native=native)
    say("replay: oracle")
    o = oracle.replay([tp, t1], truth, **P, max_steps=60)
    for f in ("accept", "hits", "lookups", "pos"):
        assert (g[f] == o[f]).all(), f
    assert g["acc_len"] == o["acc_len"] and g["acc_len"] > 2.0


@pytest.mark.parametrize("native", [True, False], ids=["engine", "driver"])
def test_replay_cache_eviction(native):
    """Periodic streams that never match: one token per step, contexts cycle
    through 20 keys; LRU sizes above and below the cycle (device engine and
    host-driven loop)."""
    store = np.full(5000, 7, np.uint16)
    period = (np.arange(20) * 13 % 97 + 100).astype(np.uint16)
    truth = np.stack([np.tile(np.roll(period, r), 12) for r in range(3)])
    st = gpu_store(store)
    for lru in (10, 20, 32):
        p = dict(n_max=16, n_min=2, k=50, m=4, c=8, alpha=(1,))
        g = GpuReplay([st], truth, lru=lru, **p).run(max_steps=1000, native=native)
        o = oracle.replay([store], truth, lru=lru, **p, max_steps=1000)
        for f in ("accept", "hits", "lookups", "pos"):
            assert (g[f] == o[f]).all(), (lru, f)
        assert (g["hits"] == (truth.shape[1] - 16 - 20 if lru >= 20 else 0)).all()


# -------------------------------------------------------------- edge cases --

def test_large_batch():
    """4,200 queries: the kept-slot offsets no longer fit the gather's LDS
    table (a scan kernel of its own) and the light launch scans 17 queries
    per thread; random contexts match short and fill the heavy class."""
    texts = [synth.random_text(7, 20000, 8, 0.02), synth.random_text(8, 30000, 8, 0.02)]
    rng = np.random.default_rng(1)
    B = 4200
    # windows of the stores match long (light); a token the stores lack then
    # a pair of theirs matches two tokens only, with ~1,000 occurrences
    ctx = np.stack([texts[b % 2][j:j + 12] if b % 5 else
                    np.concatenate([np.full(10, 39, np.uint16), rng.integers(1, 8, 2).astype(np.uint16)])
                    for b, j in enumerate(rng.integers(0, 19000, B))])
    p = dict(n_max=12, n_min=2, k=400, m=10)
    say(f"large batch B={B}")
    g = gpu_pipeline([gpu_store(t) for t in texts], ctx, p, (1, 2), 16)
    o = oracle_pipeline(texts, ctx, p, (1, 2), 16)
    assert (o["taken"].sum(1) > 256).sum() > 100  # the heavy launch has work
    compare_retrieve(g, o)
    compare_tree(g, o)
    _check_accept(g, o, p["m"], 5)


@pytest.mark.parametrize("seed", range(6))
def test_fuzz_small_stores(seed):
    rng = np.random.default_rng(seed)
    S = 1 + seed % 4
    vocab = [3, 5, 12, 40, 300, 32256][seed]
    texts = [synth.random_text(100 * seed + s, int(rng.integers(0, 6000)), vocab, 0.02) for s in range(S)]
    if seed == 0:
        texts[0] = np.zeros(0, np.uint16)  # an empty store
    pv = vocab if seed % 2 else None
    stores = [gpu_store(t, pv, records=seed % 4 == 1) if len(t) else fc.Store(dev(np.zeros(1, np.uint16))[:0],
                                                    dev(np.zeros(1, np.uint32))[:0],
                                                    fc.fc_store_prepare(dev(np.zeros(1, np.uint16))[:0],
                                                                        dev(np.zeros(1, np.uint32))[:0]))
              for t in texts]
    rows = []
    for b in range(70):
        src = texts[int(rng.integers(S))]
        L = int(rng.integers(1, 20))
        if len(src) > L and rng.random() < 0.8:
            j = int(rng.integers(0, len(src) - L))
            rows.append(src[j:j + L].copy())
        else:
            rows.append(rng.integers(0, vocab, size=L).astype(np.uint16))
    Lmax = 19
    ctx = np.stack([np.concatenate([np.full(Lmax - len(r), 1, np.uint16), r]) for r in rows])
    for (n_max, n_min, k, m, c) in ((16, 2, 5000, 10, 64), (8, 1, 37, 4, 9), (3, 3, 300, 17, 200), (16, 2, 1, 1, 1)):
        say(f"fuzz seed={seed} S={S} n={n_max}..{n_min} k={k} m={m} c={c}")
        p = dict(n_max=n_max, n_min=n_min, k=k, m=m)
        alpha = (1, 2, 3, 5)[:S]
        g = gpu_pipeline(stores, ctx, p, alpha, c)
        o = oracle_pipeline(texts, ctx, p, alpha, c)
        compare_retrieve(g, o)
        compare_tree(g, o)
        _check_accept(g, o, m, seed)
    for L in (1, 2, 3):
        say(f"fuzz seed={seed} L={L}")
        p = dict(n_max=16, n_min=1 if L == 1 else 2, k=64, m=5)
        g = gpu_pipeline(stores, ctx[:, -L:], p, (1,) * S, 16)
        o = oracle_pipeline(texts, ctx[:, -L:], p, (1,) * S, 16)
        compare_retrieve(g, o)
        compare_tree(g, o)


def test_fuzz_many_tiny_cases():
    """About 1.2e4 query cases on tiny adversarial stores: 48 seeded store
    sets (one to four stores, vocabularies of 2 to 300 tokens, empty and
    one-token stores, with and without pair tables, records and the records'
    top-level sample) x 64 queries
    of 1 to 19 tokens x four parameter sets (the paper's n and budgets
    scaled down, n_min = 1, m > 16 through the any-m gather and tree, and
    k = m = c = 1).  Every retrieval, tree and acceptance output against the
    oracle."""
    params = ((16, 2, 64, 10, 16), (8, 1, 9, 4, 5), (5, 3, 300, 17, 40), (16, 2, 1, 1, 1))
    cases = 0
    for seed in range(48):
        rng = np.random.default_rng(1000 + seed)
        S = 1 + seed % 4
        vocab = (2, 3, 5, 12, 40, 300)[seed % 6]
        lens = [int(rng.integers(0, 800)) for _ in range(S)]
        if seed % 7 == 0:
            lens[0] = 1
        texts = [synth.random_text(5000 + 10 * seed + s, n, vocab, 0.03) for s, n in enumerate(lens)]
        stores = []
        for t in texts:
            if len(t) == 0:
                t = np.zeros(0, np.uint16)
                stores.append(fc.Store(dev(np.zeros(1, np.uint16))[:0], dev(np.zeros(1, np.uint32))[:0],
                                       fc.fc_store_prepare(dev(np.zeros(1, np.uint16))[:0],
                                                           dev(np.zeros(1, np.uint32))[:0])))
            else:
                # records with their top-level sample (seed % 4 == 1) and without it (== 3)
                stores.append(gpu_store(t, vocab if seed % 2 else None, records=seed % 2 == 1,
                                        top=seed % 4 == 1 if seed % 2 else None))
        rows = []
        for b in range(64):
            src = texts[int(rng.integers(S))]
            L = int(rng.integers(1, 20))
            if len(src) > L and rng.random() < 0.7:
                j = int(rng.integers(0, len(src) - L))
                rows.append(src[j:j + L].copy())
            else:
                rows.append(rng.integers(0, vocab, size=L).astype(np.uint16))
        ctx = np.stack([np.concatenate([np.full(19 - len(r), 1, np.uint16), r]) for r in rows])
        alpha = (1, 2, 3, 5)[:S]
        for (n_max, n_min, k, m, c) in params:
            say(f"tiny fuzz seed={seed} S={S} vocab={vocab} n={n_max}..{n_min} k={k} m={m} c={c}")
            p = dict(n_max=n_max, n_min=n_min, k=k, m=m)
            g = gpu_pipeline(stores, ctx, p, alpha, c)
            o = oracle_pipeline(texts, ctx, p, alpha, c)
            compare_retrieve(g, o)
            compare_tree(g, o)
            _check_accept(g, o, m, seed)
            cases += len(ctx)
    assert cases >= 12000


def test_results_do_not_depend_on_batching():
    """The same queries give the same per-query bytes whatever launch shape
    the batch leads to: one batch of 300 (the tree's heaviest-first planning
    launch, a full gather grid), batches of 1, 7, 41 and 251 (other gather
    grids and slot pieces, no planning launch), and the batch reversed
    through a row map (other workgroup-to-query assignment)."""
    t = synth.store(1, "single")
    st = gpu_store(t, synth.VOCAB, records=True)
    base = synth.queries(1)
    rng = np.random.default_rng(3)
    ctx = base[rng.integers(0, len(base), 300)]
    p = dict(P)
    fields = ("match_n", "range_lo", "range_cnt", "taken", "num_nodes", "node_tok", "parent", "weight",
              "pos_ids", "mask")
    ref = gpu_pipeline([st], ctx, p, (1,), p["c"])

    def same(got, lo, hi):
        for f in fields:
            assert (got[f] == ref[f][lo:hi]).all(), (f, lo, hi)
        for b in range(hi - lo):
            used = int(ref["taken"][lo + b].sum())
            for f in ("cont_pos", "cont_src", "cont_len", "cont_tok"):
                assert (got[f][b, :used] == ref[f][lo + b, :used]).all(), (f, lo + b)

    for size in (1, 7, 41, 251):
        say(f"batching: batches of {size}")
        for lo in range(0, 300, size):
            hi = min(300, lo + size)
            same(gpu_pipeline([st], ctx[lo:hi], p, (1,), p["c"]), lo, hi)
    say("batching: reversed through a row map")
    cx = dev(ctx[::-1].astype(np.uint16))
    rows = dev(np.arange(299, -1, -1, dtype=np.int32))
    r = fc.fc_retrieve([st], cx, n_max=p["n_max"], n_min=p["n_min"], k=p["k"], m=p["m"], rows=rows,
                       out=fc.retrieve_outputs(300, 1, p["k"], p["m"], cx.device))
    tr = fc.fc_build_tree(r["taken"], r["cont_len"], r["cont_tok"], dev(ctx.astype(np.uint16)), c=p["c"],
                          alpha=(1,))
    torch.cuda.synchronize()
    got = {f: host(v) for f, v in r.items()}
    got.update({f: host(v) for f, v in tr.items()})
    same(got, 0, 300)


def test_targets_from_truth_edges():
    """fc_targets_from_truth against its definition: a stream map that
    permutes and repeats streams, starts at the stream's last token (every
    deeper row falls past the end), at 0, in the middle, and malformed trees
    (num_nodes -1) whose rows all read -1."""
    t = synth.store(1, "single")
    ctx = synth.queries(1)[:24]
    st = gpu_store(t)
    g = gpu_pipeline([st], ctx, P, (1,), 16)
    num_nodes = g["num_nodes"].copy()
    num_nodes[5] = -1
    truth = synth.truth(n_seq=6, length=300)
    rng = np.random.default_rng(9)
    seq = rng.integers(0, truth.shape[0], size=ctx.shape[0]).astype(np.int32)
    start = rng.integers(0, 300, size=ctx.shape[0]).astype(np.int32)
    start[:4] = (299, 298, 0, 150)
    tree = {"num_nodes": dev(num_nodes), "pos_ids": dev(g["pos_ids"]), "node_tok": dev(g["node_tok"])}
    got = host(fc.fc_targets_from_truth(dev(truth), dev(start), tree, seq=dev(seq)))
    want = targets_from_truth(g["pos_ids"], num_nodes, truth[seq], start)
    assert (got == want).all()
    assert (got[5] == -1).all() and (got[0, 1:] == -1).all()


def _decoy_trees(rng, B: int, R: int, m: int) -> tuple:
    """Random trees (depth <= m, distinct sibling tokens) whose rows at and
    past num_nodes are decoys: each hangs under a live row u and carries a
    fresh token that is also u's target, so a walk that reads a row past
    the node count would step into it.  Node counts include 0, 1 and R."""
    nn = rng.integers(0, R + 1, size=B).astype(np.int32)
    nn[:4] = (0, 1, 2, R)
    tok = np.full((B, R), 7, np.int32)
    par = np.full((B, R), -1, np.int32)
    pos = np.zeros((B, R), np.int32)
    tgt = rng.integers(-1, 50, size=(B, R)).astype(np.int32)
    for b in range(B):
        n = max(int(nn[b]), 1)
        used = {}
        for v in range(1, n):
            u = int(rng.integers(0, v))
            while pos[b, u] >= m:
                u = int(par[b, u])
            t = int(rng.integers(0, 12))
            while t in used.setdefault(u, set()):
                t += 1
            used[u].add(t)
            par[b, v], tok[b, v], pos[b, v] = u, t, pos[b, u] + 1
            if rng.random() < 0.7:  # follow this child from u
                tgt[b, u] = t
        for v in range(n, R):
            u = int(rng.integers(0, n))
            fresh = 1000 + v
            par[b, v], tok[b, v], pos[b, v] = u, fresh, pos[b, u] + 1
            tgt[b, u] = fresh if rng.random() < 0.5 else tgt[b, u]
    return nn, tok, par, pos, tgt


@pytest.mark.parametrize("m", [3, 10])
def test_accept_ignores_rows_past_the_node_count(m):
    """fc_verify_accept against the oracle on trees whose rows past
    num_nodes (0, 1, 2, R and random counts) hold decoys that match the
    targets: only live rows may be walked."""
    rng = np.random.default_rng(40 + m)
    B, R = 96, 65
    nn, tok, par, pos, tgt = _decoy_trees(rng, B, R, m)
    tree = {"num_nodes": dev(nn), "node_tok": dev(tok), "parent": dev(par), "pos_ids": dev(pos)}
    got = fc.fc_verify_accept(tree, dev(tgt), m=m)
    torch.cuda.synchronize()
    want = oracle.verify_accept(dict(num_nodes=nn, node_tok=tok, parent=par, pos_ids=pos), tgt, m=m)
    for f in ("accept_len", "accept_tok", "last_node"):
        assert (host(got[f]) == want[f]).all(), f
    assert (want["last_node"] < np.maximum(nn, 1)).all()


@pytest.mark.parametrize("extra", [0, 1, 5])
def test_accept_on_trees_deeper_than_m(extra):
    """Chains of depth m + extra (a built tree is at most m deep) whose
    targets follow them: the walk stops at m + 1 accepted tokens on both
    sides and nothing is written past accept_tok's m + 1 entries."""
    m, R = 4, 16
    depth = m + extra
    B = 3
    nn = np.full(B, depth + 1, np.int32)
    tok = np.zeros((B, R), np.int32)
    par = np.full((B, R), -1, np.int32)
    pos = np.zeros((B, R), np.int32)
    tok[:, :depth + 1] = np.arange(10, 11 + depth)
    par[:, 1:depth + 1] = np.arange(depth)
    pos[:, :depth + 1] = np.arange(depth + 1)
    tgt = np.full((B, R), -1, np.int32)
    tgt[:, :depth] = np.arange(11, 11 + depth)
    tgt[:, depth] = 99
    tgt[1, 2] = 5  # the second tree stops at depth 2
    tree = {"num_nodes": dev(nn), "node_tok": dev(tok), "parent": dev(par), "pos_ids": dev(pos)}
    got = fc.fc_verify_accept(tree, dev(tgt), m=m)
    torch.cuda.synchronize()
    want = oracle.verify_accept(dict(num_nodes=nn, node_tok=tok, parent=par, pos_ids=pos), tgt, m=m)
    for f in ("accept_len", "accept_tok", "last_node"):
        assert (host(got[f]) == want[f]).all(), f
    assert want["accept_len"].tolist() == [min(depth + 1, m + 1), 3, min(depth + 1, m + 1)]


def test_unsorted_slots_are_flagged():
    """A query whose store slots are out of order gets num_nodes = -1 and
    padding rows; the other queries are unaffected."""
    taken = np.array([[3], [2]], np.int32)
    lens = np.array([[1, 1, 1], [2, 1, 0]], np.uint8)
    toks = np.array([[[5, 0], [4, 0], [6, 0]], [[1, 2], [3, 0], [0, 0]]], np.uint16)
    ctx = np.array([[9, 9], [8, 8]], np.uint16)
    t = fc.fc_build_tree(dev(taken), dev(lens), dev(toks), dev(ctx), c=4, alpha=(1,))
    torch.cuda.synchronize()
    assert host(t["num_nodes"]).tolist() == [-1, 4]
    assert (host(t["mask"])[0] == 0).all() and (host(t["parent"])[0] == -1).all()
    o = oracle.build_tree(taken[1:], lens[1:], toks[1:], ctx[1:], c=4, alpha=(1,))
    for f in ("node_tok", "parent", "weight", "pos_ids", "mask"):
        assert (host(t[f])[1] == o[f][0]).all()


def _sorted_slots(rng, T: int, m: int, vocab: int) -> tuple:
    """T continuations of lengths 0..m over a small vocabulary (long shared
    prefixes), in the order a store hands them over: lexicographic, a
    prefix before its extensions."""
    rows = []
    for _ in range(T):
        n = m if rng.random() < 0.7 else int(rng.integers(0, m + 1))
        rows.append(tuple(int(x) for x in rng.integers(1, vocab + 1, size=n)))
    rows.sort()
    lens = np.array([len(r) for r in rows], np.uint8)
    toks = np.zeros((T, m), np.uint16)
    for i, r in enumerate(rows):
        toks[i, :len(r)] = r
    return lens, toks


def _largest_k(m: int, S: int, alpha) -> int:
    """The largest k whose LDS layouts the tree kernels accept for m, S
    stores and these store weights (found through the entry point itself:
    past it the call is refused before any launch)."""
    def ok(k):
        taken = dev(np.zeros((1, S), np.int32))
        try:
            fc.fc_build_tree(taken, dev(np.zeros((1, k), np.uint8)), dev(np.zeros((1, k, m), np.uint16)),
                             dev(np.ones((1, 2), np.uint16)), c=4, alpha=alpha)
            return True
        except fc.FcError as e:
            assert "UNSUPPORTED" in str(e), e
            return False
    lo, hi = 1, 65535
    assert ok(lo)
    while lo < hi:
        mid = (lo + hi + 1) // 2
        if ok(mid):
            lo = mid
        else:
            hi = mid - 1
    return lo


@pytest.mark.parametrize("m", [2, 10, 255])
def test_tree_at_maximum_sizes(m):
    """c = 255 (256 rows: four row groups), k at the largest LDS layout the
    kernels take for m and two stores (about 12,000 slots; for m = 2 the
    one-workgroup layout cannot hold half of them as short strings, so the
    evenly split queries go to the full-LDS kernel through its list; m = 255
    is the general kernel), with unequal weights and with equal ones (unequal
    weights need a larger layout, so k is the largest they take); k + 1 is
    refused."""
    torch.cuda.synchronize()
    c, S, B = 255, 2, 5
    k = _largest_k(m, S, (3, 1))
    say(f"tree maximum sizes m={m}: k={k}")
    assert k >= 200
    rng = np.random.default_rng(m)
    totals = [k, k - 1, min(k, 300), min(k, 257), 2]
    taken = np.zeros((B, S), np.int32)
    lens = np.zeros((B, k), np.uint8)
    toks = np.zeros((B, k, m), np.uint16)
    for b, T in enumerate(totals):
        t0 = int(rng.integers(0, T + 1)) if b % 2 else T // 2
        taken[b] = (t0, T - t0)
        at = 0
        for s in range(S):
            ln, tk = _sorted_slots(rng, int(taken[b, s]), m, 3 if b < 2 else 5)
            lens[b, at:at + len(ln)] = ln
            toks[b, at:at + len(ln)] = tk
            at += len(ln)
    ctx = rng.integers(1, 6, size=(B, 4)).astype(np.uint16)
    for alpha in ((1, 1), (3, 1)):
        t = fc.fc_build_tree(dev(taken), dev(lens), dev(toks), dev(ctx), c=c, alpha=alpha)
        torch.cuda.synchronize()
        o = oracle.build_tree(taken, lens, toks, ctx, c=c, alpha=alpha)
        compare_tree({f: host(v) for f, v in t.items()}, o)
        if m >= 10:
            assert (o["num_nodes"][:2] == c + 1).all()
    with pytest.raises(fc.FcError):
        fc.fc_build_tree(dev(np.zeros((1, S), np.int32)), dev(np.zeros((1, k + 1), np.uint8)),
                         dev(np.zeros((1, k + 1, m), np.uint16)), dev(np.ones((1, 2), np.uint16)), c=c, alpha=(3, 1))


def test_repeat_runs_are_identical():
    """Same call twice gives the same bytes (no order-dependent races)."""
    t = synth.store(1, "single")
    ctx = synth.queries(1)
    st = gpu_store(t)
    a = gpu_pipeline([st], ctx, P, (1,), P["c"])
    b = gpu_pipeline([st], ctx, P, (1,), P["c"])
    for f in ("match_n", "range_lo", "range_cnt", "taken", "num_nodes", "node_tok", "parent", "weight", "mask"):
        assert (a[f] == b[f]).all(), f
    sa2 = host(fc.fc_datastore_build(dev(t)))
    assert (sa2 == host(st.sa)).all()


# ------------------------------------------------------------------- CACHE --

def _cache_texts(seed: int, n_texts: int, vocab: int, max_len: int) -> list:
    """Texts shaped like CACHE contents: short sequences of a small
    vocabulary (long repeats, many ties) joined by single 0 tokens."""
    rng = np.random.default_rng(seed)
    out = []
    for t in range(n_texts):
        target = int(rng.integers(0, max_len + 1))
        toks = []
        while len(toks) < target:
            n = int(rng.integers(3, 30))
            seq = synth.random_text(1000 * seed + 17 * t + len(toks), n, vocab).tolist()
            toks += ([0] if toks else []) + seq
        out.append(np.array(toks[:target], np.uint16))
    return out


def test_cache_retrieve_matches_oracle():
    """fc_cache_retrieve equals the oracle's retrieval over a one-store
    datastore holding each CACHE text, field by field: empty texts, texts at
    the 16,384-token limit, more occurrences than k (strided), short and
    long contexts, a text row map and an output row map."""
    stride = fc.FC_MAX_CACHE_TOKENS
    for seed, (vocab, max_len, k, m, n_max, n_min) in enumerate([
            (4, 400, 30, 4, 16, 2), (9, 3000, 5000, 10, 16, 2), (3, stride, 200, 10, 16, 2),
            (50, stride, 5000, 16, 8, 1), (6, 800, 7, 3, 5, 3), (7, 5000, 5000, 10, 16, 2)]):
        texts = _cache_texts(seed, 6, vocab, max_len)
        if seed == 0:
            texts[0] = np.zeros(0, np.uint16)
        if seed == 2:
            texts[1] = np.resize(synth.random_text(5, 50, vocab), stride).astype(np.uint16)  # full and periodic
        if seed == 5:
            # periodic texts whose patterns occur ~40 and ~80 times (the ranked
            # tiers above 32 occurrences), one with sparse noise so that the
            # occurrences' suffixes part at varied depths
            rng5 = np.random.default_rng(55)
            texts[0] = np.resize(synth.random_text(50, 60, vocab), 5000).astype(np.uint16)
            texts[1] = np.resize(synth.random_text(51, 120, vocab), 5000).astype(np.uint16)
            t2 = np.resize(synth.random_text(52, 70, vocab), 5600).astype(np.uint16)
            flip = rng5.random(len(t2)) < 0.003
            t2[flip] = rng5.integers(1, vocab, size=int(flip.sum()))
            texts[2] = t2
        buf = np.zeros((len(texts), stride), np.uint16)
        lens = np.zeros(len(texts), np.int32)
        for i, t in enumerate(texts):
            buf[i, :len(t)] = t
            lens[i] = len(t)
        rng = np.random.default_rng(100 + seed)
        B, Lq = 40, 16
        trow = rng.integers(0, len(texts), size=B).astype(np.int32)
        ctx = np.zeros((B, Lq), np.uint16)
        for b in range(B):
            t = texts[trow[b]]
            if len(t) > Lq and rng.random() < 0.8:
                j = int(rng.integers(0, len(t) - Lq))
                ctx[b] = t[j:j + Lq]
            else:
                ctx[b] = rng.integers(1, vocab, size=Lq)
        out_rows = rng.permutation(B + 5)[:B].astype(np.int32)  # results land in a larger buffer
        say(f"cache retrieve seed={seed} vocab={vocab} k={k} m={m} n={n_max}..{n_min}")
        out = fc.retrieve_outputs(B + 5, 1, k, m, torch.device("cuda"))
        fc.fc_cache_retrieve(dev(buf), dev(lens), dev(ctx), n_max=n_max, n_min=n_min, k=k, m=m,
                             text_row=dev(trow), out=out, rows=dev(out_rows))
        torch.cuda.synchronize()
        g = {f: host(v) for f, v in out.items()}
        for b in range(B):
            o = oracle.retrieve([texts[trow[b]]], ctx[b:b + 1], n_max=n_max, n_min=n_min, k=k, m=m)
            compare_retrieve(g, o, rows=[int(out_rows[b])])


@pytest.mark.parametrize("native", [True, False], ids=["engine", "driver"])
@pytest.mark.parametrize("cache_l,cap", [(50, fc.FC_MAX_CACHE_TOKENS), (4, 300)])
def test_replay_with_cache_matches_oracle(cache_l, cap, native):
    """Decode-trace replay with the CACHE branch of Alg. 1: every accepted
    length, final position, LRU count and CACHE-served count equal the
    oracle's; the small-cap case evicts and rewrites CACHE texts."""
    tp, t1 = synth.store(3, "project"), synth.store(1, "single")
    truth = synth.truth(n_seq=12, length=500)
    stores = [gpu_store(tp, synth.VOCAB, records=True), gpu_store(t1)]
    say(f"replay+cache l={cache_l} cap={cap}: gpu")
    g = GpuReplay(stores, truth, cache_l=cache_l, cache_cap=cap, **P).run(max_steps=400, native=native)
    say(f"replay+cache l={cache_l} cap={cap}: oracle")
    o = oracle.replay([tp, t1], truth, cache_l=cache_l, cache_cap=cap, **P, max_steps=400)
    for f in ("accept", "hits", "lookups", "pos", "cache_served"):
        assert (g[f] == o[f]).all(), f
    assert g["cache_served"].sum() > 0


def test_replay_cache_with_unequal_store_weights():
    """The engine builds a served stream's tree from its CACHE result as the
    first store's slots, weighted by that store's alpha (3 here) instead of
    1: the same nodes in the same order, so every accepted length and count
    still equals the oracle's."""
    tp, t1 = synth.store(3, "project"), synth.store(1, "single")
    truth = synth.truth(n_seq=8, length=400)
    stores = [gpu_store(tp, synth.VOCAB, records=True), gpu_store(t1)]
    kw = dict(P, alpha=(3, 1))
    say("replay+cache alpha=(3, 1): gpu")
    g = GpuReplay(stores, truth, cache_l=4, cache_cap=300, **kw).run(max_steps=300, native=True)
    say("replay+cache alpha=(3, 1): oracle")
    o = oracle.replay([tp, t1], truth, cache_l=4, cache_cap=300, **kw, max_steps=300)
    for f in ("accept", "hits", "lookups", "pos", "cache_served"):
        assert (g[f] == o[f]).all(), f
    assert g["cache_served"].sum() > 0


@pytest.mark.parametrize("native", [True, False], ids=["engine", "driver"])
@pytest.mark.parametrize("case", ["project-streams", "recurring-misses"])
def test_replay_with_retrieval_control_matches_oracle(case, native):
    """Alg. 1 in full (CACHE branch, missing table, skip gate with p = 0.5
    on the streams' most frequent token): every accepted length, position
    and branch count equal the oracle's.  The second case replays periodic
    streams over stores they rarely match, so failed contexts recur and the
    missing table bypasses them."""
    if case == "project-streams":
        texts = [synth.store(3, "project"), synth.store(1, "single")]
        truth = synth.truth(n_seq=12, length=500)
        stores = [gpu_store(texts[0], synth.VOCAB, records=True), gpu_store(texts[1])]
    else:
        texts = [synth.random_text(41, 200_000, synth.VOCAB, 0.01), synth.store(1, "single")]
        truth = np.stack([np.resize(synth.random_text(50 + i, 37, synth.VOCAB), 400) for i in range(8)])
        stores = [gpu_store(texts[0], synth.VOCAB, records=True), gpu_store(texts[1])]
    tok = int(np.bincount(truth.ravel()).argmax())
    draws = np.stack([synth.uniform(31, 30, step, truth.shape[0], 0, 2 ** 31 - 1) for step in range(400)])
    kw = dict(cache_l=50, missing=True, skip_tok=tok, skip_p=0.5, skip_draws=draws)
    say(f"replay+control {case}: gpu")
    g = GpuReplay(stores, truth, **kw, **P).run(max_steps=400, native=native)
    say(f"replay+control {case}: oracle")
    o = oracle.replay(texts, truth, **kw, **P, max_steps=400)
    for f in ("accept", "hits", "lookups", "pos", "cache_served", "missing_skips", "gate_skips"):
        assert (g[f] == o[f]).all(), f
    assert g["gate_skips"].sum() > 0
    if case == "recurring-misses":
        assert g["missing_skips"].sum() > 0


@pytest.mark.parametrize("mode", ["lru1", "tiny-cache", "cache0-control"])
def test_replay_engine_edge_cases(mode):
    """The device engine against the oracle replay on small-vocabulary
    stores and streams (long matches, many ties): an LRU of one slot, a
    40-token CACHE of 3-token chunks that evicts almost every step, and a
    CACHE searched from the first step (cache_l = 0, empty texts) with the
    missing table and the skip gate on."""
    texts = [synth.random_text(71, 3000, 6, 0.01), synth.random_text(72, 5000, 6, 0.01)]
    # random streams, one repeating a single token (the same context every
    # step: LRU hits), one of a token the stores lack (empty results: the
    # missing table), one of period 3
    truth = np.stack([synth.random_text(80 + i, 120, 6) for i in range(4)] +
                     [np.full(120, 3, np.uint16), np.full(120, 9, np.uint16),
                      np.resize(np.array([2, 4, 1], np.uint16), 120)])
    p = dict(n_max=8, n_min=1, k=40, m=4, c=12, alpha=(1, 2), ctx_len=8)
    kw = {"lru1": dict(lru=1),
          "tiny-cache": dict(lru=3, cache_l=2, cache_every=3, cache_cap=40),
          "cache0-control": dict(lru=3, cache_l=0, cache_every=5, cache_cap=200, missing=True,
                                 skip_tok=int(np.bincount(truth.ravel()).argmax()), skip_p=0.5,
                                 skip_draws=np.stack([synth.uniform(33, 30, st, truth.shape[0], 0, 2 ** 31 - 1)
                                                      for st in range(300)]))}[mode]
    say(f"replay engine edge case {mode}")
    g = GpuReplay([gpu_store(t) for t in texts], truth, **kw, **p).run(max_steps=300)
    o = oracle.replay(texts, truth, **kw, **p, max_steps=300)
    for f in ("accept", "hits", "lookups", "pos", "cache_served", "missing_skips", "gate_skips"):
        assert (g[f] == o[f]).all(), (mode, f)
    assert g["steps"] == o["accept"].shape[0]
    assert g["hits"].sum() > 0
    if mode == "cache0-control":
        assert g["missing_skips"].sum() > 0 and g["gate_skips"].sum() > 0


# ---------------------------------------------------------- tree attention --

def _bf16(rng, *shape, scale=1.0):
    return torch.from_numpy(rng.uniform(-scale, scale, size=shape)).to(torch.bfloat16)


def _attention_bound(q, kt, kc, vt, vc, P, tree, base):
    """Per-row error bound of the bf16 matrix-core evaluation against the
    exact result on the same inputs: rotated queries and keys are rounded to
    bf16 (relative 2^-9 each), so a score moves by at most
    2^-8 * sum_d |q_d k_d| / sqrt(D) (plus fp32 accumulation, < 1e-5); a
    softmax whose scores move by at most delta moves its weighted mean by at
    most 2*delta*max|v|; the bf16 weights in the value product add 2^-8 *
    max|v|."""
    B, R, H, D = q.shape
    Hkv = kt.shape[2]
    bound = np.zeros((B, R, H))
    for b in range(B):
        n = int(tree["num_nodes"][b])
        p = int(P[b])
        if n <= 0:
            continue
        pos = p + tree["pos_ids"][b][:n].astype(np.int64)
        for h in range(H):
            g = h // (H // Hkv)
            qh = np.abs(oracle.rope(q[b, :n, h], pos, base))
            keys = np.abs(np.concatenate([kc[b, :p, g], oracle.rope(kt[b, :n, g], pos, base)]))
            vmax = max(np.abs(vc[b, :p, g]).max() if p else 0.0, np.abs(vt[b, :n, g]).max())
            for i in range(n):
                allowed = np.concatenate([np.ones(p, bool), tree["mask"][b][i][:n] == 1])
                delta = 2.0 ** -8 * (keys[allowed] @ qh[i]).max() / np.sqrt(D) + 1e-5
                bound[b, i, h] = 2 * delta * vmax + 2.0 ** -8 * vmax + 1e-6
    return bound


def _tree_attention_case(trees: dict, rows, H, Hkv, P, Pmax, seed, base=10000.0, qscale=1.0):
    rng = np.random.default_rng(seed)
    B = len(rows)
    R = trees["mask"].shape[1]
    D = fc.FC_TREE_ATTN_HEAD_DIM
    tsub = {f: np.ascontiguousarray(trees[f][rows]) for f in ("num_nodes", "mask", "pos_ids")}
    q = _bf16(rng, B, R, H, D, scale=qscale)
    kt, vt = _bf16(rng, B, R, Hkv, D), _bf16(rng, B, R, Hkv, D)
    kc, vc = _bf16(rng, B, max(Pmax, 1), Hkv, D), _bf16(rng, B, max(Pmax, 1), Hkv, D)
    Pn = np.asarray(P, np.int32)
    g = fc.fc_tree_attention(q.cuda(), kt.cuda(), vt.cuda(), kc.cuda(), vc.cuda(), dev(Pn),
                             {f: dev(v) for f, v in tsub.items()}, rope_base=base)
    torch.cuda.synchronize()
    g = host(g).astype(np.float64)
    f64 = lambda t: t.float().numpy().astype(np.float64)  # noqa: E731
    o = oracle.tree_attention(f64(q), f64(kt), f64(vt), f64(kc), f64(vc), Pn, tsub["num_nodes"], tsub["mask"],
                              tsub["pos_ids"], rope_base=base)
    bound = _attention_bound(f64(q), f64(kt), f64(kc), f64(vt), f64(vc), Pn, tsub, base)
    err = np.abs(g - o).max(axis=3)
    assert (err <= bound).all(), (err.max(), float((err - bound).max()))
    for b in range(B):  # rows past the tree are exactly zero
        assert (g[b, max(int(tsub["num_nodes"][b]), 0):] == 0).all()
    return err, bound


def test_tree_attention_matches_oracle():
    """Tree attention on real draft trees (the 1M-token workload's batch):
    prefixes of 0 to 300 cached tokens across block edges, multi-head and
    grouped heads, every output within the derived bf16 bound of the exact
    result, rows past the tree zero."""
    t = synth.store(1, "single")
    ctx = synth.queries(1)
    st = gpu_store(t)
    for c in (64, 8, 200):  # 200: the 1024-thread instance (more than 128 rows)
        g = gpu_pipeline([st], ctx, P, (1,), c)
        trees = {f: g[f] for f in ("num_nodes", "mask", "pos_ids")}
        for (B, H, Hkv, seed) in ((16, 4, 4, 1), (16, 4, 2, 2), (3, 3, 1, 3)):
            rows = list(range(3 * seed, 3 * seed + B))
            P_ = [(0, 1, 31, 32, 33, 100, 300)[i % 7] for i in range(B)]
            say(f"tree attention c={c} B={B} H={H} Hkv={Hkv}")
            err, bound = _tree_attention_case(trees, rows, H, Hkv, P_, 320, seed)
            assert err.mean() < 0.25 * bound.mean()  # typical error well inside the bound


def test_tree_attention_masks_and_edge_cases():
    """No prefix and sharp scores, so every row attends to a handful of its
    ancestors and a wrong mask entry would move it far outside the bound; a
    malformed tree (num_nodes = -1) gives zeros; large positions."""
    t = synth.store(1, "single")
    ctx = synth.queries(1)
    g = gpu_pipeline([gpu_store(t)], ctx, P, (1,), 64)
    trees = {f: g[f].copy() for f in ("num_nodes", "mask", "pos_ids")}
    trees["num_nodes"][5] = -1
    err, bound = _tree_attention_case(trees, list(range(0, 24)), 2, 2, [0] * 24, 0, 11, qscale=3.0)
    assert (err[5] == 0).all()
    err, bound = _tree_attention_case(trees, list(range(24, 32)), 2, 1, [4000] * 8, 4000, 12, base=1e6)
