"""Pins for the oracle's weighted trie, top-c selection and emission
(Section IV-D, eq. (3)-(4)): brute-force prefix counting, trie invariants,
ancestor closure, slot-order independence and the worked examples."""
import numpy as np
import pytest

import brute
import oracle
import synth


def _random_slots(rng, S, k, m, vocab, fill=0.8):
    taken = np.zeros((1, S), np.int32)
    used = 0
    for s in range(S):
        t = int(rng.integers(0, int(k * fill / S) + 1))
        taken[0, s] = t
        used += t
    lens = np.zeros((1, k), np.uint8)
    toks = np.zeros((1, k, m), np.uint16)
    for i in range(used):
        ln = int(rng.integers(0, m + 1))
        lens[0, i] = ln
        toks[0, i, :ln] = rng.integers(1, vocab, size=ln)
    return taken, lens, toks


def _conts(taken, lens, toks):
    out = []
    slot = 0
    for s in range(taken.shape[1]):
        for _ in range(int(taken[0, s])):
            out.append((s, toks[0, slot, :lens[0, slot]].tolist()))
            slot += 1
    return out


def _check_vs_brute(taken, lens, toks, c, alpha, root_tok=7):
    ctx = np.array([[1, root_tok]], np.uint16)
    tr = oracle.build_tree(taken, lens, toks, ctx, c=c, alpha=alpha)
    want = brute.draft_tree(_conts(taken, lens, toks), alpha, c, root_tok)
    n = len(want["rows"])
    assert tr["num_nodes"][0] == n
    for i, (tok, par, w, pos) in enumerate(want["rows"]):
        assert (tr["node_tok"][0, i], tr["parent"][0, i], tr["weight"][0, i], tr["pos_ids"][0, i]) == \
            (tok, par, w, pos), i
    R = c + 1
    assert not tr["node_tok"][0, n:].any() and (tr["parent"][0, n:] == -1).all()
    assert not tr["weight"][0, n:].any() and not tr["pos_ids"][0, n:].any()
    mask = tr["mask"][0]
    for i in range(R):
        for j in range(R):
            anc = False
            if i < n:
                v = i
                while v >= 0:
                    if v == j:
                        anc = True
                    v = want["rows"][v][1]
            assert mask[i, j] == int(anc), (i, j)
    return tr


@pytest.mark.parametrize("seed", range(8))
@pytest.mark.parametrize("S", [1, 2])
def test_tree_vs_brute(seed, S):
    rng = np.random.default_rng(seed + 10 * S)
    vocab = [2, 3, 6, 50][seed % 4]
    taken, lens, toks = _random_slots(rng, S, 40, 5, vocab)
    alpha = (1, 1) if seed % 2 == 0 else (3, 2)
    for c in (1, 2, 5, 17, 64, 300):
        _check_vs_brute(taken, lens, toks, c, alpha[:S])


def test_invariants_full_trie():
    """With c above the node count the whole trie is emitted: check the
    weight identities of eq. (3)."""
    rng = np.random.default_rng(5)
    taken, lens, toks = _random_slots(rng, 2, 60, 6, 3)
    alpha = (2, 5)
    tr = oracle.build_tree(taken, lens, toks, np.array([[3]], np.uint16), c=500, alpha=alpha)
    n = int(tr["num_nodes"][0])
    par = tr["parent"][0, :n]
    w = tr["weight"][0, :n].astype(np.int64)
    pos = tr["pos_ids"][0, :n]
    conts = _conts(taken, lens, toks)
    # root weight = sum of alpha over non-empty continuations
    assert w[0] == sum(alpha[s] for s, cc in conts if cc)
    assert w[1:][par[1:] == 0].sum() == w[0]
    # weight(v) = children + alpha of continuations ending at v
    ends = {}
    for s, cc in conts:
        if cc:
            ends[tuple(cc)] = ends.get(tuple(cc), 0) + alpha[s]
    paths = {0: ()}
    for i in range(1, n):
        paths[i] = paths[par[i]] + (int(tr["node_tok"][0, i]),)
    for v in range(1, n):
        assert w[v] == w[1:][par[1:] == v].sum() + ends.get(paths[v], 0)
        assert w[v] <= w[par[v]]
        assert pos[v] == pos[par[v]] + 1
    assert w[1:].sum() == sum(alpha[s] * len(cc) for s, cc in conts)
    # number of non-root nodes = number of distinct non-empty prefixes
    assert n - 1 == len({tuple(cc[:d]) for _, cc in conts for d in range(1, len(cc) + 1)})


def test_ancestor_closed_and_preorder():
    rng = np.random.default_rng(11)
    taken, lens, toks = _random_slots(rng, 2, 80, 6, 4)
    for c in range(1, 40):
        tr = oracle.build_tree(taken, lens, toks, np.array([[3]], np.uint16), c=c, alpha=(1, 1))
        n = int(tr["num_nodes"][0])
        par = tr["parent"][0, :n]
        assert all(0 <= par[i] < i for i in range(1, n))  # parent emitted before child
        paths = [()]
        for i in range(1, n):
            paths.append(paths[par[i]] + (int(tr["node_tok"][0, i]),))
        assert paths[1:] == sorted(paths[1:])  # preorder = sorted paths
        # row sum of the mask = depth + 1
        assert (tr["mask"][0, :n].sum(axis=1) == tr["pos_ids"][0, :n] + 1).all()


def test_slot_order_does_not_matter():
    rng = np.random.default_rng(2)
    taken, lens, toks = _random_slots(rng, 2, 100, 5, 3)
    ctx = np.array([[9]], np.uint16)
    base = oracle.build_tree(taken, lens, toks, ctx, c=20, alpha=(2, 1))
    t0 = int(taken[0, 0])
    used = int(taken.sum())
    for rep in range(5):
        perm = np.concatenate([rng.permutation(t0), t0 + rng.permutation(used - t0),
                               np.arange(used, lens.shape[1])])
        tr = oracle.build_tree(taken, lens[:, perm], toks[:, perm], ctx, c=20, alpha=(2, 1))
        for f in base:
            assert (tr[f] == base[f]).all(), f


def test_ties_break_by_path():
    # three single-token continuations of equal weight: the smaller tokens win
    taken = np.array([[3]], np.int32)
    lens = np.array([[1, 1, 1]], np.uint8)
    toks = np.array([[[30], [10], [20]]], np.uint16)
    tr = oracle.build_tree(taken, lens, toks, np.array([[5]], np.uint16), c=2, alpha=(1,))
    assert tr["node_tok"][0].tolist() == [5, 10, 20]
    # a prefix beats its extension at equal weight
    taken = np.array([[1]], np.int32)
    lens = np.array([[3]], np.uint8)
    toks = np.array([[[4, 2, 9]]], np.uint16)
    tr = oracle.build_tree(taken, lens, toks, np.array([[5]], np.uint16), c=2, alpha=(1,))
    assert tr["node_tok"][0].tolist() == [5, 4, 2]


def test_empty_and_degenerate():
    taken = np.array([[2, 0]], np.int32)
    lens = np.zeros((1, 4), np.uint8)
    toks = np.zeros((1, 4, 3), np.uint16)
    tr = oracle.build_tree(taken, lens, toks, np.array([[8, 6]], np.uint16), c=4, alpha=(1, 1))
    assert tr["num_nodes"][0] == 1 and tr["node_tok"][0, 0] == 6 and tr["weight"][0, 0] == 0
    assert tr["mask"][0].sum() == 1


def test_examples(golden):
    g = golden("example_a.json")
    p = g["params"]
    t = np.array(g["text"], np.uint16)
    ctx = np.array([g["ctx"]], np.uint16)
    r = oracle.retrieve([t], ctx, n_max=p["n_max"], n_min=p["n_min"], k=3, m=p["m"])
    for c, key in ((2, "tree_k3_c2"), (3, "tree_k3_c3")):
        tr = oracle.build_tree(r["taken"], r["cont_len"], r["cont_tok"], ctx, c=c, alpha=(1,))
        for f, v in g[key].items():
            assert tr[f][0].tolist() == v, (key, f)
    gb = golden("example_b.json")
    p = gb["params"]
    ctx = np.array([gb["ctx"]], np.uint16)
    r = oracle.retrieve([np.array(gb["project"], np.uint16), np.array(gb["general"], np.uint16)], ctx,
                        n_max=p["n_max"], n_min=p["n_min"], k=p["k"], m=p["m"])
    tr = oracle.build_tree(r["taken"], r["cont_len"], r["cont_tok"], ctx, c=p["c"], alpha=(1, 1))
    for f, v in gb["tree"].items():
        assert tr[f][0].tolist() == v, f


def test_on_store_sample():
    """A batch of real-shaped queries through retrieve + tree, checked
    against the brute-force prefix count."""
    t = synth.store(1, "single")[:40_000]
    rng = np.random.default_rng(0)
    rows = [t[j:j + 16] for j in rng.integers(0, len(t) - 16, size=3)]
    ctx = np.stack(rows).astype(np.uint16)
    r = oracle.retrieve([t], ctx, n_max=16, n_min=2, k=200, m=10)
    for b in range(3):
        _check_vs_brute(r["taken"][b:b + 1], r["cont_len"][b:b + 1], r["cont_tok"][b:b + 1], 64, (1,),
                        root_tok=int(ctx[b, -1]))
