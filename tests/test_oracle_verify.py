"""Pins for the oracle's acceptance rule (Section IV-D): brute-force path
enumeration and the worked examples."""
import numpy as np
import pytest

import brute
import oracle


def _random_tree(rng, c, vocab):
    taken = np.array([[int(rng.integers(0, 30))]], np.int32)
    k, m = 30, 4
    lens = np.zeros((1, k), np.uint8)
    toks = np.zeros((1, k, m), np.uint16)
    for i in range(int(taken[0, 0])):
        ln = int(rng.integers(0, m + 1))
        lens[0, i] = ln
        toks[0, i, :ln] = rng.integers(1, vocab, size=ln)
    return oracle.build_tree(taken, lens, toks, np.array([[7]], np.uint16), c=c, alpha=(1,)), m


@pytest.mark.parametrize("seed", range(30))
def test_accept_vs_enumeration(seed):
    rng = np.random.default_rng(seed)
    c = int(rng.integers(1, 20))
    tree, m = _random_tree(rng, c, 3)
    n = int(tree["num_nodes"][0])
    rows = [(int(tree["node_tok"][0, i]), int(tree["parent"][0, i])) for i in range(n)]
    for _ in range(10):
        target = rng.integers(-1, 3, size=(1, c + 1)).astype(np.int32)
        # bias towards following the tree
        for i in range(n):
            kids = [v for v in range(n) if rows[v][1] == i]
            if kids and rng.random() < 0.7:
                target[0, i] = rows[kids[int(rng.integers(0, len(kids)))]][0]
        got = oracle.verify_accept(tree, target, m=m)
        ln, toks, u = brute.accept(rows, target[0].tolist())
        assert got["accept_len"][0] == ln
        assert got["last_node"][0] == u
        assert got["accept_tok"][0, :ln].tolist() == toks
        assert (got["accept_tok"][0, ln:] == -1).all()
        assert 0 <= ln <= m + 1


def test_examples(golden):
    g = golden("example_a.json")
    tr = {f: np.array([v]) for f, v in g["tree_k3_c2"].items()}
    tr["num_nodes"] = np.array([g["tree_k3_c2"]["num_nodes"]])
    for case in g["accept_c2"]:
        got = oracle.verify_accept(tr, np.array([case["target"]], np.int32), m=2)
        assert got["accept_len"][0] == case["accept_len"]
        assert got["accept_tok"][0].tolist() == case["accept_tok"]
        assert got["last_node"][0] == case["last_node"]
    gb = golden("example_b.json")
    tr = {f: np.array([v]) for f, v in gb["tree"].items()}
    tr["num_nodes"] = np.array([gb["tree"]["num_nodes"]])
    a = gb["accept"]
    got = oracle.verify_accept(tr, np.array([a["target"]], np.int32), m=2)
    assert got["accept_len"][0] == a["accept_len"]
    assert got["accept_tok"][0].tolist() == a["accept_tok"]
    assert got["last_node"][0] == a["last_node"]


def test_root_only_and_exhausted_truth():
    tr = dict(num_nodes=np.array([1]), node_tok=np.array([[5, 0, 0]]), parent=np.array([[-1, -1, -1]]),
              pos_ids=np.zeros((1, 3), np.int32))
    got = oracle.verify_accept(tr, np.array([[9, -1, -1]], np.int32), m=2)
    assert got["accept_len"][0] == 1 and got["accept_tok"][0].tolist() == [9, -1, -1]
    got = oracle.verify_accept(tr, np.array([[-1, -1, -1]], np.int32), m=2)
    assert got["accept_len"][0] == 0 and got["last_node"][0] == 0


@pytest.mark.parametrize("extra", [0, 1, 3])
def test_tree_deeper_than_m_stops_at_m_plus_one(extra):
    """A chain of depth m + extra whose every edge matches: the walk takes
    m + 1 tokens at most and writes nothing past accept_tok's m + 1 slots
    (a chain of depth m, extra = 0, is the deepest a built tree can be)."""
    m = 4
    depth = m + extra
    R = depth + 1
    tr = dict(num_nodes=np.array([R, R]), node_tok=np.tile(np.arange(10, 10 + R, dtype=np.int32), (2, 1)),
              parent=np.tile(np.arange(-1, R - 1, dtype=np.int32), (2, 1)),
              pos_ids=np.tile(np.arange(R, dtype=np.int32), (2, 1)))
    target = np.tile(np.concatenate([np.arange(11, 10 + R, dtype=np.int32), [99]]), (2, 1))
    got = oracle.verify_accept(tr, target, m=m)
    want_path = min(depth, m + 1)
    want_len = min(depth + 1, m + 1)
    assert (got["accept_len"] == want_len).all()
    assert (got["last_node"] == want_path).all()
    toks = list(range(11, 11 + want_path)) + ([99] if depth < m + 1 else [])
    assert got["accept_tok"][0, :want_len].tolist() == toks[:want_len]
    assert (got["accept_tok"][:, want_len:] == -1).all()
