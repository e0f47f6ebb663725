"""Brute-force restatements of the method for tiny inputs (pure Python).

These pin the oracle from outside: each one computes the same result by a
different, naive route (materialised suffix lists, substring scans per n,
prefix counting in a dict, path enumeration), so a mistake in the oracle's
arithmetic shows up as a disagreement.  They are written from the paper's
definitions (Section III-A, Section IV-A, Section IV-C, Section IV-D) with the
readings the oracle documents.
"""
from __future__ import annotations


def suffix_array(text) -> list:
    """Sort start positions by the suffix as a Python list (lexicographic,
    a proper prefix first)."""
    t = [int(x) for x in text]
    return sorted(range(len(t)), key=lambda i: t[i:])


def query_limit(row, n_max: int) -> int:
    row = [int(x) for x in row]
    tail = 0
    for x in reversed(row):
        if x == 0:
            break
        tail += 1
    return min(n_max, len(row), tail)


def match(text, row, n_max: int, n_min: int):
    """(match_n, range_lo, occ in suffix order) by scanning every n."""
    t = [int(x) for x in text]
    r = [int(x) for x in row]
    hi = query_limit(r, n_max)
    for n in range(hi, n_min - 1, -1):
        q = r[len(r) - n:]
        occ = [j for j in range(len(t) - n + 1) if t[j:j + n] == q]
        if occ:
            order = suffix_array(t)
            occ_sorted = sorted(occ, key=lambda j: t[j:])
            lo = order.index(occ_sorted[0])
            assert order[lo:lo + len(occ)] == occ_sorted
            return n, lo, occ_sorted
    return 0, 0, []


def retrieve(texts, row, n_max: int, n_min: int, k: int, m: int) -> dict:
    """Per-query retrieval over prioritised stores, as flat Python lists."""
    out = dict(match_n=[], range_lo=[], range_cnt=[], taken=[], slots=[])
    used = 0
    for s, text in enumerate(texts):
        t = [int(x) for x in text]
        n, lo, occ = match(t, row, n_max, n_min)
        budget = k - used
        take = min(budget, len(occ))
        if len(occ) > budget:
            picks = [occ[(i * len(occ)) // budget] for i in range(budget)]
        else:
            picks = occ[:take]
        for j in picks:
            start = j + n
            cont = []
            while len(cont) < m and start + len(cont) < len(t) and t[start + len(cont)] != 0:
                cont.append(t[start + len(cont)])
            out["slots"].append((s, start, cont))
        out["match_n"].append(n)
        out["range_lo"].append(lo)
        out["range_cnt"].append(len(occ))
        out["taken"].append(take)
        used += take
    return out


def trie_weights(conts, alpha) -> dict:
    """{prefix tuple: weight} over (source, continuation) pairs (eq. (3))."""
    w = {}
    for s, cont in conts:
        for d in range(1, len(cont) + 1):
            p = tuple(cont[:d])
            w[p] = w.get(p, 0) + alpha[s]
    return w


def draft_tree(conts, alpha, c: int, root_token: int) -> dict:
    """Top-c prefixes by (weight desc, prefix asc), emitted in preorder."""
    w = trie_weights(conts, alpha)
    ranked = sorted(w, key=lambda p: (-w[p], p))
    chosen = sorted(ranked[:c])  # preorder of a trie = sorted prefixes
    index = {p: i + 1 for i, p in enumerate(chosen)}
    root_w = sum(alpha[s] for s, cont in conts if cont)
    rows = [(root_token, -1, root_w, 0)]
    for p in chosen:
        rows.append((p[-1], index[p[:-1]] if len(p) > 1 else 0, w[p], len(p)))
    return dict(rows=rows, chosen=chosen)


def accept(rows, target) -> tuple:
    """Longest root path whose every edge matches the parent's target, by
    enumerating all nodes; returns (accept_len, tokens, last_node)."""
    n = len(rows)
    best = (0, 0)  # (depth, node)
    for u in range(n):
        path = []
        v = u
        ok = True
        while v != 0:
            par = rows[v][1]
            if target[par] != rows[v][0]:
                ok = False
            path.append(rows[v][0])
            v = par
        if ok and (len(path), -u) > (best[0], -best[1]):
            best = (len(path), u)
    depth, u = best
    toks = []
    v = u
    while v != 0:
        toks.append(rows[v][0])
        v = rows[v][1]
    toks.reverse()
    if target[u] >= 0:
        toks.append(target[u])
    return len(toks), toks, u
