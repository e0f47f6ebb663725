"""Oracle for the draft-stage hot path (TEST INFRASTRUCTURE ONLY).

A plain CPU implementation, in C (fc_oracle.c, built with gcc), of what the
method computes: suffix array (Section III-A), suffix-match retrieval over
prioritised stores (Section III-A, Section IV-A, Section IV-C), weighted trie
and top-c draft tree with mask and position ids (Section IV-D, eq. (3)-(4)),
and greedy acceptance (Section IV-D).  Only the tests, the smoke check and the
benchmark's CPU baseline may import this package; the GPU library never does.

Every function takes and returns numpy arrays; the array layouts match the C
library's entry points so results compare element by element.
"""
from __future__ import annotations

import ctypes
import functools
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# FC_ORACLE_LIB names another build of fc_oracle.c to load (e.g. one built
# with -fsanitize=address,undefined for a checked run of the pins).
_LIB_PATH = os.environ.get("FC_ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")


def build() -> None:
    """Compile fc_oracle.c into liboracle.so (gcc, OpenMP over queries)."""
    tmp = _LIB_PATH + ".tmp"
    subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-o", tmp,
                           os.path.join(_HERE, "fc_oracle.c")])
    os.replace(tmp, _LIB_PATH)


@functools.lru_cache(maxsize=1)
def _lib():
    if not os.path.exists(_LIB_PATH):
        build()
    lib = ctypes.CDLL(_LIB_PATH)
    vp, u64, i32 = ctypes.c_void_p, ctypes.c_uint64, ctypes.c_int
    lib.oracle_suffix_cmp.restype = i32
    lib.oracle_suffix_cmp.argtypes = [vp, u64, u64, u64]
    lib.oracle_suffix_array.restype = None
    lib.oracle_suffix_array.argtypes = [vp, u64, vp]
    lib.oracle_check_sa.restype = i32
    lib.oracle_check_sa.argtypes = [vp, u64, vp, vp, ctypes.POINTER(ctypes.c_uint64)]
    lib.oracle_retrieve.restype = None
    lib.oracle_retrieve.argtypes = [i32, vp, vp, vp, i32, i32, i32, i32, i32, i32,
                                    vp, vp, vp, vp, vp, vp, vp, vp]
    lib.oracle_retrieve_batched.restype = None
    lib.oracle_retrieve_batched.argtypes = lib.oracle_retrieve.argtypes
    lib.oracle_build_tree.restype = None
    lib.oracle_build_tree.argtypes = [i32, i32, i32, i32, i32, vp, vp, vp, vp, vp, i32,
                                      vp, vp, vp, vp, vp, vp]
    lib.oracle_verify_accept.restype = None
    lib.oracle_verify_accept.argtypes = [i32, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp]
    lib.oracle_max_threads.restype = i32
    lib.oracle_max_threads.argtypes = []
    return lib


def _p(a: np.ndarray) -> ctypes.c_void_p:
    assert a.flags.c_contiguous
    return ctypes.c_void_p(a.ctypes.data)


def _u16(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.uint16)


def max_threads() -> int:
    """Threads the oracle's OpenMP loops use."""
    return int(_lib().oracle_max_threads())


def suffix_cmp(text, i: int, j: int) -> int:
    t = _u16(text)
    return int(_lib().oracle_suffix_cmp(_p(t), len(t), i, j))


def suffix_array(text) -> np.ndarray:
    """Suffix array of `text` by a plain comparison sort (uint32[N])."""
    t = _u16(text)
    sa = np.empty(max(len(t), 1), dtype=np.uint32)
    _lib().oracle_suffix_array(_p(t), len(t), _p(sa))
    return sa[:len(t)]


def check_sa(text, sa) -> tuple[int, int]:
    """Linear-time check; returns (code, index): code 0 valid, 1 not a
    permutation, 2 order violation at SA index `index`."""
    t = _u16(text)
    s = np.ascontiguousarray(sa, dtype=np.uint32)
    if len(s) != len(t):
        return 1, min(len(s), len(t))
    ws = np.empty(max(len(t), 1), dtype=np.uint32)
    where = ctypes.c_uint64(0)
    code = _lib().oracle_check_sa(_p(t), len(t), _p(s), _p(ws), ctypes.byref(where))
    return int(code), int(where.value)


def retrieve(texts, ctx, n_max: int = 16, n_min: int = 2, k: int = 5000, m: int = 10,
             batched: bool = False) -> dict:
    """Batched suffix-match retrieval over stores in priority order.

    texts: list of uint16 arrays (store 0 = repository store first);
    ctx: uint16 [B][L].  Returns dict of match_n, range_lo, range_cnt, taken
    ([B][S]) and cont_pos, cont_src, cont_len ([B][k]), cont_tok ([B][k][m]).

    batched=False runs the definition query by query (three scans of every
    store per query); batched=True computes the same result with each scan
    shared by the whole batch (one pass over a store per scan), which the
    tests pin against the per-query form.
    """
    ts = [_u16(t) for t in texts]
    S = len(ts)
    c = _u16(ctx)
    if c.ndim != 2:
        raise ValueError("ctx must be [B][L]")
    B, L = c.shape
    ptrs = (ctypes.c_void_p * S)(*[t.ctypes.data for t in ts])
    lens = np.array([len(t) for t in ts], dtype=np.uint64)
    out = dict(
        match_n=np.zeros((B, S), np.int32), range_lo=np.zeros((B, S), np.uint32),
        range_cnt=np.zeros((B, S), np.uint32), taken=np.zeros((B, S), np.int32),
        cont_pos=np.zeros((B, k), np.uint32), cont_src=np.zeros((B, k), np.uint8),
        cont_len=np.zeros((B, k), np.uint8), cont_tok=np.zeros((B, k, m), np.uint16))
    fn = _lib().oracle_retrieve_batched if batched else _lib().oracle_retrieve
    fn(S, ctypes.cast(ptrs, ctypes.c_void_p), _p(lens), _p(c), B, L, n_max, n_min, k, m,
       _p(out["match_n"]), _p(out["range_lo"]), _p(out["range_cnt"]), _p(out["taken"]),
       _p(out["cont_pos"]), _p(out["cont_src"]), _p(out["cont_len"]), _p(out["cont_tok"]))
    return out


def build_tree(taken, cont_len, cont_tok, ctx, c: int = 64, alpha=(1, 1)) -> dict:
    """Weighted trie -> top-c draft tree per query.

    taken [B][S], cont_len [B][k], cont_tok [B][k][m], ctx [B][L].  Returns
    num_nodes [B], node_tok, parent, pos_ids (int32) and weight (uint32)
    [B][c+1], mask int32 [B][c+1][c+1].
    """
    tk = np.ascontiguousarray(taken, dtype=np.int32)
    ln = np.ascontiguousarray(cont_len, dtype=np.uint8)
    tok = _u16(cont_tok)
    cx = _u16(ctx)
    B, S = tk.shape
    k, m = tok.shape[1], tok.shape[2]
    L = cx.shape[1]
    a = np.ascontiguousarray(list(alpha)[:S], dtype=np.uint32)
    if len(a) != S:
        raise ValueError("need one alpha per store")
    R = c + 1
    out = dict(num_nodes=np.zeros(B, np.int32), node_tok=np.zeros((B, R), np.int32),
               parent=np.zeros((B, R), np.int32), weight=np.zeros((B, R), np.uint32),
               pos_ids=np.zeros((B, R), np.int32), mask=np.zeros((B, R, R), np.int32))
    _lib().oracle_build_tree(B, S, k, m, c, _p(a), _p(tk), _p(ln), _p(tok), _p(cx), L,
                             _p(out["num_nodes"]), _p(out["node_tok"]), _p(out["parent"]), _p(out["weight"]),
                             _p(out["pos_ids"]), _p(out["mask"]))
    return out


def verify_accept(tree: dict, target, m: int = 10) -> dict:
    """Greedy acceptance of a draft tree against per-row target tokens.

    tree: output of build_tree; target int32 [B][c+1] (-1 = none).  Returns
    accept_len [B], accept_tok [B][m+1], last_node [B].
    """
    nn = np.ascontiguousarray(tree["num_nodes"], dtype=np.int32)
    tok = np.ascontiguousarray(tree["node_tok"], dtype=np.int32)
    par = np.ascontiguousarray(tree["parent"], dtype=np.int32)
    pos = np.ascontiguousarray(tree["pos_ids"], dtype=np.int32)
    tg = np.ascontiguousarray(target, dtype=np.int32)
    B, R = tok.shape
    out = dict(accept_len=np.zeros(B, np.int32), accept_tok=np.zeros((B, m + 1), np.int32),
               last_node=np.zeros(B, np.int32))
    _lib().oracle_verify_accept(B, R - 1, m, _p(nn), _p(tok), _p(par), _p(pos), _p(tg),
                                _p(out["accept_len"]), _p(out["accept_tok"]), _p(out["last_node"]))
    return out


class Cache:
    """The context- and LLM preference-aware CACHE of one stream (Section
    IV-B), as the oracle keeps it.

    It holds token sequences; `size` is their number.  Its text, the
    sequences joined by single 0 tokens (the separator of a datastore), is
    searched exactly like a store (Section III-A).  Reading for a bounded
    device buffer: when adding a sequence would make the text longer than
    `cap` tokens, the oldest sequences are dropped first (a sequence longer
    than `cap` on its own is cut to its last `cap` tokens).
    """

    def __init__(self, cap: int):
        self.cap = cap
        self.seqs = []

    @property
    def size(self) -> int:
        return len(self.seqs)

    def text_len(self) -> int:
        return sum(len(x) for x in self.seqs) + max(len(self.seqs) - 1, 0)

    def add(self, seq) -> None:
        seq = [int(x) for x in seq][-self.cap:]
        if not seq:
            return
        self.seqs.append(seq)
        while self.text_len() > self.cap:
            self.seqs.pop(0)

    def text(self) -> np.ndarray:
        out = []
        for i, x in enumerate(self.seqs):
            if i:
                out.append(0)
            out.extend(x)
        return np.array(out, dtype=np.uint16)


def replay(texts, truth, n_max: int = 16, n_min: int = 2, k: int = 5000, m: int = 10, c: int = 64, alpha=(1, 1),
           lru: int = 32, ctx_len: int = 16, max_steps: int = 512, cache_l: int | None = None,
           cache_every: int = 20, cache_cap: int = 16384, missing: bool = False, skip_tok: int | None = None,
           skip_p: float = 0.5, skip_draws=None) -> dict:
    """Decode-trace replay over known streams (reading of the average
    acceptance length setting, Section V-C eq. (7)).

    Every stream starts with its first ctx_len tokens as context at position
    p = ctx_len.  Each step, for every stream with p below its length: the
    key is the last ctx_len tokens; an LRU of `lru` entries per stream maps
    keys to stored retrieval results (a hit reuses the result and becomes most
    recent; a miss retrieves, inserts as most recent and drops the least
    recent beyond `lru`); the draft tree is built; the target after tree row
    i is truth[p + pos_ids[i]] (-1 past the stream); the accepted length is
    added to p.

    With cache_l set, each stream also keeps the CACHE of Section IV-B and
    follows the cache branch of Alg. 1:
      - when the CACHE holds at least cache_l sequences (Alg. 1's test; the
        prose says "exceeds", read as the listing's >=), the context is first
        searched in the CACHE's text as a single store; a non-empty result is
        the retrieval result R and the datastores are not consulted;
      - otherwise (or on an empty CACHE result) the datastores are searched
        as above (through the LRU);
      - after verification, when R is non-empty and at least one draft token
        was accepted, the context followed by the accepted draft tokens is
        added to the CACHE (the verified retrieved sequence);
      - the stream's output (every token accepted from p = ctx_len on,
        bonus tokens included) is added in consecutive chunks of
        cache_every tokens, each when it completes (the LLM output
        truncated every 20 tokens, Section V-D).
    The CACHE's trie uses weight 1 (one source).

    Alg. 1's retrieval-timing control, for a context that the CACHE did not
    serve:
      - missing=True keeps a missing table M per stream: a context whose
        datastore retrieval found no occurrence in any store is added to M
        (the prose's reading: only an actual, empty retrieval adds), and a
        context found in M later is not retrieved at all;
      - skip_tok set enables the skip gate: when the context ends with
        skip_tok, the datastores are searched only when the step's draw
        skip_draws[step][stream] (uniform integers in [0, 2^31)) is below
        skip_p * 2^31;
      - a context that is not retrieved gets an empty R: a bare root, so the
        step accepts the target model's own token only.

    Returns accept [steps][n_streams] (-1 for finished streams), hits and
    lookups of the LRU per stream, cache_served (steps whose R came from the
    CACHE), missing_skips and gate_skips (contexts not retrieved because of
    M or of the gate) per stream, final positions, the mean accepted length
    per live step, and the step count.
    """
    from collections import OrderedDict

    truth = np.ascontiguousarray(truth, dtype=np.uint16)
    nseq, tlen = truth.shape
    pos = [ctx_len] * nseq
    caches = [OrderedDict() for _ in range(nseq)]
    hits = [0] * nseq
    lookups = [0] * nseq
    served = [0] * nseq
    m_skips = [0] * nseq
    g_skips = [0] * nseq
    mtab = [set() for _ in range(nseq)]
    cch = [Cache(cache_cap) for _ in range(nseq)] if cache_l is not None else None
    chunks_done = [0] * nseq
    fields = ("taken", "cont_len", "cont_tok")
    steps = []
    for step in range(max_steps):
        act = [b for b in range(nseq) if pos[b] < tlen]
        if not act:
            break
        ctx = np.stack([truth[b, pos[b] - ctx_len:pos[b]] for b in act])
        got = [None] * len(act)
        from_cache = [False] * len(act)
        if cch is not None:
            for j, b in enumerate(act):
                if cch[b].size >= cache_l:
                    r = retrieve([cch[b].text()], ctx[j:j + 1], n_max=n_max, n_min=n_min, k=k, m=m)
                    if int(r["taken"][0].sum()) > 0:
                        got[j] = {f: r[f][0].copy() for f in fields}
                        from_cache[j] = True
                        served[b] += 1
        need = []
        empty = {"taken": np.zeros(len(texts), np.int32), "cont_len": np.zeros(k, np.uint8),
                 "cont_tok": np.zeros((k, m), np.uint16)}
        for j in range(len(act)):
            if got[j] is not None:
                continue
            b = act[j]
            if missing and ctx[j].tobytes() in mtab[b]:
                got[j] = empty
                m_skips[b] += 1
            elif (skip_tok is not None and int(ctx[j][-1]) == skip_tok
                  and not int(skip_draws[step][b]) < int(skip_p * 2 ** 31)):
                got[j] = empty
                g_skips[b] += 1
            else:
                need.append(j)
        keys = {j: ctx[j].tobytes() for j in need}
        misses = []
        for j in need:
            b = act[j]
            lookups[b] += 1
            if keys[j] in caches[b]:
                caches[b].move_to_end(keys[j])
                hits[b] += 1
            else:
                misses.append(j)
        if misses:
            r = retrieve(texts, ctx[misses], n_max=n_max, n_min=n_min, k=k, m=m, batched=True)
            for i, j in enumerate(misses):
                b = act[j]
                if len(caches[b]) >= lru:
                    caches[b].popitem(last=False)
                caches[b][keys[j]] = {f: r[f][i].copy() for f in fields}
        for j in need:
            got[j] = caches[act[j]][keys[j]]
            if missing and int(np.asarray(got[j]["taken"]).sum()) == 0:
                mtab[act[j]].add(keys[j])
        acc = np.zeros(len(act), np.int64)
        depth = np.zeros(len(act), np.int64)
        for group, al in ((True, (1,)), (False, tuple(alpha))):
            idx = [j for j in range(len(act)) if from_cache[j] == group]
            if not idx:
                continue
            tree = build_tree(np.stack([got[j]["taken"] for j in idx]), np.stack([got[j]["cont_len"] for j in idx]),
                              np.stack([got[j]["cont_tok"] for j in idx]), ctx[idx], c=c, alpha=al)
            target = np.full(tree["node_tok"].shape, -1, np.int32)
            for i, j in enumerate(idx):
                b = act[j]
                for r_ in range(int(tree["num_nodes"][i])):
                    at = pos[b] + int(tree["pos_ids"][i, r_])
                    if at < tlen:
                        target[i, r_] = int(truth[b, at])
            va = verify_accept(tree, target, m=m)
            for i, j in enumerate(idx):
                acc[j] = int(va["accept_len"][i])
                depth[j] = int(tree["pos_ids"][i, int(va["last_node"][i])])
        row = np.full(nseq, -1, np.int64)
        for j, b in enumerate(act):
            if cch is not None:
                if int(np.asarray(got[j]["taken"]).sum()) > 0 and depth[j] >= 1:
                    cch[b].add(list(ctx[j]) + list(truth[b, pos[b]:pos[b] + depth[j]]))
            row[b] = int(acc[j])
            pos[b] += int(acc[j])
            if cch is not None:
                while ctx_len + cache_every * (chunks_done[b] + 1) <= min(pos[b], tlen):
                    lo = ctx_len + cache_every * chunks_done[b]
                    cch[b].add(list(truth[b, lo:lo + cache_every]))
                    chunks_done[b] += 1
        steps.append(row)
    accept = np.stack(steps) if steps else np.zeros((0, nseq), np.int64)
    live = accept >= 0
    return dict(accept=accept, hits=np.array(hits), lookups=np.array(lookups), pos=np.array(pos),
                cache_served=np.array(served), missing_skips=np.array(m_skips), gate_skips=np.array(g_skips),
                acc_len=float(accept[live].sum() / max(live.sum(), 1)), steps=len(steps))


def rope(x: np.ndarray, positions: np.ndarray, base: float) -> np.ndarray:
    """Rotary position embedding, rotate-half form: for d < D/2 the pair
    (x_d, x_{d+D/2}) is rotated by the angle position * base^(-2d/D).
    x [..., n, D] (float64), positions [n]."""
    x = np.asarray(x, dtype=np.float64)
    D = x.shape[-1]
    half = D // 2
    inv = base ** (-2.0 * np.arange(half) / D)
    ang = np.asarray(positions, dtype=np.float64)[:, None] * inv[None, :]
    c, s = np.cos(ang), np.sin(ang)
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def tree_attention(q, k_tree, v_tree, k_cache, v_cache, prefix_len, num_nodes, mask, pos_ids,
                   rope_base: float = 10000.0) -> np.ndarray:
    """Attention of a draft tree's rows in one target-model forward (Section
    IV-D, eq. (4)): row i of tree b sits at position prefix_len[b] +
    pos_ids[b][i] (the root, depth 0, right after the cached prefix) and
    attends to every cached prefix token and to the tree rows j with
    mask[b][i][j] = 1.  Queries and tree keys are rotated by their
    positions (rotary embedding, rotate-half form); cached keys are stored
    rotated.  Scores are q.k / sqrt(D); the output is the softmax-weighted
    sum of values.  Rows at or past num_nodes[b] are 0.

    q [B][R][H][D], k_tree/v_tree [B][R][Hkv][D], k_cache/v_cache
    [B][Pmax][Hkv][D] (any float dtype; computed in float64), prefix_len and
    num_nodes [B], mask [B][R][R], pos_ids [B][R]; query head h reads key
    head h // (H // Hkv).  Returns float64 [B][R][H][D].
    """
    q = np.asarray(q, dtype=np.float64)
    B, R, H, D = q.shape
    Hkv = k_tree.shape[2]
    grp = H // Hkv
    out = np.zeros((B, R, H, D), np.float64)
    for b in range(B):
        P = int(prefix_len[b])
        n = int(num_nodes[b])
        if n <= 0:
            continue
        pos = P + np.asarray(pos_ids[b][:n], dtype=np.int64)
        for h in range(H):
            g = h // grp
            qh = rope(q[b, :n, h, :], pos, rope_base)
            kt = rope(np.asarray(k_tree[b, :n, g, :], dtype=np.float64), pos, rope_base)
            vt = np.asarray(v_tree[b, :n, g, :], dtype=np.float64)
            kc = np.asarray(k_cache[b, :P, g, :], dtype=np.float64)
            vc = np.asarray(v_cache[b, :P, g, :], dtype=np.float64)
            keys = np.concatenate([kc, kt], axis=0)
            vals = np.concatenate([vc, vt], axis=0)
            for i in range(n):
                allowed = np.concatenate([np.ones(P, bool), np.asarray(mask[b][i][:n]) == 1])
                s = keys[allowed] @ qh[i] / np.sqrt(D)
                w = np.exp(s - s.max())
                out[b, i, h] = (w / w.sum()) @ vals[allowed]
    return out
