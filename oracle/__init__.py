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
_LIB_PATH = os.path.join(_HERE, "liboracle.so")


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


def retrieve(texts, ctx, n_max: int = 16, n_min: int = 2, k: int = 5000, m: int = 10) -> dict:
    """Batched suffix-match retrieval over stores in priority order.

    texts: list of uint16 arrays (store 0 = repository store first);
    ctx: uint16 [B][L].  Returns dict of match_n, range_lo, range_cnt, taken
    ([B][S]) and cont_pos, cont_src, cont_len ([B][k]), cont_tok ([B][k][m]).
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
    _lib().oracle_retrieve(S, ctypes.cast(ptrs, ctypes.c_void_p), _p(lens), _p(c), B, L, n_max, n_min, k, m,
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


def replay(texts, truth, n_max: int = 16, n_min: int = 2, k: int = 5000, m: int = 10, c: int = 64, alpha=(1, 1),
           lru: int = 32, ctx_len: int = 16, max_steps: int = 512) -> dict:
    """Decode-trace replay over known streams (reading of the average
    acceptance length setting, Section V-C eq. (7)).

    Every stream starts with its first ctx_len tokens as context at position
    p = ctx_len.  Each step, for every stream with p below its length: the
    key is the last ctx_len tokens; an LRU of `lru` entries per stream maps
    keys to stored retrieval results (a hit reuses the result and becomes most
    recent; a miss retrieves, inserts as most recent and drops the least
    recent beyond `lru`); the draft tree is built; the target after tree row
    i is truth[p + pos_ids[i]] (-1 past the stream); the accepted length is
    added to p.  Returns accept [steps][n_streams] (-1 for finished streams),
    hits and lookups per stream, final positions, the mean accepted length
    per live step, and the step count.
    """
    from collections import OrderedDict

    truth = np.ascontiguousarray(truth, dtype=np.uint16)
    nseq, tlen = truth.shape
    pos = [ctx_len] * nseq
    caches = [OrderedDict() for _ in range(nseq)]
    hits = [0] * nseq
    lookups = [0] * nseq
    fields = ("taken", "cont_len", "cont_tok")
    steps = []
    for _ in range(max_steps):
        act = [b for b in range(nseq) if pos[b] < tlen]
        if not act:
            break
        ctx = np.stack([truth[b, pos[b] - ctx_len:pos[b]] for b in act])
        keys = [ctx[j].tobytes() for j in range(len(act))]
        missing = []
        for j, b in enumerate(act):
            lookups[b] += 1
            if keys[j] in caches[b]:
                caches[b].move_to_end(keys[j])
                hits[b] += 1
            else:
                missing.append(j)
        if missing:
            r = retrieve(texts, ctx[missing], n_max=n_max, n_min=n_min, k=k, m=m)
            for i, j in enumerate(missing):
                b = act[j]
                if len(caches[b]) >= lru:
                    caches[b].popitem(last=False)
                caches[b][keys[j]] = {f: r[f][i].copy() for f in fields}
        got = [caches[b][keys[j]] for j, b in enumerate(act)]
        tree = build_tree(np.stack([g["taken"] for g in got]), np.stack([g["cont_len"] for g in got]),
                          np.stack([g["cont_tok"] for g in got]), ctx, c=c, alpha=alpha)
        target = np.full(tree["node_tok"].shape, -1, np.int32)
        for j, b in enumerate(act):
            for i in range(int(tree["num_nodes"][j])):
                at = pos[b] + int(tree["pos_ids"][j, i])
                if at < tlen:
                    target[j, i] = int(truth[b, at])
        acc = verify_accept(tree, target, m=m)["accept_len"]
        row = np.full(nseq, -1, np.int64)
        for j, b in enumerate(act):
            row[b] = int(acc[j])
            pos[b] += int(acc[j])
        steps.append(row)
    accept = np.stack(steps) if steps else np.zeros((0, nseq), np.int64)
    live = accept >= 0
    return dict(accept=accept, hits=np.array(hits), lookups=np.array(lookups), pos=np.array(pos),
                acc_len=float(accept[live].sum() / max(live.sum(), 1)), steps=len(steps))
