"""Helpers for the GPU parity tests: run the HIP path through the C ABI and
the oracle side by side on the same seeded inputs, and compare every output
element by element.  The two sides never exchange values: each computes its
own retrieval, tree and acceptance from the seeded inputs."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
import paper_2502_17139_amd as fc


def say(*a) -> None:
    print(*a, flush=True)
    sys.stdout.flush()


def dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t: torch.Tensor) -> np.ndarray:
    return t.cpu().numpy()


def gpu_store(tokens: np.ndarray, pair_vocab: int | None = None, records: bool = False,
              top: bool | None = None) -> fc.Store:
    return fc.Store(dev(tokens.astype(np.uint16)), pair_vocab=pair_vocab, records=records, top=top)


def gpu_pipeline(stores, ctx: np.ndarray, p: dict, alpha, c: int) -> dict:
    """fc_retrieve -> fc_build_tree on the GPU; host copies of every output."""
    cx = dev(ctx.astype(np.uint16))
    r = fc.fc_retrieve(stores, cx, n_max=p["n_max"], n_min=p["n_min"], k=p["k"], m=p["m"])
    t = fc.fc_build_tree(r["taken"], r["cont_len"], r["cont_tok"], cx, c=c, alpha=alpha)
    torch.cuda.synchronize()
    out = {f: host(v) for f, v in r.items()}
    out.update({f: host(v) for f, v in t.items()})
    out["_tree_dev"] = t
    return out


def oracle_pipeline(texts, ctx: np.ndarray, p: dict, alpha, c: int) -> dict:
    r = oracle.retrieve(texts, ctx, n_max=p["n_max"], n_min=p["n_min"], k=p["k"], m=p["m"])
    t = oracle.build_tree(r["taken"], r["cont_len"], r["cont_tok"], ctx, c=c, alpha=alpha)
    out = dict(r)
    out.update(t)
    return out


def compare_retrieve(g: dict, o: dict, rows=None) -> None:
    """Bit-exact on every per-store field and every slot below the query's
    total taken (slots past it are not written by the GPU path)."""
    B = o["taken"].shape[0]
    rows = range(B) if rows is None else rows
    for i, b in enumerate(rows):
        for f in ("match_n", "range_lo", "range_cnt", "taken"):
            assert (g[f][b] == o[f][i]).all(), (f, b, g[f][b].tolist(), o[f][i].tolist())
        used = int(o["taken"][i].sum())
        for f in ("cont_pos", "cont_src", "cont_len", "cont_tok"):
            assert (g[f][b, :used] == o[f][i, :used]).all(), (f, b)


def compare_tree(g: dict, o: dict, rows=None) -> None:
    B = o["num_nodes"].shape[0]
    rows = range(B) if rows is None else rows
    for i, b in enumerate(rows):
        for f in ("num_nodes", "node_tok", "parent", "weight", "pos_ids", "mask"):
            assert (g[f][b] == o[f][i]).all(), (f, b)


def targets_from_truth(pos_ids: np.ndarray, num_nodes: np.ndarray, truth_rows: np.ndarray,
                       start: np.ndarray) -> np.ndarray:
    """target[i] = truth[start + pos_ids[i]] (the true next token after row i
    when the tree row's path is right), -1 past the stream or in padding."""
    B, R = pos_ids.shape
    out = np.full((B, R), -1, np.int32)
    for b in range(B):
        for i in range(max(int(num_nodes[b]), 0)):
            j = int(start[b]) + int(pos_ids[b, i])
            if j < truth_rows.shape[1]:
                out[b, i] = int(truth_rows[b, j])
    return out
