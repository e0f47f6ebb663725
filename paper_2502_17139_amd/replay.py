"""Decode-trace replay on the GPU.

Drives the draft stage over known token streams as a stand-in for a
decoding loop: every step each live stream retrieves (or reuses a cached
retrieval for the same 16-token context), builds its draft tree, receives
the true next tokens as the target model's outputs, and advances by the
accepted length.  The mean advance per step is the paper's average
acceptance length (Section V-C, eq. (7)).

Per stream, an LRU cache of 32 recent retrievals is keyed by the exact
16-token context; a hit reuses the stored retrieval and becomes most
recent, a miss retrieves into the least recent slot.  The cache lives on the
GPU: its slots are rows of the retrieval output arrays, misses are retrieved
straight into their slot (fc_retrieve's row map) and the tree reads each
stream's slot in place (fc_build_tree's row map), so cached results are
never copied.  Only the cache keys and positions are kept on the host; one
small copy of the accepted lengths comes back per step.
"""
from __future__ import annotations

from collections import OrderedDict

import numpy as np
import torch

from . import (accept_outputs, fc_build_tree, fc_build_tree_workspace_bytes, fc_retrieve,
               fc_retrieve_workspace_bytes, fc_targets_from_truth, fc_verify_accept, retrieve_outputs,
               tree_outputs)


class GpuReplay:
    """Replay state for `truth` (uint16 [n_streams][length]) over `stores`."""

    def __init__(self, stores, truth: np.ndarray, n_max=16, n_min=2, k=5000, m=10, c=64, alpha=(1, 1), lru=32,
                 ctx_len=16, device="cuda"):
        self.stores = stores
        self.truth_np = np.ascontiguousarray(truth, dtype=np.uint16)
        self.nseq, self.tlen = self.truth_np.shape
        self.truth = torch.from_numpy(self.truth_np).to(device)
        self.p = dict(n_max=n_max, n_min=n_min, k=k, m=m)
        self.c, self.alpha, self.lru, self.ctx_len = c, tuple(alpha)[:len(stores)], lru, ctx_len
        self.device = torch.device(device)
        S = len(stores)
        self.cache = retrieve_outputs(self.nseq * lru, S, k, m, self.device)
        self.rws = torch.empty(max(fc_retrieve_workspace_bytes(self.nseq, S, n_max, n_min, k, m), 1),
                               dtype=torch.uint8, device=self.device)
        self.tws = torch.empty(max(fc_build_tree_workspace_bytes(self.nseq), 1), dtype=torch.uint8,
                               device=self.device)
        self.tout = tree_outputs(self.nseq, c, self.device)
        self.aout = accept_outputs(self.nseq, m, self.device)
        self.tgt = torch.empty((self.nseq, c + 1), dtype=torch.int32, device=self.device)
        self.reset()

    def reset(self):
        self.pos = np.full(self.nseq, self.ctx_len, np.int64)
        self.lru_state = [OrderedDict() for _ in range(self.nseq)]
        self.hits = np.zeros(self.nseq, np.int64)
        self.lookups = np.zeros(self.nseq, np.int64)

    def step(self) -> np.ndarray | None:
        """One step for every live stream; returns accepted lengths per stream
        (-1 for finished streams) or None when every stream is done."""
        act = np.nonzero(self.pos < self.tlen)[0]
        if len(act) == 0:
            return None
        L = self.ctx_len
        ctx = np.stack([self.truth_np[b, self.pos[b] - L:self.pos[b]] for b in act])
        slots = np.empty(len(act), np.int64)
        miss = []
        for j, b in enumerate(act):
            d = self.lru_state[b]
            key = ctx[j].tobytes()
            self.lookups[b] += 1
            if key in d:
                d.move_to_end(key)
                slots[j] = d[key]
                self.hits[b] += 1
            else:
                if len(d) >= self.lru:
                    _, slot = d.popitem(last=False)
                else:
                    slot = len(d)
                d[key] = slot
                slots[j] = slot
                miss.append(j)
        rows = (act * self.lru + slots).astype(np.int32)
        dev = self.device
        if miss:
            fc_retrieve(self.stores, torch.from_numpy(ctx[miss]).to(dev), out=self.cache, workspace=self.rws,
                        rows=torch.from_numpy(rows[miss]).to(dev), **self.p)
        B = len(act)
        ctx_d = torch.from_numpy(ctx).to(dev)
        tree = {f: v[:B] for f, v in self.tout.items()}
        fc_build_tree(self.cache["taken"], self.cache["cont_len"], self.cache["cont_tok"], ctx_d, c=self.c,
                      alpha=self.alpha, out=tree, workspace=self.tws, rows=torch.from_numpy(rows).to(dev))
        tgt = fc_targets_from_truth(self.truth, torch.from_numpy(self.pos[act].astype(np.int32)).to(dev), tree,
                                    seq=torch.from_numpy(act.astype(np.int32)).to(dev), out=self.tgt[:B])
        acc = fc_verify_accept(tree, tgt, m=self.p["m"], out={f: v[:B] for f, v in self.aout.items()})
        a = acc["accept_len"].cpu().numpy().astype(np.int64)
        out = np.full(self.nseq, -1, np.int64)
        out[act] = a
        self.pos[act] += a
        return out

    def run(self, max_steps: int = 512) -> dict:
        steps = []
        for _ in range(max_steps):
            a = self.step()
            if a is None:
                break
            steps.append(a)
        acc = np.stack(steps) if steps else np.zeros((0, self.nseq), np.int64)
        live = acc >= 0
        return dict(accept=acc, hits=self.hits.copy(), lookups=self.lookups.copy(), pos=self.pos.copy(),
                    acc_len=float(acc[live].sum() / max(live.sum(), 1)), steps=len(steps))
