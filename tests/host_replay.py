"""Decode-trace replay driven from the host: a second implementation of the
replay, for the tests only.

It drives the draft stage over known token streams as a stand-in for a
decoding loop, through the library's entry points one call at a time: every
step each live stream retrieves (or reuses a cached retrieval for the same
16-token context), builds its draft tree, receives the true next tokens as
the target model's outputs, and advances by the accepted length.  The mean
advance per step is the paper's average acceptance length (Section V-C,
eq. (7)).  The product's replay is the device-resident engine
(paper_2502_17139_amd.ReplayEngine, fc_replay_init / fc_replay_run); the
tests run both and compare each with the oracle.

Per stream, an LRU cache of 32 recent retrievals is keyed by the exact
16-token context; a hit reuses the stored retrieval and becomes most recent,
a miss retrieves into the least recent slot.  The slots are rows of the
retrieval output arrays on the GPU: misses are retrieved straight into their
slot (fc_retrieve's row map) and the tree reads each stream's slot in place
(fc_build_tree's row map).  The cache keys and positions are kept on the
host; one small copy of the accepted lengths comes back per step.

With cache_l set, each stream also keeps the paper's CACHE (Section IV-B)
and follows the cache branch of Alg. 1: once the CACHE holds cache_l
sequences, the context is searched there first (fc_cache_retrieve) and a
non-empty result replaces the datastore retrieval; after verification the
context plus the accepted draft tokens, and every completed chunk of
cache_every output tokens, are added.  The CACHE texts live on the GPU (one
row of FC_MAX_CACHE_TOKENS tokens per stream, sequences joined by 0); the
host keeps the sequence lists, decides evictions (oldest sequences first
when a text would outgrow its row) and ships each step's appended tokens in
one batched fc_cache_write.

Alg. 1's retrieval-timing control (for contexts the CACHE did not serve):
with missing=True a per-stream missing table holds the contexts whose
datastore retrieval found nothing, and such a context is not retrieved
again; with skip_tok set, a context ending with skip_tok is retrieved only
when the step's draw (skip_draws[step][stream], uniform in [0, 2^31)) is
below skip_p * 2^31.  A context that is not retrieved gets an empty result
(a bare root).  Both tables are host-side sets next to the LRU keys.

GpuReplay.run(native=True) hands the replay to the device engine with the
same parameters; run(native=False) steps this loop.
"""
from __future__ import annotations

from collections import OrderedDict

import numpy as np
import torch

from paper_2502_17139_amd import (FC_MAX_CACHE_TOKENS, ReplayEngine, accept_outputs, fc_build_tree,
                                  fc_build_tree_workspace_bytes, fc_cache_retrieve, fc_cache_write, fc_retrieve,
                                  fc_retrieve_workspace_bytes, fc_targets_from_truth, fc_verify_accept,
                                  retrieve_outputs, tree_outputs)


class _Sequences:
    """One stream's CACHE sequences and the text they make (joined by 0),
    bounded by `cap` tokens: the oldest sequences go first.  The text is
    kept as one flat list, so an append costs its own length."""

    def __init__(self, cap: int):
        self.cap = cap
        self.lens = []  # sequence lengths, oldest first
        self.flat = []  # the text

    @property
    def tokens(self) -> int:
        return len(self.flat)

    def add(self, seq) -> bool:
        """Append a sequence; True when older sequences had to go."""
        seq = [int(x) for x in seq][-self.cap:]
        if not seq:
            return False
        if self.flat:
            self.flat.append(0)
        self.flat.extend(seq)
        self.lens.append(len(seq))
        cut = 0
        while len(self.flat) - cut > self.cap:
            cut += self.lens.pop(0) + 1  # the sequence and the separator after it
        if cut:
            self.flat = self.flat[cut:]
        return cut > 0

    def text(self) -> list:
        return self.flat


class GpuReplay:
    """Replay state for `truth` (uint16 [n_streams][length]) over `stores`."""

    def __init__(self, stores, truth: np.ndarray, n_max=16, n_min=2, k=5000, m=10, c=64, alpha=(1, 1), lru=32,
                 ctx_len=16, device="cuda", cache_l=None, cache_every=20, cache_cap=FC_MAX_CACHE_TOKENS,
                 missing=False, skip_tok=None, skip_p=0.5, skip_draws=None):
        self.stores = stores
        self.kw = dict(n_max=n_max, n_min=n_min, k=k, m=m, c=c, alpha=alpha, lru=lru, ctx_len=ctx_len)
        self.truth_np = np.ascontiguousarray(truth, dtype=np.uint16)
        self.nseq, self.tlen = self.truth_np.shape
        self.truth = torch.from_numpy(self.truth_np).to(device)
        self.p = dict(n_max=n_max, n_min=n_min, k=k, m=m)
        self.c, self.alpha, self.lru, self.ctx_len = c, tuple(alpha)[:len(stores)], lru, ctx_len
        self.device = torch.device(device)
        S = len(stores)
        # LRU slots, plus one last row that stays empty (taken 0): the input
        # row of contexts that are not retrieved
        self.cache = retrieve_outputs(self.nseq * lru + 1, S, k, m, self.device)
        self.cache["taken"][-1].zero_()
        self.empty_row = self.nseq * lru
        self.rws = torch.empty(max(fc_retrieve_workspace_bytes(self.nseq, S, n_max, n_min, k, m), 1),
                               dtype=torch.uint8, device=self.device)
        self.tws = torch.empty(max(fc_build_tree_workspace_bytes(self.nseq), 1), dtype=torch.uint8,
                               device=self.device)
        self.tout = tree_outputs(self.nseq, c, self.device)
        self.aout = accept_outputs(self.nseq, m, self.device)
        self.tgt = torch.empty((self.nseq, c + 1), dtype=torch.int32, device=self.device)
        self.cache_l, self.cache_every, self.cache_cap = cache_l, cache_every, cache_cap
        self.missing, self.skip_tok = missing, skip_tok
        self.skip_p, self.skip_thr = skip_p, int(skip_p * 2 ** 31)
        self.skip_draws = None if skip_draws is None else np.asarray(skip_draws)
        if cache_l is not None:
            self.ctext = torch.zeros((self.nseq, cache_cap), dtype=torch.uint16, device=self.device)
            self.clen = torch.zeros(self.nseq, dtype=torch.int32, device=self.device)
            self.cres = retrieve_outputs(self.nseq, 1, k, m, self.device)
        self.reset()

    def reset(self):
        self.pos = np.full(self.nseq, self.ctx_len, np.int64)
        self.lru_state = [OrderedDict() for _ in range(self.nseq)]
        self.hits = np.zeros(self.nseq, np.int64)
        self.lookups = np.zeros(self.nseq, np.int64)
        self.served = np.zeros(self.nseq, np.int64)
        self.m_skips = np.zeros(self.nseq, np.int64)
        self.g_skips = np.zeros(self.nseq, np.int64)
        self.mtab = [set() for _ in range(self.nseq)]
        self.step_i = 0
        if self.cache_l is not None:
            self.seqs = [_Sequences(self.cache_cap) for _ in range(self.nseq)]
            self.chunks = np.zeros(self.nseq, np.int64)
            self.clen.zero_()

    def _cache_upload(self, changed: dict) -> None:
        """Ship the CACHE texts of the streams in `changed` (stream -> text
        length on the device before this step's additions, or -1 when the
        whole text must be rewritten) in one batched write."""
        rows, offs, lens, src_off, src_len, parts = [], [], [], [], [], []
        at = 0
        for b, old in changed.items():
            text = self.seqs[b].text()
            start = 0 if old < 0 else old
            piece = text[start:]
            rows.append(b)
            offs.append(start)
            lens.append(len(text))
            src_off.append(at)
            src_len.append(len(piece))
            parts.extend(piece)
            at += len(piece)
        if not rows:
            return
        dev = self.device

        def d(x, dt):
            return torch.from_numpy(np.asarray(x, dtype=dt)).to(dev)

        fc_cache_write(self.ctext, self.clen, d(rows, np.int32), d(offs, np.int32), d(lens, np.int32),
                       d(src_off, np.int64), d(src_len, np.int32), d(parts if parts else [0], np.uint16))

    def step(self) -> np.ndarray | None:
        """One step for every live stream; returns accepted lengths per stream
        (-1 for finished streams) or None when every stream is done."""
        act = np.nonzero(self.pos < self.tlen)[0]
        if len(act) == 0:
            return None
        L = self.ctx_len
        dev = self.device
        ctx = np.stack([self.truth_np[b, self.pos[b] - L:self.pos[b]] for b in act])
        ctx_d = torch.from_numpy(ctx).to(dev)
        # Alg. 1: the CACHE first, once it holds cache_l sequences
        served = np.zeros(len(act), bool)
        if self.cache_l is not None:
            elig = np.array([j for j, b in enumerate(act) if len(self.seqs[b].lens) >= self.cache_l], np.int64)
            if len(elig):
                sid = torch.from_numpy(act[elig].astype(np.int32)).to(dev)
                fc_cache_retrieve(self.ctext, self.clen, torch.from_numpy(ctx[elig]).to(dev), text_row=sid,
                                  out=self.cres, rows=sid, **self.p)
                tk = self.cres["taken"][sid.long(), 0].cpu().numpy()
                served[elig[tk > 0]] = True
        # Alg. 1's timing control for the rest: the missing table, then the
        # skip gate
        skip = np.zeros(len(act), bool)
        if self.missing or self.skip_tok is not None:
            for j, b in enumerate(act):
                if served[j]:
                    continue
                if self.missing and ctx[j].tobytes() in self.mtab[b]:
                    skip[j] = True
                    self.m_skips[b] += 1
                elif (self.skip_tok is not None and int(ctx[j][-1]) == self.skip_tok
                      and not int(self.skip_draws[self.step_i][b]) < self.skip_thr):
                    skip[j] = True
                    self.g_skips[b] += 1
        self.step_i += 1
        srv = np.nonzero(served)[0]
        need = np.nonzero(~served & ~skip)[0]
        skp = np.nonzero(skip)[0]
        slots = np.empty(len(need), np.int64)
        miss = []
        for i, j in enumerate(need):
            b = act[j]
            d = self.lru_state[b]
            key = ctx[j].tobytes()
            self.lookups[b] += 1
            if key in d:
                d.move_to_end(key)
                slots[i] = d[key]
                self.hits[b] += 1
            else:
                if len(d) >= self.lru:
                    _, slot = d.popitem(last=False)
                else:
                    slot = len(d)
                d[key] = slot
                slots[i] = slot
                miss.append(i)
        rows = (act[need] * self.lru + slots).astype(np.int32)
        if miss:
            fc_retrieve(self.stores, torch.from_numpy(ctx[need[miss]]).to(dev), out=self.cache, workspace=self.rws,
                        rows=torch.from_numpy(rows[miss]).to(dev), **self.p)
        if self.missing and len(need):
            tot = self.cache["taken"][torch.from_numpy(rows).long().to(dev)].sum(1).cpu().numpy()
            for i, j in enumerate(need):
                if tot[i] == 0:
                    self.mtab[act[j]].add(ctx[j].tobytes())
        # trees: CACHE-served streams first (one source), then the rest, the
        # contexts that were not retrieved reading the empty row
        rows = np.concatenate([rows, np.full(len(skp), self.empty_row, np.int32)])
        need = np.concatenate([need, skp]).astype(np.int64)
        order = np.concatenate([srv, need]).astype(np.int64)
        B, Bs = len(order), len(srv)
        tree = {f: v[:B] for f, v in self.tout.items()}
        if Bs:
            fc_build_tree(self.cres["taken"], self.cres["cont_len"], self.cres["cont_tok"],
                          torch.from_numpy(ctx[srv]).to(dev), c=self.c, alpha=(1,),
                          out={f: v[:Bs] for f, v in tree.items()}, workspace=self.tws,
                          rows=torch.from_numpy(act[srv].astype(np.int32)).to(dev))
        if len(need):
            fc_build_tree(self.cache["taken"], self.cache["cont_len"], self.cache["cont_tok"],
                          ctx_d if np.array_equal(need, np.arange(len(act))) else torch.from_numpy(ctx[need]).to(dev),
                          c=self.c, alpha=self.alpha,
                          out={f: v[Bs:] for f, v in tree.items()}, workspace=self.tws,
                          rows=torch.from_numpy(rows).to(dev))
        seq_o = act[order]
        tgt = fc_targets_from_truth(self.truth, torch.from_numpy(self.pos[seq_o].astype(np.int32)).to(dev), tree,
                                    seq=torch.from_numpy(seq_o.astype(np.int32)).to(dev), out=self.tgt[:B])
        acc = fc_verify_accept(tree, tgt, m=self.p["m"], out={f: v[:B] for f, v in self.aout.items()})
        a = acc["accept_len"].cpu().numpy().astype(np.int64)
        out = np.full(self.nseq, -1, np.int64)
        out[seq_o] = a
        if self.cache_l is None:
            self.pos[seq_o] += a
            return out
        last = acc["last_node"].long()
        depth = tree["pos_ids"].gather(1, last[:, None])[:, 0].cpu().numpy().astype(np.int64)
        self.served[act[srv]] += 1
        changed = {}
        for i, b in enumerate(seq_o):
            p = int(self.pos[b])
            old = int(self.seqs[b].tokens)
            ev = False
            if depth[i] >= 1:  # a verified draft (R non-empty)
                ev |= self.seqs[b].add(list(self.truth_np[b, p - L:p]) + list(self.truth_np[b, p:p + depth[i]]))
            self.pos[b] = p + a[i]
            while L + self.cache_every * (self.chunks[b] + 1) <= min(self.pos[b], self.tlen):
                lo = L + self.cache_every * int(self.chunks[b])
                ev |= self.seqs[b].add(self.truth_np[b, lo:lo + self.cache_every])
                self.chunks[b] += 1
            if self.seqs[b].tokens != old or ev:
                changed[int(b)] = -1 if ev else old
        self._cache_upload(changed)
        return out

    def run(self, max_steps: int = 512, native: bool = True) -> dict:
        """Replays for at most max_steps steps: from the start on the device
        engine (native), or from the current state with step()."""
        if native:
            if not hasattr(self, "_engine") or self._engine.max_steps < max_steps:
                steps = max(max_steps, 512)
                ckw = {}
                if self.cache_l is not None:
                    ckw.update(cache_l=self.cache_l, cache_every=self.cache_every, cache_cap=self.cache_cap)
                if self.missing:
                    ckw.update(missing=True)
                if self.skip_tok is not None:
                    draws = np.zeros((steps, self.nseq), np.int64)
                    have = min(steps, len(self.skip_draws))
                    draws[:have] = np.asarray(self.skip_draws)[:have, :self.nseq]
                    ckw.update(skip_tok=self.skip_tok, skip_p=self.skip_p, skip_draws=draws)
                self._engine = ReplayEngine(self.stores, self.truth, max_steps=steps, **self.kw, **ckw)
            return self._engine.run(limit=max_steps)
        steps = []
        for _ in range(max_steps):
            a = self.step()
            if a is None:
                break
            steps.append(a)
        acc = np.stack(steps) if steps else np.zeros((0, self.nseq), np.int64)
        live = acc >= 0
        return dict(accept=acc, hits=self.hits.copy(), lookups=self.lookups.copy(), pos=self.pos.copy(),
                    cache_served=self.served.copy(), missing_skips=self.m_skips.copy(),
                    gate_skips=self.g_skips.copy(), acc_len=float(acc[live].sum() / max(live.sum(), 1)),
                    steps=len(steps))
