#!/usr/bin/env python3
"""Draft-stage hot-path benchmark on one MI355X.

One step = one batch of queries through the whole draft-stage path on the
GPU: fc_retrieve (longest-suffix match in both stores + continuation gather),
fc_build_tree (weighted trie, top-c, mask, position ids) and fc_verify_accept
(longest accepted path against the true next tokens).  Stores, suffix arrays,
first-token and two-token tables, inline-prefix records, query contexts and
target tokens are
resident in HBM before the timed region; the suffix arrays and tables are
built once, untimed, with fc_datastore_build / fc_store_prepare(_pairs) (the
paper builds its datastores offline).

Default workload: the 1,024-query batch over a 10M-token project store and a
1B-token general store (k = 5000, m = 10, c = 64, n = 16..2).  Prints ONE JSON
line.  Timing uses HIP events on the stream the kernels run on.
"""
from __future__ import annotations

import argparse
import gc
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, published peak
WORKLOADS = {"headline": 3, "two-store": 2, "single": 1, "replay": 3, "replay-cache": 3, "replay-control": 3,
             "build": 3, "build-repos": 0, "extend": 3, "copy": 0, "tree-attention": 1, "gather-probe": 0}
# kernels each entry point launches (rocprofv3 kernel names start with these)
ENTRY_KERNELS = {
    "fc_retrieve": ("k_search", "k_offsets", "k_gather"),
    "fc_build_tree": ("k_tree_plan", "k_tree_flat", "k_tree_fast", "k_tree_any"),
    "fc_verify_accept": ("k_verify",),
}
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_headline_10M_1B.txt")
BUILD_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_sa_build_1B_10M.txt")


def kernel_source_hash() -> str:
    """SHA-256 over the HIP sources and the ABI header: measured hardware
    traffic is only reported for the sources it was measured on."""
    import glob
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2502_17139_amd", "csrc")
    files = sorted(glob.glob(os.path.join(csrc, "*.hip")) + glob.glob(os.path.join(csrc, "*.h")) +
                   glob.glob(os.path.join(csrc, "*.cpp"))) + [os.path.join(ROOT, "include", "fastcoder.h")]
    for f in files:
        h.update(os.path.basename(f).encode())
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(path: str) -> dict:
    """HBM bytes per launch from a committed counter summary (FETCH_SIZE and
    WRITE_SIZE, scaled by a plain copy's readings), or {} when it is missing
    or was taken on other kernel sources."""
    try:
        with open(path) as f:
            lines = f.read().splitlines()
    except OSError:
        return {}
    out, sha = {}, None
    for ln in lines:
        parts = ln.split()
        if len(parts) == 2 and parts[0] == "source_sha256":
            sha = parts[1]
        elif len(parts) == 4 and parts[0] == "entry" and parts[2] == "bytes":
            out[parts[1]] = float(parts[3])
    return out if sha == kernel_source_hash() else {}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def algorithmic_bytes(taken, cont_len, match_n, ctx_nhi, store_sizes, k, m, c, n_min, L=16):
    """Bytes the method must move per launch, from the batch's own outputs.

    search (per query, per store, for every suffix length tried - n_hi down
    to the match, or down to n_min when nothing matches): two binary
    searches over the whole suffix array, ceil(log2(N_s + 1)) probes each, a
    probe being a 4-byte suffix-array entry plus up to 2n bytes of text.
    `search_bucketed` is the same with the first-token bucket narrowing each
    search first (8 bytes of table, ranges of N_s / 32256).
    io (per query): the context (2L) read, the four per-store fields (16 per
    store) written.
    gather (per kept slot): 4-byte suffix-array entry + 2*len text bytes
    read; 4 + 1 + 1 + 2*m bytes written.
    tree (per query): taken (4*S) + cont_len (1 per kept slot) + cont_tok
    (2*m per kept slot) + root token (2) read; rows 4*4*(c+1) + num_nodes 4
    + mask 4*(c+1)^2 written.
    verify (per query): num_nodes 4 + node_tok/parent/target 3*4*(c+1) read;
    4 + 4*(m+1) + 4 written.
    """
    B, S = taken.shape
    R = c + 1
    search = search_b = 0.0
    for s in range(S):
        full = int(np.ceil(np.log2(store_sizes[s] + 1.0)))
        buck = int(np.ceil(np.log2(store_sizes[s] / 32256.0 + 1)))
        lo = np.where(match_n[:, s] > 0, match_n[:, s], n_min).astype(np.int64)
        hi = ctx_nhi.astype(np.int64)
        for n in range(n_min, 17):
            tried = (hi >= n) & (lo <= n)
            cnt = int(tried.sum())
            search += cnt * 2 * full * (4 + 2 * n)
            search_b += cnt * (8 + 2 * buck * (4 + 2 * n))
    io = B * (2 * L + 16 * S)
    used = taken.sum(axis=1)
    kept = int(used.sum())
    lens = sum(int(cont_len[b, :used[b]].astype(np.int64).sum()) for b in range(B))
    gather = kept * (4 + 4 + 1 + 1 + 2 * m) + 2 * lens
    tree = B * (4 * S + 2) + kept * (1 + 2 * m) + B * (4 + 16 * R + 4 * R * R)
    verify = B * (4 + 12 * R + 4 + 4 * (m + 1) + 4)
    return dict(search=float(search), search_bucketed=float(search_b), io=float(io), gather=float(gather),
                tree=float(tree), verify=float(verify), kept=kept)


def n_hi_of(ctx: np.ndarray, n_max: int) -> np.ndarray:
    out = np.zeros(ctx.shape[0], np.int64)
    for b in range(ctx.shape[0]):
        t = 0
        while t < ctx.shape[1] and ctx[b, ctx.shape[1] - 1 - t] != 0:
            t += 1
        out[b] = min(n_max, ctx.shape[1], t)
    return out


def targets_for(pos_ids, num_nodes, nxt):
    """target[b][i] = the true token after the path to row i (-1 if none)."""
    B, R = pos_ids.shape
    out = np.full((B, R), -1, np.int32)
    for b in range(B):
        n = int(num_nodes[b])
        for i in range(max(n, 0)):
            j = int(pos_ids[b, i])
            if j < nxt.shape[1]:
                out[b, i] = int(nxt[b, j])
    return out


def host_info() -> dict:
    """Cores this process may use, the oracle's thread count and the CPU model."""
    import oracle
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    model = ln.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"affinity_cores": len(os.sched_getaffinity(0)), "nproc": os.cpu_count(),
            "oracle_threads": oracle.max_threads(), "cpu_model": model}


def oracle_batch(texts, ctx, nxt, p, alpha, c):
    """The oracle (test infrastructure) on a whole batch: retrieval (its
    batched form), tree and acceptance; returns seconds."""
    import oracle
    t0 = time.perf_counter()
    r = oracle.retrieve(texts, ctx, n_max=p["n_max"], n_min=p["n_min"], k=p["k"], m=p["m"], batched=True)
    t = oracle.build_tree(r["taken"], r["cont_len"], r["cont_tok"], ctx, c=c, alpha=alpha)
    oracle.verify_accept(t, targets_for(t["pos_ids"], t["num_nodes"], nxt), m=p["m"])
    return time.perf_counter() - t0


class Batch:
    """One query batch resident on the GPU with its own output buffers."""

    def __init__(self, fc, torch, dev, ctx_np, nxt_np, S, p, c):
        B = ctx_np.shape[0]
        self.B, self.ctx_np, self.nxt_np = B, ctx_np, nxt_np
        self.ctx = torch.from_numpy(ctx_np).to(dev)
        self.rout = fc.retrieve_outputs(B, S, p["k"], p["m"], dev)
        self.tout = fc.tree_outputs(B, c, dev)
        self.aout = fc.accept_outputs(B, p["m"], dev)
        self.target = None


def make_pipeline(fc, torch, dev, stores, p, alpha, c, Bmax):
    rws = torch.empty(max(fc.fc_retrieve_workspace_bytes(Bmax, len(stores), p["n_max"], p["n_min"], p["k"], p["m"]),
                          1), dtype=torch.uint8, device=dev)
    tws = torch.empty(max(fc.fc_build_tree_workspace_bytes(Bmax), 1), dtype=torch.uint8, device=dev)

    def retrieve(bt):
        fc.fc_retrieve(stores, bt.ctx, n_max=p["n_max"], n_min=p["n_min"], k=p["k"], m=p["m"], out=bt.rout,
                       workspace=rws)

    def tree(bt):
        fc.fc_build_tree(bt.rout["taken"], bt.rout["cont_len"], bt.rout["cont_tok"], bt.ctx, c=c, alpha=alpha,
                         out=bt.tout, workspace=tws)

    def verify(bt):
        fc.fc_verify_accept(bt.tout, bt.target, m=p["m"], out=bt.aout)

    return retrieve, tree, verify


def prepare_targets(torch, dev, batches, retrieve, tree):
    """First pass over every batch: its tree fixes the target tokens (the
    target model's outputs: the true tokens after each row's path)."""
    for bt in batches:
        retrieve(bt)
        tree(bt)
    torch.cuda.synchronize()
    for bt in batches:
        tgt = targets_for(bt.tout["pos_ids"].cpu().numpy(), bt.tout["num_nodes"].cpu().numpy(), bt.nxt_np)
        bt.target = torch.from_numpy(tgt).to(dev)


def timed_steps(torch, stream, K, order, batches, fns):
    """K steps back to back, step i on batches[order(i)]; one event pair."""
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for i in range(K):
        bt = batches[order(i)]
        for f in fns:
            f(bt)
    end.record(stream)
    torch.cuda.synchronize()
    return start.elapsed_time(end)


def timed_phases(torch, stream, K, order, batches, fns):
    """K steps with an event at every entry-point boundary; per-entry lists
    of milliseconds per launch."""
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(len(fns) + 1)] for _ in range(K)]
    torch.cuda.synchronize()
    for i in range(K):
        bt = batches[order(i)]
        ev[i][0].record(stream)
        for j, f in enumerate(fns):
            f(bt)
            ev[i][j + 1].record(stream)
    torch.cuda.synchronize()
    return [[ev[i][j].elapsed_time(ev[i][j + 1]) for i in range(K)] for j in range(len(fns))]


def small_config(args, cfg, fc, torch, synth, dev, p, c, with_oracle, retrieve_bytes=False):
    """One of the smaller configurations (1M single store, 2M + 100M): the
    whole step (retrieve + tree + accept) timed over K steps of its batch,
    and the oracle on the same batch."""
    roles = synth.store_roles(cfg)
    alpha = tuple(p["alpha"])[:len(roles)]
    texts = [synth.store(cfg, r) for r in roles]
    ctx_np, nxt_np = synth.queries(cfg, next_tokens=p["m"] + 1)
    stores = [fc.Store(torch.from_numpy(t).to(dev), pair_vocab=synth.VOCAB, records=True) for t in texts]
    bt = Batch(fc, torch, dev, ctx_np, nxt_np, len(stores), p, c)
    retrieve, tree, verify = make_pipeline(fc, torch, dev, stores, p, alpha, c, bt.B)
    prepare_targets(torch, dev, [bt], retrieve, tree)
    stream = torch.cuda.current_stream()
    K = max(args.steps, 10)
    for _ in range(args.warmup):
        retrieve(bt), tree(bt), verify(bt)
    ms = timed_steps(torch, stream, K, lambda i: 0, [bt], (retrieve, tree, verify))
    ph = timed_phases(torch, stream, K, lambda i: 0, [bt], (retrieve, tree, verify))
    out = {"workload": synth.WORKLOADS[cfg]["name"], "stores_tokens": [len(t) for t in texts], "batch": bt.B,
           "retrievals_per_s": bt.B * K / (ms * 1e-3), "ms_per_step": ms / K,
           "phases_ms_mean": {n: float(np.mean(v)) for n, v in zip(("fc_retrieve", "fc_build_tree",
                                                                    "fc_verify_accept"), ph)},
           "accept_len_mean": float(bt.aout["accept_len"].float().mean().item())}
    if retrieve_bytes:
        nb = algorithmic_bytes(bt.rout["taken"].cpu().numpy(), bt.rout["cont_len"].cpu().numpy(),
                               bt.rout["match_n"].cpu().numpy(), n_hi_of(ctx_np, p["n_max"]), [len(t) for t in texts],
                               p["k"], p["m"], c, p["n_min"])
        rb = nb["search"] + nb["io"] + nb["gather"]
        out["fc_retrieve_algorithmic_GBps"] = rb / (np.mean(ph[0]) * 1e-3) / 1e9
        out["fc_retrieve_frac"] = out["fc_retrieve_algorithmic_GBps"] / HBM_PEAK_GBS
    if with_oracle:
        sec = oracle_batch(texts, ctx_np, nxt_np, p, alpha, c)
        out["oracle"] = {"retrievals_per_s": bt.B / sec, "seconds": sec, "sample": f"the whole batch ({bt.B} queries)"}
    del stores, bt
    torch.cuda.empty_cache()
    return out


def replay_config(args, fc, torch, synth, dev, stores, texts, p, with_oracle):
    """Decode-trace replay on the headline stores: 128 streams of 4,096
    tokens, 512 steps, LRU of 32, on the device engine."""
    truth = synth.truth()
    eng = fc.ReplayEngine(stores, torch.from_numpy(truth).to(dev), max_steps=512, **p)
    eng.run(limit=max(args.warmup, 1))
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    res = eng.run(limit=512)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    live = res["accept"] >= 0
    out = {"workload": "decode-trace replay, 128 streams x 4096 tokens over project 10M + general 1B, LRU 32",
           "steps": res["steps"], "steps_per_s": res["steps"] / wall, "ms_per_step": 1e3 * wall / res["steps"],
           "accepted_tokens_per_s": float(res["accept"][live].sum()) / wall, "acc_len": res["acc_len"],
           "lru_hit_rate": float(res["hits"].sum() / max(res["lookups"].sum(), 1))}
    if with_oracle:
        import oracle
        n = 4
        t0 = time.perf_counter()
        o = oracle.replay(texts, truth, **p, max_steps=n)
        sec = time.perf_counter() - t0
        out["oracle"] = {"steps_per_s": n / sec, "seconds": sec,
                         "sample": f"the first {n} steps of all 128 streams (batched retrieval per step)",
                         "acc_len_first_steps": o["acc_len"]}
    return out


def build_config(args, fc, torch, synth, dev, texts_by_role, with_oracle):
    """Suffix-array builds of the 1B-token general store and the 10M-token
    project store: seconds, doubling rounds, suffixes still tied after each
    round, the longest common prefix bracket, and the floor bandwidth of any
    build (read 2n, write 4n bytes)."""
    out = {}
    traffic = measured_traffic(BUILD_TRAFFIC_FILE)
    for role in ("project", "general"):
        t = texts_by_role[role]
        n = len(t)
        tok = torch.from_numpy(t).to(dev)
        sa = torch.empty(n, dtype=torch.uint32, device=dev)
        ws = torch.empty(fc.fc_datastore_build_workspace_bytes(n), dtype=torch.uint8, device=dev)
        times, stats = [], None
        for i in range(3):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            _, stats = fc.fc_datastore_build_stats(tok, sa_out=sa, workspace=ws)
            torch.cuda.synchronize()
            if i:
                times.append(time.perf_counter() - t0)
        sec = float(np.median(times))
        pl = stats["prefix_len"]
        rec = {"tokens": n, "seconds": sec, "floor_GBps": 6 * n / sec / 1e9, "rounds": stats["rounds"],
               "sort_passes": stats["sort_passes"], "prefix_len": pl, "sorted_per_round": stats["sorted"],
               "unresolved_per_round": stats["unresolved"],
               "max_lcp": {"at_least": int(pl[-2]) if len(pl) > 1 else 0, "below": int(pl[-1])}}
        tb = traffic.get(role)
        rec["counter_bytes"] = tb
        rec["counter_GBps"] = None if tb is None else tb / sec / 1e9
        out[role] = rec
        del ws, sa, tok
        torch.cuda.empty_cache()
    if with_oracle:
        import oracle
        t = texts_by_role["project"]
        t0 = time.perf_counter()
        oracle.suffix_array(t)
        sec = time.perf_counter() - t0
        n1 = len(texts_by_role["general"])
        n0 = len(t)
        out["oracle"] = {"project_seconds": sec, "threads": 1, "kind": "naive comparison sort",
                         "general_seconds_extrapolated": sec * (n1 * np.log2(n1)) / (n0 * np.log2(n0)),
                         "general_note": "not run: extrapolated from the 10M-token sort by n log n"}
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", choices=sorted(WORKLOADS), default="headline")
    ap.add_argument("--rotations", type=int, default=8, help="distinct query batches cycled by the timed steps")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-latency", action="store_true",
                    help="skip the single-query latency runs (profiles then hold batch dispatches only)")
    ap.add_argument("--no-configs", action="store_true",
                    help="headline only: skip the other configurations' sub-records")
    args = ap.parse_args()
    # No garbage-collector pauses inside timed regions: a pause stalls the
    # host while the GPU drains its queue, and the stall would be timed.
    gc.disable()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU (no sharded stores or collectives); "
                                   "--gpus must be 1", "n_gpus": args.gpus}))
        sys.exit(2)

    if args.workload in ("replay", "replay-cache", "replay-control"):
        return run_replay(args, cache=args.workload != "replay", control=args.workload == "replay-control")
    if args.workload == "build":
        return run_build(args)
    if args.workload == "build-repos":
        return run_build_repos(args)
    if args.workload == "extend":
        return run_extend(args)
    if args.workload == "tree-attention":
        return run_tree_attention(args)
    if args.workload == "copy":
        return run_copy(args)
    if args.workload == "gather-probe":
        return run_gather_probe(args)
    return run_headline(args)


def run_headline(args):
    import torch
    import paper_2502_17139_amd as fc
    import synth

    cfg = WORKLOADS[args.workload]
    p = dict(synth.PARAMS)
    c, alpha = p["c"], tuple(p["alpha"])
    roles = synth.store_roles(cfg)
    alpha = alpha[:len(roles)]
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    k, m = p["k"], p["m"]

    t0 = time.perf_counter()
    texts = [synth.store(cfg, r) for r in roles]
    R = max(args.rotations, 1)
    qs = [synth.queries(cfg, next_tokens=m + 1, rotation=r) for r in range(R)]
    log(f"generated stores {[len(t) for t in texts]} and {R} batches of {qs[0][0].shape[0]} queries "
        f"in {time.perf_counter() - t0:.1f}s")

    stream = torch.cuda.current_stream()
    stores, build_s = [], []
    for t in texts:
        tok = torch.from_numpy(t).to(dev)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        st = fc.Store(tok, pair_vocab=synth.VOCAB, records=True)
        torch.cuda.synchronize()
        build_s.append(time.perf_counter() - t1)
        stores.append(st)
    log(f"suffix arrays + tables built in {[round(x, 3) for x in build_s]} s")

    batches = [Batch(fc, torch, dev, cq, nq, len(stores), p, c) for cq, nq in qs]
    B = batches[0].B
    retrieve, tree, verify = make_pipeline(fc, torch, dev, stores, p, alpha, c, B)
    prepare_targets(torch, dev, batches, retrieve, tree)
    fns = (retrieve, tree, verify)
    rot = lambda i: i % R  # noqa: E731
    same = lambda i: 0  # noqa: E731
    for i in range(args.warmup):
        for f in fns:
            f(batches[rot(i)])
    torch.cuda.synchronize()

    K = args.steps
    gc.collect()
    # Timed region 1: K steps back to back over the rotation of distinct
    # batches (each step's contexts, continuations and trees live in buffers
    # the previous R - 1 steps did not touch), one event pair around them; an
    # event between entry points costs a few microseconds of queue time, so
    # the throughput is timed without them.  Then the same with one batch
    # repeated (its lines stay warm in L2 and the MALL).
    wall0 = time.perf_counter()
    total_ms = timed_steps(torch, stream, K, rot, batches, fns)
    wall = time.perf_counter() - wall0
    repeat_ms = timed_steps(torch, stream, K, same, batches, fns)
    # Timed region 2: K more rotating steps with an event at every
    # entry-point boundary, for each entry point's time per launch.
    ph = timed_phases(torch, stream, K, rot, batches, fns)
    names = ("fc_retrieve", "fc_build_tree", "fc_verify_accept")
    phase_mean = {n: float(np.mean(v)) for n, v in zip(names, ph)}
    phase_med = {n: float(np.median(v)) for n, v in zip(names, ph)}

    # single-query latency (B = 1): one query's retrieve + tree + accept on
    # its own, event-timed, over the first batch's first queries
    lat = []
    if not args.no_latency:
        one = Batch(fc, torch, dev, qs[0][0][:1], qs[0][1][:1], len(stores), p, c)
        r1, t1f, v1 = make_pipeline(fc, torch, dev, stores, p, alpha, c, 1)
        for qi in range(min(64, B) + 3):
            one.ctx.copy_(batches[0].ctx[qi % B:qi % B + 1])
            one.target = batches[0].target[qi % B:qi % B + 1]
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            r1(one), t1f(one), v1(one)
            e1.record(stream)
            torch.cuda.synchronize()
            if qi >= 3:  # the first three warm up
                lat.append(e0.elapsed_time(e1))

    # byte models per batch, averaged over the launches of the timed rotation
    sizes = [len(t) for t in texts]
    per = []
    for bt in batches:
        per.append(algorithmic_bytes(bt.rout["taken"].cpu().numpy(), bt.rout["cont_len"].cpu().numpy(),
                                     bt.rout["match_n"].cpu().numpy(), n_hi_of(bt.ctx_np, p["n_max"]), sizes, k, m, c,
                                     p["n_min"]))
    w = np.bincount([rot(i) for i in range(K)], minlength=R) / K
    nb = {key: float(sum(w[r] * per[r][key] for r in range(R))) for key in per[0]}
    entry_bytes = {"fc_retrieve": nb["search"] + nb["io"] + nb["gather"], "fc_build_tree": nb["tree"],
                   "fc_verify_accept": nb["verify"]}
    traffic = measured_traffic(TRAFFIC_FILE)
    roofs = {}
    for name in names:
        ms = phase_mean[name]
        gbs = entry_bytes[name] / (ms * 1e-3) / 1e9
        t = traffic.get(name)
        roofs[name] = {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                       "frac": gbs / HBM_PEAK_GBS, "traffic": t, "kernel": name, "kernels": list(ENTRY_KERNELS[name]),
                       "algorithmic_bytes": entry_bytes[name], "us_per_launch": ms * 1e3,
                       "us_per_launch_median": phase_med[name] * 1e3,
                       "traffic_GBps": None if t is None else t / (ms * 1e-3) / 1e9}
    rr = roofs["fc_retrieve"]
    rr["byte_model"] = ("search: 2*ceil(log2(N_s+1))*(4+2n) per store and tried n; io: context 2L + 16 per store; "
                        "gather: 4 + 2*len read and 26 written per kept slot")
    rr["algorithmic_bytes_bucketed_search"] = nb["search_bucketed"] + nb["io"] + nb["gather"]
    rr["frac_bucketed_search"] = rr["algorithmic_bytes_bucketed_search"] / (phase_mean["fc_retrieve"] * 1e-3) / 1e9 / HBM_PEAK_GBS

    footprint = sum(bt.ctx.numel() * 2 + sum(v.numel() * v.element_size() for v in bt.rout.values())
                    + sum(v.numel() * v.element_size() for v in bt.tout.values()) for bt in batches)

    with_oracle = not args.no_cpu_baseline
    info = host_info() if with_oracle else None
    cpu = None
    if with_oracle:
        sec = oracle_batch(texts, batches[0].ctx_np, batches[0].nxt_np, p, alpha, c)
        cpu = {"value": B / sec, "unit": "retrievals/s", "cores": info["oracle_threads"], "kind": "oracle",
               "sample": f"the whole first batch ({B} queries: batched retrieval, tree, acceptance), {sec:.1f} s",
               "host": info}

    configs = None
    if not args.no_configs:
        configs = {}
        log("configuration 4: replay")
        configs["replay_128x4096"] = replay_config(args, fc, torch, synth, dev, stores, texts, p, with_oracle)
        del stores, batches
        torch.cuda.empty_cache()
        log("configuration 5: builds")
        configs["sa_build_1B_and_10M"] = build_config(args, fc, torch, synth, dev, dict(zip(roles, texts)), with_oracle)
        synth.drop_cache()
        del texts
        log("configuration 1")
        configs["single_1M"] = small_config(args, 1, fc, torch, synth, dev, p, c, with_oracle)
        log("configuration 2")
        configs["two_store_2M_100M"] = small_config(args, 2, fc, torch, synth, dev, p, c, with_oracle,
                                                    retrieve_bytes=True)
        synth.drop_cache()

    line = {
        "metric": "draft retrievals/sec (match+gather+trie) at 1B-token datastore; HBM GB/s vs peak",
        "value": B * K / (total_ms * 1e-3),
        "unit": "retrievals/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": total_ms / K,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u16/u32 (integer)",
        "data": "synthetic (seeded template/Zipf/noise token stores; no dataset)",
        "config": {"workload": synth.WORKLOADS[cfg]["name"], "stores_tokens": sizes, "batch": B,
                   "n_max": p["n_max"], "n_min": p["n_min"], "k": k, "m": m, "c": c, "alpha": list(alpha),
                   "parallelism": "none (1 GPU)", "batches_rotated": R},
        "cache_state": (f"value: steps cycle {R} distinct seeded batches, each with its own output buffers "
                        f"({footprint / 1e9:.2f} GB of contexts and outputs in the rotation, above the 256 MB MALL); "
                        "value_repeat_batch: one batch repeated (warm L2 and MALL)"),
        "value_repeat_batch": B * K / (repeat_ms * 1e-3),
        "ms_per_step_repeat_batch": repeat_ms / K,
        "roofline": roofs["fc_retrieve"],
        "roofline_by_entry": roofs,
        "cpu_baseline": cpu,
        "phases_ms": phase_mean,
        "phases_ms_median": phase_med,
        "single_query_latency_ms": None if not lat else {
            "median": float(np.median(lat)), "p90": float(np.percentile(lat, 90)), "queries": len(lat)},
        "ms_per_step_with_phase_events": float(sum(phase_mean.values())),
        "algorithmic_bytes_per_step": nb,
        "step_GBps_algorithmic": (nb["search"] + nb["io"] + nb["gather"] + nb["tree"] + nb["verify"])
        / (total_ms / K * 1e-3) / 1e9,
        "slots_kept_mean": nb["kept"] / B,
        "sa_build_s": build_s,
        "wall_s_timed": wall,
        "configs": configs,
    }
    print(json.dumps(line), flush=True)


def run_replay(args, cache: bool = False, control: bool = False):
    """Decode-trace replay: 128 streams of 4096 tokens drawn like the 10M-token
    project store, over the 10M + 1B stores, up to 512 steps, LRU(32).  With
    cache, each stream also keeps the CACHE of Section IV-B (activation at
    l = 50 sequences, output added every 20 tokens, Section V-D) and Alg. 1
    searches it first.  With control, Alg. 1's missing table and skip gate
    (p = 0.5) are on too; the synthetic streams have no line breaks, so the
    skip token is their most frequent token and the gate's draws come from
    the seeded generator."""
    import torch
    import paper_2502_17139_amd as fc
    import synth

    p = dict(synth.PARAMS)
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    texts = [synth.store(3, r) for r in synth.store_roles(3)]
    stores = [fc.Store(torch.from_numpy(t).to(dev), pair_vocab=synth.VOCAB, records=True) for t in texts]
    truth = synth.truth()
    ckw = dict(cache_l=50, cache_every=20) if cache else {}
    if control:
        tok = int(np.bincount(truth.ravel()).argmax())
        draws = np.stack([synth.uniform(31, 30, step, truth.shape[0], 0, 2 ** 31 - 1) for step in range(1024)])
        ckw.update(missing=True, skip_tok=tok, skip_p=0.5, skip_draws=draws)
    eng = fc.ReplayEngine(stores, torch.from_numpy(truth).to(dev), max_steps=512, **p, **ckw)
    eng.run(limit=args.warmup)  # warm-up steps; every run replays from the start
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    res = eng.run(limit=512)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    live = res["accept"] >= 0
    tokens = int(res["accept"][live].sum())
    line = {
        "metric": ("decode-trace replay with Alg. 1 (CACHE, missing table, skip gate) steps/sec (128 streams)"
                   if control else
                   "decode-trace replay with CACHE steps/sec (128 streams; CACHE or datastore retrieval + tree + "
                   "accept per step)" if cache else
                   "decode-trace replay steps/sec (128 streams; retrieve + tree + accept per step)"),
        "value": res["steps"] / wall, "unit": "steps/s", "n_gpus": 1, "steps": res["steps"], "warmup": args.warmup,
        "ms_per_step": 1e3 * wall / max(res["steps"], 1), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "u16/u32 (integer)",
        "data": "synthetic (seeded streams from the project pool; no dataset)",
        "config": {"workload": "replay over project 10M + general 1B" + (" with CACHE (l=50, every 20)" if cache else ""),
                   "streams": int(truth.shape[0]), "stream_len": int(truth.shape[1]), "lru": 32,
                   **{kk: p[kk] for kk in ("n_max", "n_min", "k", "m", "c")}},
        "roofline": None,
        "accepted_tokens_per_s": tokens / wall,
        "acc_len": res["acc_len"],
        "lru_hit_rate": float(res["hits"].sum() / max(res["lookups"].sum(), 1)),
        "retrievals": int(res["lookups"].sum() - res["hits"].sum()),
        "cache_served": int(res["cache_served"].sum()),
        "cache_served_share": float(res["cache_served"].sum() / max(res["cache_served"].sum() + res["lookups"].sum(), 1)),
        "missing_skips": int(res["missing_skips"].sum()),
        "gate_skips": int(res["gate_skips"].sum()),
    }
    print(json.dumps(line), flush=True)


def run_build(args):
    """Suffix-array construction of the 1B-token general store and the
    10M-token project store (plus both stores' first-token tables)."""
    import torch
    import paper_2502_17139_amd as fc
    import synth

    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    out = {}
    for role in ("project", "general"):
        t = synth.store(3, role)
        tok = torch.from_numpy(t).to(dev)
        sa = torch.empty(len(t), dtype=torch.uint32, device=dev)
        ws = torch.empty(fc.fc_datastore_build_workspace_bytes(len(t)), dtype=torch.uint8, device=dev)
        times = []
        for i in range(max(args.warmup, 1) + args.steps):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            fc.fc_datastore_build(tok, sa_out=sa, workspace=ws)
            torch.cuda.synchronize()
            if i >= max(args.warmup, 1):
                times.append(time.perf_counter() - t0)
        sec = float(np.median(times))
        n = len(t)
        # floor traffic of any build: read the text, write the array
        out[role] = {"tokens": n, "seconds": sec, "floor_GBps": (2 * n + 4 * n) / sec / 1e9}
        del ws, sa, tok
        torch.cuda.empty_cache()
    line = {
        "metric": "suffix-array build seconds (1B-token general store)", "value": out["general"]["seconds"],
        "unit": "s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": 1e3 * out["general"]["seconds"], "higher_is_better": False, "scaling": "weak",
        "vs_baseline": None, "dtype": "u16/u32/u64 (integer)", "data": "synthetic (seeded store; no dataset)",
        "config": {"workload": "SA build, 1B general + 10M project stores"}, "roofline": None, "builds": out,
    }
    print(json.dumps(line), flush=True)


def run_build_repos(args):
    """Per-repository stores: 64 repositories of 60..2000 files each
    (log-uniform, 16.9M tokens in all) built by one batched call, against one
    fc_datastore_build call per repository on the same stream."""
    import torch
    import paper_2502_17139_amd as fc
    import synth

    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    t, off = synth.repos(12, 64, 60, 2000)
    n, R = len(t), len(off) - 1
    tok = torch.from_numpy(t).to(dev)
    sa = torch.empty(n, dtype=torch.uint32, device=dev)
    ws = torch.empty(fc.fc_datastore_build_batched_workspace_bytes(n, R), dtype=torch.uint8, device=dev)
    lens = np.diff(off).astype(np.int64)

    def batched():
        fc.fc_datastore_build_batched(tok, off, sa_out=sa, workspace=ws)

    def per_repo():
        for r in range(R):
            a, b = int(off[r]), int(off[r + 1])
            if b > a:
                fc.fc_datastore_build(tok[a:b], sa_out=sa[a:b], workspace=ws)

    def timed(fn):
        times = []
        for i in range(max(args.warmup, 1) + args.steps):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            fn()
            torch.cuda.synchronize()
            if i >= max(args.warmup, 1):
                times.append(time.perf_counter() - t0)
        return float(np.median(times))

    sec_b = timed(batched)
    sec_p = timed(per_repo)
    line = {
        "metric": "per-repository store build seconds (64 repositories, batched)", "value": sec_b, "unit": "s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": 1e3 * sec_b,
        "higher_is_better": False, "scaling": "weak", "vs_baseline": None, "dtype": "u16/u32/u64 (integer)",
        "data": "synthetic (seeded repositories; no dataset)",
        "config": {"workload": "SA builds of 64 repositories, 60..2000 files, 16.9M tokens", "tokens": n,
                   "repositories": R, "smallest": int(lens.min()), "largest": int(lens.max())},
        "roofline": None,
        "per_repository_calls_s": sec_p, "speedup_vs_per_repository": sec_p / sec_b,
        "tokens_per_s": n / sec_b,
    }
    print(json.dumps(line), flush=True)


def run_extend(args):
    """New files in front of an existing store (fc_datastore_extend) against
    a full rebuild of the grown store: 1 and 200 new files on the 10M-token
    project store, 2,000 new files (1M tokens) on the 1B-token general store.
    The new files are the store's next files (same template pool, later file
    indexes), so they share its code; each case is timed with the inverse
    computed inside the call and with a kept inverse."""
    import torch
    import paper_2502_17139_amd as fc
    import synth

    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)

    def timed(fn):
        times = []
        for i in range(max(args.warmup, 1) + args.steps):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            fn()
            torch.cuda.synchronize()
            if i >= max(args.warmup, 1):
                times.append(time.perf_counter() - t0)
        return float(np.median(times))

    spec = {r: (seed, nt, zs, nf) for r, seed, nt, zs, nf in synth.WORKLOADS[3]["stores"]}
    cases = []
    for role, files in (("project", 1), ("project", 200), ("general", 2000)):
        seed, nt, zs, nf = spec[role]
        old = synth.store(3, role)
        new = synth.pool(seed, nt, zs).files(seed, nf, files, synth.FILE_LEN, sep=True)
        t = np.concatenate([new, np.zeros(1, np.uint16), old])
        n, n_new = len(t), len(new) + 1
        tt = torch.from_numpy(t).to(dev)
        old_sa = fc.fc_datastore_build(tt[n_new:])
        old_isa = torch.empty(n - n_new, dtype=torch.uint32, device=dev)
        fc.fc_datastore_extend(tt[n_new:], 0, old_sa, isa_out=old_isa)   # the old store's inverse
        sa = torch.empty(n, dtype=torch.uint32, device=dev)
        isa = torch.empty(n, dtype=torch.uint32, device=dev)
        ws = torch.empty(max(fc.fc_datastore_extend_workspace_bytes(n, n_new),
                             fc.fc_datastore_build_workspace_bytes(n)), dtype=torch.uint8, device=dev)
        sec_e = timed(lambda: fc.fc_datastore_extend(tt, n_new, old_sa, sa_out=sa, workspace=ws))
        sec_k = timed(lambda: fc.fc_datastore_extend(tt, n_new, old_sa, old_isa=old_isa, sa_out=sa, isa_out=isa,
                                                     workspace=ws))
        sec_b = timed(lambda: fc.fc_datastore_build(tt, sa_out=sa, workspace=ws))
        cases.append({"store": role, "old_tokens": n - n_new, "new_files": files, "new_tokens": n_new,
                      "extend_s": sec_e, "extend_kept_inverse_s": sec_k, "rebuild_s": sec_b,
                      "speedup": sec_b / sec_e, "speedup_kept_inverse": sec_b / sec_k})
        del tt, old_sa, old_isa, sa, isa, ws
        torch.cuda.empty_cache()
    big = cases[-1]
    line = {
        "metric": "store extension seconds (2,000 new files on the 1B-token store)", "value": big["extend_s"],
        "unit": "s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": 1e3 * big["extend_s"],
        "higher_is_better": False, "scaling": "weak", "vs_baseline": None, "dtype": "u16/u32/u64 (integer)",
        "data": "synthetic (seeded stores and their next files; no dataset)",
        "config": {"workload": "SA extension: new files in front of the 10M project and 1B general stores"},
        "roofline": None, "cases": cases,
    }
    print(json.dumps(line), flush=True)


def run_tree_attention(args):
    """One layer's attention step over 64 draft trees (the 1M-token
    workload's batch, c = 64, so 65 rows each) after a 2,048-token cached
    prefix, 32 heads of 128 dims (a 7B-class code model's attention shape),
    bf16 inputs from a seeded generator."""
    import torch
    import paper_2502_17139_amd as fc
    import synth

    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    p = dict(synth.PARAMS)
    t = synth.store(1, "single")
    ctx = torch.from_numpy(synth.queries(1)).to(dev)
    st = fc.Store(torch.from_numpy(t).to(dev), pair_vocab=synth.VOCAB, records=True)
    r = fc.fc_retrieve([st], ctx, n_max=p["n_max"], n_min=p["n_min"], k=p["k"], m=p["m"])
    tree = fc.fc_build_tree(r["taken"], r["cont_len"], r["cont_tok"], ctx, c=p["c"], alpha=(1,))
    B, R = tree["mask"].shape[0], tree["mask"].shape[1]
    H, Hkv, D, Pn = 32, 32, fc.FC_TREE_ATTN_HEAD_DIM, 2048
    gen = torch.Generator(device=dev)
    gen.manual_seed(5)
    rnd = lambda *shape: (torch.rand(*shape, generator=gen, device=dev) * 2 - 1).to(torch.bfloat16)  # noqa: E731
    q, kt, vt = rnd(B, R, H, D), rnd(B, R, Hkv, D), rnd(B, R, Hkv, D)
    kc, vc = rnd(B, Pn, Hkv, D), rnd(B, Pn, Hkv, D)
    prefix = torch.full((B,), Pn, dtype=torch.int32, device=dev)
    out = torch.empty((B, R, H, D), dtype=torch.float32, device=dev)
    run = lambda: fc.fc_tree_attention(q, kt, vt, kc, vc, prefix, tree, out=out)  # noqa: E731
    for _ in range(max(args.warmup, 1)):
        run()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    K = args.steps
    e0.record(stream)
    for _ in range(K):
        run()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / K
    nn = tree["num_nodes"].cpu().numpy()
    rows = int(nn.sum())
    # algorithmic bytes: each head reads its queries, its key/value head's
    # prefix and tree rows, the mask once per tree, and writes its outputs
    hb = R * D * 2 + (Pn + R) * D * 2 * 2 + R * D * 4
    byts = B * H * hb + B * R * R * 4 + B * R * 4
    flops = float(sum(4 * int(n) * (Pn + int(n)) * D for n in nn)) * H
    gbs = byts / (ms * 1e-3) / 1e9
    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        f64 = lambda x: x[:1].float().cpu().numpy().astype(np.float64)  # noqa: E731
        t0 = time.perf_counter()
        oracle.tree_attention(f64(q), f64(kt), f64(vt), f64(kc), f64(vc), np.array([Pn], np.int32), nn[:1],
                              tree["mask"][:1].cpu().numpy(), tree["pos_ids"][:1].cpu().numpy())
        spent = time.perf_counter() - t0
        cpu = {"value": int(nn[0]) * H / spent, "unit": "row-heads/s", "cores": 1, "kind": "oracle",
               "sample": f"tree 0 ({int(nn[0])} rows x {H} heads), {spent:.1f} s"}
    print(json.dumps({
        "metric": "tree-attention row-heads/sec (64 trees x 65 rows, 2,048-token prefix, 32 heads x 128)",
        "value": rows * H / (ms * 1e-3), "unit": "row-heads/s", "n_gpus": 1, "steps": K, "warmup": args.warmup,
        "ms_per_step": ms, "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded bf16 tensors; trees from the 1M-token workload)",
        "config": {"workload": "tree attention, 64 trees, prefix 2048, H 32, Hkv 32, D 128", "trees": B, "rows": R,
                   "prefix": Pn, "heads": H, "kv_heads": Hkv, "head_dim": D},
        "roofline": {"bound": "hbm", "kernel": "fc_tree_attention", "achieved": gbs, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": gbs / HBM_PEAK_GBS, "traffic": None,
                     "algorithmic_bytes": byts, "mfma_tflops": flops / (ms * 1e-3) / 1e12,
                     "mfma_frac_bf16": flops / (ms * 1e-3) / 2.5e15},
        "cpu_baseline": cpu,
    }), flush=True)


def run_gather_probe(args):
    """Known-bytes random reads for checking the traffic counters' scale on
    the access pattern of the retrieval: rows of 64 bytes (then 32 bytes) at
    uniformly random row indexes of a 64 GiB buffer, 4M rows per launch,
    gathered into a dense output.  Per launch it reads 8 bytes of index and
    one row per index, and writes one row per index."""
    import torch

    dev = torch.device("cuda", 0)
    span = 64 << 30
    buf = torch.empty(span // 4, dtype=torch.int32, device=dev)
    rows = 4 << 20
    gen = torch.Generator(device=dev)
    gen.manual_seed(11)
    out = {}
    for row_bytes in (64, 32):
        src = buf.view(-1, row_bytes // 4)
        idx = torch.randint(0, src.shape[0], (rows,), generator=gen, device=dev)
        dst = torch.empty((rows, row_bytes // 4), dtype=torch.int32, device=dev)
        for _ in range(max(args.warmup, 1)):
            torch.index_select(src, 0, idx, out=dst)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(args.steps):
            torch.index_select(src, 0, idx, out=dst)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / max(args.steps, 1)
        read = rows * (8 + row_bytes)
        out[f"rows_{row_bytes}B"] = {"rows": rows, "bytes_read": read, "bytes_written": rows * row_bytes,
                                     "us_per_launch": ms * 1e3,
                                     "GBps": (read + rows * row_bytes) / (ms * 1e-3) / 1e9}
    print(json.dumps({"metric": "random row gather over a 64 GiB buffer (known bytes per launch)", "cases": out,
                      "steps": args.steps, "warmup": args.warmup, "n_gpus": 1}), flush=True)


def run_copy(args):
    """A plain device-to-device copy of 1 GiB: the reference for scaling
    hardware traffic counters to bytes."""
    import torch

    dev = torch.device("cuda", 0)
    src = torch.ones(1 << 30, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    for _ in range(args.warmup):
        dst.copy_(src)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        dst.copy_(src)
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / max(args.steps, 1)
    print(json.dumps({"metric": "device copy GB/s (1 GiB read + 1 GiB written per copy)", "value": 2 * (1 << 30) / dt / 1e9,
                      "unit": "GB/s", "bytes_read_per_copy": 1 << 30, "bytes_written_per_copy": 1 << 30,
                      "steps": args.steps, "warmup": args.warmup, "n_gpus": 1}), flush=True)


if __name__ == "__main__":
    main()
