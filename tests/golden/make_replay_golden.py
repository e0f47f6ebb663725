#!/usr/bin/env python3
"""Writes tests/golden/replay_10M_1B_128x512.json: the oracle's decode-trace
replay over the 10M-token project store and the 1B-token general store, 128
streams of 4,096 tokens, 512 steps, LRU of 32 (Section V-C, eq. (7)).

Only the oracle and the seeded generator are called.  The file records the
SHA-256 of every input (both stores, the streams) and the parameters, so a
test can tell that it compares against the same inputs.  Each stream's
accepted lengths are one character per step: the length in base 36, '.'
once the stream has ended.

Takes about 40 minutes on 8 CPU cores (two passes over the 1B-token store
per step).
"""
from __future__ import annotations

import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import oracle  # noqa: E402
import synth  # noqa: E402

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "replay_10M_1B_128x512.json")
DIGITS = "0123456789abcdefghijklmnopqrstuvwxyz"


def sha(a: np.ndarray) -> str:
    return hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()


def encode(col: np.ndarray) -> str:
    return "".join("." if int(v) < 0 else DIGITS[int(v)] for v in col)


def main() -> None:
    p = dict(synth.PARAMS)
    t0 = time.time()
    tp, tg = synth.store(3, "project"), synth.store(3, "general")
    truth = synth.truth()
    print(f"inputs in {time.time() - t0:.1f} s", flush=True)
    t0 = time.time()
    r = oracle.replay([tp, tg], truth, **p, lru=32, max_steps=512)
    print(f"replay in {time.time() - t0:.1f} s, {r['steps']} steps, AccLen {r['acc_len']:.4f}", flush=True)
    out = {
        "what": "oracle decode-trace replay, project 10M + general 1B, 128 streams x 4096 tokens, 512 steps, LRU 32",
        "sha256": {"project": sha(tp), "general": sha(tg), "truth": sha(truth)},
        "params": {kk: (list(v) if isinstance(v, tuple) else v) for kk, v in p.items()},
        "lru": 32, "max_steps": 512, "steps": int(r["steps"]), "acc_len": r["acc_len"],
        "hits": r["hits"].tolist(), "lookups": r["lookups"].tolist(), "pos": r["pos"].tolist(),
        "accept": [encode(r["accept"][:, b]) for b in range(truth.shape[0])],
    }
    with open(OUT, "w") as f:
        json.dump(out, f, indent=0)
        f.write("\n")
    print("wrote", OUT, flush=True)


if __name__ == "__main__":
    main()
