"""Seeded synthetic inputs shared by the oracle's tests, the GPU path's tests
and the benchmark.

The paper's datastores are built from code files: a common store from a
subset of The Stack and a repository store from the current project's files
(Section IV-A, Section V-D).  Neither corpus is available here, so stores are
made of template n-grams drawn with Zipf reuse plus 10% token noise, which
gives the repeated-n-gram ("localness") structure the method relies on
(Section III-B).  Tokens are uint16, the vocabulary is 32256 ids, token 0
separates files.

This module holds no part of the retrieval method; it only produces inputs.
The C core (gen.c) is built by :func:`build` with gcc.
"""
from __future__ import annotations

import ctypes
import functools
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libsynth.so")

VOCAB = 32256
FILE_LEN = 500
CTX_LEN = 16

# Stream roles used from Python (gen.c owns roles 1-3).
ROLE_QUERY = 10
ROLE_SHUFFLE = 11
ROLE_FRESH = 12
ROLE_REPOS = 13

# Synthetic workloads by size.  A store is (seed, n_templates, zipf_s, n_files).
WORKLOADS = {
    1: dict(name="single-source 1M", stores=[("single", 0, 5000, 1.2, 2000)],
            qseed=0, batch=64, project_share=None),
    2: dict(name="project 2M + general 100M",
            stores=[("project", 1, 500, 1.2, 4000), ("general", 2, 200_000, 1.2, 200_000)],
            qseed=3, batch=256, project_share=0.7),
    3: dict(name="project 10M + general 1B",
            stores=[("project", 5, 2000, 1.2, 20_000), ("general", 4, 2_000_000, 1.1, 2_000_000)],
            qseed=6, batch=1024, project_share=0.7),
}
# Retrieval and tree parameters shared by every configuration.
PARAMS = dict(n_max=16, n_min=2, k=5000, m=10, c=64, alpha=(1, 1))
NOISE = 0.1
TEMPLATE_LEN = (4, 32)
TRUTH = dict(seed=7, n_seq=128, length=4096, pool=("project", 5, 2000, 1.2))


def build() -> None:
    """Compile gen.c into libsynth.so (gcc, OpenMP)."""
    src = os.path.join(_HERE, "gen.c")
    tmp = _LIB_PATH + ".tmp"
    subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-o", tmp, src, "-lm"])
    os.replace(tmp, _LIB_PATH)


@functools.lru_cache(maxsize=1)
def _lib():
    if not os.path.exists(_LIB_PATH):
        build()
    lib = ctypes.CDLL(_LIB_PATH)
    u64, u32, i32, dbl, vp = ctypes.c_uint64, ctypes.c_uint32, ctypes.c_int, ctypes.c_double, ctypes.c_void_p
    lib.synth_stream_key.restype = u64
    lib.synth_stream_key.argtypes = [u64, u64, u64]
    lib.synth_pool_lengths.restype = u64
    lib.synth_pool_lengths.argtypes = [u64, u64, u32, u32, vp]
    lib.synth_pool_tokens.restype = None
    lib.synth_pool_tokens.argtypes = [u64, u64, u32, vp, vp]
    lib.synth_zipf_table.restype = None
    lib.synth_zipf_table.argtypes = [u64, dbl, vp]
    lib.synth_files.restype = None
    lib.synth_files.argtypes = [vp, vp, u64, vp, dbl, u32, u64, u64, u64, u32, i32, vp]
    lib.synth_uniform.restype = None
    lib.synth_uniform.argtypes = [u64, u64, u64, u64, u32, u32, vp]
    return lib


def _ptr(a: np.ndarray) -> ctypes.c_void_p:
    return ctypes.c_void_p(a.ctypes.data)


class Pool:
    """A template pool with its Zipf table."""

    def __init__(self, seed: int, n_templates: int, zipf_s: float, vocab: int = VOCAB):
        lib = _lib()
        self.seed, self.n_templates, self.zipf_s, self.vocab = seed, n_templates, zipf_s, vocab
        self.offsets = np.empty(n_templates + 1, dtype=np.uint64)
        total = lib.synth_pool_lengths(seed, n_templates, TEMPLATE_LEN[0], TEMPLATE_LEN[1], _ptr(self.offsets))
        self.tokens = np.empty(max(total, 1), dtype=np.uint16)
        lib.synth_pool_tokens(seed, n_templates, vocab, _ptr(self.offsets), _ptr(self.tokens))
        self.cum = np.empty(n_templates, dtype=np.float64)
        lib.synth_zipf_table(n_templates, zipf_s, _ptr(self.cum))

    def files(self, file_seed: int, first_index: int, n_files: int, file_len: int, sep: bool,
              noise: float = NOISE) -> np.ndarray:
        n = n_files * file_len + (n_files - 1 if sep and n_files > 0 else 0)
        out = np.empty(max(n, 1), dtype=np.uint16)
        _lib().synth_files(_ptr(self.offsets), _ptr(self.tokens), self.n_templates, _ptr(self.cum), noise,
                           self.vocab, file_seed, first_index, n_files, file_len, 1 if sep else 0, _ptr(out))
        return out[:n]


def uniform(seed: int, role: int, index: int, n: int, lo: int, hi: int) -> np.ndarray:
    out = np.empty(max(n, 1), dtype=np.uint32)
    _lib().synth_uniform(seed, role, index, n, lo, hi, _ptr(out))
    return out[:n]


@functools.lru_cache(maxsize=4)
def pool(seed: int, n_templates: int, zipf_s: float) -> Pool:
    return Pool(seed, n_templates, zipf_s)


def make_store(seed: int, n_templates: int, zipf_s: float, n_files: int) -> np.ndarray:
    """Files of FILE_LEN tokens from pool `seed`, joined by single 0 tokens."""
    return pool(seed, n_templates, zipf_s).files(seed, 0, n_files, FILE_LEN, sep=True)


_STORE_CACHE: dict = {}


def store(cfg: int, role: str) -> np.ndarray:
    """The store named `role` ('single', 'project' or 'general') of a configuration."""
    key = (cfg, role)
    if key not in _STORE_CACHE:
        for r, seed, nt, s, nf in WORKLOADS[cfg]["stores"]:
            if r == role:
                _STORE_CACHE[key] = make_store(seed, nt, s, nf)
                break
        else:
            raise KeyError(f"config {cfg} has no store {role!r}")
    return _STORE_CACHE[key]


def store_roles(cfg: int) -> list:
    """Store roles of a configuration in priority order (project first)."""
    return [r for r, *_ in WORKLOADS[cfg]["stores"]]


def drop_cache() -> None:
    _STORE_CACHE.clear()


def _window_random(text_files: int, qseed: int, q: int, src_text: np.ndarray, extra: int) -> np.ndarray:
    f, off = uniform(qseed, ROLE_QUERY, q, 2, 0, 0x7FFFFFFF)
    f = int(f) % text_files
    off = int(off) % (FILE_LEN - CTX_LEN + 1)
    start = f * (FILE_LEN + 1) + off
    w = src_text[start:start + CTX_LEN + extra]
    return np.concatenate([w, np.zeros(CTX_LEN + extra - len(w), np.uint16)])


def _window_fresh(p: Pool, qseed: int, q: int, extra: int) -> np.ndarray:
    text = p.files(qseed + 1_000_003, 1_000_000_000 + q, 1, FILE_LEN + extra, sep=False)
    off = int(uniform(qseed, ROLE_FRESH, q, 1, 0, FILE_LEN - CTX_LEN)[0])
    return text[off:off + CTX_LEN + extra].copy()


def query_seed(cfg: int, rotation: int = 0) -> int:
    """Seed of a configuration's query batch; rotation r > 0 names the r-th
    further batch drawn the same way (distinct windows of the same stores),
    for timing over batches that do not repeat."""
    return WORKLOADS[cfg]["qseed"] + 1_000_033 * rotation


def query_plan(cfg: int, rotation: int = 0) -> list:
    """(kind, role) of every query, in batch order.

    kind is 'random' (a 16-token window at a uniform file and offset of the
    store) or 'fresh' (a window of a newly drawn file from the same pool:
    unseen text from the same distribution).  Two-source batches draw
    `project_share` of the queries from the project store's pool, the rest
    from the general store's; each group is half random, half fresh.  The
    order is a seeded shuffle.
    """
    c = WORKLOADS[cfg]
    b = c["batch"]
    if c["project_share"] is None:
        groups = [(store_roles(cfg)[0], b)]
    else:
        n_proj = (int(round(c["project_share"] * 10)) * b + 5) // 10
        groups = [("project", n_proj), ("general", b - n_proj)]
    plan = []
    for role, g in groups:
        n_rand = (g + 1) // 2
        plan += [("random", role)] * n_rand + [("fresh", role)] * (g - n_rand)
    # Fisher-Yates with the configuration's shuffle stream.
    r = uniform(query_seed(cfg, rotation), ROLE_SHUFFLE, 0, len(plan), 0, 0x7FFFFFFF)
    for i in range(len(plan) - 1, 0, -1):
        j = int(r[i]) % (i + 1)
        plan[i], plan[j] = plan[j], plan[i]
    return plan


def queries(cfg: int, count: int | None = None, next_tokens: int = 0, rotation: int = 0):
    """Query contexts, uint16 [B][16] (the first `count` of the batch if given;
    batch `rotation` of the configuration, see query_seed).

    With next_tokens > 0 also returns the tokens that truly follow each
    window, uint16 [B][next_tokens] (the store's own text for a random
    window, 0-padded at the end of the store; the fresh file's continuation
    for a fresh one): the ground truth a target model would reproduce.
    """
    c = WORKLOADS[cfg]
    plan = query_plan(cfg, rotation)
    if count is not None:
        plan = plan[:count]
    qseed = query_seed(cfg, rotation)
    stores = {r: (seed, nt, s, nf) for r, seed, nt, s, nf in c["stores"]}
    out = np.empty((len(plan), CTX_LEN + next_tokens), dtype=np.uint16)
    for q, (kind, role) in enumerate(plan):
        seed, nt, s, nf = stores[role]
        if kind == "random":
            out[q] = _window_random(nf, qseed, q, store(cfg, role), next_tokens)
        else:
            out[q] = _window_fresh(pool(seed, nt, s), qseed, q, next_tokens)
    if next_tokens:
        return np.ascontiguousarray(out[:, :CTX_LEN]), np.ascontiguousarray(out[:, CTX_LEN:])
    return out


def truth(n_seq: int | None = None, length: int | None = None) -> np.ndarray:
    """Ground-truth token streams for decode-trace replay, uint16 [n_seq][length].

    Drawn like the 10M-token project store (same pool and Zipf exponent) but
    from their own file streams and without separators.
    """
    t = TRUTH
    n_seq = t["n_seq"] if n_seq is None else n_seq
    length = t["length"] if length is None else length
    _, seed, nt, s = t["pool"]
    flat = pool(seed, nt, s).files(t["seed"], 0, n_seq, length, sep=False)
    return flat.reshape(n_seq, length)


def repos(seed: int, n_repos: int, min_files: int, max_files: int, n_templates: int = 2000,
          zipf_s: float = 1.2) -> tuple:
    """Many per-repository stores laid back to back: repository r holds a
    log-uniform number of files in [min_files, max_files] (FILE_LEN tokens
    each, joined by 0 tokens), drawn from one template pool shared by every
    repository (common library code), each with its own file seed.  Returns
    (tokens, offsets) with repository r at tokens[offsets[r]:offsets[r+1]]."""
    u = uniform(seed, ROLE_REPOS, 0, n_repos, 0, 999_999).astype(np.float64) / 1e6
    lo, hi = np.log(min_files), np.log(max_files + 1)
    n_files = np.minimum(np.exp(lo + u * (hi - lo)).astype(np.int64), max_files)
    p = pool(seed, n_templates, zipf_s)
    parts = [p.files(seed * 1_000_003 + r, 0, int(f), FILE_LEN, sep=True) for r, f in enumerate(n_files)]
    off = np.zeros(n_repos + 1, np.uint64)
    off[1:] = np.cumsum([len(x) for x in parts])
    return (np.concatenate(parts) if parts else np.zeros(0, np.uint16)), off


def random_text(seed: int, n: int, vocab: int, sep_prob: float = 0.0) -> np.ndarray:
    """Uniform tokens in [1, vocab-1] with each position a 0 separator with
    probability sep_prob; for small adversarial tests (tiny vocabularies make
    long repeats and many ties)."""
    toks = uniform(seed, 20, 0, n, 1, max(vocab - 1, 1)).astype(np.uint16)
    if sep_prob > 0:
        u = uniform(seed, 21, 0, n, 0, 999_999)
        toks[u < int(sep_prob * 1_000_000)] = 0
    return toks
