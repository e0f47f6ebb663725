"""MI355X (gfx950) draft-stage retrieval library for retrieval-based
speculative decoding after FastCoder (arXiv 2502.17139).

The compute lives in libfastcoder.so (hand-written HIP kernels behind the C
ABI of include/fastcoder.h).  This module is the thin Python binding: the
functions carry the C entry points' names, take torch tensors on the GPU for
device memory and the current torch stream for ordering, and only marshal
arguments.  There is no CPU path: without the built library every call
raises.
"""
from __future__ import annotations

import ctypes
import functools
import os

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libfastcoder.so")

FC_MAX_SOURCES = 4
FC_MAX_NMAX = 16
FC_MAX_TREE_ROWS = 256
FC_BUCKETS = 65537
FC_MAX_CACHE_TOKENS = 16384
FC_TREE_ATTN_HEAD_DIM = 128

STATUS = {0: "FC_OK", 1: "FC_ERR_INVALID", 2: "FC_ERR_WORKSPACE", 3: "FC_ERR_DEVICE", 4: "FC_ERR_UNSUPPORTED"}

# Names of every entry point the header declares.
EXPORTS = (
    "fc_abi_version", "fc_status_string",
    "fc_datastore_build_workspace_bytes", "fc_datastore_build", "fc_datastore_build_batched_workspace_bytes",
    "fc_datastore_build_batched", "fc_datastore_extend_workspace_bytes", "fc_datastore_extend", "fc_store_prepare",
    "fc_pair_table_entries", "fc_store_prepare_pairs", "fc_record_bytes", "fc_store_prepare_records",
    "fc_store_top_bytes", "fc_store_prepare_top",
    "fc_retrieve_workspace_bytes", "fc_retrieve", "fc_build_tree_workspace_bytes", "fc_build_tree",
    "fc_verify_accept", "fc_targets_from_truth", "fc_cache_lds_bytes", "fc_cache_retrieve", "fc_cache_write",
    "fc_tree_attention", "fc_replay_init", "fc_replay_run", "fc_retrieve_noalloc_max_bytes", "fc_retrieve_noalloc",
    "fc_datastore_build_stats",
)


class FcError(RuntimeError):
    """A non-OK status from the library."""

    def __init__(self, fn: str, code: int, text: str):
        super().__init__(f"{fn} failed: {text}")
        self.code = code


class FcStore(ctypes.Structure):
    _fields_ = [("tokens", ctypes.c_void_p), ("sa", ctypes.c_void_p), ("bucket", ctypes.c_void_p),
                ("n", ctypes.c_uint64), ("pair", ctypes.c_void_p), ("pair_vocab", ctypes.c_uint32),
                ("rec", ctypes.c_void_p), ("top", ctypes.c_void_p)]


FC_MAX_BUILD_ROUNDS = 40


class FcBuildStats(ctypes.Structure):
    _fields_ = [("rounds", ctypes.c_int32), ("sort_passes", ctypes.c_int32),
                ("prefix_len", ctypes.c_uint64 * FC_MAX_BUILD_ROUNDS), ("sorted", ctypes.c_uint64 * FC_MAX_BUILD_ROUNDS),
                ("unresolved", ctypes.c_uint64 * FC_MAX_BUILD_ROUNDS)]


class FcRetrieveParams(ctypes.Structure):
    _fields_ = [("n_max", ctypes.c_int32), ("n_min", ctypes.c_int32), ("k", ctypes.c_int32), ("m", ctypes.c_int32)]


class FcTreeParams(ctypes.Structure):
    _fields_ = [("c", ctypes.c_int32), ("alpha", ctypes.c_uint32 * FC_MAX_SOURCES)]


_P = ctypes.c_void_p


class FcReplay(ctypes.Structure):
    _fields_ = [("truth", _P), ("truth_stride", ctypes.c_int64), ("truth_len", ctypes.c_int32),
                ("n_streams", ctypes.c_int32), ("ctx_len", ctypes.c_int32), ("lru", ctypes.c_int32),
                ("max_steps", ctypes.c_int32), ("rp", FcRetrieveParams), ("tp", FcTreeParams)] + [
        (f, _P) for f in ("pos", "lru_key", "lru_used", "lru_count", "hits", "lookups", "ctx", "rows_retrieve",
                          "rows_tree", "live", "history", "match_n", "range_lo", "range_cnt", "taken", "cont_pos",
                          "cont_src", "cont_len", "cont_tok", "retrieve_ws")] + [
        ("retrieve_ws_bytes", ctypes.c_size_t)] + [
        (f, _P) for f in ("num_nodes", "node_tok", "parent", "weight", "pos_ids", "mask", "tree_ws")] + [
        ("tree_ws_bytes", ctypes.c_size_t)] + [
        (f, _P) for f in ("target", "accept_len", "accept_tok", "last_node")] + [
        (f, ctypes.c_int32) for f in ("cache_l", "cache_every", "cache_cap", "max_seqs")] + [
        (f, _P) for f in ("ctext", "clen", "seq_len", "seq_head", "seq_count", "chunks", "served", "rows_cache",
                          "state", "c_match_n", "c_range_lo", "c_range_cnt", "c_taken", "c_cont_pos", "c_cont_src",
                          "c_cont_len", "c_cont_tok", "c_num_nodes", "c_node_tok", "c_parent", "c_weight",
                          "c_pos_ids", "c_mask")] + [
        ("missing", ctypes.c_int32), ("miss_cap", ctypes.c_int32), ("miss_key", _P), ("miss_used", _P),
        ("m_skips", _P), ("skip_tok", ctypes.c_int32), ("skip_thr", ctypes.c_uint32), ("skip_draws", _P),
        ("g_skips", _P)]


@functools.lru_cache(maxsize=1)
def lib() -> ctypes.CDLL:
    """Load libfastcoder.so (torch is imported first so its HIP runtime is the
    one the library binds to)."""
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                           "(hipcc --offload-arch=gfx950); there is no CPU fallback")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, u32, u64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_size_t
    L.fc_abi_version.restype = i32
    L.fc_abi_version.argtypes = []
    L.fc_status_string.restype = ctypes.c_char_p
    L.fc_status_string.argtypes = [ctypes.c_int]
    L.fc_datastore_build_workspace_bytes.restype = sz
    L.fc_datastore_build_workspace_bytes.argtypes = [u64]
    L.fc_datastore_build.restype = ctypes.c_int
    L.fc_datastore_build.argtypes = [vp, u64, vp, vp, sz, vp]
    L.fc_datastore_build_stats.restype = ctypes.c_int
    L.fc_datastore_build_stats.argtypes = [vp, u64, vp, vp, sz, ctypes.POINTER(FcBuildStats), vp]
    L.fc_datastore_build_batched_workspace_bytes.restype = sz
    L.fc_datastore_build_batched_workspace_bytes.argtypes = [u64, i32]
    L.fc_datastore_build_batched.restype = ctypes.c_int
    L.fc_datastore_build_batched.argtypes = [vp, vp, i32, vp, vp, sz, vp]
    L.fc_datastore_extend_workspace_bytes.restype = sz
    L.fc_datastore_extend_workspace_bytes.argtypes = [u64, u64, i32]
    L.fc_datastore_extend.restype = ctypes.c_int
    L.fc_datastore_extend.argtypes = [vp, u64, u64, vp, vp, vp, vp, vp, sz, vp]
    L.fc_store_prepare.restype = ctypes.c_int
    L.fc_store_prepare.argtypes = [vp, vp, u64, vp, vp]
    L.fc_pair_table_entries.restype = u64
    L.fc_pair_table_entries.argtypes = [u32]
    L.fc_store_prepare_pairs.restype = ctypes.c_int
    L.fc_store_prepare_pairs.argtypes = [vp, vp, u64, u32, vp, vp]
    L.fc_record_bytes.restype = u64
    L.fc_record_bytes.argtypes = [u64]
    L.fc_store_prepare_records.restype = ctypes.c_int
    L.fc_store_prepare_records.argtypes = [vp, vp, u64, vp, vp]
    L.fc_store_top_bytes.restype = u64
    L.fc_store_top_bytes.argtypes = [u64]
    L.fc_store_prepare_top.restype = ctypes.c_int
    L.fc_store_prepare_top.argtypes = [vp, u64, vp, vp]
    L.fc_retrieve_workspace_bytes.restype = sz
    L.fc_retrieve_workspace_bytes.argtypes = [i32, i32, FcRetrieveParams]
    L.fc_retrieve.restype = ctypes.c_int
    L.fc_retrieve.argtypes = [ctypes.POINTER(FcStore), i32, vp, i32, i32, FcRetrieveParams,
                              vp, vp, vp, vp, vp, vp, vp, vp, vp, i32, vp, sz, vp]
    L.fc_retrieve_noalloc_max_bytes.restype = sz
    L.fc_retrieve_noalloc_max_bytes.argtypes = []
    L.fc_retrieve_noalloc.restype = ctypes.c_int
    L.fc_retrieve_noalloc.argtypes = [ctypes.POINTER(FcStore), i32, vp, i32, i32, FcRetrieveParams,
                                      vp, vp, vp, vp, vp, vp, vp, vp, vp, i32, vp]
    L.fc_cache_lds_bytes.restype = sz
    L.fc_cache_lds_bytes.argtypes = [ctypes.c_int64]
    L.fc_cache_retrieve.restype = ctypes.c_int
    L.fc_cache_retrieve.argtypes = [vp, ctypes.c_int64, i32, vp, vp, vp, i32, i32, FcRetrieveParams,
                                    vp, vp, vp, vp, vp, vp, vp, vp, vp, i32, vp]
    L.fc_cache_write.restype = ctypes.c_int
    L.fc_cache_write.argtypes = [vp, ctypes.c_int64, i32, vp, i32, vp, vp, vp, vp, vp, vp, vp]
    L.fc_tree_attention.restype = ctypes.c_int
    L.fc_tree_attention.argtypes = [vp] * 9 + [i32] * 6 + [ctypes.c_float, vp, vp]
    L.fc_build_tree_workspace_bytes.restype = sz
    L.fc_build_tree_workspace_bytes.argtypes = [i32]
    L.fc_build_tree.restype = ctypes.c_int
    L.fc_build_tree.argtypes = [vp, vp, vp, vp, i32, i32, i32, i32, i32, FcTreeParams,
                                vp, vp, vp, vp, vp, vp, vp, i32, vp, sz, vp]
    L.fc_verify_accept.restype = ctypes.c_int
    L.fc_verify_accept.argtypes = [vp, vp, vp, vp, vp, i32, i32, i32, vp, vp, vp, vp]
    L.fc_replay_init.restype = ctypes.c_int
    L.fc_replay_init.argtypes = [ctypes.POINTER(FcReplay), vp]
    L.fc_replay_run.restype = ctypes.c_int
    L.fc_replay_run.argtypes = [ctypes.POINTER(FcStore), i32, ctypes.POINTER(FcReplay), i32, i32, vp]
    L.fc_targets_from_truth.restype = ctypes.c_int
    L.fc_targets_from_truth.argtypes = [vp, i32, ctypes.c_int64, vp, vp, vp, vp, i32, i32, vp, vp]
    return L


def _check(fn: str, code: int) -> None:
    if code != 0:
        raise FcError(fn, code, lib().fc_status_string(code).decode())


def _ptr(t: torch.Tensor | None) -> ctypes.c_void_p:
    if t is None:
        return ctypes.c_void_p(0)
    if not t.is_cuda:
        raise ValueError("device tensor expected")
    if not t.is_contiguous():
        raise ValueError("contiguous tensor expected")
    return ctypes.c_void_p(t.data_ptr())


def _expect(name: str, t: torch.Tensor | None, dtype, shape=None, optional: bool = False) -> None:
    """The library trusts the sizes it is given, so a tensor of the wrong
    type or shape is refused here, before any launch."""
    if t is None:
        if optional:
            return
        raise ValueError(f"{name} is required")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, not {t.dtype}")
    if shape is not None and t.shape != shape:
        raise ValueError(f"{name} must have shape {tuple(int(x) for x in shape)}, not {tuple(t.shape)}")


def _expect_outputs(out: dict, fields, shapes: dict, dtypes: dict) -> None:
    for f in fields:
        _expect(f, out.get(f), dtypes[f], shapes[f])


_RETRIEVE_DTYPES = dict(match_n=torch.int32, range_lo=torch.uint32, range_cnt=torch.uint32, taken=torch.int32,
                        cont_pos=torch.uint32, cont_src=torch.uint8, cont_len=torch.uint8, cont_tok=torch.uint16)


def _retrieve_shapes(n_rows: int, S: int, k: int, m: int) -> dict:
    return dict(match_n=(n_rows, S), range_lo=(n_rows, S), range_cnt=(n_rows, S), taken=(n_rows, S),
                cont_pos=(n_rows, k), cont_src=(n_rows, k), cont_len=(n_rows, k), cont_tok=(n_rows, k, m))


def _stream(stream) -> ctypes.c_void_p:
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _empty(shape, dtype, device) -> torch.Tensor:
    return torch.empty(shape, dtype=dtype, device=device)


# ---------------------------------------------------------------- index ----

def fc_datastore_build_workspace_bytes(n: int) -> int:
    return int(lib().fc_datastore_build_workspace_bytes(n))


def fc_datastore_build_batched_workspace_bytes(n: int, n_seg: int) -> int:
    return int(lib().fc_datastore_build_batched_workspace_bytes(n, n_seg))


def fc_datastore_build(tokens: torch.Tensor, sa_out: torch.Tensor | None = None,
                       workspace: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Suffix array (uint32[n]) of a uint16 token tensor on the GPU."""
    if tokens.dtype != torch.uint16 or tokens.dim() != 1:
        raise ValueError("tokens must be a 1-D uint16 tensor")
    n = tokens.numel()
    if sa_out is None:
        sa_out = _empty(n, torch.uint32, tokens.device)
    need = fc_datastore_build_workspace_bytes(n)
    if workspace is None:
        workspace = _empty(max(need, 1), torch.uint8, tokens.device)
    _check("fc_datastore_build", lib().fc_datastore_build(_ptr(tokens), n, _ptr(sa_out), _ptr(workspace),
                                                         workspace.numel(), _stream(stream)))
    return sa_out


def fc_datastore_build_stats(tokens: torch.Tensor, sa_out: torch.Tensor | None = None,
                             workspace: torch.Tensor | None = None, stream=None) -> tuple:
    """fc_datastore_build that also returns the doubling rounds: (sa, dict of
    rounds, sort_passes and per-round prefix_len, sorted, unresolved)."""
    if tokens.dtype != torch.uint16 or tokens.dim() != 1:
        raise ValueError("tokens must be a 1-D uint16 tensor")
    n = tokens.numel()
    if sa_out is None:
        sa_out = _empty(n, torch.uint32, tokens.device)
    need = fc_datastore_build_workspace_bytes(n)
    if workspace is None:
        workspace = _empty(max(need, 1), torch.uint8, tokens.device)
    st = FcBuildStats()
    _check("fc_datastore_build_stats", lib().fc_datastore_build_stats(
        _ptr(tokens), n, _ptr(sa_out), _ptr(workspace), workspace.numel(), ctypes.byref(st), _stream(stream)))
    r = int(st.rounds)
    return sa_out, dict(rounds=r, sort_passes=int(st.sort_passes), prefix_len=list(st.prefix_len[:r]),
                        sorted=list(st.sorted[:r]), unresolved=list(st.unresolved[:r]))


def fc_datastore_build_batched(tokens: torch.Tensor, seg_off, sa_out: torch.Tensor | None = None,
                               workspace: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Suffix arrays of many stores laid back to back in `tokens` (store r
    at [seg_off[r], seg_off[r+1])), each local to its store, in one build."""
    if tokens.dtype != torch.uint16 or tokens.dim() != 1:
        raise ValueError("tokens must be a 1-D uint16 tensor")
    off = np.ascontiguousarray(seg_off, dtype=np.uint64)
    R = len(off) - 1
    n = tokens.numel()
    if sa_out is None:
        sa_out = _empty(n, torch.uint32, tokens.device)
    need = fc_datastore_build_batched_workspace_bytes(n, R) if R >= 1 else 0
    if workspace is None:
        workspace = _empty(max(need, 1), torch.uint8, tokens.device)
    _check("fc_datastore_build_batched", lib().fc_datastore_build_batched(
        _ptr(tokens), ctypes.c_void_p(off.ctypes.data), R, _ptr(sa_out), _ptr(workspace), workspace.numel(),
        _stream(stream)))
    return sa_out


def fc_datastore_extend_workspace_bytes(n: int, n_new: int, isa_given: bool = False) -> int:
    return int(lib().fc_datastore_extend_workspace_bytes(n, n_new, 1 if isa_given else 0))


def fc_datastore_extend(tokens: torch.Tensor, n_new: int, old_sa: torch.Tensor, old_isa: torch.Tensor | None = None,
                        sa_out: torch.Tensor | None = None, isa_out: torch.Tensor | None = None,
                        workspace: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Suffix array of tokens = new (n_new tokens, ending with the joining 0)
    followed by an old store whose suffix array is old_sa (and, optionally,
    whose inverse is old_isa); isa_out, if given, receives the new inverse."""
    if tokens.dtype != torch.uint16 or tokens.dim() != 1:
        raise ValueError("tokens must be a 1-D uint16 tensor")
    n = tokens.numel()
    for name, t in (("old_sa", old_sa), ("old_isa", old_isa)):
        if t is not None and (t.dtype != torch.uint32 or t.numel() != n - n_new):
            raise ValueError(f"{name} must be a uint32 tensor of n - n_new entries")
    if sa_out is None:
        sa_out = _empty(n, torch.uint32, tokens.device)
    if workspace is None:
        need = fc_datastore_extend_workspace_bytes(n, n_new, old_isa is not None)
        workspace = _empty(max(need, 1), torch.uint8, tokens.device)
    _check("fc_datastore_extend", lib().fc_datastore_extend(
        _ptr(tokens), n, n_new, _ptr(old_sa), _ptr(old_isa), _ptr(sa_out), _ptr(isa_out), _ptr(workspace),
        workspace.numel(), _stream(stream)))
    return sa_out


def fc_store_prepare(tokens: torch.Tensor, sa: torch.Tensor, bucket_out: torch.Tensor | None = None,
                     stream=None) -> torch.Tensor:
    """First-token table (uint32[FC_BUCKETS]) of a store."""
    if bucket_out is None:
        bucket_out = _empty(FC_BUCKETS, torch.uint32, tokens.device)
    _check("fc_store_prepare", lib().fc_store_prepare(_ptr(tokens), _ptr(sa), tokens.numel(), _ptr(bucket_out),
                                                     _stream(stream)))
    return bucket_out


def fc_pair_table_entries(V: int) -> int:
    return int(lib().fc_pair_table_entries(V))


def fc_store_prepare_pairs(tokens: torch.Tensor, sa: torch.Tensor, V: int, pair_out: torch.Tensor | None = None,
                           stream=None) -> torch.Tensor:
    """Two-token prefix table (uint32[V*(V+1)+1]) of a store; V > every token."""
    if pair_out is None:
        pair_out = _empty(fc_pair_table_entries(V), torch.uint32, tokens.device)
    _check("fc_store_prepare_pairs", lib().fc_store_prepare_pairs(_ptr(tokens), _ptr(sa), tokens.numel(), V,
                                                                 _ptr(pair_out), _stream(stream)))
    return pair_out


def fc_record_bytes(n: int) -> int:
    return int(lib().fc_record_bytes(n))


def fc_store_prepare_records(tokens: torch.Tensor, sa: torch.Tensor, rec_out: torch.Tensor | None = None,
                             stream=None) -> torch.Tensor:
    """Inline-prefix records (uint8[64*n]: sa[i] then T[sa[i]+2 .. sa[i]+32))."""
    if rec_out is None:
        rec_out = _empty(max(fc_record_bytes(tokens.numel()), 1), torch.uint8, tokens.device)
    _check("fc_store_prepare_records", lib().fc_store_prepare_records(_ptr(tokens), _ptr(sa), tokens.numel(),
                                                                     _ptr(rec_out), _stream(stream)))
    return rec_out


def fc_store_prepare_top(rec: torch.Tensor, n: int, top_out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Top-level sample of the records (uint8[32 * ceil(n / 256)]): the first
    32 bytes of every 256th record."""
    if top_out is None:
        top_out = _empty(max(int(lib().fc_store_top_bytes(n)), 1), torch.uint8, rec.device)
    _check("fc_store_prepare_top", lib().fc_store_prepare_top(_ptr(rec), n, _ptr(top_out), _stream(stream)))
    return top_out


class Store:
    """A datastore resident on the GPU: tokens, suffix array, bucket table and,
    with pair_vocab = V, the optional two-token table; with records = True
    (needs pair_vocab) also the inline-prefix records and, unless top = False,
    their top-level sample."""

    def __init__(self, tokens: torch.Tensor, sa: torch.Tensor | None = None, bucket: torch.Tensor | None = None,
                 pair_vocab: int | None = None, records: bool = False, top: bool | None = None, stream=None):
        if tokens.dtype != torch.uint16 or tokens.dim() != 1 or not tokens.is_cuda or not tokens.is_contiguous():
            raise ValueError("tokens must be a contiguous 1-D uint16 device tensor")
        for name, t, shape in (("sa", sa, (tokens.numel(),)), ("bucket", bucket, (FC_BUCKETS,))):
            _expect(name, t, torch.uint32, shape, optional=True)
            if t is not None and (not t.is_cuda or not t.is_contiguous()):
                raise ValueError(f"{name} must be a contiguous device tensor")
        self.tokens = tokens
        self.sa = fc_datastore_build(tokens, stream=stream) if sa is None else sa
        self.bucket = fc_store_prepare(tokens, self.sa, stream=stream) if bucket is None else bucket
        self.pair_vocab = pair_vocab or 0
        self.pair = (fc_store_prepare_pairs(tokens, self.sa, pair_vocab, stream=stream)
                     if pair_vocab else None)
        if records and not pair_vocab:
            raise ValueError("records need the two-token table (pair_vocab)")
        self.rec = fc_store_prepare_records(tokens, self.sa, stream=stream) if records else None
        if top and not records:
            raise ValueError("the top-level sample needs the records")
        use_top = records if top is None else top
        self.top = fc_store_prepare_top(self.rec, self.n, stream=stream) if use_top and self.n > 0 else None

    @property
    def n(self) -> int:
        return self.tokens.numel()

    def view(self) -> FcStore:
        return FcStore(self.tokens.data_ptr(), self.sa.data_ptr(), self.bucket.data_ptr(), self.n,
                       None if self.pair is None else self.pair.data_ptr(), self.pair_vocab,
                       None if self.rec is None else self.rec.data_ptr(),
                       None if self.top is None else self.top.data_ptr())


# ------------------------------------------------------------ retrieval ----

RETRIEVE_FIELDS = ("match_n", "range_lo", "range_cnt", "taken", "cont_pos", "cont_src", "cont_len", "cont_tok")


def retrieve_outputs(B: int, S: int, k: int, m: int, device) -> dict:
    return dict(
        match_n=_empty((B, S), torch.int32, device), range_lo=_empty((B, S), torch.uint32, device),
        range_cnt=_empty((B, S), torch.uint32, device), taken=_empty((B, S), torch.int32, device),
        cont_pos=_empty((B, k), torch.uint32, device), cont_src=_empty((B, k), torch.uint8, device),
        cont_len=_empty((B, k), torch.uint8, device), cont_tok=_empty((B, k, m), torch.uint16, device))


def fc_retrieve_workspace_bytes(B: int, S: int, n_max: int = 16, n_min: int = 2, k: int = 5000,
                                m: int = 10) -> int:
    return int(lib().fc_retrieve_workspace_bytes(B, S, FcRetrieveParams(n_max, n_min, k, m)))


def fc_retrieve(stores, ctx: torch.Tensor, n_max: int = 16, n_min: int = 2, k: int = 5000, m: int = 10,
                out: dict | None = None, workspace: torch.Tensor | None = None, rows: torch.Tensor | None = None,
                stream=None) -> dict:
    """Batched longest-suffix retrieval; ctx is uint16 [B][L] on the GPU.
    With rows (int32 [B]), query b's results go to row rows[b] of `out`."""
    if ctx.dtype != torch.uint16 or ctx.dim() != 2:
        raise ValueError("ctx must be a 2-D uint16 tensor")
    B, L = ctx.shape
    S = len(stores)
    views = (FcStore * max(S, 1))(*[s.view() for s in stores])
    p = FcRetrieveParams(n_max, n_min, k, m)
    if out is None:
        out = retrieve_outputs(B, S, k, m, ctx.device)
    n_rows = out["taken"].shape[0] if "taken" in out else B
    if rows is None and n_rows != B:
        raise ValueError("without a row map the outputs need one row per query")
    _expect_outputs(out, RETRIEVE_FIELDS, _retrieve_shapes(n_rows, S, k, m), _RETRIEVE_DTYPES)
    _expect("rows", rows, torch.int32, (B,), optional=True)
    _expect("workspace", workspace, torch.uint8, optional=True)
    need = int(lib().fc_retrieve_workspace_bytes(B, S, p))
    if workspace is None and need > 0:
        workspace = _empty(need, torch.uint8, ctx.device)
    _check("fc_retrieve", lib().fc_retrieve(
        views, S, _ptr(ctx), B, L, p, *[_ptr(out[f]) for f in RETRIEVE_FIELDS], _ptr(rows), n_rows,
        _ptr(workspace), 0 if workspace is None else workspace.numel(), _stream(stream)))
    return out


def fc_retrieve_noalloc_max_bytes() -> int:
    return int(lib().fc_retrieve_noalloc_max_bytes())


def fc_retrieve_noalloc(stores, ctx: torch.Tensor, n_max: int = 16, n_min: int = 2, k: int = 5000, m: int = 10,
                        out: dict | None = None, rows: torch.Tensor | None = None, stream=None) -> dict:
    """fc_retrieve with the library's static per-GPU workspace (no workspace
    argument; the call allocates nothing when `out` is given).  Calls that
    overlap on one GPU share that workspace and race."""
    if ctx.dtype != torch.uint16 or ctx.dim() != 2:
        raise ValueError("ctx must be a 2-D uint16 tensor")
    B, L = ctx.shape
    S = len(stores)
    views = (FcStore * max(S, 1))(*[s.view() for s in stores])
    p = FcRetrieveParams(n_max, n_min, k, m)
    if out is None:
        out = retrieve_outputs(B, S, k, m, ctx.device)
    n_rows = out["taken"].shape[0] if "taken" in out else B
    if rows is None and n_rows != B:
        raise ValueError("without a row map the outputs need one row per query")
    _expect_outputs(out, RETRIEVE_FIELDS, _retrieve_shapes(n_rows, S, k, m), _RETRIEVE_DTYPES)
    _expect("rows", rows, torch.int32, (B,), optional=True)
    _check("fc_retrieve_noalloc", lib().fc_retrieve_noalloc(
        views, S, _ptr(ctx), B, L, p, *[_ptr(out[f]) for f in RETRIEVE_FIELDS], _ptr(rows), n_rows,
        _stream(stream)))
    return out


# ---------------------------------------------------------------- CACHE ----

def fc_cache_lds_bytes(stride: int) -> int:
    return int(lib().fc_cache_lds_bytes(stride))


def fc_cache_retrieve(texts: torch.Tensor, text_len: torch.Tensor, ctx: torch.Tensor, n_max: int = 16,
                      n_min: int = 2, k: int = 5000, m: int = 10, text_row: torch.Tensor | None = None,
                      out: dict | None = None, rows: torch.Tensor | None = None, stream=None) -> dict:
    """Retrieval from CACHE texts (uint16 [n_texts][stride], lengths int32
    [n_texts]) as single stores; outputs as fc_retrieve with S = 1."""
    if texts.dtype != torch.uint16 or texts.dim() != 2 or text_len.dtype != torch.int32:
        raise ValueError("texts must be 2-D uint16 and text_len int32")
    if ctx.dtype != torch.uint16 or ctx.dim() != 2:
        raise ValueError("ctx must be a 2-D uint16 tensor")
    B, L = ctx.shape
    n_texts, stride = texts.shape
    _expect("text_len", text_len, torch.int32, (n_texts,))
    _expect("text_row", text_row, torch.int32, (B,), optional=True)
    if out is None:
        out = retrieve_outputs(B, 1, k, m, ctx.device)
    n_rows = out["taken"].shape[0] if "taken" in out else B
    if rows is None and n_rows != B:
        raise ValueError("without a row map the outputs need one row per query")
    _expect_outputs(out, RETRIEVE_FIELDS, _retrieve_shapes(n_rows, 1, k, m), _RETRIEVE_DTYPES)
    _expect("rows", rows, torch.int32, (B,), optional=True)
    _check("fc_cache_retrieve", lib().fc_cache_retrieve(
        _ptr(texts), stride, n_texts, _ptr(text_len), _ptr(text_row), _ptr(ctx), B, L,
        FcRetrieveParams(n_max, n_min, k, m), *[_ptr(out[f]) for f in RETRIEVE_FIELDS], _ptr(rows),
        out["taken"].shape[0], _stream(stream)))
    return out


def fc_cache_write(texts: torch.Tensor, text_len: torch.Tensor, dst_row: torch.Tensor, dst_off: torch.Tensor,
                   new_len: torch.Tensor, src_off: torch.Tensor, src_len: torch.Tensor, src_tok: torch.Tensor,
                   stream=None) -> None:
    """Segment copies into CACHE texts (see include/fastcoder.h)."""
    if texts.dtype != torch.uint16 or texts.dim() != 2:
        raise ValueError("texts must be a 2-D uint16 tensor")
    n_texts, stride = texts.shape
    n_seg = dst_row.numel()
    _expect("text_len", text_len, torch.int32, (n_texts,))
    for name, t, dt in (("dst_row", dst_row, torch.int32), ("dst_off", dst_off, torch.int32),
                        ("new_len", new_len, torch.int32), ("src_off", src_off, torch.int64),
                        ("src_len", src_len, torch.int32)):
        _expect(name, t, dt, (n_seg,))
    _expect("src_tok", src_tok, torch.uint16)
    _check("fc_cache_write", lib().fc_cache_write(
        _ptr(texts), stride, n_texts, _ptr(text_len), dst_row.numel(), _ptr(dst_row), _ptr(dst_off),
        _ptr(new_len), _ptr(src_off), _ptr(src_len), _ptr(src_tok), _stream(stream)))


# ------------------------------------------------------- tree attention ----

def fc_tree_attention(q: torch.Tensor, k_tree: torch.Tensor, v_tree: torch.Tensor, k_cache: torch.Tensor,
                      v_cache: torch.Tensor, prefix_len: torch.Tensor, tree: dict, rope_base: float = 10000.0,
                      out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Tree attention (bf16 q [B][R][H][D], k/v_tree [B][R][Hkv][D],
    k/v_cache [B][Pmax][Hkv][D]) with the tree's num_nodes, mask and pos_ids;
    returns fp32 [B][R][H][D]."""
    for t in (q, k_tree, v_tree, k_cache, v_cache):
        if t.dtype != torch.bfloat16 or t.dim() != 4:
            raise ValueError("q, k_tree, v_tree, k_cache, v_cache must be 4-D bfloat16")
    B, R, H, D = q.shape
    Hkv, Pmax = k_tree.shape[2], k_cache.shape[1]
    for name, t, shape in (("k_tree", k_tree, (B, R, Hkv, D)), ("v_tree", v_tree, (B, R, Hkv, D)),
                           ("k_cache", k_cache, (B, Pmax, Hkv, D)), ("v_cache", v_cache, (B, Pmax, Hkv, D))):
        _expect(name, t, torch.bfloat16, shape)
    _expect("prefix_len", prefix_len, torch.int32, (B,))
    _expect("num_nodes", tree["num_nodes"], torch.int32, (B,))
    _expect("pos_ids", tree["pos_ids"], torch.int32, (B, R))
    _expect("mask", tree["mask"], torch.int32, (B, R, R))
    _expect("out", out, torch.float32, (B, R, H, D), optional=True)
    if out is None:
        out = _empty((B, R, H, D), torch.float32, q.device)
    u16 = lambda t: _ptr(t.view(torch.uint16))  # noqa: E731
    _check("fc_tree_attention", lib().fc_tree_attention(
        u16(q), u16(k_tree), u16(v_tree), u16(k_cache), u16(v_cache), _ptr(prefix_len), _ptr(tree["num_nodes"]),
        _ptr(tree["mask"]), _ptr(tree["pos_ids"]), B, R, H, Hkv, D, Pmax, rope_base, _ptr(out), _stream(stream)))
    return out


# ----------------------------------------------------------------- tree ----

TREE_FIELDS = ("num_nodes", "node_tok", "parent", "weight", "pos_ids", "mask")


def tree_outputs(B: int, c: int, device) -> dict:
    R = c + 1
    return dict(num_nodes=_empty(B, torch.int32, device), node_tok=_empty((B, R), torch.int32, device),
                parent=_empty((B, R), torch.int32, device), weight=_empty((B, R), torch.uint32, device),
                pos_ids=_empty((B, R), torch.int32, device), mask=_empty((B, R, R), torch.int32, device))


def fc_build_tree_workspace_bytes(B: int) -> int:
    return int(lib().fc_build_tree_workspace_bytes(B))


def fc_build_tree(taken: torch.Tensor, cont_len: torch.Tensor, cont_tok: torch.Tensor, ctx: torch.Tensor,
                  c: int = 64, alpha=(1, 1), out: dict | None = None, workspace: torch.Tensor | None = None,
                  rows: torch.Tensor | None = None, stream=None) -> dict:
    """Weighted draft trie pruned to c nodes, with mask and position ids.
    With rows (int32 [B]), query b reads row rows[b] of taken/cont_*."""
    if taken.dim() != 2 or cont_tok.dim() != 3 or ctx.dim() != 2:
        raise ValueError("taken [rows][S], cont_tok [rows][k][m] and ctx [B][L] expected")
    n_rows, S = taken.shape
    B = n_rows if rows is None else rows.numel()
    k, m = cont_tok.shape[1], cont_tok.shape[2]
    L = ctx.shape[1]
    _expect("taken", taken, torch.int32)
    _expect("cont_len", cont_len, torch.uint8, (n_rows, k))
    _expect("cont_tok", cont_tok, torch.uint16, (n_rows, k, m))
    _expect("ctx", ctx, torch.uint16, (B, L))
    _expect("rows", rows, torch.int32, (B,), optional=True)
    a = list(alpha)[:S]
    if len(a) != S:
        raise ValueError("need one alpha per store")
    tp = FcTreeParams(c, (ctypes.c_uint32 * FC_MAX_SOURCES)(*(a + [0] * (FC_MAX_SOURCES - S))))
    if out is None:
        out = tree_outputs(B, c, ctx.device)
    R = c + 1
    _expect_outputs(out, TREE_FIELDS, dict(num_nodes=(B,), node_tok=(B, R), parent=(B, R), weight=(B, R),
                                           pos_ids=(B, R), mask=(B, R, R)),
                    dict(num_nodes=torch.int32, node_tok=torch.int32, parent=torch.int32, weight=torch.uint32,
                         pos_ids=torch.int32, mask=torch.int32))
    need = fc_build_tree_workspace_bytes(B)
    if workspace is None and need > 0:
        workspace = _empty(need, torch.uint8, ctx.device)
    _check("fc_build_tree", lib().fc_build_tree(
        _ptr(taken), _ptr(cont_len), _ptr(cont_tok), _ptr(ctx), B, L, S, k, m, tp,
        *[_ptr(out[f]) for f in TREE_FIELDS], _ptr(rows), n_rows, _ptr(workspace),
        0 if workspace is None else workspace.numel(), _stream(stream)))
    return out


# ----------------------------------------------------------- acceptance ----

ACCEPT_FIELDS = ("accept_len", "accept_tok", "last_node")


def accept_outputs(B: int, m: int, device) -> dict:
    return dict(accept_len=_empty(B, torch.int32, device), accept_tok=_empty((B, m + 1), torch.int32, device),
                last_node=_empty(B, torch.int32, device))


def fc_verify_accept(tree: dict, target: torch.Tensor, m: int = 10, out: dict | None = None, stream=None) -> dict:
    """Longest accepted root path against per-row target tokens ([B][c+1])."""
    B, R = tree["node_tok"].shape
    _expect("num_nodes", tree["num_nodes"], torch.int32, (B,))
    for f in ("node_tok", "parent", "pos_ids"):
        _expect(f, tree[f], torch.int32, (B, R))
    _expect("target", target, torch.int32, (B, R))
    if out is not None:
        _expect_outputs(out, ACCEPT_FIELDS, dict(accept_len=(B,), accept_tok=(B, m + 1), last_node=(B,)),
                        dict(accept_len=torch.int32, accept_tok=torch.int32, last_node=torch.int32))
    if out is None:
        out = accept_outputs(B, m, target.device)
    _check("fc_verify_accept", lib().fc_verify_accept(
        _ptr(tree["num_nodes"]), _ptr(tree["node_tok"]), _ptr(tree["parent"]), _ptr(tree["pos_ids"]),
        _ptr(target), B, R - 1, m, *[_ptr(out[f]) for f in ACCEPT_FIELDS], _stream(stream)))
    return out


def fc_targets_from_truth(truth: torch.Tensor, start: torch.Tensor, tree: dict, seq: torch.Tensor | None = None,
                          out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Target tokens [B][c+1] from true streams (uint16 [n_streams][len])."""
    B, R = tree["node_tok"].shape
    if truth.dtype != torch.uint16 or truth.dim() != 2:
        raise ValueError("truth must be a 2-D uint16 tensor")
    _expect("start", start, torch.int32, (B,))
    _expect("seq", seq, torch.int32, (B,), optional=True)
    _expect("num_nodes", tree["num_nodes"], torch.int32, (B,))
    _expect("pos_ids", tree["pos_ids"], torch.int32, (B, R))
    _expect("out", out, torch.int32, (B, R), optional=True)
    if out is None:
        out = _empty((B, R), torch.int32, truth.device)
    _check("fc_targets_from_truth", lib().fc_targets_from_truth(
        _ptr(truth), truth.shape[1], truth.stride(0), _ptr(seq), _ptr(start), _ptr(tree["num_nodes"]),
        _ptr(tree["pos_ids"]), B, R - 1, _ptr(out), _stream(stream)))
    return out


class ReplayEngine:
    """Device-resident decode-trace replay (fc_replay_init / fc_replay_run):
    owns the device state for `truth` (uint16 [n_streams][length] on the
    GPU) over `stores`; run() replays until every stream is finished.  With
    cache_l, the CACHE of Section IV-B comes first (Alg. 1's cache branch);
    missing and skip_tok switch on Alg. 1's retrieval-timing control, with
    the gate's draws from skip_draws (int [>= max_steps][n_streams])."""

    def __init__(self, stores, truth: torch.Tensor, n_max=16, n_min=2, k=5000, m=10, c=64, alpha=(1, 1), lru=32,
                 ctx_len=16, max_steps=512, chunk=16, cache_l=None, cache_every=20, cache_cap=FC_MAX_CACHE_TOKENS,
                 missing=False, skip_tok=None, skip_p=0.5, skip_draws=None):
        if truth.dtype != torch.uint16 or truth.dim() != 2 or not truth.is_contiguous() or not truth.is_cuda:
            raise ValueError("truth must be a contiguous 2-D uint16 device tensor")
        dev = truth.device
        self.stores, self.truth, self.chunk = stores, truth, chunk
        n, tlen = truth.shape
        S = len(stores)
        self.views = (FcStore * S)(*[st.view() for st in stores])
        i32 = torch.int32
        self.t = dict(pos=_empty(n, i32, dev), lru_key=_empty((n, lru, ctx_len), torch.uint16, dev),
                      lru_used=_empty((n, lru), i32, dev), lru_count=_empty(n, i32, dev), hits=_empty(n, i32, dev),
                      lookups=_empty(n, i32, dev), ctx=_empty((n, ctx_len), torch.uint16, dev),
                      rows_retrieve=_empty(n, i32, dev), rows_tree=_empty(n, i32, dev), live=_empty(2, i32, dev),
                      history=_empty((max_steps, n), i32, dev), target=_empty((n, c + 1), i32, dev),
                      state=_empty(n, i32, dev))
        self.cache_on = cache_l is not None
        # the LRU slots, one empty row (the bare root of skipped contexts) and,
        # with the CACHE, one row per stream for its served CACHE result
        self.t.update(retrieve_outputs(n * lru + 1 + (n if self.cache_on else 0), S, k, m, dev))
        self.t.update(tree_outputs(n, c, dev))
        self.t.update(accept_outputs(n, m, dev))
        self.control_on = bool(missing) or skip_tok is not None
        if self.cache_on:
            max_seqs = (cache_cap + 1) // 2 + 1
            self.t.update(ctext=_empty((n, cache_cap), torch.uint16, dev), clen=_empty(n, i32, dev),
                          seq_len=_empty((n, max_seqs), i32, dev), seq_head=_empty(n, i32, dev),
                          seq_count=_empty(n, i32, dev), chunks=_empty(n, i32, dev), served=_empty(n, i32, dev),
                          rows_cache=_empty(n, i32, dev))
            self.t.update({"c_" + f: v for f, v in retrieve_outputs(n, 1, k, m, dev).items()})
        miss_cap = 64
        while miss_cap <= max_steps:
            miss_cap *= 2
        if missing:
            self.t.update(miss_key=_empty((n, miss_cap, ctx_len), torch.uint16, dev),
                          miss_used=_empty((n, miss_cap), torch.uint8, dev))
        if self.control_on:
            self.t.update(m_skips=_empty(n, i32, dev), g_skips=_empty(n, i32, dev))
        if skip_tok is not None:
            d = np.ascontiguousarray(np.asarray(skip_draws)[:max_steps], dtype=np.int32)
            if d.shape != (max_steps, n):
                raise ValueError("skip_draws must hold max_steps rows of n_streams draws")
            self.t["skip_draws"] = torch.from_numpy(d).to(dev)
        rp = FcRetrieveParams(n_max, n_min, k, m)
        self.rws = _empty(max(int(lib().fc_retrieve_workspace_bytes(n, S, rp)), 1), torch.uint8, dev)
        self.tws = _empty(max(fc_build_tree_workspace_bytes(n), 1), torch.uint8, dev)
        al = (ctypes.c_uint32 * FC_MAX_SOURCES)(*([int(a) for a in tuple(alpha)[:S]] + [0] * (FC_MAX_SOURCES - S)))
        r = FcReplay()
        r.truth, r.truth_stride, r.truth_len = truth.data_ptr(), truth.stride(0), tlen
        r.n_streams, r.ctx_len, r.lru, r.max_steps = n, ctx_len, lru, max_steps
        r.rp, r.tp = rp, FcTreeParams(c, al)
        for f, v in self.t.items():
            setattr(r, f, v.data_ptr())
        r.retrieve_ws, r.retrieve_ws_bytes = self.rws.data_ptr(), self.rws.numel()
        r.tree_ws, r.tree_ws_bytes = self.tws.data_ptr(), self.tws.numel()
        r.cache_l = -1 if cache_l is None else int(cache_l)
        r.cache_every, r.cache_cap = int(cache_every), int(cache_cap)
        r.max_seqs = (int(cache_cap) + 1) // 2 + 1
        r.missing, r.miss_cap = (1 if missing else 0), miss_cap
        r.skip_tok = -1 if skip_tok is None else int(skip_tok)
        r.skip_thr = int(skip_p * 2 ** 31)
        self.r, self.max_steps = r, max_steps

    def run(self, limit: int | None = None, stream=None) -> dict:
        """Replays from the start for at most `limit` (default max_steps)
        steps; returns the per-step accepted lengths ([steps][n_streams], -1
        for finished streams), LRU hits and lookups, final positions, the
        mean accepted length and the CACHE / timing-control counters."""
        st = _stream(stream)
        cap = self.max_steps if limit is None else min(limit, self.max_steps)
        _check("fc_replay_init", lib().fc_replay_init(ctypes.byref(self.r), st))
        step = 0
        while step < cap:
            n = min(self.chunk, cap - step)
            _check("fc_replay_run", lib().fc_replay_run(self.views, len(self.stores), ctypes.byref(self.r), step, n,
                                                        st))
            step += n
            if int(self.t["live"][(step - 1) & 1].item()) == 0:
                break
        hist = self.t["history"][:step].cpu().numpy().astype(np.int64)
        steps = int((hist >= 0).any(axis=1).sum())
        acc = hist[:steps]
        live = acc >= 0
        nn = self.r.n_streams

        def host(name):
            return self.t[name].cpu().numpy().astype(np.int64) if name in self.t else np.zeros(nn, np.int64)

        return dict(accept=acc, hits=host("hits"), lookups=host("lookups"), pos=host("pos"),
                    acc_len=float(acc[live].sum() / max(live.sum(), 1)), steps=steps, cache_served=host("served"),
                    missing_skips=host("m_skips"), gate_skips=host("g_skips"))
