"""The C ABI library loads, exports every entry point include/fastcoder.h
declares, and rejects bad arguments on the host before touching a GPU."""
import ctypes
import os
import re

import pytest

import paper_2502_17139_amd as fc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(fc.LIB_PATH):
        from paper_2502_17139_amd import build
        build.build()
    return fc.lib()


def _declared():
    with open(os.path.join(ROOT, "include", "fastcoder.h")) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(fc_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported(L):
    names = _declared()
    assert set(names) == set(fc.EXPORTS)
    for name in names:
        assert hasattr(L, name), name


def test_status_strings(L):
    assert L.fc_abi_version() == 4
    for code, name in fc.STATUS.items():
        assert L.fc_status_string(code).decode().startswith(name)
    assert L.fc_status_string(99).decode() == "FC_ERR_UNKNOWN"


def test_workspace_sizes(L):
    assert fc.fc_datastore_build_workspace_bytes(1000) < fc.fc_datastore_build_workspace_bytes(2000)
    # about 28.6 bytes per token below 2^26 tokens (rank, two key and two
    # value buffers, per-tile status); from 2^26 on, 8 more for the rank
    # pairs (about 36.6 for the 1B-token store)
    n = (1 << 26) - 1
    assert 28 * n < fc.fc_datastore_build_workspace_bytes(n) < 29 * n
    n = 1_001_999_999
    assert 36 * n < fc.fc_datastore_build_workspace_bytes(n) < 37 * n
    # the batch's slot offsets
    assert L.fc_retrieve_workspace_bytes(1024, 2, fc.FcRetrieveParams(16, 2, 5000, 10)) == 4 * 1025
    assert L.fc_retrieve_workspace_bytes(0, 2, fc.FcRetrieveParams(16, 2, 5000, 10)) == 0


def _retrieve_args(S=1, B=1, L_=4, p=(16, 2, 5000, 10), ws_bytes=0):
    views = (fc.FcStore * 4)(*[fc.FcStore(1, 1, 1, 10, None, 0) for _ in range(4)])
    one = ctypes.c_void_p(8)
    return [views, S, one, B, L_, fc.FcRetrieveParams(*p)] + [one] * 8 + [None, 0, None, ws_bytes, None]


@pytest.mark.parametrize("change,code", [
    (dict(S=0), 1), (dict(S=5), 1), (dict(B=-1), 1), (dict(L_=0), 1),
    (dict(p=(17, 2, 10, 10)), 1), (dict(p=(4, 5, 10, 10)), 1), (dict(p=(4, 0, 10, 10)), 1),
    (dict(p=(4, 2, 0, 10)), 1), (dict(p=(4, 2, 10, 0)), 1), (dict(p=(4, 2, 10, 256)), 1),
])
def test_retrieve_rejects(L, change, code):
    assert L.fc_retrieve(*_retrieve_args(**change)) == code


def test_retrieve_rejects_batches_past_31_bit_slots(L):
    # 430,000 queries x 5,000 slots number more than 2^31
    assert L.fc_retrieve(*_retrieve_args(B=430_000)) == 4


def _noalloc_args(**change):
    a = _retrieve_args(**change)
    return a[:-3] + [a[-1]]  # fc_retrieve's arguments without the workspace pointer and size


def test_retrieve_noalloc_rejects_on_the_host(L):
    """The no-allocation retrieval takes fc_retrieve's checks, and refuses a
    batch whose workspace exceeds its static array, before any device call."""
    assert L.fc_retrieve_noalloc_max_bytes() == 1 << 20
    for change, code in ((dict(S=0), 1), (dict(B=-1), 1), (dict(L_=0), 1), (dict(p=(4, 2, 10, 256)), 1),
                         (dict(B=430_000), 4)):
        assert L.fc_retrieve_noalloc(*_noalloc_args(**change)) == code
    # 4 * (B + 1) bytes of offsets: 262,143 queries fit in 1 MiB, 262,144 do not
    assert L.fc_retrieve_noalloc(*_noalloc_args(B=262_144, p=(16, 2, 8, 10))) == 4
    assert L.fc_retrieve_noalloc(*_noalloc_args(B=0)) == 0  # nothing to do, no device call


def test_retrieve_rejects_missing_workspace(L):
    assert L.fc_retrieve(*_retrieve_args(ws_bytes=0)) == 2
    args = _retrieve_args(ws_bytes=4)  # 4*(B+1) = 8 needed
    args[-3] = ctypes.c_void_p(8)
    assert L.fc_retrieve(*args) == 2


def test_retrieve_rejects_null_outputs_and_big_store(L):
    args = _retrieve_args()
    args[6] = None  # match_n
    assert L.fc_retrieve(*args) == 1
    views = (fc.FcStore * 1)(fc.FcStore(1, 1, 1, 1 << 32, None, 0))
    args = _retrieve_args()
    args[0] = views
    assert L.fc_retrieve(*args) == 1
    views = (fc.FcStore * 1)(fc.FcStore(1, None, 1, 10, None, 0))
    args[0] = views
    assert L.fc_retrieve(*args) == 1
    views = (fc.FcStore * 1)(fc.FcStore(1, 1, 1, 10, 1, 70000))  # pair vocabulary out of range
    args[0] = views
    assert L.fc_retrieve(*args) == 1
    views = (fc.FcStore * 1)(fc.FcStore(1, 1, 1, 10, None, 0, 64))  # records without a two-token table
    args[0] = views
    assert L.fc_retrieve(*args) == 1
    views = (fc.FcStore * 1)(fc.FcStore(1, 1, 1, 10, 1, 100, 48))  # records not 64-byte aligned
    args[0] = views
    assert L.fc_retrieve(*args) == 1
    views = (fc.FcStore * 1)(fc.FcStore(1, 1, 1, 10, None, 0, None, 32))  # a sample without records
    args[0] = views
    assert L.fc_retrieve(*args) == 1
    views = (fc.FcStore * 1)(fc.FcStore(1, 1, 1, 10, 1, 100, 64, 48))  # a sample not 32-byte aligned
    args[0] = views
    assert L.fc_retrieve(*args) == 1


def _tree_args(B=1, L_=2, S=2, k=10, m=4, c=8, alpha=(1, 1, 0, 0)):
    one = ctypes.c_void_p(8)
    tp = fc.FcTreeParams(c, (ctypes.c_uint32 * 4)(*alpha))
    return [one, one, one, one, B, L_, S, k, m, tp] + [one] * 6 + [None, 0, one, 1 << 20, None]


@pytest.mark.parametrize("change,code", [
    (dict(B=-1), 1), (dict(L_=0), 1), (dict(S=0), 1), (dict(S=5), 1), (dict(k=0), 1), (dict(m=0), 1),
    (dict(m=256), 1), (dict(c=0), 1), (dict(c=255 + 1), 1), (dict(k=65536), 4),
    (dict(k=60000, alpha=(1 << 20, 1, 0, 0)), 4), (dict(k=5000, m=255), 4),
])
def test_build_tree_rejects(L, change, code):
    if change == dict(k=5000, m=255):
        # about 2.6 MB of LDS per query: larger than any workgroup can hold; this
        # check reads the device's limit, so it needs a GPU
        pytest.skip("LDS limit check queries the device")
    assert L.fc_build_tree(*_tree_args(**change)) == code


def test_build_tree_rejects_missing_workspace(L):
    args = _tree_args()
    args[-2] = 8  # 4*(2B+2) = 16 needed
    assert L.fc_build_tree(*args) == 2
    args = _tree_args()
    args[-3] = None
    assert L.fc_build_tree(*args) == 2
    assert L.fc_build_tree_workspace_bytes(1024) == 4 * 2050


def test_row_maps_and_targets_reject(L):
    args = _retrieve_args(ws_bytes=1 << 20)
    args[-3] = ctypes.c_void_p(8)
    args[-5] = ctypes.c_void_p(8)  # a row map with no rows
    args[-4] = 0
    assert L.fc_retrieve(*args) == 1
    targs = _tree_args()
    targs[-5] = ctypes.c_void_p(8)
    targs[-4] = 0
    assert L.fc_build_tree(*targs) == 1
    one = ctypes.c_void_p(8)
    assert L.fc_targets_from_truth(one, 100, 50, None, one, one, one, 2, 8, one, None) == 1  # stride < len
    assert L.fc_targets_from_truth(one, 100, 100, None, one, one, one, 2, 256, one, None) == 1
    assert L.fc_targets_from_truth(None, 100, 100, None, one, one, one, 2, 8, one, None) == 1
    assert L.fc_targets_from_truth(None, 0, 0, None, None, None, None, 0, 8, None, None) == 0


def test_pair_table_size_and_rejects(L):
    assert L.fc_pair_table_entries(32256) == 32256 * 32257 + 1
    assert L.fc_pair_table_entries(3) == 13
    one = ctypes.c_void_p(8)
    assert L.fc_store_prepare_pairs(one, one, 10, 0, one, None) == 1
    assert L.fc_store_prepare_pairs(one, one, 10, 65537, one, None) == 1
    assert L.fc_store_prepare_pairs(one, one, 10, 5, None, None) == 1
    assert L.fc_store_prepare_pairs(None, one, 10, 5, one, None) == 1


def test_record_size_and_rejects(L):
    assert L.fc_record_bytes(1_001_999_999) == 64 * 1_001_999_999
    assert L.fc_record_bytes(0) == 0
    one, aligned = ctypes.c_void_p(8), ctypes.c_void_p(64)
    assert L.fc_store_prepare_records(one, one, 10, ctypes.c_void_p(48), None) == 1  # misaligned
    assert L.fc_store_prepare_records(one, one, 10, None, None) == 1
    assert L.fc_store_prepare_records(None, one, 10, aligned, None) == 1
    assert L.fc_store_prepare_records(one, None, 10, aligned, None) == 1
    assert L.fc_store_prepare_records(one, one, 1 << 32, aligned, None) == 1
    assert L.fc_store_prepare_records(None, None, 0, None, None) == 0  # nothing to write


def test_top_sample_size_and_rejects(L):
    # one 32-byte entry per started stride of 256 suffixes
    assert L.fc_store_top_bytes(1_001_999_999) == 32 * 3_914_063
    assert L.fc_store_top_bytes(256) == 32 and L.fc_store_top_bytes(257) == 64 and L.fc_store_top_bytes(0) == 0
    rec, top = ctypes.c_void_p(64), ctypes.c_void_p(32)
    assert L.fc_store_prepare_top(None, 10, top, None) == 1
    assert L.fc_store_prepare_top(rec, 10, None, None) == 1
    assert L.fc_store_prepare_top(ctypes.c_void_p(32), 10, top, None) == 1  # records misaligned
    assert L.fc_store_prepare_top(rec, 10, ctypes.c_void_p(16), None) == 1  # sample misaligned
    assert L.fc_store_prepare_top(rec, 1 << 32, top, None) == 1
    assert L.fc_store_prepare_top(None, 0, None, None) == 0  # nothing to write


def test_verify_and_build_reject(L):
    one = ctypes.c_void_p(8)
    assert L.fc_verify_accept(one, one, one, one, one, 1, -1, 4, one, one, one, None) == 1
    assert L.fc_verify_accept(one, one, one, one, one, 1, 255 + 1, 4, one, one, one, None) == 1
    assert L.fc_verify_accept(None, one, one, one, one, 1, 8, 4, one, one, one, None) == 1
    assert L.fc_datastore_build(one, 1 << 32, one, one, 1 << 40, None) == 1
    assert L.fc_datastore_build(one, 100, one, None, 0, None) == 2
    assert L.fc_datastore_build(one, 100, one, one, 16, None) == 2
    assert L.fc_datastore_build(None, 100, one, one, 1 << 30, None) == 1
    assert L.fc_store_prepare(one, one, 100, None, None) == 1
    # empty requests succeed without launching anything
    assert L.fc_datastore_build(None, 0, None, None, 0, None) == 0
    assert L.fc_retrieve(*_retrieve_args(B=0)) == 0
    assert L.fc_verify_accept(None, None, None, None, None, 0, 8, 4, None, None, None, None) == 0


def test_binding_has_no_cpu_path(monkeypatch, tmp_path):
    """Without the built library every call raises instead of computing."""
    monkeypatch.setattr(fc, "LIB_PATH", str(tmp_path / "missing.so"))
    fc.lib.cache_clear()
    try:
        with pytest.raises(RuntimeError, match="no CPU fallback"):
            fc.lib()
    finally:
        monkeypatch.undo()
        fc.lib.cache_clear()


def test_cache_entry_points_reject(L):
    assert L.fc_cache_lds_bytes(16384) == 32768 + 65536
    assert L.fc_cache_lds_bytes(1) == 16 + 4
    assert L.fc_cache_lds_bytes(0) == 0 and L.fc_cache_lds_bytes(16385) == 0
    one = ctypes.c_void_p(8)
    p = fc.FcRetrieveParams(16, 2, 5000, 10)

    def call(stride=100, n_texts=2, B=1, L_=4, params=p, ctx=one):
        return L.fc_cache_retrieve(one, stride, n_texts, one, None, ctx, B, L_, params, *([one] * 8), None, 0, None)

    assert call(stride=0) == 1 and call(stride=16385) == 1 and call(n_texts=0) == 1
    assert call(B=-1) == 1 and call(L_=0) == 1 and call(ctx=None) == 1
    assert call(params=fc.FcRetrieveParams(17, 2, 10, 10)) == 1
    assert call(params=fc.FcRetrieveParams(4, 2, 0, 10)) == 1
    assert call(params=fc.FcRetrieveParams(4, 2, 10, 256)) == 1
    assert call(B=0) == 0
    assert L.fc_cache_write(one, 100, 2, one, -1, one, one, one, one, one, one, None) == 1
    assert L.fc_cache_write(one, 0, 2, one, 1, one, one, one, one, one, one, None) == 1
    assert L.fc_cache_write(None, 100, 2, one, 1, one, one, one, one, one, one, None) == 1
    assert L.fc_cache_write(one, 100, 2, one, 0, one, one, one, one, one, one, None) == 0


def test_batched_build_rejects(L):
    one = ctypes.c_void_p(8)
    off = lambda *v: (ctypes.c_uint64 * len(v))(*v)  # noqa: E731
    assert L.fc_datastore_build_batched(one, off(0, 5), 0, one, one, 1 << 30, None) == 1   # no segment
    assert L.fc_datastore_build_batched(one, None, 1, one, one, 1 << 30, None) == 1
    assert L.fc_datastore_build_batched(one, off(1, 5), 1, one, one, 1 << 30, None) == 1   # must start at 0
    assert L.fc_datastore_build_batched(one, off(0, 5, 3), 2, one, one, 1 << 30, None) == 1  # decreasing
    assert L.fc_datastore_build_batched(one, off(0, 1 << 32), 1, one, one, 1 << 30, None) == 1
    assert L.fc_datastore_build_batched(one, off(0, 5), 1, one, one, 8, None) == 2  # workspace too small
    assert L.fc_datastore_build_batched(None, off(0, 0, 0), 2, None, None, 0, None) == 0  # nothing to build
    assert (L.fc_datastore_build_batched_workspace_bytes(1000, 3) >
            L.fc_datastore_build_workspace_bytes(1000))


def test_extend_rejects(L):
    one = ctypes.c_void_p(8)
    big = 1 << 34
    assert L.fc_datastore_extend(one, 10, 11, one, None, one, None, one, big, None) == 1   # more new than all
    assert L.fc_datastore_extend(one, 1 << 32, 5, one, None, one, None, one, big, None) == 1
    assert L.fc_datastore_extend(one, 10, 4, None, None, one, None, one, big, None) == 1   # old store, no array
    assert L.fc_datastore_extend(None, 10, 4, one, None, one, None, one, big, None) == 1
    assert L.fc_datastore_extend(one, 10, 4, one, None, None, None, one, big, None) == 1   # no output
    assert L.fc_datastore_extend(one, 10, 4, one, None, one, None, one, 8, None) == 2      # workspace too small
    assert L.fc_datastore_extend(None, 0, 0, None, None, None, None, None, 0, None) == 0   # nothing to build
    assert L.fc_datastore_extend_workspace_bytes(10, 11, 0) == 0
    # without a given inverse the workspace holds one: 4 bytes per old token
    assert (L.fc_datastore_extend_workspace_bytes(1_000_000, 1000, 0) -
            L.fc_datastore_extend_workspace_bytes(1_000_000, 1000, 1)) >= 4 * 999_000


def test_struct_layouts_match_header(tmp_path):
    """The binding's ctypes structs have the header's field offsets (a C
    program built against include/fastcoder.h prints them)."""
    import shutil
    import subprocess
    import paper_2502_17139_amd as fc
    if shutil.which("gcc") is None:
        pytest.skip("no C compiler")
    structs = {"fc_replay": fc.FcReplay, "fc_store": fc.FcStore, "fc_retrieve_params": fc.FcRetrieveParams,
               "fc_tree_params": fc.FcTreeParams, "fc_build_stats": fc.FcBuildStats}
    lines = ["#include <stdio.h>", '#include "fastcoder.h"', "int main(void) {"]
    for name, cls in structs.items():
        lines.append(f'  printf("{name} sizeof %zu\\n", sizeof({name}));')
        for f, _ in cls._fields_:
            lines.append(f'  printf("{name} {f} %zu\\n", offsetof({name}, {f}));')
    lines += ["  return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    subprocess.run(["gcc", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", "-I" + os.path.join(root, "include"),
                    str(src), "-o", str(exe)], check=True)
    got = {}
    for line in subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.splitlines():
        name, f, v = line.split()
        got[(name, f)] = int(v)
    for name, cls in structs.items():
        assert got[(name, "sizeof")] == ctypes.sizeof(cls), name
        for f, _ in cls._fields_:
            assert got[(name, f)] == getattr(cls, f).offset, (name, f)
