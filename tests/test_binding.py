"""The binding refuses tensors of the wrong type or shape before anything
reaches the library (whose kernels trust the sizes they are given).  These
run on the CPU: the checks come before any device pointer is taken."""
import pytest
import torch

import paper_2502_17139_amd as fc


def _tree_inputs(n_rows=3, S=2, k=8, m=4, L=5):
    return (torch.zeros((n_rows, S), dtype=torch.int32), torch.zeros((n_rows, k), dtype=torch.uint8),
            torch.zeros((n_rows, k, m), dtype=torch.uint16), torch.zeros((n_rows, L), dtype=torch.uint16))


def test_build_tree_refuses_mismatched_slots():
    taken, lens, toks, ctx = _tree_inputs()
    with pytest.raises(ValueError, match="cont_len"):
        fc.fc_build_tree(taken, lens[:, :7], toks, ctx, c=4)
    with pytest.raises(ValueError, match="cont_tok"):
        fc.fc_build_tree(taken, lens, toks.to(torch.int32), ctx, c=4)
    with pytest.raises(ValueError, match="ctx"):
        fc.fc_build_tree(taken, lens, toks, ctx[:2], c=4)
    with pytest.raises(ValueError, match="rows"):
        fc.fc_build_tree(taken, lens, toks, ctx[:2], c=4, rows=torch.zeros(2, dtype=torch.int64))


def test_build_tree_refuses_small_outputs():
    taken, lens, toks, ctx = _tree_inputs()
    out = fc.tree_outputs(3, 4, "cpu")
    out["mask"] = out["mask"][:, :4]
    with pytest.raises(ValueError, match="mask"):
        fc.fc_build_tree(taken, lens, toks, ctx, c=4, out=out)


def test_verify_refuses_mismatched_target():
    tree = fc.tree_outputs(2, 4, "cpu")
    with pytest.raises(ValueError, match="target"):
        fc.fc_verify_accept(tree, torch.zeros((2, 4), dtype=torch.int32), m=3)
    with pytest.raises(ValueError, match="target"):
        fc.fc_verify_accept(tree, torch.zeros((2, 5), dtype=torch.int64), m=3)


class _NoStore:
    """Stands in for a Store: only its (empty) view is read before the checks."""

    def view(self):
        return fc.FcStore()


def test_retrieve_refuses_short_outputs():
    ctx = torch.zeros((4, 16), dtype=torch.uint16)
    out = fc.retrieve_outputs(4, 1, 10, 3, "cpu")
    out["cont_tok"] = out["cont_tok"][:, :9]
    with pytest.raises(ValueError, match="cont_tok"):
        fc.fc_retrieve([_NoStore()], ctx, k=10, m=3, out=out)
    out = fc.retrieve_outputs(3, 1, 10, 3, "cpu")
    with pytest.raises(ValueError, match="one row per query"):
        fc.fc_retrieve([_NoStore()], ctx, k=10, m=3, out=out)


def test_tree_attention_refuses_mismatched_cache():
    B, R, H, Hkv, D, P = 2, 5, 4, 2, 128, 16
    bf = torch.bfloat16
    q = torch.zeros((B, R, H, D), dtype=bf)
    kt = torch.zeros((B, R, Hkv, D), dtype=bf)
    kc = torch.zeros((B, P, Hkv, D), dtype=bf)
    tree = fc.tree_outputs(B, R - 1, "cpu")
    plen = torch.zeros(B, dtype=torch.int32)
    with pytest.raises(ValueError, match="v_cache"):
        fc.fc_tree_attention(q, kt, kt, kc, kc[:, :8], plen, tree)
    with pytest.raises(ValueError, match="prefix_len"):
        fc.fc_tree_attention(q, kt, kt, kc, kc, plen.to(torch.int64), tree)


def test_cache_write_refuses_mismatched_segments():
    texts = torch.zeros((2, 32), dtype=torch.uint16)
    tl = torch.zeros(2, dtype=torch.int32)
    i32 = lambda n: torch.zeros(n, dtype=torch.int32)  # noqa: E731
    with pytest.raises(ValueError, match="src_off"):
        fc.fc_cache_write(texts, tl, i32(3), i32(3), i32(3), i32(3), i32(3), torch.zeros(5, dtype=torch.uint16))
    with pytest.raises(ValueError, match="dst_off"):
        fc.fc_cache_write(texts, tl, i32(3), i32(2), i32(3), torch.zeros(3, dtype=torch.int64), i32(3),
                          torch.zeros(5, dtype=torch.uint16))
