"""Pins for the oracle's tree attention (Section IV-D, eq. (4)) and its
rotary embedding: closed forms, invariances, and agreement with a library
causal attention where the tree is a chain."""
import numpy as np
import torch

import oracle


def _rand(rng, *shape):
    return rng.uniform(-1, 1, size=shape)


def test_rope_identity_norm_and_relative_position():
    rng = np.random.default_rng(1)
    x = _rand(rng, 5, 16)
    assert np.allclose(oracle.rope(x, np.zeros(5), 10000.0), x)
    y = oracle.rope(x, np.arange(5) * 7, 10000.0)
    assert np.allclose(np.linalg.norm(y, axis=1), np.linalg.norm(x, axis=1))
    # <rope(q, m), rope(k, n)> depends on m - n only
    q, k = _rand(rng, 1, 16), _rand(rng, 1, 16)
    a = oracle.rope(q, [10], 500.0) @ oracle.rope(k, [3], 500.0).T
    b = oracle.rope(q, [107], 500.0) @ oracle.rope(k, [100], 500.0).T
    assert np.allclose(a, b)
    # one pair by hand: D = 2, angle = position
    assert np.allclose(oracle.rope(np.array([[1.0, 0.0]]), [0.5], 10.0), [[np.cos(0.5), np.sin(0.5)]])


def _inputs(rng, B, R, H, Hkv, D, Pmax):
    return (_rand(rng, B, R, H, D), _rand(rng, B, R, Hkv, D), _rand(rng, B, R, Hkv, D),
            _rand(rng, B, Pmax, Hkv, D), _rand(rng, B, Pmax, Hkv, D))


def test_chain_tree_is_causal_attention():
    """A chain (every row's ancestors are the rows before it) over a cached
    prefix is causal attention over prefix + chain: checked against torch's
    scaled_dot_product_attention in float64 on the rotated inputs."""
    rng = np.random.default_rng(2)
    B, R, H, D, P = 2, 7, 3, 8, 5
    q, kt, vt, kc, vc = _inputs(rng, B, R, H, H, D, P)
    mask = np.tril(np.ones((R, R), np.int32))[None].repeat(B, 0)
    pos = np.arange(R)[None].repeat(B, 0)
    out = oracle.tree_attention(q, kt, vt, kc, vc, [P, P], [R, R], mask, pos, rope_base=100.0)
    for b in range(B):
        p = P + np.arange(R)
        for h in range(H):
            qq = oracle.rope(q[b, :, h], p, 100.0)
            keys = np.concatenate([kc[b, :, h], oracle.rope(kt[b, :, h], p, 100.0)])
            vals = np.concatenate([vc[b, :, h], vt[b, :, h]])
            allowed = torch.ones(R, P + R, dtype=torch.bool)
            allowed[:, P:] = torch.tril(torch.ones(R, R, dtype=torch.bool))
            ref = torch.nn.functional.scaled_dot_product_attention(
                torch.from_numpy(qq)[None], torch.from_numpy(keys)[None], torch.from_numpy(vals)[None],
                attn_mask=allowed[None])[0]
            assert np.allclose(out[b, :, h], ref.numpy(), atol=1e-12)


def test_closed_forms():
    rng = np.random.default_rng(3)
    B, R, H, D, P = 1, 4, 2, 8, 3
    q, kt, vt, kc, vc = _inputs(rng, B, R, H, H, D, P)
    # zero queries: uniform weights, the mean of the allowed values
    mask = np.array([[[1, 0, 0, 0], [1, 1, 0, 0], [1, 0, 1, 0], [1, 0, 1, 1]]], np.int32)
    pos = np.array([[0, 1, 1, 2]])
    out = oracle.tree_attention(np.zeros_like(q), kt, vt, kc, vc, [P], [R], mask, pos)
    for i in range(R):
        vals = np.concatenate([vc[0, :, 0], vt[0, mask[0, i] == 1, 0]])
        assert np.allclose(out[0, i, 0], vals.mean(axis=0))
    # no prefix: the root sees only itself
    out = oracle.tree_attention(q, kt, vt, kc, vc, [0], [R], mask, pos)
    assert np.allclose(out[0, 0, 1], vt[0, 0, 1])
    # rows past num_nodes are zero, and a tree of n rows ignores rows >= n
    out2 = oracle.tree_attention(q, kt, vt, kc, vc, [P], [2], mask, pos)
    assert (out2[0, 2:] == 0).all()
    full = oracle.tree_attention(q, kt, vt, kc, vc, [P], [R], mask, pos)
    assert np.allclose(out2[0, :2], full[0, :2])
    # shifting every position (no prefix) leaves tree-only attention unchanged
    a = oracle.tree_attention(q, kt, vt, kc, vc, [0], [R], mask, pos)
    b = oracle.tree_attention(q, kt, vt, kc, vc, [0], [R], mask, pos + 40)
    assert np.allclose(a, b)


def test_grouped_heads_share_key_heads():
    """With H = 4 query heads over Hkv = 2 key heads, heads 0-1 read key head
    0 and heads 2-3 key head 1: equal to two single-head calls."""
    rng = np.random.default_rng(4)
    B, R, D, P = 1, 3, 8, 4
    q, kt, vt, kc, vc = _inputs(rng, B, R, 4, 2, D, P)
    mask = np.tril(np.ones((R, R), np.int32))[None]
    pos = np.arange(R)[None]
    out = oracle.tree_attention(q, kt, vt, kc, vc, [P], [R], mask, pos)
    for h in range(4):
        g = h // 2
        one = oracle.tree_attention(q[:, :, h:h + 1], kt[:, :, g:g + 1], vt[:, :, g:g + 1], kc[:, :, g:g + 1],
                                    vc[:, :, g:g + 1], [P], [R], mask, pos)
        assert np.allclose(out[:, :, h], one[:, :, 0])
