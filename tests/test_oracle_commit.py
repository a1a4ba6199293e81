"""Pins of the oracle's accepted-path KV commit (section 5.1: verified tokens
are stored back for the next iteration).

* a hand-worked case (tests/golden/commit_hand_worked.json) with a page
  boundary, a missing page, a node outside the tree and a malformed request;
* consistency with attention: after committing the path root..parent(i*), a
  one-node tree holding i* over the longer prefix sees exactly the keys i*
  saw in the original tree, in the same order, so the fp64 oracle gives the
  same output bit for bit;
* the copy is bit-exact for bf16 patterns and touches no other slot.
"""
import json
import os

import numpy as np
import pytest

import oracle
from paper_2501_12162_amd.workload import make_batch, random_tree, chain_tree

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "commit_hand_worked.json")


def test_hand_worked_commit():
    g = json.load(open(GOLDEN))
    ps, P, D = g["page_size"], g["num_pages"], g["head_dim"]
    indptr = np.array(g["node_indptr"], np.int32)
    T = int(indptr[-1])
    base = 1000 + 10 * np.arange(T)[:, None] + np.arange(D)[None, :]
    k_tree = base.astype(np.float32)[:, None, :]
    v_tree = (-base).astype(np.float32)[:, None, :]
    k_pages = np.full((P, 1, ps, D), 0.5, np.float32)
    v_pages = np.full((P, 1, ps, D), 0.5, np.float32)
    kp, vp, new_len = oracle.commit_kv(
        node_indptr=indptr, accept_len=g["accept_len"], accept_nodes=np.array(g["accept_nodes"]),
        k_tree=k_tree, v_tree=v_tree, k_pages=k_pages, v_pages=v_pages,
        block_table=np.array(g["block_table"]), prefix_len=g["prefix_len"], page_size=ps)
    assert new_len.tolist() == g["expected_new_prefix_len"]
    ek, ev = k_pages.copy(), v_pages.copy()
    for c in g["expected_changes"]:
        ek[c["page"], 0, c["slot"], :] = 1000 + 10 * c["row"] + np.arange(D)
        ev[c["page"], 0, c["slot"], :] = -(1000 + 10 * c["row"] + np.arange(D))
    np.testing.assert_array_equal(kp, ek)
    np.testing.assert_array_equal(vp, ev)


def _path(parent, i):
    out = [i]
    while out[-1] != 0:
        out.append(int(parent[out[-1]]))
    return out[::-1]


@pytest.mark.parametrize("shape", ["random", "chain"])
def test_commit_then_decode_equals_tree_attention(shape):
    """Committing root..parent(i*) and decoding i* alone over the longer
    prefix reproduces i*'s tree-attention output exactly (fp64 oracle)."""
    rng = np.random.Generator(np.random.PCG64(41))
    n, L, ps = 24, 37, 16
    par = random_tree(rng, n, 6) if shape == "random" else chain_tree(n)
    b = make_batch(parents=[par], prefix_lens=[L], num_q_heads=4, num_kv_heads=2, head_dim=64,
                   page_size=ps, dtype="f32", vocab=64, seed=7, reserve_tokens=n)
    i_star = n - 1 if shape == "chain" else int(np.argmax([len(_path(par, i)) for i in range(n)]))
    path = _path(par, i_star)                       # root .. i*
    d = len(path) - 1
    nodes = np.full((1, n + 1), -1, np.int32)
    nodes[0, :d] = path[:-1]                        # commit root .. parent(i*)
    kp, vp, new_len = oracle.commit_kv(
        node_indptr=b.node_indptr, accept_len=[d], accept_nodes=nodes, k_tree=b.k_tree,
        v_tree=b.v_tree, k_pages=b.k_pages, v_pages=b.v_pages, block_table=b.block_table,
        prefix_len=b.prefix_len, page_size=ps)
    assert new_len.tolist() == [L + d]
    full = oracle.tree_attn(node_indptr=b.node_indptr, parent=b.parent, prefix_len=b.prefix_len,
                            block_table=b.block_table, q=b.q, k_tree=b.k_tree, v_tree=b.v_tree,
                            k_pages=b.k_pages, v_pages=b.v_pages, dtype="f32", num_q_heads=4,
                            num_kv_heads=2, head_dim=64, page_size=ps, sm_scale=b.sm_scale,
                            nodes=[i_star])
    one = oracle.tree_attn(node_indptr=np.array([0, 1], np.int32), parent=np.array([-1], np.int32),
                           prefix_len=new_len, block_table=b.block_table, q=b.q[i_star:i_star + 1],
                           k_tree=b.k_tree[i_star:i_star + 1], v_tree=b.v_tree[i_star:i_star + 1],
                           k_pages=kp, v_pages=vp, dtype="f32", num_q_heads=4, num_kv_heads=2,
                           head_dim=64, page_size=ps, sm_scale=b.sm_scale, nodes=[0])
    np.testing.assert_array_equal(full[0], one[0])


def test_commit_is_bit_exact_and_local():
    rng = np.random.Generator(np.random.PCG64(5))
    parents = [random_tree(rng, 20, 5), chain_tree(9), random_tree(rng, 3, 2)]
    b = make_batch(parents=parents, prefix_lens=[40, 15, 0], num_q_heads=8, num_kv_heads=2,
                   head_dim=128, vocab=64, seed=3, reserve_tokens=24)
    alen, _, nodes = oracle.tree_accept(b.node_indptr, b.parent, b.draft_tokens,
                                        b.planted_argmax, 12)
    kp, vp, new_len = oracle.commit_kv(
        node_indptr=b.node_indptr, accept_len=alen, accept_nodes=nodes, k_tree=b.k_tree,
        v_tree=b.v_tree, k_pages=b.k_pages, v_pages=b.v_pages, block_table=b.block_table,
        prefix_len=b.prefix_len, page_size=16)
    assert (new_len == b.prefix_len + alen).all()
    touched = np.zeros(b.k_pages.shape[:1] + b.k_pages.shape[2:3], bool)   # [page, slot]
    for r in range(3):
        for k in range(alen[r]):
            t = b.prefix_len[r] + k
            page = b.block_table[r, t // 16]
            row = b.node_indptr[r] + nodes[r, k]
            assert kp[page, :, t % 16, :].tobytes() == b.k_tree[row].tobytes()
            assert vp[page, :, t % 16, :].tobytes() == b.v_tree[row].tobytes()
            touched[page, t % 16] = True
    untouched = ~touched
    assert kp.transpose(0, 2, 1, 3)[untouched].tobytes() == b.k_pages.transpose(0, 2, 1, 3)[untouched].tobytes()
    assert vp.transpose(0, 2, 1, 3)[untouched].tobytes() == b.v_pages.transpose(0, 2, 1, 3)[untouched].tobytes()


def test_commit_stops_at_missing_page_and_skips_malformed():
    rng = np.random.Generator(np.random.PCG64(9))
    b = make_batch(parents=[chain_tree(8), chain_tree(8)], prefix_lens=[14, 3], num_q_heads=2,
                   num_kv_heads=1, head_dim=64, vocab=64, seed=1)   # no reserve: one page each
    nodes = np.tile(np.arange(8, dtype=np.int32), (2, 1))
    kp, vp, new_len = oracle.commit_kv(
        node_indptr=b.node_indptr, accept_len=[5, -1], accept_nodes=nodes, k_tree=b.k_tree,
        v_tree=b.v_tree, k_pages=b.k_pages, v_pages=b.v_pages, block_table=b.block_table,
        prefix_len=b.prefix_len, page_size=16)
    assert new_len.tolist() == [16, 3]    # positions 14, 15 fit the one page; 16 has none
