"""Pins for the oracle's tree attention (CPU only).

Nothing here re-types the oracle's loops.  Each test checks the oracle
against something the mathematics fixes:

* a chain-shaped tree is ordinary causal attention over prefix + chain
  (torch's scaled_dot_product_attention, fp64, bottom-right causal mask);
* a one-node tree is decode attention over the prefix plus the root;
* any node equals attention of its query over the sequence "prefix, then
  its root-to-node path" (the draft-token-tree definition, section 2);
* closed forms: zero queries average the visible values; constant values
  come back unchanged; a hand-worked 3-node example (tests/golden);
* invariances: non-ancestor tree K/V, NaN in unused page slots, physical
  page placement and topological relabelling do not change the result.
"""
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2501_12162_amd.workload import (bf16_bits_to_f32, chain_tree, make_batch,
                                            random_tree)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _f64(a, dtype):
    return (bf16_bits_to_f32(a) if dtype == "bf16" else np.asarray(a, np.float32)).astype(np.float64)


def _prefix_kv(b, r):
    """Contiguous [L, Hkv, D] prefix K and V of request r, read page by page."""
    L, ps = int(b.prefix_len[r]), b.page_size
    if L == 0:
        z = np.zeros((0, b.num_kv_heads, b.head_dim))
        return z, z
    pages = b.block_table[r, :(L + ps - 1) // ps]
    k = _f64(b.k_pages[pages], b.dtype).transpose(0, 2, 1, 3).reshape(-1, b.num_kv_heads, b.head_dim)[:L]
    v = _f64(b.v_pages[pages], b.dtype).transpose(0, 2, 1, 3).reshape(-1, b.num_kv_heads, b.head_dim)[:L]
    return k, v


def _path(par, i):
    out = []
    while i != -1:
        out.append(i)
        i = int(par[i])
    return out[::-1]


def _sdpa(q, k, v, scale, mask=None):
    """torch SDPA in fp64; q [Hq, M, D], k/v [Hkv, N, D] with kv heads
    repeated to the q heads in contiguous groups."""
    G = q.shape[0] // k.shape[0]
    kt = torch.from_numpy(k).repeat_interleave(G, dim=0)
    vt = torch.from_numpy(v).repeat_interleave(G, dim=0)
    m = None if mask is None else torch.from_numpy(mask)
    return torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q), kt, vt, attn_mask=m, scale=scale).numpy()


def _node_reference(b, node):
    """SDPA of one node's query over prefix + its root-to-node path."""
    r = int(np.searchsorted(b.node_indptr, node, side="right") - 1)
    base = int(b.node_indptr[r])
    par = b.parent[base:int(b.node_indptr[r + 1])]
    kp, vp = _prefix_kv(b, r)
    path = [base + j for j in _path(par, node - base)]
    kt = _f64(b.k_tree[path], b.dtype)
    vt = _f64(b.v_tree[path], b.dtype)
    k = np.concatenate([kp, kt], 0).transpose(1, 0, 2).copy()
    v = np.concatenate([vp, vt], 0).transpose(1, 0, 2).copy()
    q = _f64(b.q[node], b.dtype)[:, None, :].copy()
    return _sdpa(q, k, v, b.sm_scale)[:, 0, :]


@pytest.mark.parametrize("dtype,L,n", [("f32", 40, 7), ("bf16", 37, 9), ("f32", 0, 5), ("bf16", 16, 1)])
def test_chain_equals_causal_attention(dtype, L, n):
    b = make_batch(parents=[chain_tree(n)], prefix_lens=[L], num_q_heads=4, num_kv_heads=2,
                   head_dim=32, dtype=dtype, vocab=64, seed=11 + n)
    got = oracle.tree_attn_batch(b)
    kp, vp = _prefix_kv(b, 0)
    k = np.concatenate([kp, _f64(b.k_tree, dtype)], 0).transpose(1, 0, 2).copy()
    v = np.concatenate([vp, _f64(b.v_tree, dtype)], 0).transpose(1, 0, 2).copy()
    q = _f64(b.q, dtype).transpose(1, 0, 2).copy()
    mask = np.arange(L + n)[None, :] <= (L + np.arange(n))[:, None]   # bottom-right causal
    ref = _sdpa(q, k, v, b.sm_scale, mask).transpose(1, 0, 2)
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_single_node_equals_decode_attention(dtype):
    b = make_batch(parents=[chain_tree(1), chain_tree(1)], prefix_lens=[50, 129], num_q_heads=8,
                   num_kv_heads=2, head_dim=64, dtype=dtype, vocab=64, seed=5)
    got = oracle.tree_attn_batch(b)
    for r in range(2):
        kp, vp = _prefix_kv(b, r)
        k = np.concatenate([kp, _f64(b.k_tree[r:r + 1], dtype)], 0).transpose(1, 0, 2).copy()
        v = np.concatenate([vp, _f64(b.v_tree[r:r + 1], dtype)], 0).transpose(1, 0, 2).copy()
        q = _f64(b.q[r], dtype)[:, None, :].copy()
        ref = _sdpa(q, k, v, b.sm_scale)[:, 0, :]
        np.testing.assert_allclose(got[r], ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_every_node_is_attention_over_prefix_plus_root_path(seed):
    rng = np.random.Generator(np.random.PCG64(100 + seed))
    parents = [random_tree(rng, int(rng.integers(1, 24)), max_depth=int(rng.integers(1, 7)))
               for _ in range(4)]
    lens = [int(x) for x in rng.integers(0, 70, size=4)]
    b = make_batch(parents=parents, prefix_lens=lens, num_q_heads=8, num_kv_heads=2,
                   head_dim=32, dtype="bf16" if seed % 2 else "f32", vocab=64, seed=seed)
    got = oracle.tree_attn_batch(b)
    for node in range(b.total_nodes):
        np.testing.assert_allclose(got[node], _node_reference(b, node), rtol=0, atol=1e-12)


def test_sampled_nodes_match_full_evaluation():
    b = make_batch(parents=[random_tree(np.random.default_rng(3), 20)] * 2, prefix_lens=[33, 64],
                   num_q_heads=4, num_kv_heads=4, head_dim=16, dtype="f32", vocab=32, seed=9)
    full = oracle.tree_attn_batch(b)
    sel = [39, 0, 21, 5]
    np.testing.assert_array_equal(oracle.tree_attn_batch(b, nodes=sel), full[sel])


def test_zero_query_averages_visible_values():
    rng = np.random.Generator(np.random.PCG64(77))
    par = random_tree(rng, 12, max_depth=4)
    b = make_batch(parents=[par], prefix_lens=[21], num_q_heads=2, num_kv_heads=1,
                   head_dim=8, dtype="f32", vocab=16, seed=1)
    b.q[:] = 0.0
    got = oracle.tree_attn_batch(b)
    kp, vp = _prefix_kv(b, 0)
    for i in range(12):
        vis = np.concatenate([vp, b.v_tree[_path(par, i)].astype(np.float64)], 0)
        np.testing.assert_allclose(got[i], np.broadcast_to(vis.mean(0)[0], (2, 8)), atol=1e-12)


def test_constant_values_come_back_exactly():
    rng = np.random.Generator(np.random.PCG64(78))
    b = make_batch(parents=[random_tree(rng, 10)], prefix_lens=[45], num_q_heads=4,
                   num_kv_heads=2, head_dim=8, dtype="f32", vocab=16, seed=2)
    b.v_pages[np.isfinite(b.v_pages)] = 1.25
    b.v_tree[:] = 1.25
    got = oracle.tree_attn_batch(b)
    np.testing.assert_allclose(got, 1.25, rtol=1e-14)


def test_non_ancestor_kv_does_not_matter():
    rng = np.random.Generator(np.random.PCG64(79))
    par = random_tree(rng, 16)
    b = make_batch(parents=[par], prefix_lens=[30], num_q_heads=4, num_kv_heads=2,
                   head_dim=16, dtype="f32", vocab=16, seed=3)
    base = oracle.tree_attn_batch(b)
    for i in range(16):
        anc = set(_path(par, i))
        others = [j for j in range(16) if j not in anc]
        if not others:
            continue
        k2, v2 = b.k_tree.copy(), b.v_tree.copy()
        k2[others] = 1e3 * rng.standard_normal(k2[others].shape)
        v2[others] = 1e3 * rng.standard_normal(v2[others].shape)
        got = oracle.tree_attn(node_indptr=b.node_indptr, parent=b.parent, prefix_len=b.prefix_len,
                               block_table=b.block_table, q=b.q, k_tree=k2, v_tree=v2,
                               k_pages=b.k_pages, v_pages=b.v_pages, dtype="f32",
                               num_q_heads=4, num_kv_heads=2, head_dim=16, page_size=16,
                               sm_scale=b.sm_scale, nodes=[i])
        np.testing.assert_array_equal(got[0], base[i])


def test_poisoned_slots_and_page_placement_do_not_matter():
    rng = np.random.Generator(np.random.PCG64(80))
    b = make_batch(parents=[random_tree(rng, 9), chain_tree(3)], prefix_lens=[37, 18],
                   num_q_heads=4, num_kv_heads=2, head_dim=16, dtype="bf16", vocab=16, seed=4)
    assert np.isnan(bf16_bits_to_f32(b.k_pages)).any()      # NaN tails and spare pages exist
    base = oracle.tree_attn_batch(b)
    assert np.isfinite(base).all()
    # move every page to a new physical slot
    P = b.num_pages
    perm = rng.permutation(P)
    kp = np.empty_like(b.k_pages)
    vp = np.empty_like(b.v_pages)
    kp[perm] = b.k_pages
    vp[perm] = b.v_pages
    bt = np.where(b.block_table >= 0, perm[np.maximum(b.block_table, 0)], -1).astype(np.int32)
    got = oracle.tree_attn(node_indptr=b.node_indptr, parent=b.parent, prefix_len=b.prefix_len,
                           block_table=bt, q=b.q, k_tree=b.k_tree, v_tree=b.v_tree,
                           k_pages=kp, v_pages=vp, dtype="bf16", num_q_heads=4, num_kv_heads=2,
                           head_dim=16, page_size=16, sm_scale=b.sm_scale)
    np.testing.assert_array_equal(got, base)


def test_topological_relabelling_permutes_outputs():
    rng = np.random.Generator(np.random.PCG64(81))
    n = 14
    par = random_tree(rng, n)
    b = make_batch(parents=[par], prefix_lens=[20], num_q_heads=2, num_kv_heads=1,
                   head_dim=8, dtype="f32", vocab=16, seed=6)
    base = oracle.tree_attn_batch(b)
    # a random order in which every parent still precedes its children
    order, ready = [0], list(np.nonzero(par == 0)[0])
    while ready:
        j = ready.pop(int(rng.integers(0, len(ready))))
        order.append(int(j))
        ready.extend(int(c) for c in np.nonzero(par == j)[0])
    new_of = np.empty(n, dtype=np.int32)
    new_of[order] = np.arange(n)
    par2 = np.array([-1] + [new_of[par[o]] for o in order[1:]], dtype=np.int32)
    got = oracle.tree_attn(node_indptr=b.node_indptr, parent=par2, prefix_len=b.prefix_len,
                           block_table=b.block_table, q=b.q[order], k_tree=b.k_tree[order],
                           v_tree=b.v_tree[order], k_pages=b.k_pages, v_pages=b.v_pages,
                           dtype="f32", num_q_heads=2, num_kv_heads=1, head_dim=8,
                           page_size=16, sm_scale=b.sm_scale)
    np.testing.assert_allclose(got, base[order], rtol=0, atol=1e-13)


def test_golden_hand_worked_tree():
    with open(os.path.join(GOLDEN, "tree_attn_hand_worked.json")) as f:
        g = json.load(f)
    f32 = lambda x: np.asarray(x, dtype=np.float32)
    ps, D = g["page_size"], g["head_dim"]
    k_pages = np.full((1, 1, ps, D), np.nan, np.float32)
    v_pages = np.full((1, 1, ps, D), np.nan, np.float32)
    L = len(g["prefix_k"])
    k_pages[0, 0, :L] = f32(g["prefix_k"])
    v_pages[0, 0, :L] = f32(g["prefix_v"])
    n = len(g["parent"])
    q = np.repeat(f32(g["q"])[None, None, :], n, 0)
    got = oracle.tree_attn(node_indptr=[0, n], parent=g["parent"], prefix_len=[L],
                           block_table=[[0]], q=q, k_tree=f32(g["tree_k"])[:, None, :],
                           v_tree=f32(g["tree_v"])[:, None, :], k_pages=k_pages, v_pages=v_pages,
                           dtype="f32", num_q_heads=1, num_kv_heads=1, head_dim=D, page_size=ps,
                           sm_scale=g["sm_scale"])
    np.testing.assert_allclose(got[:, 0, :], np.asarray(g["expected_out"]), rtol=1e-6)


def test_malformed_tree_is_rejected():
    with pytest.raises(ValueError):
        oracle.tree_attn(node_indptr=[0, 3], parent=[-1, 2, 0], prefix_len=[0],
                         block_table=[[0]], q=np.zeros((3, 1, 4), np.float32),
                         k_tree=np.zeros((3, 1, 4), np.float32), v_tree=np.zeros((3, 1, 4), np.float32),
                         k_pages=np.zeros((1, 1, 16, 4), np.float32),
                         v_pages=np.zeros((1, 1, 16, 4), np.float32), dtype="f32",
                         num_q_heads=1, num_kv_heads=1, head_dim=4, page_size=16, sm_scale=1.0)
