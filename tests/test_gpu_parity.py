"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Bars (attention against the fp64 oracle):
  * fp32: max |err| <= 1e-4;
  * bf16: max |err| <= 2e-2 AND max |err| / max |ref| <= 1e-2 (the absolute
    bar alone is loose for near-uniform softmaxes, whose outputs are small);
  * every output finite although unused page slots and pages hold NaN;
  * a mask-discriminating case where the masked and unmasked answers differ
    by far more than the tolerance.
Argmax indices, accept lengths, tokens and nodes: bit-exact.
"""
import numpy as np
import pytest

import oracle
from conftest import cached_config
from paper_2501_12162_amd.workload import (bf16_bits_to_f32, chain_tree, f32_to_bf16_bits,
                                            make_batch, make_tie_logits, random_tree)

pytestmark = pytest.mark.gpu

BF16_ABS, BF16_REL, F32_ABS = 2e-2, 1e-2, 1e-4


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2501_12162_amd as ada
    ada.load_library()
    return torch


def run_device(b, max_accept=128):
    from paper_2501_12162_amd.device import DeviceBatch
    d = DeviceBatch(b, max_accept=max_accept)
    d.step()
    return d, d.results()


def check_attention(b, out, nodes=None):
    assert np.isfinite(out).all(), "non-finite attention output"
    ref = oracle.tree_attn_batch(b, nodes=nodes)
    got = out if nodes is None else out[np.asarray(nodes)]
    err = float(np.abs(got - ref).max())
    scale = float(np.abs(ref).max())
    if b.dtype == "f32":
        assert err <= F32_ABS, err
    else:
        assert err <= BF16_ABS, err
        assert err <= BF16_REL * scale, (err, scale)
    return err


def check_argmax_accept(b, amax, alen, tok, nodes, max_accept=128):
    ref_amax = oracle.node_argmax(b.logits, b.vocab, b.dtype)
    np.testing.assert_array_equal(amax, ref_amax)
    np.testing.assert_array_equal(amax, b.planted_argmax)
    ra, rt, rn = oracle.tree_accept(b.node_indptr, b.parent, b.draft_tokens, ref_amax, max_accept)
    np.testing.assert_array_equal(alen, ra)
    np.testing.assert_array_equal(tok, rt)
    np.testing.assert_array_equal(nodes, rn)


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_named_workload(torch_cuda, cfg):
    """Every node and every head of the named workload against the oracle;
    the bf16 workloads' logits tie at the maximum in some rows."""
    b = cached_config(cfg)
    print("workload", cfg, b.name, "T", b.total_nodes, flush=True)
    _, (out, amax, alen, tok, nodes) = run_device(b)
    check_attention(b, out)
    check_argmax_accept(b, amax, alen, tok, nodes)
    if b.dtype == "bf16":
        assert (b.planted_ties > 1).sum() >= 0.04 * b.total_nodes


def test_tensor_parallel_rank_share(torch_cuda):
    """One rank's share of the 70B-shaped workload under 4-way tensor
    parallelism (16 q-heads, 2 kv-heads, a quarter of the vocabulary): every
    node against the oracle."""
    from paper_2501_12162_amd.workload import make_config
    b = make_config(4, tp=4)
    assert (b.num_q_heads, b.num_kv_heads, b.vocab) == (16, 2, 32064)
    _, (out, amax, alen, tok, nodes) = run_device(b)
    check_attention(b, out)
    check_argmax_accept(b, amax, alen, tok, nodes)


def _ragged_batch(dtype, head_dim, seed, hq=8, hkv=2):
    rng = np.random.Generator(np.random.PCG64(seed))
    sizes = [1, 5, 33, 64, 100, 128]
    lens = [0, 15, 64, 333, 1500, 5000]
    parents = [chain_tree(1), random_tree(rng, 5), random_tree(rng, 33, 6), chain_tree(64),
               random_tree(rng, 100, 10), random_tree(rng, 128)]
    assert [len(p) for p in parents] == sizes
    return make_batch(parents=parents, prefix_lens=lens, num_q_heads=hq, num_kv_heads=hkv,
                      head_dim=head_dim, dtype=dtype, vocab=5003, seed=seed, row_pad=5)


@pytest.mark.parametrize("dtype,head_dim,hq,hkv", [("bf16", 128, 8, 2), ("bf16", 64, 16, 2),
                                                   ("bf16", 128, 16, 16), ("bf16", 128, 4, 2),
                                                   ("bf16", 128, 32, 2), ("bf16", 64, 16, 1),
                                                   ("f32", 128, 4, 2), ("f32", 64, 8, 8),
                                                   ("f32", 64, 32, 2)])
def test_ragged_tiles_chunks_and_tails(torch_cuda, dtype, head_dim, hq, hkv):
    b = _ragged_batch(dtype, head_dim, seed=31 + head_dim + hq, hq=hq, hkv=hkv)
    d, (out, amax, alen, tok, nodes) = run_device(b)
    if dtype == "bf16":
        assert d.workspace_bytes > 0          # the long prefixes were split
    check_attention(b, out)
    check_argmax_accept(b, amax, alen, tok, nodes)


def test_balanced_splits_with_uneven_prefixes(torch_cuda):
    """Llama-3-8B head shapes with prefix lengths on every side of the block,
    page and chunk sizes (0 .. 17000, past the 8192-key chunk cap), so the
    planner cuts each request's prefix into its own chunk length."""
    rng = np.random.Generator(np.random.PCG64(57))
    lens = [0, 1, 31, 32, 33, 300, 1000, 1024, 1025, 2047, 3000, 4096, 5000, 8192, 8193, 17000]
    sizes = [1, 128, 64, 7, 40, 2, 33, 128, 16, 64, 9, 100, 50, 31, 80, 20]
    parents = [random_tree(rng, n, 8) for n in sizes]
    b = make_batch(parents=parents, prefix_lens=lens, num_q_heads=32, num_kv_heads=8, head_dim=128,
                   dtype="bf16", vocab=1000, seed=57)
    d, (out, amax, alen, tok, nodes) = run_device(b)
    assert d.workspace_bytes > 0
    check_attention(b, out)
    check_argmax_accept(b, amax, alen, tok, nodes)


@pytest.mark.parametrize("tree", [1, 40])
def test_every_loop_boundary_of_the_step_pipeline(torch_cuda, tree):
    """Prefixes of 1 .. 16 whole 32-key blocks, each also one key short and
    one key long, so every request runs a different mix of the five-step
    loop, the single fast steps, the branchy tail steps and the masked
    steps (and, with 40-node trees, two tree blocks after the prefix)."""
    lens = sorted({32 * k + d for k in range(1, 17) for d in (-1, 0, 1)})
    rng = np.random.Generator(np.random.PCG64(83 + tree))
    parents = [random_tree(rng, tree, 8) for _ in lens]
    b = make_batch(parents=parents, prefix_lens=lens, num_q_heads=32, num_kv_heads=8, head_dim=128,
                   dtype="bf16", vocab=1000, seed=83 + tree)
    _, (out, amax, alen, tok, nodes) = run_device(b)
    check_attention(b, out)
    check_argmax_accept(b, amax, alen, tok, nodes)


def test_out_of_pool_pages_read_as_zero_pages(torch_cuda):
    """Block-table entries outside [0, num_pages) -- negative or past the pool
    -- act as all-zero pages: the call equals, bit for bit, the same batch
    whose entries point at a real zero page appended to the pool, and the
    oracle checks that batch.  The entries sit in the start-up blocks, inside
    long runs of whole prefix blocks (the steady-state fetch path), on both
    pages of one block, and in the partial last page."""
    import dataclasses
    rng = np.random.Generator(np.random.PCG64(71))
    lens = [5000, 3001, 700, 40]
    sizes = [128, 20, 64, 5]
    parents = [random_tree(rng, n, 8) for n in sizes]
    b = make_batch(parents=parents, prefix_lens=lens, num_q_heads=32, num_kv_heads=8, head_dim=128,
                   dtype="bf16", vocab=1000, seed=71)
    P = b.num_pages
    bad, zero = b.block_table.copy(), b.block_table.copy()
    marked = 0
    for r, L in enumerate(lens):
        npg = -(-L // 16)
        for k, e in enumerate(sorted({0, 7, 40, 41, 100, npg // 2, npg // 2 + 1, npg - 1})):
            if e < npg:
                bad[r, e] = -1 if k % 2 == 0 else P + 3
                zero[r, e] = P
                marked += 1
    assert marked >= 20
    zpage = np.zeros((1,) + b.k_pages.shape[1:], dtype=b.k_pages.dtype)
    b_bad = dataclasses.replace(b, block_table=bad)
    b_zero = dataclasses.replace(b, block_table=zero, k_pages=np.concatenate([b.k_pages, zpage]),
                                 v_pages=np.concatenate([b.v_pages, zpage]))
    d, (out_bad, *_) = run_device(b_bad)
    assert d.workspace_bytes > 0
    _, (out_zero, *_) = run_device(b_zero)
    np.testing.assert_array_equal(out_bad, out_zero)
    check_attention(b_zero, out_zero)


def test_verification_step_replayed_from_a_graph(torch_cuda):
    """The whole step (attention with its split-KV merge, argmax, acceptance)
    captured once in a HIP graph, as a serving loop replays it: every replay
    reproduces the eager outputs bit for bit, with eager steps between the
    replays and the outputs poisoned before each."""
    from paper_2501_12162_amd.device import DeviceBatch
    torch = torch_cuda
    b = cached_config(2)
    d = DeviceBatch(b, max_accept=16)
    assert d.workspace_bytes > 0           # the plan splits prefixes: the merge kernel runs too
    d.step()
    torch.cuda.synchronize()
    outs = (d.out, d.target_argmax, d.accept_len, d.accept_tokens, d.accept_nodes)
    eager = [t.clone() for t in outs]
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        d.step(stream=s)   # warm-up on the side stream before capture
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        d.step(stream=torch.cuda.current_stream())
    for rep in range(4):
        d.out.fill_(float("nan"))
        for t in outs[1:]:
            t.fill_(-5)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for got, ref in zip(outs, eager):
            assert torch.equal(got.view(torch.int16) if got.dtype == torch.bfloat16 else got,
                               ref.view(torch.int16) if ref.dtype == torch.bfloat16 else ref), rep
        d.step()   # eager work between replays
        torch.cuda.synchronize()
    out, amax, alen, tok, nodes = d.results()
    check_attention(b, out)
    check_argmax_accept(b, amax, alen, tok, nodes, max_accept=16)


def test_mask_discriminating_case(torch_cuda):
    rng = np.random.Generator(np.random.PCG64(41))
    parents = [random_tree(rng, 96, 8), random_tree(rng, 40)]
    b = make_batch(parents=parents, prefix_lens=[24, 70], num_q_heads=8, num_kv_heads=2,
                   head_dim=128, dtype="bf16", vocab=64, seed=41, qkv_std=1.0)
    vt = bf16_bits_to_f32(b.v_tree) * 0.25 + 1.0       # tree values offset from the prefix's
    b.v_tree = f32_to_bf16_bits(vt)
    _, (out, *_rest) = run_device(b)
    err = check_attention(b, out)
    # the answer if every node could see every tree node of its request
    far = 0.0
    for r in range(b.num_requests):
        a, e = int(b.node_indptr[r]), int(b.node_indptr[r + 1])
        L = int(b.prefix_len[r])
        pages = b.block_table[r, :(L + 15) // 16]
        kp = bf16_bits_to_f32(b.k_pages[pages]).transpose(1, 0, 2, 3).reshape(2, -1, 128)[:, :L]
        vp = bf16_bits_to_f32(b.v_pages[pages]).transpose(1, 0, 2, 3).reshape(2, -1, 128)[:, :L]
        k = np.concatenate([kp, bf16_bits_to_f32(b.k_tree[a:e]).transpose(1, 0, 2)], 1).astype(np.float64)
        v = np.concatenate([vp, bf16_bits_to_f32(b.v_tree[a:e]).transpose(1, 0, 2)], 1).astype(np.float64)
        qh = bf16_bits_to_f32(b.q[a:e]).astype(np.float64)            # [n, 8, D]
        kk = np.repeat(k, 4, axis=0)
        vv = np.repeat(v, 4, axis=0)
        s = np.einsum("nhd,hkd->nhk", qh, kk) * b.sm_scale
        p = np.exp(s - s.max(-1, keepdims=True))
        p /= p.sum(-1, keepdims=True)
        unmasked = np.einsum("nhk,hkd->nhd", p, vv)
        far = max(far, float(np.abs(out[a:e] - unmasked).max()))
    assert far >= 10 * err, (far, err)


@pytest.mark.parametrize("dtype,vocab,pad", [("bf16", 128256, 0), ("bf16", 3001, 2),
                                             ("f32", 1024, 0), ("f32", 777, 3), ("bf16", 5, 0),
                                             ("bf16", 1, 0)])
def test_argmax_ties_and_alignment(torch_cuda, dtype, vocab, pad):
    import torch
    import paper_2501_12162_amd as ada
    from paper_2501_12162_amd.device import to_device
    rng = np.random.Generator(np.random.PCG64(vocab + pad))
    logits, pos = make_tie_logits(rng, 97, vocab, dtype=dtype, max_ties=min(6, vocab), row_pad=pad)
    dev = to_device(logits, dtype, "cuda")
    out = torch.empty(97, dtype=torch.int32, device="cuda")
    ada.adaserve_node_argmax(dev, vocab, out)
    got = out.cpu().numpy()
    np.testing.assert_array_equal(got, oracle.node_argmax(logits, vocab, dtype))
    np.testing.assert_array_equal(got, [int(np.min(p)) for p in pos])


def _accept_on_device(indptr, parent, draft, amax, max_accept):
    import torch
    import paper_2501_12162_amd as ada
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()
    B = len(indptr) - 1
    alen = torch.empty(B, dtype=torch.int32, device="cuda")
    tok = torch.empty(B, max_accept, dtype=torch.int32, device="cuda")
    nodes = torch.empty(B, max_accept, dtype=torch.int32, device="cuda")
    ada.adaserve_tree_accept(node_indptr=t(indptr), parent=t(parent), draft_tokens=t(draft),
                             target_argmax=t(amax), max_accept=max_accept, accept_len=alen,
                             accept_tokens=tok, accept_nodes=nodes)
    return alen.cpu().numpy(), tok.cpu().numpy(), nodes.cpu().numpy()


def test_accept_exhaustive_small_trees(torch_cuda):
    from test_oracle_accept import _exhaustive_batch
    indptr, parent, draft, amax = _exhaustive_batch(7)
    got = _accept_on_device(indptr, parent, draft, amax, 8)
    ref = oracle.tree_accept(indptr, parent, draft, amax, 8)
    for x, y in zip(got, ref):
        np.testing.assert_array_equal(x, y)


@pytest.mark.parametrize("max_accept", [128, 70, 9])
def test_accept_large_trees_chains_and_depth_limit(torch_cuda, max_accept):
    rng = np.random.Generator(np.random.PCG64(max_accept))
    parents = [random_tree(rng, int(rng.integers(1, 129))) for _ in range(300)]
    parents += [chain_tree(128), chain_tree(128), chain_tree(1), chain_tree(64)]
    indptr = np.concatenate([[0], np.cumsum([len(p) for p in parents])]).astype(np.int32)
    parent = np.concatenate(parents)
    T = int(indptr[-1])
    amax = rng.integers(0, 2, size=T).astype(np.int32)
    draft = rng.integers(0, 2, size=T).astype(np.int32)
    # make the two long chains match all the way down
    for r in (300, 301):
        a = indptr[r]
        draft[a + 1:a + 128] = amax[a:a + 127]
    got = _accept_on_device(indptr, parent, draft, amax, max_accept)
    ref = oracle.tree_accept(indptr, parent, draft, amax, max_accept)
    for x, y in zip(got, ref):
        np.testing.assert_array_equal(x, y)
    if max_accept == 128:
        assert got[0][300] == 128


def test_accept_malformed_trees(torch_cuda):
    ptr = np.array([0, 3, 6, 10, 11, 11, 140], np.int32)
    parent = np.concatenate([[-1, 2, 0], [0, 0, 1], [-1, 0, 1, 2], [-1], np.arange(-1, 128)]).astype(np.int32)
    T = parent.size
    draft = np.zeros(T, np.int32)
    amax = np.zeros(T, np.int32)
    got = _accept_on_device(ptr, parent, draft, amax, 3)
    # child before parent; no root; too deep; fine; empty; 129 nodes
    assert got[0].tolist() == [-1, -1, -1, 1, -1, -1]
    ref = oracle.tree_accept(ptr[:5], parent[:11], draft[:11], amax[:11], 3)
    for x, y in zip(got, ref):
        np.testing.assert_array_equal(x[:4], y[:4])


def test_empty_calls_are_noops(torch_cuda):
    import torch
    import paper_2501_12162_amd as ada
    out = torch.empty(0, dtype=torch.int32, device="cuda")
    ada.adaserve_node_argmax(torch.empty(0, 8, dtype=torch.bfloat16, device="cuda"), 8, out)
    torch.cuda.synchronize()


def test_native_library_is_the_in_tree_build(torch_cuda):
    import os
    import paper_2501_12162_amd as ada
    with open("/proc/self/maps") as f:
        maps = f.read()
    assert os.path.realpath(ada.library_path()) in maps


def test_many_requests_use_the_scan_path(torch_cuda):
    """More requests than the kernel-argument plan holds: attention units and
    split-KV merge blocks are found by scanning node_indptr / prefix_len on
    the device.  A quarter of the requests have prefixes of 2000-6000 keys,
    which the planner splits, so the merge kernel's scan branch runs too."""
    rng = np.random.Generator(np.random.PCG64(77))
    parents = [random_tree(rng, int(rng.integers(1, 12))) for _ in range(260)]
    lens = [int(x) for x in rng.integers(0, 300, size=260)]
    for r in range(0, 260, 4):
        lens[r] = int(rng.integers(2000, 6001))
    b = make_batch(parents=parents, prefix_lens=lens, num_q_heads=8, num_kv_heads=2, head_dim=128,
                   dtype="bf16", vocab=256, seed=77)
    d, (out, amax, alen, tok, nodes) = run_device(b)
    assert d.workspace_bytes > 0
    check_attention(b, out)
    check_argmax_accept(b, amax, alen, tok, nodes)


def test_workspace_reuse_across_calls(torch_cuda):
    # split prefixes leave their arrival counters at zero: a second call on the
    # same workspace (and a call after a different batch) gives the same result
    from paper_2501_12162_amd.device import DeviceBatch
    b = _ragged_batch("bf16", 128, seed=5)
    d = DeviceBatch(b)
    assert d.workspace_bytes > 0
    d.attention()
    first = d.results()[0].copy()
    d.attention()
    d.attention()
    np.testing.assert_array_equal(d.results()[0], first)
    check_attention(b, first)
