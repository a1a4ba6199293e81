"""GPU parity of sampled-decoding tree verification (adaserve_tree_accept_sampled)
against the oracle's tree_accept_sampled (float64), on the same uniforms.

Every decision is a floating-point comparison: an acceptance test
u * q(t) < p_res(t), or where the bonus uniform falls in the cumulative
distribution of the residual.  The kernel takes them in fp32, the oracle in
fp64.
* Acceptance tests: the oracle reports each request's smallest relative
  margin; requests whose margin exceeds MARGIN (far above the ~1e-6 relative
  fp32 error of a softmax over 128K logits) must take exactly the oracle's
  path with exactly its tokens.
* The bonus token: it must be the oracle's, or lie within CDF_TOL of the
  bonus uniform in the oracle's cumulative distribution (the kernel's fp32
  cumulative mass is a 6-level prefix over at most 64 token ranges, each a
  sum of 16 wave sums; then, inside the range that holds the target, a
  10-level scan over 1024 threads' sequential sums of at most a few hundred
  terms: a few hundred roundings of ~6e-8 at most, < 1e-5 of the total mass;
  a diffuse residual has many tokens narrower than that, so such
  near-boundary draws are expected).
* Requests with a near-tie acceptance test are checked for validity only.
"""
import numpy as np
import pytest

import oracle
from paper_2501_12162_amd.workload import (bf16_bits_to_f32, chain_tree, make_config, make_draft_logits,
                                           make_uniforms, random_tree)

pytestmark = pytest.mark.gpu

MARGIN = 1e-3
CDF_TOL = 2e-5


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2501_12162_amd as ada
    ada.load_library()
    return torch


def _dev(torch, a):
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(a).cuda()


def _run(torch, indptr, parent, draft, tl, dl, vocab, ua, ub, max_accept):
    import paper_2501_12162_amd as ada
    B = len(indptr) - 1
    alen = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    tok = torch.full((B, max_accept), -7, dtype=torch.int32, device="cuda")
    nodes = torch.full((B, max_accept), -7, dtype=torch.int32, device="cuda")
    T = len(parent)
    ws = torch.empty(max(16, ada.adaserve_tree_accept_sampled_workspace_bytes(T)), dtype=torch.uint8, device="cuda")
    ada.adaserve_tree_accept_sampled(
        node_indptr=_dev(torch, np.asarray(indptr, np.int32)), parent=_dev(torch, np.asarray(parent, np.int32)),
        draft_tokens=_dev(torch, np.asarray(draft, np.int32)), target_logits=_dev(torch, tl),
        draft_logits=_dev(torch, dl), vocab=vocab, u_accept=_dev(torch, np.asarray(ua, np.float32)),
        u_bonus=_dev(torch, np.asarray(ub, np.float32)), max_accept=max_accept, accept_len=alen,
        accept_tokens=tok, accept_nodes=nodes, workspace=ws)
    torch.cuda.synchronize()
    return alen.cpu().numpy(), tok.cpu().numpy(), nodes.cpu().numpy()


def check(torch, indptr, parent, draft, tl, dl, vocab, ua, ub, max_accept, dtype):
    widen = (lambda a: bf16_bits_to_f32(a).astype(np.float64)) if dtype == "bf16" else (
        lambda a: np.asarray(a, np.float64))
    # the oracle consumes the same fp32 uniforms, widened exactly
    ref = oracle.tree_accept_sampled(node_indptr=indptr, parent=parent, draft_tokens=draft,
                                     target_logits=widen(tl), draft_logits=widen(dl), vocab=vocab,
                                     u_accept=np.asarray(ua, np.float32).astype(np.float64),
                                     u_bonus=np.asarray(ub, np.float32).astype(np.float64),
                                     max_accept=max_accept)
    got = _run(torch, indptr, parent, draft, tl, dl, vocab, ua, ub, max_accept)
    exact = 0
    for r in range(len(indptr) - 1):
        k = int(got[0][r])
        if ref[0][r] == -1:
            assert k == -1 and (got[1][r] == -1).all() and (got[2][r] == -1).all()
            exact += 1
            continue
        base = int(indptr[r])
        assert 1 <= k <= max_accept
        path = got[2][r][:k]
        assert path[0] == 0
        for i in range(1, k):
            assert parent[base + path[i]] == path[i - 1]
            assert got[1][r][i - 1] == draft[base + path[i]]
        assert 0 <= got[1][r][k - 1] < vocab
        assert (got[1][r][k:] == -1).all() and (got[2][r][k:] == -1).all()
        if ref[3][r] <= MARGIN:
            continue   # a near-tie acceptance test: valid path is all that is asked
        assert k == ref[0][r], (r, k, ref[0][r], ref[3][r])
        np.testing.assert_array_equal(got[2][r], ref[2][r])
        np.testing.assert_array_equal(got[1][r][:k - 1], ref[1][r][:k - 1])
        v, v_ref = int(got[1][r][k - 1]), int(ref[1][r][k - 1])
        if v != v_ref:
            cdf = ref[4][r]
            u = float(np.float32(ub[base + path[-1]]))
            lo = cdf[v - 1] if v > 0 else 0.0
            assert lo - CDF_TOL <= u < cdf[v] + CDF_TOL, (r, v, v_ref, u, lo, cdf[v])
        exact += 1
    return exact


def _batch(rng, B, vocab, dtype, max_nodes, depth, noise, row_pad=0):
    parents = [random_tree(rng, int(rng.integers(1, max_nodes + 1)), depth) for _ in range(B)]
    indptr = np.cumsum([0] + [p.size for p in parents]).astype(np.int32)
    parent = np.concatenate(parents)
    T = int(indptr[-1])
    x = rng.standard_normal((T, vocab + row_pad), dtype=np.float32) * np.float32(2)
    # a few strongly preferred tokens per row, so drafts get accepted
    hot = rng.integers(0, vocab, size=(T, 3))
    np.put_along_axis(x, hot, np.float32(9.0), axis=1)
    if dtype == "bf16":
        from paper_2501_12162_amd.workload import f32_to_bf16_bits
        tl = f32_to_bf16_bits(x)
    else:
        tl = x
    dl = make_draft_logits(rng, tl, vocab, dtype, noise)
    draft = np.zeros(T, np.int32)
    for r in range(B):
        base, par = indptr[r], parents[r]
        for i in range(1, par.size):
            p = base + par[i]
            draft[base + i] = hot[p, rng.integers(0, 3)] if rng.random() < 0.8 else rng.integers(0, vocab)
    return indptr, parent, draft, tl, dl, make_uniforms(rng, T), make_uniforms(rng, T)


@pytest.mark.parametrize("seed,dtype,vocab,noise", [(0, "bf16", 32000, 0.3), (1, "bf16", 1000, 1.5),
                                                    (2, "f32", 5003, 0.5), (3, "bf16", 128256, 0.5),
                                                    (4, "f32", 17, 1.0), (7, "bf16", 1, 1.0), (8, "f32", 3, 0.5),
                                                    (9, "bf16", 65537, 0.5), (10, "f32", 98305, 0.8)])
def test_random_batches(torch_cuda, seed, dtype, vocab, noise):
    """Random trees of up to 40 nodes over vocabularies from 1 token to 128256;
    65537 (bf16: two token ranges of four statistics parts each, one token
    past the last vector) and 98305 (f32: six ranges of two parts) split the
    rows unevenly."""
    rng = np.random.Generator(np.random.PCG64(500 + seed))
    pad = (-vocab) % (8 if dtype == "bf16" else 4)
    args = _batch(rng, 12, vocab, dtype, 40, 6, noise, row_pad=pad)
    exact = check(torch_cuda, *args[:5], vocab, *args[5:], 8, dtype)
    assert exact >= 10


@pytest.mark.parametrize("seed,dtype,vocab", [(5, "f32", 1_100_003), (6, "bf16", 2_200_007),
                                              (7, "bf16", 2_097_151)])
def test_vocabularies_past_64_vector_groups(torch_cuda, seed, dtype, vocab):
    """Vocabularies whose rows hold more than 64 groups of 4096 vectors, so a
    bonus draw's token ranges span two groups each and the last one ends in a
    partial group and a few tokens past the last whole vector; and one of
    exactly 64 groups (the most token ranges, and statistics parts, a node
    takes)."""
    rng = np.random.Generator(np.random.PCG64(500 + seed))
    pad = (-vocab) % (8 if dtype == "bf16" else 4)
    args = _batch(rng, 4, vocab, dtype, 4, 3, 0.5, row_pad=pad)
    exact = check(torch_cuda, *args[:5], vocab, *args[5:], 8, dtype)
    assert exact >= 3


@pytest.mark.parametrize("seed,B,parts", [(11, 40, 2), (12, 80, 1)])
def test_statistics_parts_of_large_batches(torch_cuda, seed, B, parts):
    """The statistics pass splits each token range of a node's rows (one
    range at this vocabulary) into ceil(4096 / T) parts (at most 8), which the
    walk merges and a draw from p reads: these batches take two parts per
    node and one (no merge); the smaller batches above take 8, and at vocab
    128256 two parts in each of four ranges."""
    rng = np.random.Generator(np.random.PCG64(900 + seed))
    args = _batch(rng, B, 64, "bf16", 128, 12, 0.5)
    T = int(args[0][-1])
    assert -(-4096 // T) == parts if parts > 1 else T >= 4096
    exact = check(torch_cuda, *args[:5], 64, *args[5:], 16, "bf16")
    assert exact >= B - 3


def test_llama3_8b_batch(torch_cuda):
    """The Llama-3-8B-shaped verification batch: its trees, logits (vocab
    128256, bf16) and draft tokens; draft logits a noisy copy of the target's."""
    b = make_config(2)
    rng = np.random.Generator(np.random.PCG64(77))
    dl = make_draft_logits(rng, b.logits, b.vocab, b.dtype, 0.5)
    T = b.total_nodes
    exact = check(torch_cuda, b.node_indptr, b.parent, b.draft_tokens, b.logits, dl, b.vocab,
                  make_uniforms(rng, T), make_uniforms(rng, T), 16, "bf16")
    assert exact >= b.num_requests - 2


def test_one_hot_target_matches_greedy_kernels(torch_cuda):
    """With one-hot target distributions and distinct sibling tokens, sampled
    verification is greedy verification: compare with adaserve_node_argmax +
    adaserve_tree_accept on the same batch."""
    import paper_2501_12162_amd as ada
    torch = torch_cuda
    rng = np.random.Generator(np.random.PCG64(8))
    V, B = 4096, 16
    parents = [random_tree(rng, int(rng.integers(1, 30)), 6) for _ in range(B)]
    indptr = np.cumsum([0] + [p.size for p in parents]).astype(np.int32)
    parent = np.concatenate(parents)
    T = int(indptr[-1])
    amax = rng.integers(0, V, size=T).astype(np.int32)
    tl = np.full((T, V), -np.inf, np.float32)
    tl[np.arange(T), amax] = 0.0
    dl = rng.standard_normal((T, V)).astype(np.float32)
    draft = np.zeros(T, np.int32)
    for r in range(B):
        base, par = indptr[r], parents[r]
        for u in range(par.size):
            kids = [i for i in range(par.size) if par[i] == u]
            if kids:
                toks = rng.choice(V, size=len(kids), replace=False)
                if rng.random() < 0.7 and amax[base + u] not in toks:
                    toks[rng.integers(0, len(kids))] = amax[base + u]
                draft[base + np.asarray(kids)] = toks
    got = _run(torch, indptr, parent, draft, tl, dl, V, make_uniforms(rng, T), make_uniforms(rng, T), 12)
    ga = torch.empty(T, dtype=torch.int32, device="cuda")
    ada.adaserve_node_argmax(_dev(torch, tl), V, ga)
    alen = torch.empty(B, dtype=torch.int32, device="cuda")
    tok = torch.empty(B, 12, dtype=torch.int32, device="cuda")
    nodes = torch.empty(B, 12, dtype=torch.int32, device="cuda")
    ada.adaserve_tree_accept(node_indptr=_dev(torch, indptr), parent=_dev(torch, parent),
                             draft_tokens=_dev(torch, draft), target_argmax=ga, max_accept=12, accept_len=alen,
                             accept_tokens=tok, accept_nodes=nodes)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(got[0], alen.cpu().numpy())
    np.testing.assert_array_equal(got[1], tok.cpu().numpy())
    np.testing.assert_array_equal(got[2], nodes.cpu().numpy())


def test_roots_only_and_chains(torch_cuda):
    rng = np.random.Generator(np.random.PCG64(9))
    V = 2048
    parents = [chain_tree(1)] * 5 + [chain_tree(6)] * 3
    indptr = np.cumsum([0] + [p.size for p in parents]).astype(np.int32)
    parent = np.concatenate(parents)
    T = int(indptr[-1])
    tl = (rng.standard_normal((T, V)) * 3).astype(np.float32)
    dl = make_draft_logits(rng, tl, V, "f32", 0.2)
    draft = rng.integers(0, V, size=T).astype(np.int32)
    check(torch_cuda, indptr, parent, draft, tl, dl, V, make_uniforms(rng, T), make_uniforms(rng, T), 8, "f32")


def test_malformed_requests(torch_cuda):
    V = 64
    rng = np.random.Generator(np.random.PCG64(10))
    indptr = np.array([0, 3, 6, 9, 12, 13], np.int32)
    parent = np.array([-1, 0, 2, 0, 0, 1, -1, 0, 1, -1, 0, 1, -1], np.int32)   # bad parent; bad root; ok; deep; ok
    draft = np.array([0, 1, 2, 0, 1, 2, 0, 1, 99, 0, 1, 2, 5], np.int32)       # request 2: token out of range
    tl = rng.standard_normal((13, V)).astype(np.float32)
    dl = tl + 0.1
    got = _run(torch_cuda, indptr, parent, draft, tl, dl, V, make_uniforms(rng, 13), make_uniforms(rng, 13), 2)
    assert got[0][:4].tolist() == [-1, -1, -1, -1] and got[0][4] == 1
    assert (got[1][:4] == -1).all() and (got[2][:4] == -1).all()


def test_rejection_that_leaves_no_mass(torch_cuda):
    """Target and draft one-hot at the same token A, every child proposing
    another token: each child is rejected (its q is 0), and the rejection
    leaves no mass (p - q = 0 everywhere), so the bonus is drawn from p
    itself: A, with nothing accepted.  Roots with one child take the path
    where the rejected child is the last one; roots with 2-4 children take
    it after a pass that finds no mass.  Decided exactly on both sides (all
    probabilities are 0 or 1), so every request must match."""
    rng = np.random.Generator(np.random.PCG64(12))
    V, B = 3000, 8
    parents = [np.array([-1] + [0] * k, np.int32) for k in (1, 2, 3, 4, 1, 2, 3, 4)]
    indptr = np.cumsum([0] + [p.size for p in parents]).astype(np.int32)
    parent = np.concatenate(parents)
    T = int(indptr[-1])
    hot = rng.integers(0, V, size=T)
    tl = np.full((T, V), -np.inf, np.float32)
    tl[np.arange(T), hot] = 0.0
    dl = tl.copy()
    draft = np.zeros(T, np.int32)
    for r in range(B):
        a = hot[indptr[r]]
        for i in range(indptr[r] + 1, indptr[r + 1]):
            draft[i] = (a + 1 + rng.integers(0, V - 1)) % V   # never the root's hot token
    ua, ub = make_uniforms(rng, T), make_uniforms(rng, T)
    alen, tok, nodes = _run(torch_cuda, indptr, parent, draft, tl, dl, V, ua, ub, 6)
    ref = oracle.tree_accept_sampled(node_indptr=indptr, parent=parent, draft_tokens=draft,
                                     target_logits=tl.astype(np.float64), draft_logits=dl.astype(np.float64),
                                     vocab=V, u_accept=np.asarray(ua, np.float32).astype(np.float64),
                                     u_bonus=np.asarray(ub, np.float32).astype(np.float64), max_accept=6)
    for r in range(B):
        a = int(hot[indptr[r]])
        assert alen[r] == 1 and tok[r][0] == a and nodes[r][0] == 0, (r, alen[r], tok[r], a)
        assert (tok[r][1:] == -1).all() and (nodes[r][1:] == -1).all()
        assert ref[0][r] == 1 and ref[1][r][0] == a


def test_depth_limit_boundary(torch_cuda):
    """Chains of six nodes (depth 5): walked with six output rows, refused
    (-1) with five; the same on the oracle."""
    rng = np.random.Generator(np.random.PCG64(13))
    V = 512
    parents = [chain_tree(6)] * 4
    indptr = np.cumsum([0] + [p.size for p in parents]).astype(np.int32)
    parent = np.concatenate(parents)
    T = int(indptr[-1])
    tl = (rng.standard_normal((T, V)) * 3).astype(np.float32)
    dl = make_draft_logits(rng, tl, V, "f32", 0.2)
    draft = rng.integers(0, V, size=T).astype(np.int32)
    ua, ub = make_uniforms(rng, T), make_uniforms(rng, T)
    for K, ok in ((6, True), (5, False)):
        alen, tok, nodes = _run(torch_cuda, indptr, parent, draft, tl, dl, V, ua, ub, K)
        ref = oracle.tree_accept_sampled(node_indptr=indptr, parent=parent, draft_tokens=draft,
                                         target_logits=tl.astype(np.float64), draft_logits=dl.astype(np.float64),
                                         vocab=V, u_accept=np.asarray(ua, np.float32).astype(np.float64),
                                         u_bonus=np.asarray(ub, np.float32).astype(np.float64), max_accept=K)
        assert ((alen >= 1) == ok).all() and ((ref[0] >= 1) == ok).all(), (K, alen, ref[0])
        if not ok:
            assert (tok == -1).all() and (nodes == -1).all()


def test_passing_first_children_at_every_depth(torch_cuda):
    """A draft row equal to its target row passes every first child's test
    (u q(t) < p(t) whenever u < 1), so the walk follows first children down to
    a leaf: a 128-node chain to the full depth limit, and random trees of up to
    128 nodes.  The other requests keep a noisy draft, so links that pass sit
    next to rejections and later children in the same batch."""
    rng = np.random.Generator(np.random.PCG64(13))
    V, K = 4096, 128
    parents = [chain_tree(128), chain_tree(2)] + [random_tree(rng, int(n), d) for n, d in
                                                  [(128, 40), (128, 127), (90, 8), (64, 3), (128, 20), (33, 32)]]
    indptr = np.cumsum([0] + [p.size for p in parents]).astype(np.int32)
    parent = np.concatenate(parents)
    T = int(indptr[-1])
    tl = (rng.standard_normal((T, V)) * 2).astype(np.float32)
    hot = rng.integers(0, V, size=T)
    tl[np.arange(T), hot] = 9.0
    dl = make_draft_logits(rng, tl, V, "f32", 1.0)
    equal = [0, 1, 2, 3, 6]
    for r in equal:
        dl[indptr[r]:indptr[r + 1]] = tl[indptr[r]:indptr[r + 1]]
    draft = np.zeros(T, np.int32)
    for i in range(T):
        if parent[i] >= 0:
            p = int(np.searchsorted(indptr, i, side="right") - 1)
            pr = indptr[p] + parent[i]
            draft[i] = hot[pr] if rng.random() < 0.7 else rng.integers(0, V)
    ua, ub = make_uniforms(rng, T), make_uniforms(rng, T)
    check(torch_cuda, indptr, parent, draft, tl, dl, V, ua, ub, K, "f32")
    got = _run(torch_cuda, indptr, parent, draft, tl, dl, V, ua, ub, K)
    assert got[0][0] == 128 and (got[2][0] == np.arange(128)).all()
    for r in equal:   # every first child passes: the path is the first-child chain to a leaf
        base, n = int(indptr[r]), int(indptr[r + 1] - indptr[r])
        kids = [[c for c in range(1, n) if parent[base + c] == v] for v in range(n)]
        v, path = 0, [0]
        while kids[v]:
            v = kids[v][0]
            path.append(v)
        assert got[0][r] == len(path) and list(got[2][r][:len(path)]) == path


def test_draft_rows_of_leaves_are_not_read(torch_cuda):
    """The statistics pass skips every leaf's draft row (q at a leaf enters no
    test and no residual): leaves' draft rows of NaN leave every output bit
    unchanged.  An internal node whose draft row has no finite logit (q
    undefined) fails its request alone."""
    rng = np.random.Generator(np.random.PCG64(31))
    V, K = 1000, 8
    indptr, parent, draft, tl, dl, ua, ub = _batch(rng, 10, V, "f32", 40, 6, 0.5)
    check(torch_cuda, indptr, parent, draft, tl, dl, V, ua, ub, K, "f32")
    ref = _run(torch_cuda, indptr, parent, draft, tl, dl, V, ua, ub, K)
    internal = np.zeros(len(parent), bool)
    for r in range(len(indptr) - 1):
        for i in range(indptr[r] + 1, indptr[r + 1]):
            internal[indptr[r] + parent[i]] = True
    assert (~internal).sum() > 10
    dl_nan = dl.copy()
    dl_nan[~internal] = np.nan
    got = _run(torch_cuda, indptr, parent, draft, tl, dl_nan, V, ua, ub, K)
    for a, b in zip(ref, got):
        np.testing.assert_array_equal(a, b)
    r = next(r for r in range(len(indptr) - 1) if indptr[r + 1] - indptr[r] > 1)
    dl_inf = dl.copy()
    dl_inf[indptr[r]] = -np.inf   # the root of request r has children
    got = _run(torch_cuda, indptr, parent, draft, tl, dl_inf, V, ua, ub, K)
    assert got[0][r] == -1 and (got[1][r] == -1).all() and (got[2][r] == -1).all()
    others = np.arange(len(indptr) - 1) != r
    for a, b in zip(ref, got):
        np.testing.assert_array_equal(a[others], b[others])
    check(torch_cuda, indptr, parent, draft, tl, dl_inf, V, ua, ub, K, "f32")   # the oracle fails it too


def test_overlapping_requests(torch_cuda):
    """A node_indptr that is not increasing (request 1 has a negative node
    count, so requests 0 and 2 share nodes 0-2): request 1 fails, and each of
    the others either fails or matches the oracle on its own nodes -- the
    statistics pass may take a shared node for a leaf of one of them."""
    rng = np.random.Generator(np.random.PCG64(32))
    V, K = 512, 6
    parent = np.array([-1, 0, 0, 1, 2], np.int32)
    draft = np.array([0, 5, 9, 7, 3], np.int32)
    tl = (rng.standard_normal((5, V)) * 2).astype(np.float32)
    tl[np.arange(5), [5, 7, 3, 1, 2]] = 8.0
    dl = make_draft_logits(rng, tl, V, "f32", 0.3)
    ua, ub = make_uniforms(rng, 5), make_uniforms(rng, 5)
    indptr = np.array([0, 5, 0, 3], np.int32)
    got = _run(torch_cuda, indptr, parent, draft, tl, dl, V, ua, ub, K)
    assert got[0][1] == -1
    for r, (lo, hi) in ((0, (0, 5)), (2, (0, 3))):
        if got[0][r] == -1:
            continue
        alone = _run(torch_cuda, np.array([0, hi - lo], np.int32), parent[lo:hi], draft[lo:hi], tl[lo:hi],
                     dl[lo:hi], V, ua[lo:hi], ub[lo:hi], K)
        assert got[0][r] == alone[0][0]
        np.testing.assert_array_equal(got[1][r], alone[1][0])
        np.testing.assert_array_equal(got[2][r], alone[2][0])


@pytest.mark.parametrize("seed", range(24))
def test_drawn_batches(torch_cuda, seed):
    """Drawn shapes: 1-12 requests of 1-64 nodes, depth caps 1-12, output rows
    from the deepest node's need up to 16, vocabularies 1-40000 in either
    dtype (so the statistics parts, the first-child links, the leaves'
    skipped draft rows and both kinds of bonus draw all vary), draft noise
    0.1-2."""
    rng = np.random.Generator(np.random.PCG64(4000 + seed))
    B = int(rng.integers(1, 13))
    vocab = int(rng.choice([1, 2, 7, 8, 9, 100, 1000, 4097, 32768, 32769, int(rng.integers(1, 40001))]))
    dtype = "bf16" if rng.random() < 0.5 else "f32"
    depth = int(rng.integers(1, 13))
    noise = float(rng.uniform(0.1, 2.0))
    pad = (-vocab) % (8 if dtype == "bf16" else 4)
    args = _batch(rng, B, vocab, dtype, 64, depth, noise, row_pad=pad)
    K = int(rng.integers(depth + 1, 17)) if depth + 1 < 17 else 16
    exact = check(torch_cuda, *args[:5], vocab, *args[5:], K, dtype)
    assert exact >= B - 2
