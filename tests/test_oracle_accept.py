"""Pins for the oracle's longest-accepted-path acceptance (CPU only).

* Exhaustive: every tree with up to 7 nodes (every parent array with
  parent[i] < i) under every pattern of matching draft tokens, topological
  pass vs enumeration of all root-to-leaf paths.
* Hand-worked trees (tests/golden/accept_hand_worked.json).
* Theorem 1 (section 3) in the setting it describes (siblings carry
  distinct tokens, so at most one child of a node can match): the mean
  accepted length over many draws equals the sum of path probabilities
  f(v), root included.
* A chain with independent matches has E[accept_len] = sum_k p^k.
* Structural invariants of every emitted path (root-connected, Appendix B;
  each emitted token is the target's argmax at the previous path node).
"""
import itertools
import json
import os

import numpy as np
import pytest

import oracle
from paper_2501_12162_amd.workload import random_tree

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _all_parent_arrays(n):
    for choice in itertools.product(*[range(i) for i in range(1, n)]):
        yield np.array((-1,) + choice, dtype=np.int32)


def _exhaustive_batch(max_n):
    parents, drafts, amaxes = [], [], []
    for n in range(1, max_n + 1):
        for par in _all_parent_arrays(n):
            for mask in range(1 << (n - 1)):
                amax = 1000 + np.arange(n, dtype=np.int32)
                draft = 5000 + np.arange(n, dtype=np.int32)
                draft[0] = 777
                for j in range(1, n):
                    if mask >> (j - 1) & 1:
                        draft[j] = amax[par[j]]
                parents.append(par)
                drafts.append(draft)
                amaxes.append(amax)
    sizes = [len(p) for p in parents]
    indptr = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    return indptr, np.concatenate(parents), np.concatenate(drafts), np.concatenate(amaxes)


def _check_structure(indptr, parent, draft, amax, alen, tok, nodes):
    for r in range(indptr.size - 1):
        base = indptr[r]
        n = alen[r]
        assert n >= 1
        path = nodes[r, :n]
        assert path[0] == 0
        for k in range(1, n):
            assert parent[base + path[k]] == path[k - 1]          # root-connected
            assert draft[base + path[k]] == amax[base + path[k - 1]]
        np.testing.assert_array_equal(tok[r, :n], amax[base + path])  # greedy-lossless tokens
        assert (tok[r, n:] == -1).all() and (nodes[r, n:] == -1).all()


def test_exhaustive_small_trees_topological_vs_bruteforce():
    indptr, parent, draft, amax = _exhaustive_batch(7)
    assert indptr.size - 1 == 1 + 1 * 2 + 2 * 4 + 6 * 8 + 24 * 16 + 120 * 32 + 720 * 64
    a = oracle.tree_accept(indptr, parent, draft, amax, 8)
    b = oracle.tree_accept_bruteforce(indptr, parent, draft, amax, 8)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)
    sel = np.arange(0, indptr.size - 1, 37)
    sub_ptr = np.concatenate([[0], np.cumsum(np.diff(indptr)[sel])]).astype(np.int32)
    take = np.concatenate([np.arange(indptr[r], indptr[r + 1]) for r in sel])
    _check_structure(sub_ptr, parent[take], draft[take], amax[take],
                     a[0][sel], a[1][sel], a[2][sel])


def test_random_larger_trees_with_colliding_tokens():
    rng = np.random.Generator(np.random.PCG64(21))
    parents = [random_tree(rng, int(rng.integers(1, 40))) for _ in range(3000)]
    indptr = np.concatenate([[0], np.cumsum([len(p) for p in parents])]).astype(np.int32)
    parent = np.concatenate(parents)
    T = int(indptr[-1])
    amax = rng.integers(0, 3, size=T).astype(np.int32)      # tiny vocab: many duplicate matches
    draft = rng.integers(0, 3, size=T).astype(np.int32)
    a = oracle.tree_accept(indptr, parent, draft, amax, 40)
    b = oracle.tree_accept_bruteforce(indptr, parent, draft, amax, 40)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)
    _check_structure(indptr, parent, draft, amax, *a)


def test_golden_hand_worked_cases():
    with open(os.path.join(GOLDEN, "accept_hand_worked.json")) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        par = np.asarray(c["parent"], np.int32)
        ptr = np.array([0, par.size], np.int32)
        for fn in (oracle.tree_accept, oracle.tree_accept_bruteforce):
            alen, tok, nodes = fn(ptr, par, c["draft"], c["argmax"], c["max_accept"])
            assert alen[0] == c["accept_len"], c["name"]
            assert tok[0].tolist() == c["accept_tokens"], c["name"]
            assert nodes[0].tolist() == c["accept_nodes"], c["name"]


def test_theorem1_expected_accepted_equals_sum_of_path_probabilities():
    rng = np.random.Generator(np.random.PCG64(22))
    n = 24
    par = random_tree(rng, n, max_depth=5)
    children = [np.nonzero(par == u)[0] for u in range(n)]
    # per-child probability of being the one child that matches its parent
    pi = np.zeros(n)
    for u in range(n):
        c = children[u]
        if c.size:
            w = rng.random(c.size + 1)
            pi[c] = 0.9 * w[:-1] / w.sum()
    f = np.ones(n)
    for v in range(1, n):
        f[v] = f[par[v]] * pi[v]
    trials = 40000
    amax = np.tile(1000 + np.arange(n, dtype=np.int32), trials)
    draft = np.tile(5000 + np.arange(n, dtype=np.int32), trials)
    for u in range(n):
        c = children[u]
        if not c.size:
            continue
        probs = np.append(pi[c], 1.0 - pi[c].sum())
        pick = rng.choice(c.size + 1, size=trials, p=probs)
        for j, child in enumerate(c):
            hit = np.nonzero(pick == j)[0]
            draft[hit * n + child] = 1000 + u
    indptr = (np.arange(trials + 1) * n).astype(np.int32)
    alen, _, _ = oracle.tree_accept(indptr, np.tile(par, trials), draft, amax, n)
    mean, se = alen.mean(), alen.std() / np.sqrt(trials)
    assert abs(mean - f.sum()) < 4.5 * se, (mean, f.sum(), se)


@pytest.mark.parametrize("p,n", [(0.7, 8), (0.6, 11), (0.8, 32)])
def test_chain_closed_form(p, n):
    rng = np.random.Generator(np.random.PCG64(int(p * 100) + n))
    trials = 30000
    amax = np.tile(np.arange(n, dtype=np.int32), trials)
    draft = np.tile(np.arange(-1, n - 1, dtype=np.int32), trials)      # all match ...
    miss = rng.random(trials * n) >= p
    draft[miss] = -7                                                      # ... unless drawn off
    indptr = (np.arange(trials + 1) * n).astype(np.int32)
    par = np.tile(np.arange(-1, n - 1, dtype=np.int32), trials)
    alen, _, _ = oracle.tree_accept(indptr, par, draft, amax, n)
    expect = sum(p ** k for k in range(n))
    se = alen.std() / np.sqrt(trials)
    assert abs(alen.mean() - expect) < 4.5 * se, (alen.mean(), expect)


def test_malformed_and_too_deep_trees():
    ptr = np.array([0, 3, 6, 10, 11, 11], np.int32)
    parent = np.array([-1, 2, 0,  0, 0, 1,  -1, 0, 1, 2,  -1], np.int32)
    T = parent.size
    draft = np.zeros(T, np.int32)
    amax = np.zeros(T, np.int32)
    for fn in (oracle.tree_accept, oracle.tree_accept_bruteforce):
        alen, tok, nodes = fn(ptr, parent, draft, amax, 3)
        # child before parent; no root at local 0; depth 3 > max_accept-1; ok; empty tree
        assert alen.tolist() == [-1, -1, -1, 1, -1]
        assert (tok[[0, 1, 2, 4]] == -1).all() and (nodes[[0, 1, 2, 4]] == -1).all()
        assert nodes[3].tolist() == [0, -1, -1] and tok[3].tolist() == [0, -1, -1]
