"""GPU parity of the draft-tree selection (adaserve_select_trees) against the
oracle's select_trees: tree sizes, parents and candidate indices must match
exactly (the only floating-point decision, the SLO phase's float32 sum, is
taken in the same order and precision on both sides)."""
import numpy as np
import pytest

import oracle
from paper_2501_12162_amd.workload import make_candidates

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2501_12162_amd as ada
    ada.load_library()
    return torch


def _run(torch, c, max_nodes=128, indptr=None):
    import paper_2501_12162_amd as ada
    dev = torch.device("cuda")
    B = c.num_requests
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    size = torch.empty(B, dtype=torch.int32, device=dev)
    tpar = torch.empty(B, max_nodes, dtype=torch.int32, device=dev)
    tcand = torch.empty(B, max_nodes, dtype=torch.int32, device=dev)
    ada.adaserve_select_trees(cand_indptr=t(c.cand_indptr if indptr is None else indptr),
                              cand_parent=t(c.cand_parent), cand_prob=t(c.cand_prob), need=t(c.need),
                              budget=c.budget, n_max=c.n_max, tree_size=size, tree_parent=tpar,
                              tree_cand=tcand)
    torch.cuda.synchronize()
    return size.cpu().numpy(), tpar.cpu().numpy(), tcand.cpu().numpy()


def _check(torch, c, indptr=None):
    ref = oracle.select_trees(cand_indptr=c.cand_indptr if indptr is None else indptr,
                              cand_parent=c.cand_parent, cand_prob=c.cand_prob, need=c.need,
                              budget=c.budget, n_max=c.n_max, max_nodes=128)
    got = _run(torch, c, indptr=indptr)
    for g, r in zip(got, ref):
        np.testing.assert_array_equal(g, r)
    return got


@pytest.mark.parametrize("seed", range(12))
def test_select_random_batches(torch_cuda, seed):
    rng = np.random.Generator(np.random.PCG64(1000 + seed))
    B = int(rng.integers(1, 70))
    d, w = int(rng.integers(1, 9)), int(rng.integers(1, 9))
    c = make_candidates(rng, B, d, w, prob_levels=[None, 3, 8][seed % 3])
    c.budget = int(rng.integers(0, B * (1 + d * w) + 5))
    c.n_max = int(rng.integers(1, 2 + d * w))
    _check(torch_cuda, c)


def test_select_large_batch_and_full_trees(torch_cuda):
    """64 requests of 127 candidates (8128 in all, near the limit)."""
    rng = np.random.Generator(np.random.PCG64(5))
    c = make_candidates(rng, 64, 1, 127)
    c.budget = 64 * 40
    size, _, _ = _check(torch_cuda, c)
    assert size.sum() == 64 * 40


def test_select_malformed_and_bad_index_array(torch_cuda):
    rng = np.random.Generator(np.random.PCG64(6))
    c = make_candidates(rng, 5, 3, 3)
    lo = c.cand_indptr
    c.cand_parent[lo[1] + 4] = 7                   # not earlier
    c.cand_prob[lo[2] + 5] = np.float32(np.nan)
    c.cand_prob[lo[3]] = np.float32(0.0)
    c.need[4] = np.float32(np.nan)
    size, _, _ = _check(torch_cuda, c)
    assert size[1] == -1 and size[2] == -1 and size[3] == -1
    bad = c.cand_indptr.copy()
    bad[-1] += 1
    size, _, _ = _check(torch_cuda, c, indptr=bad)
    assert (size == -1).all()


@pytest.mark.parametrize("B,d,w,levels,budget", [
    (512, 4, 4, 2, "third"),      # 8192 candidates, 512 requests: both limits at once, heavy ties
    (512, 16, 1, 1, "third"),     # every path probability 1: ranked by depth, request, index alone
    (64, 127, 1, 1, "third"),     # chains of 127: the deepest trees
    (8, 1, 127, 1, "third"),      # 127 siblings of probability 1
    (8, 3, 42, 1, "all"),         # budget beyond every candidate: all are taken
    (8, 3, 42, 3, "roots"),       # budget of the roots alone: nothing is added
    (33, 5, 7, None, "third"),
])
def test_select_ties_depths_and_limits(torch_cuda, B, d, w, levels, budget):
    rng = np.random.Generator(np.random.PCG64(B * 1000 + d * 10 + w))
    c = make_candidates(rng, B, d, w, prob_levels=levels)
    total = B * (1 + d * w)
    c.budget = {"third": total // 3, "all": total + 10, "roots": B}[budget]
    size, _, _ = _check(torch_cuda, c)
    assert size.sum() == min(c.budget, total)
