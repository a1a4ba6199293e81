"""The allocation-free tree-attention entry point (split-KV partials in the
library's static scratch) against the workspace entry point and the oracle:
two calls in a row on one device, the second with a smaller batch, each
bit-identical to the workspace call on the same inputs and within the bf16
bars of the oracle."""
import numpy as np
import pytest

import oracle
from paper_2501_12162_amd.workload import chain_tree, make_batch, random_tree

pytestmark = pytest.mark.gpu

BF16_ABS, BF16_REL = 2e-2, 1e-2


def _batch(seed, sizes, lens):
    rng = np.random.Generator(np.random.PCG64(seed))
    parents = [chain_tree(n) if i % 2 == 0 else random_tree(rng, n) for i, n in enumerate(sizes)]
    return make_batch(parents=parents, prefix_lens=lens, num_q_heads=32, num_kv_heads=8, head_dim=128,
                      dtype="bf16", vocab=64, seed=seed)


def test_noalloc_matches_the_workspace_entry_point():
    import torch
    import paper_2501_12162_amd as ada
    from paper_2501_12162_amd.device import DeviceBatch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    ada.load_library()
    big = _batch(91, [32] * 8, [16384, 9000, 12000, 16000, 7000, 15000, 8192, 10000])
    small = _batch(92, [12, 5, 30], [3000, 2500, 4100])
    devs = [DeviceBatch(b) for b in (big, small)]
    assert devs[0].workspace_bytes > devs[1].workspace_bytes > 0
    assert devs[0].workspace_bytes <= ada.TREE_ATTN_SCRATCH_BYTES
    refs = []
    for d in devs:
        d.attention()
        refs.append(d.out.clone())
    outs = [torch.full_like(d.out, float("nan")) for d in devs]
    for d, o in zip(devs, outs):   # two calls in a row, the second smaller
        print("noalloc call: requests", d.batch.num_requests, "workspace", d.workspace_bytes, flush=True)
        ada.adaserve_tree_attn_verify_noalloc(
            node_indptr=d.node_indptr, node_indptr_host=d.node_indptr_host, parent=d.parent, q=d.q,
            k_tree=d.k_tree, v_tree=d.v_tree, k_pages=d.k_pages, v_pages=d.v_pages,
            block_table=d.block_table, prefix_len=d.prefix_len, prefix_len_host=d.prefix_len_host,
            sm_scale=d.batch.sm_scale, out=o)
    torch.cuda.synchronize()
    for d, o, r in zip(devs, outs, refs):
        assert torch.equal(o.view(torch.int16), r.view(torch.int16))
        got = o.float().cpu().numpy()
        assert np.isfinite(got).all()
        ref = oracle.tree_attn_batch(d.batch)
        err = float(np.abs(got - ref).max())
        assert err <= BF16_ABS and err <= BF16_REL * float(np.abs(ref).max()), err


def _noalloc(ada, d, out, stream=None):
    ada.adaserve_tree_attn_verify_noalloc(
        node_indptr=d.node_indptr, node_indptr_host=d.node_indptr_host, parent=d.parent, q=d.q,
        k_tree=d.k_tree, v_tree=d.v_tree, k_pages=d.k_pages, v_pages=d.v_pages,
        block_table=d.block_table, prefix_len=d.prefix_len, prefix_len_host=d.prefix_len_host,
        sm_scale=d.batch.sm_scale, out=out, stream=stream)


def test_noalloc_replayed_from_a_graph():
    """Captured in a HIP graph (what a caller that cannot allocate does) and
    replayed three times, the output poisoned before each replay and an eager
    allocation-free call on another batch between replays (it reuses the
    same scratch): every replay and every eager call is bit-identical to the
    workspace entry point on its batch."""
    import torch
    import paper_2501_12162_amd as ada
    from paper_2501_12162_amd.device import DeviceBatch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    ada.load_library()
    d = DeviceBatch(_batch(93, [32, 20, 32, 9], [12000, 5000, 9000, 3000]))
    e = DeviceBatch(_batch(94, [7, 30], [2500, 6000]))
    for x in (d, e):
        assert 0 < x.workspace_bytes <= ada.TREE_ATTN_SCRATCH_BYTES
        x.attention()
    torch.cuda.synchronize()
    ref_d, ref_e = d.out.clone(), e.out.clone()
    out_d, out_e = torch.empty_like(d.out), torch.empty_like(e.out)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        _noalloc(ada, d, out_d, stream=side)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        _noalloc(ada, d, out_d, stream=torch.cuda.current_stream())
    for rep in range(3):
        print("graph replay", rep, flush=True)
        out_d.fill_(float("nan"))
        out_e.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out_d.view(torch.int16), ref_d.view(torch.int16)), rep
        _noalloc(ada, e, out_e)
        torch.cuda.synchronize()
        assert torch.equal(out_e.view(torch.int16), ref_e.view(torch.int16)), rep
