"""GPU parity of the one-call verification step (adaserve_tree_verify_step):
every output -- attention, argmax, accept length, tokens and nodes -- is
bit-identical to the three separate calls (attention, argmax, acceptance)
on the same inputs, and within the oracle's bars on its own."""
import numpy as np
import pytest

from conftest import cached_config
from paper_2501_12162_amd.workload import chain_tree, make_batch, random_tree
from test_gpu_parity import _ragged_batch, check_argmax_accept, check_attention

pytestmark = pytest.mark.gpu


def _outs(d):
    return (d.out, d.target_argmax, d.accept_len, d.accept_tokens, d.accept_nodes)


def _same(got, ref):
    import torch
    v = lambda t: t.view(torch.int16) if t.dtype == torch.bfloat16 else t
    return torch.equal(v(got), v(ref))


def fused_matches_separate(b, max_accept=128, check_oracle=False):
    import torch
    import paper_2501_12162_amd as ada
    from paper_2501_12162_amd.device import DeviceBatch
    ada.load_library()
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    print("step case:", b.name, "requests", b.num_requests, "T", b.total_nodes, flush=True)
    d = DeviceBatch(b, max_accept=max_accept)
    d.step()
    torch.cuda.synchronize()
    ref = [t.clone() for t in _outs(d)]
    d.out.fill_(float("nan"))
    for t in _outs(d)[1:]:
        t.fill_(-7)
    d.fused_step()
    torch.cuda.synchronize()
    for name, got, r in zip(("out", "argmax", "accept_len", "accept_tokens", "accept_nodes"), _outs(d), ref):
        assert _same(got, r), name
    if check_oracle:
        out, amax, alen, tok, nodes = d.results()
        check_attention(b, out)
        check_argmax_accept(b, amax, alen, tok, nodes, max_accept=max_accept)
    return d


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_step_on_named_workloads(cfg):
    fused_matches_separate(cached_config(cfg), check_oracle=cfg in (1, 2))


@pytest.mark.parametrize("dtype,head_dim,hq,hkv", [("bf16", 128, 8, 2), ("bf16", 64, 32, 4), ("f32", 128, 4, 2)])
def test_step_on_ragged_batches(dtype, head_dim, hq, hkv):
    b = _ragged_batch(dtype, head_dim, seed=301 + head_dim + hq, hq=hq, hkv=hkv)
    d = fused_matches_separate(b, check_oracle=True)
    if dtype == "bf16":
        assert d.workspace_bytes > 0


def test_step_without_splits_and_with_a_depth_limit():
    """Short prefixes (no split-KV merge: the second launch is acceptance
    only) and max_accept below some trees' depth (those requests get -1)."""
    rng = np.random.Generator(np.random.PCG64(311))
    parents = [chain_tree(20), random_tree(rng, 50, 4), chain_tree(3), random_tree(rng, 128)]
    b = make_batch(parents=parents, prefix_lens=[100, 0, 37, 120], num_q_heads=32, num_kv_heads=8,
                   head_dim=128, dtype="bf16", vocab=3001, seed=311)
    d = fused_matches_separate(b, max_accept=9, check_oracle=True)
    assert d.workspace_bytes == 0
    assert (d.accept_len.cpu().numpy() == -1).any()


def test_step_on_the_scan_path():
    """More requests than the kernel-argument plan table holds, some split:
    attention units, merge blocks and the appended argmax workgroups and
    acceptance waves all found without the table."""
    rng = np.random.Generator(np.random.PCG64(313))
    parents = [random_tree(rng, int(rng.integers(1, 12))) for _ in range(260)]
    lens = [int(x) for x in rng.integers(0, 300, size=260)]
    for r in range(0, 260, 4):
        lens[r] = int(rng.integers(2000, 6001))
    b = make_batch(parents=parents, prefix_lens=lens, num_q_heads=8, num_kv_heads=2, head_dim=128,
                   dtype="bf16", vocab=256, seed=313)
    d = fused_matches_separate(b, check_oracle=True)
    assert d.workspace_bytes > 0


def test_step_replayed_from_a_graph():
    """The one-call step captured in a HIP graph and replayed, eager steps
    between replays, outputs poisoned before each: every replay reproduces
    the eager outputs bit for bit."""
    import torch
    b = cached_config(2)
    d = fused_matches_separate(b, max_accept=16)
    ref = [t.clone() for t in _outs(d)]
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        d.fused_step(stream=s)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        d.fused_step(stream=torch.cuda.current_stream())
    for rep in range(4):
        d.out.fill_(float("nan"))
        for t in _outs(d)[1:]:
            t.fill_(-5)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for got, r in zip(_outs(d), ref):
            assert _same(got, r), rep
        d.fused_step()
        torch.cuda.synchronize()
