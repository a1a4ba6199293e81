"""GPU parity of one beam-search speculation step (adaserve_beam_step) against
the oracle's beam_step (float64).

The kernel computes each row's log-sum-exp in float32, so a child's score
carries a small rounding error; SCORE_TOL bounds it (float32 sums of at
most 8192 terms per slice, then at most a few dozen slices, then two
additions of magnitudes below ~100: a few 1e-6 relative, i.e. a few 1e-5
absolute at the scores used here).  The comparison is therefore exact where
the ranking is decided by more than the tolerance, and a validity check
where it is not: two children whose float64 scores lie within 2 * SCORE_TOL
may be ranked either way by float32 arithmetic.  Exact ties (equal logits in
one row; equal rows with equal beam scores) are decided identically on both
sides by the stated tie rules and are compared exactly.
"""
import numpy as np
import pytest

import oracle
from paper_2501_12162_amd.workload import bf16_bits_to_f32, f32_to_bf16_bits, make_beam_batch

pytestmark = pytest.mark.gpu

SCORE_TOL = 5e-5


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2501_12162_amd as ada
    ada.load_library()
    return torch


def _run(torch, logits, vocab, lp, w_out, dtype, calls=1):
    import paper_2501_12162_amd as ada
    dev = torch.device("cuda")
    if dtype == "bf16":
        x = torch.from_numpy(np.ascontiguousarray(logits).view(np.int16)).to(dev).view(torch.bfloat16)
    else:
        x = torch.from_numpy(np.ascontiguousarray(logits, dtype=np.float32)).to(dev)
    B, w_in = lp.shape
    code = ada.ADASERVE_BF16 if dtype == "bf16" else ada.ADASERVE_F32
    ws = torch.empty(max(1, ada.adaserve_beam_step_workspace_bytes(B, w_in, vocab, w_out, code)),
                     dtype=torch.uint8, device=dev)
    lp_d = torch.from_numpy(np.ascontiguousarray(lp, dtype=np.float32)).to(dev)
    par = torch.full((B, w_out), -7, dtype=torch.int32, device=dev)
    tok = torch.full((B, w_out), -7, dtype=torch.int32, device=dev)
    out = torch.full((B, w_out), 7.0, dtype=torch.float32, device=dev)
    for _ in range(calls):
        ada.adaserve_beam_step(logits=x, vocab=vocab, beam_logprob=lp_d, out_parent=par, out_token=tok,
                               out_logprob=out, workspace=ws)
    torch.cuda.synchronize()
    return par.cpu().numpy(), tok.cpu().numpy(), out.cpu().numpy()


def _values(logits, vocab, B, w_in, dtype):
    x = bf16_bits_to_f32(logits) if dtype == "bf16" else np.asarray(logits, np.float32)
    return x[:, :vocab].reshape(B, w_in, vocab).astype(np.float64)


def check(torch, logits, vocab, lp, w_out, dtype):
    B, w_in = lp.shape
    x = _values(logits, vocab, B, w_in, dtype)
    par, tok, out = _run(torch, logits, vocab, lp, w_out, dtype)
    score = oracle.beam_log_path_prob(x, lp.astype(np.float64))            # [B, w_in, V]
    opar, otok, olp = oracle.beam_step(logits=x, beam_logprob=lp.astype(np.float64), w_out=w_out + 1)
    exact = 0
    for r in range(B):
        kept = int(np.isfinite(olp[r, :w_out]).sum())
        got = int((par[r] >= 0).sum())
        assert got == kept, (r, got, kept)
        assert (par[r, :kept] >= 0).all() and (par[r, :kept] < w_in).all()
        assert (tok[r, :kept] >= 0).all() and (tok[r, :kept] < vocab).all()
        assert (par[r, kept:] == -1).all() and (tok[r, kept:] == -1).all()
        assert np.isneginf(out[r, kept:]).all()
        assert len(set(zip(par[r, :kept].tolist(), tok[r, :kept].tolist()))) == kept
        s_got = score[r, par[r, :kept], tok[r, :kept]]
        assert np.isfinite(s_got).all()
        tol = SCORE_TOL * np.maximum(1.0, np.abs(s_got) / 20)
        # the written score is the child's score
        np.testing.assert_array_less(np.abs(out[r, :kept] - s_got), tol)
        # the k-th pick has the k-th best score, up to rounding
        np.testing.assert_array_less(np.abs(s_got - olp[r, :kept]), 2 * tol)
        # Group the oracle's ranking into clusters of scores closer than the
        # tolerance.  A cluster of one child, or of exactly equal scores
        # (decided by the tie rules on both sides), must match exactly; a
        # cluster holding a near tie may come out in another order.
        ref = olp[r]
        k = 0
        while k < kept:
            e = k
            while e + 1 < ref.size and np.isfinite(ref[e + 1]) and abs(ref[e] - ref[e + 1]) <= 4 * tol[min(e, kept - 1)]:
                e += 1
            if all(ref[j] == ref[k] for j in range(k, e + 1)):
                for j in range(k, min(e + 1, kept)):
                    assert (par[r, j], tok[r, j]) == (opar[r, j], otok[r, j]), (r, j)
                    exact += 1
            k = e + 1
    return exact


def test_root_step_llama_vocab(torch_cuda):
    rng = np.random.Generator(np.random.PCG64(1))
    b = make_beam_batch(rng, 5, 1, 128256, root_step=True)
    assert check(torch_cuda, b.logits, b.vocab, b.beam_logprob, 8, "bf16") > 30


def test_llama_shape_with_unused_beams(torch_cuda):
    rng = np.random.Generator(np.random.PCG64(2))
    b = make_beam_batch(rng, 16, 8, 128256, dead_beams=2)
    assert check(torch_cuda, b.logits, b.vocab, b.beam_logprob, 8, "bf16") > 100


def test_long_context_batch_shape(torch_cuda):
    """8 requests x 8 beams over 128256 tokens (the long-context batch's
    beam step: 64 rows, two scan workgroups per row)."""
    rng = np.random.Generator(np.random.PCG64(4))
    b = make_beam_batch(rng, 8, 8, 128256)
    assert check(torch_cuda, b.logits, b.vocab, b.beam_logprob, 8, "bf16") > 50


def test_qwen_vocab_padded_rows(torch_cuda):
    rng = np.random.Generator(np.random.PCG64(3))
    b = make_beam_batch(rng, 4, 4, 151936, row_pad=64)
    check(torch_cuda, b.logits, b.vocab, b.beam_logprob, 16, "bf16")


@pytest.mark.parametrize("dtype,vocab,pad", [("f32", 1001, 3), ("bf16", 9000, 8), ("f32", 4097, 3),
                                             ("bf16", 8192, 0), ("bf16", 17, 7)])
def test_ragged_vocab_tails(torch_cuda, dtype, vocab, pad):
    rng = np.random.Generator(np.random.PCG64(vocab))
    b = make_beam_batch(rng, 3, 3, vocab, dtype=dtype, row_pad=pad)
    check(torch_cuda, b.logits, b.vocab, b.beam_logprob, 5, dtype)


def test_widest_beams(torch_cuda):
    rng = np.random.Generator(np.random.PCG64(4))
    b = make_beam_batch(rng, 2, 64, 20000, std=3.0)
    check(torch_cuda, b.logits, b.vocab, b.beam_logprob, 64, "bf16")


def test_fewer_children_than_slots(torch_cuda):
    x = np.array([[0.5, -0.5, 1.0, 0.0], [2.0, 0.0, 0.0, 0.0]], dtype=np.float32)  # vocab 3, stride 4
    lp = np.array([[0.0, -np.inf]], dtype=np.float32)
    par, tok, out = _run(torch_cuda, x, 3, lp, 8, "f32")
    assert par[0].tolist() == [0, 0, 0, -1, -1, -1, -1, -1]
    assert tok[0].tolist() == [2, 0, 1, -1, -1, -1, -1, -1]
    check(torch_cuda, x, 3, lp, 8, "f32")


@pytest.mark.parametrize("V", [3000, 16384])   # a ragged chunk only; whole chunks only (bf16 2, fp32 4)
def test_ties_dead_rows_and_neg_inf_logits(torch_cuda, V):
    rng = np.random.Generator(np.random.PCG64(5))
    B, w_in = 3, 4
    x = (rng.standard_normal((B * w_in, V)).astype(np.float32) * 2)
    x[0] = 0.0                                   # constant row: every token ties
    x[2] = x[1]                                  # identical rows, equal beam scores below
    x[5, ::3] = -np.inf                          # tokens of probability 0
    x[6] = -np.inf                               # a live beam whose row has no finite logit
    x[9, :] = np.round(x[9, :])                  # many equal logits in one row
    lp = np.log(rng.random((B, w_in))).astype(np.float32)
    lp[0, 2] = lp[0, 1]
    bits = f32_to_bf16_bits(x)
    check(torch_cuda, bits, V, lp, 12, "bf16")
    check(torch_cuda, x, V, lp, 12, "f32")


@pytest.mark.parametrize("order", ["increasing", "decreasing", "sawtooth"])
def test_adversarial_orders_refill_the_candidate_buffer(torch_cuda, order):
    # Increasing rows make every vector beat the running threshold, so the
    # per-wave candidate buffer is cut back many times.
    V, B, w_in = 40000, 2, 3
    base = np.linspace(-8, 8, V, dtype=np.float32)
    if order == "decreasing":
        base = base[::-1].copy()
    elif order == "sawtooth":
        base = np.tile(np.linspace(-4, 4, 1000, dtype=np.float32), V // 1000)
    x = np.stack([base + np.float32(0.01 * i) for i in range(B * w_in)])
    lp = np.log(np.linspace(0.9, 0.2, B * w_in)).reshape(B, w_in).astype(np.float32)
    check(torch_cuda, f32_to_bf16_bits(x), V, lp, 64, "bf16")
    check(torch_cuda, x, V, lp, 33, "f32")


def test_peaked_and_wide_logits(torch_cuda):
    rng = np.random.Generator(np.random.PCG64(6))
    b = make_beam_batch(rng, 4, 4, 50000, std=8.0)
    vals = bf16_bits_to_f32(b.logits)
    vals[::2, 123] = 60.0                        # one dominant token in every other row
    check(torch_cuda, f32_to_bf16_bits(vals), b.vocab, b.beam_logprob, 8, "bf16")


def test_repeated_calls_reuse_the_workspace(torch_cuda):
    rng = np.random.Generator(np.random.PCG64(7))
    b = make_beam_batch(rng, 6, 2, 30000)
    one = _run(torch_cuda, b.logits, b.vocab, b.beam_logprob, 8, "bf16")
    three = _run(torch_cuda, b.logits, b.vocab, b.beam_logprob, 8, "bf16", calls=3)
    for a, c in zip(one, three):
        np.testing.assert_array_equal(a, c)


def test_chained_steps_replayed_from_a_graph(torch_cuda):
    """d speculation steps (the first from the roots, each later one taking
    the previous step's kept children as its beams) captured once in a HIP
    graph and replayed, as the draft steps after the first are replayed from
    a captured graph (section 5.2).  Every replay must reproduce the eager
    chain exactly; eager work runs between replays."""
    import paper_2501_12162_amd as ada
    torch = torch_cuda
    rng = np.random.Generator(np.random.PCG64(11))
    B, w, V, d = 6, 4, 30000, 4
    dev = torch.device("cuda")
    logits = []
    for k in range(d):
        b = make_beam_batch(rng, B, 1 if k == 0 else w, V)
        logits.append(torch.from_numpy(b.logits.view(np.int16)).to(dev).view(torch.bfloat16))
    root_lp = torch.zeros(B, 1, dtype=torch.float32, device=dev)
    outs = [(torch.empty(B, w, dtype=torch.int32, device=dev), torch.empty(B, w, dtype=torch.int32, device=dev),
             torch.empty(B, w, dtype=torch.float32, device=dev)) for _ in range(d)]
    nbytes = max(ada.adaserve_beam_step_workspace_bytes(B, 1 if k == 0 else w, V, w, ada.ADASERVE_BF16)
                 for k in range(d))
    ws = torch.empty(nbytes, dtype=torch.uint8, device=dev)

    def chain():
        lp = root_lp
        for k in range(d):
            par, tok, out = outs[k]
            ada.adaserve_beam_step(logits=logits[k], vocab=V, beam_logprob=lp, out_parent=par, out_token=tok,
                                   out_logprob=out, workspace=ws)
            lp = out

    chain()
    torch.cuda.synchronize()
    eager = [[t.clone() for t in o] for o in outs]
    # the eager chain agrees with the oracle step by step
    lp = np.zeros((B, 1))
    for k in range(d):
        x = bf16_bits_to_f32(logits[k].view(torch.int16).cpu().numpy().view(np.uint16)).astype(np.float64)
        x = x.reshape(B, lp.shape[1], V)
        opar, otok, olp = oracle.beam_step(logits=x, beam_logprob=lp, w_out=w)
        got_lp = eager[k][2].cpu().numpy()
        np.testing.assert_allclose(got_lp, olp, rtol=0, atol=SCORE_TOL * 4)
        lp = got_lp.astype(np.float64)   # next step from the kernel's own scores
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        chain()   # warm-up on the side stream before capture
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        chain()
    for rep in range(4):
        for o in outs:
            for t in o:
                t.fill_(-5)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k in range(d):
            for a_, b_ in zip(outs[k], eager[k]):
                assert torch.equal(a_, b_), (rep, k)
        chain()   # eager work between replays
        torch.cuda.synchronize()


@pytest.mark.parametrize("w_in,w_out", [(16, 16), (17, 16), (4, 64)])
def test_final_selection_both_forms(torch_cuda, w_in, w_out):
    """W·K = 256 and 4·64 = 256 place the children by rank (one thread
    each); 17·16 = 272 takes the head merge: both give the oracle's
    children in its order."""
    rng = np.random.Generator(np.random.PCG64(w_in * 100 + w_out))
    b = make_beam_batch(rng, 3, w_in, 5000)
    check(torch_cuda, b.logits, b.vocab, b.beam_logprob, w_out, "bf16")


@pytest.mark.parametrize("seed", range(16))
def test_drawn_shapes(torch_cuda, seed):
    """Drawn shapes: 1-20 requests of 1-16 beams, 1-24 children kept,
    vocabularies of 1-200000 tokens in either dtype with padded rows (at most
    8M logits a batch), logit spreads 0.5-6, root steps and unused beams."""
    rng = np.random.Generator(np.random.PCG64(7000 + seed))
    dtype = "bf16" if rng.random() < 0.5 else "f32"
    vocab = int(rng.choice([1, 2, 15, 16, 17, 4095, 4096, 65536, 65537, int(rng.integers(1, 200001))]))
    B = int(rng.integers(1, 21))
    w_in = int(rng.integers(1, 17))
    while B * w_in * vocab > 8_000_000 and B * w_in > 1:
        B, w_in = max(1, B // 2), max(1, w_in // 2)
    w_out = int(rng.integers(1, 25))
    pad = (-vocab) % (8 if dtype == "bf16" else 4) + int(rng.integers(0, 2)) * 8
    dead = int(rng.integers(0, w_in)) if rng.random() < 0.3 else 0
    b = make_beam_batch(rng, B, w_in, vocab, dtype=dtype, std=float(rng.uniform(0.5, 6.0)), row_pad=pad,
                        root_step=rng.random() < 0.2, dead_beams=dead)
    check(torch_cuda, b.logits, b.vocab, b.beam_logprob, w_out, dtype)
