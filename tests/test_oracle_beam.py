"""Pins of the oracle's beam-search speculation step (section 4.3 step 1):

* the log-softmax agrees with torch.log_softmax in float64 (an independent
  library routine);
* brute force on tiny vocabularies: children ranked by the product
  f(b) * softmax(logits_b)[t] computed directly from probabilities (no logs);
* the root step (one beam, log f = 0) keeps the top tokens of the row;
* a beam with path probability 0 (-inf) never contributes while others can;
* ties (equal logits within a row, equal path probabilities across beams) go
  to the smaller beam, then the smaller token.
"""
import itertools

import numpy as np
import pytest

import oracle


def test_log_softmax_against_torch():
    import torch
    rng = np.random.Generator(np.random.PCG64(1))
    x = rng.normal(0, 3, size=(3, 4, 777))
    lp = np.log(rng.random((3, 4)))
    par, tok, out = oracle.beam_step(logits=x, beam_logprob=lp, w_out=5)
    ref = torch.log_softmax(torch.from_numpy(x), dim=2).numpy() + lp[:, :, None]
    for r in range(3):
        np.testing.assert_allclose(out[r], ref[r][par[r], tok[r]], rtol=0, atol=1e-12)
        assert out[r][-1] >= np.sort(ref[r].ravel())[-5] - 1e-12


@pytest.mark.parametrize("seed", range(20))
def test_brute_force_products(seed):
    rng = np.random.Generator(np.random.PCG64(50 + seed))
    w_in, V, w_out = int(rng.integers(1, 4)), int(rng.integers(2, 7)), int(rng.integers(1, 5))
    x = rng.normal(0, 2, size=(1, w_in, V))
    f = rng.random(w_in)
    par, tok, out = oracle.beam_step(logits=x, beam_logprob=np.log(f)[None], w_out=w_out)
    p = np.exp(x[0]) / np.exp(x[0]).sum(axis=1, keepdims=True)
    prod = f[:, None] * p
    cand = sorted(itertools.product(range(w_in), range(V)), key=lambda bt: (-prod[bt], bt[0], bt[1]))
    want = cand[:min(w_out, w_in * V)]
    assert list(zip(par[0], tok[0]))[:len(want)] == want
    np.testing.assert_allclose(np.exp(out[0][:len(want)]), [prod[bt] for bt in want], rtol=1e-12)


def test_root_step_keeps_the_top_tokens():
    rng = np.random.Generator(np.random.PCG64(3))
    x = rng.normal(size=(2, 1, 1000))
    par, tok, _ = oracle.beam_step(logits=x, beam_logprob=np.zeros((2, 1)), w_out=8)
    assert (par == 0).all()
    for r in range(2):
        assert tok[r].tolist() == np.argsort(-x[r, 0], kind="stable")[:8].tolist()


def test_dead_beam_and_ties():
    x = np.zeros((1, 3, 4))
    x[0, 0] = [1.0, 1.0, 0.0, 0.0]          # tie inside beam 0
    x[0, 2] = [1.0, 1.0, 0.0, 0.0]          # same row in beam 2
    lp = np.array([[0.0, -np.inf, 0.0]])    # beam 1 is dead; beams 0 and 2 tie
    par, tok, out = oracle.beam_step(logits=x, beam_logprob=lp, w_out=6)
    assert list(zip(par[0], tok[0])) == [(0, 0), (0, 1), (2, 0), (2, 1), (0, 2), (0, 3)]
    assert np.isfinite(out[0]).all()


def test_fewer_children_than_slots():
    x = np.array([[[0.5, -0.5], [2.0, 0.0]]])
    par, tok, out = oracle.beam_step(logits=x, beam_logprob=np.array([[0.0, -np.inf]]), w_out=4)
    assert par[0].tolist() == [0, 0, -1, -1] and tok[0].tolist() == [0, 1, -1, -1]
    assert np.isneginf(out[0, 2:]).all()


def test_row_without_finite_logit_is_dead():
    x = np.full((1, 2, 3), -np.inf)
    x[0, 1] = [0.0, np.log(3.0), -np.inf]
    par, tok, out = oracle.beam_step(logits=x, beam_logprob=np.zeros((1, 2)), w_out=3)
    assert par[0].tolist() == [1, 1, -1] and tok[0].tolist() == [1, 0, -1]
    np.testing.assert_allclose(np.exp(out[0, :2]), [0.75, 0.25], rtol=1e-14)
