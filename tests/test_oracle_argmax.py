"""Pins for the oracle's per-node argmax (CPU only).

The oracle's row scan is checked against numpy.argmax (first occurrence)
on the exactly widened values, against planted maxima, and on rows built
to tie at the maximum (ties go to the lowest index; +0 and -0 are equal).
"""
import numpy as np
import pytest

import oracle
from paper_2501_12162_amd.workload import (bf16_bits_to_f32, f32_to_bf16_bits, make_tie_logits)
from conftest import cached_config


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_matches_numpy_first_occurrence(dtype):
    rng = np.random.Generator(np.random.PCG64(5))
    x = rng.standard_normal((64, 4099), dtype=np.float32) * 2
    if dtype == "bf16":
        bits = f32_to_bf16_bits(x)
        ref = np.argmax(bf16_bits_to_f32(bits), axis=1)
        got = oracle.node_argmax(bits, 4099, "bf16")
    else:
        x = np.round(x * 4) / 4          # coarse grid: plenty of ties
        ref = np.argmax(x, axis=1)
        got = oracle.node_argmax(x, 4099, "f32")
    np.testing.assert_array_equal(got, ref)


def test_natural_bf16_ties_at_full_vocab():
    rng = np.random.Generator(np.random.PCG64(6))
    bits = f32_to_bf16_bits(rng.standard_normal((48, 128256), dtype=np.float32) * 2)
    wide = bf16_bits_to_f32(bits)
    tied = (wide == wide.max(1, keepdims=True)).sum(1) > 1
    assert tied.any()                     # bf16 N(0,2) rows do tie at the max
    np.testing.assert_array_equal(oracle.node_argmax(bits, 128256, "bf16"), np.argmax(wide, 1))


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_planted_ties_resolve_to_lowest_index(dtype):
    rng = np.random.Generator(np.random.PCG64(7))
    logits, pos = make_tie_logits(rng, 40, 3000, dtype=dtype, max_ties=5, row_pad=7)
    got = oracle.node_argmax(logits, 3000, dtype)
    np.testing.assert_array_equal(got, [int(np.min(p)) for p in pos])


def test_signed_zero_ties():
    row = np.full((1, 6), -1.0, np.float32)
    row[0, 2] = -0.0
    row[0, 4] = 0.0
    assert oracle.node_argmax(row, 6, "f32")[0] == 2
    row[0, 2], row[0, 4] = 0.0, -0.0
    assert oracle.node_argmax(row, 6, "f32")[0] == 2
    assert oracle.node_argmax(f32_to_bf16_bits(row), 6, "bf16")[0] == 2


def test_padding_past_vocab_is_ignored():
    rng = np.random.Generator(np.random.PCG64(8))
    logits, pos = make_tie_logits(rng, 10, 500, dtype="bf16", max_ties=1, row_pad=64)
    logits[:, 500:] = f32_to_bf16_bits(np.full((10, 64), 1e4, np.float32))
    np.testing.assert_array_equal(oracle.node_argmax(logits, 500, "bf16"), [p[0] for p in pos])


@pytest.mark.parametrize("n", [1, 2])
def test_planted_maxima_of_named_workloads(n):
    b = cached_config(n)
    rows = np.arange(0, b.total_nodes, 7)
    got = oracle.node_argmax(b.logits, b.vocab, b.dtype, rows=rows)
    np.testing.assert_array_equal(got, b.planted_argmax[rows])
    if b.dtype == "bf16":
        # ties at about the natural bf16 rate, resolved to the lowest index;
        # every row of a tie is checked
        tied = np.nonzero(b.planted_ties > 1)[0]
        assert 0.04 * b.total_nodes <= tied.size <= 0.14 * b.total_nodes, tied.size
        np.testing.assert_array_equal(oracle.node_argmax(b.logits, b.vocab, b.dtype, rows=tied),
                                      b.planted_argmax[tied])
        x = bf16_bits_to_f32(b.logits[tied, :b.vocab])
        assert ((x == x.max(axis=1, keepdims=True)).sum(axis=1) == b.planted_ties[tied]).all()


def test_single_column_and_empty():
    assert oracle.node_argmax(np.zeros((3, 1), np.float32), 1, "f32").tolist() == [0, 0, 0]
    assert oracle.node_argmax(np.zeros((0, 5), np.float32), 5, "f32").size == 0
