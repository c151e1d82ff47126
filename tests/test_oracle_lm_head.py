"""Pins of the LM-head + argmax oracle: brute-force sums, one-hot hidden
states that select a weight column, ties, chunking, the reported margin."""
import numpy as np
import pytest

import oracle
from oracle.tree_build import bf16_bits_to_f32


def bits(x):
    return (np.asarray(x, dtype=np.float32).view(np.uint32) >> 16).astype(np.uint16)


def test_brute_force_sums():
    rng = np.random.default_rng(0)
    h, w = bits(rng.standard_normal((3, 12))), bits(rng.standard_normal((9, 12)))
    hv, wv = bf16_bits_to_f32(h).astype(float), bf16_bits_to_f32(w).astype(float)
    want = [[sum(hv[r, i] * wv[v, i] for i in range(12)) for v in range(9)] for r in range(3)]
    np.testing.assert_allclose(oracle.lm_head_logits(h, w), want, rtol=1e-14, atol=1e-14)


def test_one_hot_hidden_selects_a_weight_column():
    rng = np.random.default_rng(1)
    w = bits(rng.standard_normal((500, 32)))
    h = np.zeros((32, 32), np.float32)
    np.fill_diagonal(h, 1.0)
    a, _, _ = oracle.lm_head_argmax(bits(h), w, chunk=64)
    wv = bf16_bits_to_f32(w)
    np.testing.assert_array_equal(a, np.argmax(wv, axis=0))


def test_ties_go_to_the_lowest_id():
    rng = np.random.default_rng(2)
    w = bits(rng.standard_normal((40, 16)) * 0.1)
    w[25] = w[7] = bits(np.full(16, 3.0))                 # two identical winning rows
    h = bits(np.ones((2, 16)))
    a, m, _ = oracle.lm_head_argmax(h, w, chunk=10)
    assert a.tolist() == [7, 7] and (m == 0).all()


@pytest.mark.parametrize("chunk", [1, 7, 64, 1000])
def test_chunking_and_margin(chunk):
    rng = np.random.default_rng(3)
    h, w = bits(rng.standard_normal((6, 24))), bits(rng.standard_normal((300, 24)))
    lg = oracle.lm_head_logits(h, w)
    a, m, sc = oracle.lm_head_argmax(h, w, chunk=chunk)
    np.testing.assert_array_equal(a, np.argmax(lg, axis=1))
    srt = np.sort(lg, axis=1)
    np.testing.assert_allclose(m, srt[:, -1] - srt[:, -2], rtol=1e-12)
    assert (sc >= np.abs(lg[np.arange(6), a])).all()
