"""Host checks of the seeded input generators (no GPU, no method arithmetic).

The full-size parity tests draw only the sampled rows of a configuration's
weights; these checks pin that a row drawn alone equals the same row drawn
with the whole matrix, and that the laws have the stated scales.
"""
import math

import numpy as np
import pytest

import workloads as W


@pytest.mark.parametrize("gen", [
    lambda rows: W.llama8b_weight(1, 512, 40, rows),
    lambda rows: W.sweep_weight(256, 40, rows),
    lambda rows: W.crossover_weight(256, 40, rows),
    lambda rows: W.prefill70b_weight(256, 40, 2, rows),
])
def test_rows_drawn_alone_equal_rows_of_the_whole_matrix(gen):
    full = gen(None)
    assert full.shape[0] == 40 and full.dtype == np.float32
    rows = np.array([0, 7, 39, 12])
    assert np.array_equal(gen(rows), full[rows])


def test_row_outside_the_matrix_is_refused():
    with pytest.raises(IndexError):
        W.sweep_weight(256, 40, [40])


def test_law_scales():
    # Student-t(5) scaled to std 0.02, N(0, 0.015^2), Laplace(0, 0.01) x row multiplier
    assert abs(W.crossover_weight(8192, 64, None).std() / 0.02 - 1) < 0.03
    assert abs(W.sweep_weight(8192, 64, None).std() / 0.015 - 1) < 0.01
    m = W.prefill70b_row_multipliers(64)
    assert m.min() >= 0.5 and m.max() <= 2.0
    w = W.prefill70b_weight(8192, 64, 0, None)
    ratio = w.std(axis=1) / (math.sqrt(2) * 0.01 * m)
    assert np.all(np.abs(ratio - 1) < 0.05)


def test_llama8b_outlier_channels():
    k = 4096
    w = W.llama8b_weight(2, k, 32, None).astype(np.float64)
    cols = W.llama8b_outlier_cols(2, k)
    assert len(cols) == math.ceil(0.01 * k) == len(set(cols.tolist()))
    rest = np.setdiff1d(np.arange(k), cols)
    # Laplace(0, 0.014): mean |w| = 0.014 on ordinary channels, 8x that on outliers
    assert abs(np.abs(w[:, rest]).mean() / 0.014 - 1) < 0.02
    assert abs(np.abs(w[:, cols]).mean() / (8 * 0.014) - 1) < 0.1
