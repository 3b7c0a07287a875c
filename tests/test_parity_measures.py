"""CPU checks of the GPU parity tests' row-error measure (tests/parity_measures.py)."""

import numpy as np

from parity_measures import block_row_errors, row_errors


def test_one_wrong_row_scores_about_one_where_the_block_norm_hardly_moves():
    rng = np.random.default_rng(0)
    ref = rng.standard_normal((2048, 1024))
    bad = ref.copy()
    bad[1234] = rng.standard_normal(1024)          # one gate row replaced
    block = np.linalg.norm(bad - ref) / np.linalg.norm(ref)
    assert 0.02 < block < 0.04                       # sqrt(2) / sqrt(2048) = 0.031
    assert 1.2 < row_errors(bad, ref, 2048) < 1.7    # sqrt(2) with unit-norm rows
    assert row_errors(ref, ref, 2048) == 0.0


def test_uniform_relative_noise_scores_its_size():
    rng = np.random.default_rng(1)
    ref = rng.standard_normal((512, 256))
    noisy = ref * (1 + 0.01 * rng.standard_normal(ref.shape))
    assert 0.009 < row_errors(noisy, ref, 512) < 0.015


def test_vectors_are_cut_into_rows_of_sixteen():
    def layout(_):
        return {"w": (0, (4, 3)), "b": (12, (20,))}, 32
    g = np.zeros(32)
    want = np.ones(32)
    g[:] = want
    g[12 + 17] = 5.0                                 # one element of the vector's second row
    errs = block_row_errors(g, want, None, param_layout=layout)
    assert errs["w"] == 0.0
    # second row [1,1,1,1, 0 x 12 padding] with one element off by 4; rms row
    # norm sqrt(20 / 2)
    assert abs(errs["b"] - 4.0 / np.sqrt(10.0)) < 1e-12
