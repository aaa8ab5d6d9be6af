"""The GPU's tiling and delivery plan, modelled in numpy, reproduce the
oracle's trajectory (Theorem 2 and the lazy block update of Sec. 4.3)."""
import numpy as np
import pytest

import oracle
from paper_2607_27042_amd import build, workloads as wl

from tile_model import tile_model_round


@pytest.fixture(scope="module", autouse=True)
def _lib():
    if build.is_stale():
        build.build()


@pytest.mark.parametrize("m,n,g", [(40, 30, 4), (64, 64, 1), (150, 130, 1), (150, 130, 3),
                                   (200, 70, 2), (65, 260, 4), (400, 330, 2), (330, 460, 1),
                                   (520, 200, 3)])
def test_tile_model_matches_oracle(m, n, g):
    X, A, B = wl.random_problem(m, n, 3, "f64", "wishart").widened()
    L, _, U, _ = oracle.factors(A, B)
    Zo, Yo, _, _ = oracle.round_nested(X, L, U)
    Zt, Yt = tile_model_round(X, L, U, g)
    assert np.array_equal(Zt, Zo)
    assert np.abs(Yt - Yo).max() < 1e-9
