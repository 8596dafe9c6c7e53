"""Pins of the compensation study's measures (CPU): the effective rank
(entropy of the normalised singular values) and the SQNR (eq. sqnr)."""
import numpy as np

from oracle import comparators as cmp
from paper_2603_04800_amd import study


def test_effective_rank_special_cases():
    assert abs(study.effective_rank(np.ones(7)) - 7.0) < 1e-12         # k equal values: k
    assert study.effective_rank(np.array([3.0, 0.0, 0.0])) == 1.0       # rank one
    assert study.effective_rank(np.zeros(4)) == 0.0
    s = np.array([4.0, 2.0, 1.0, 0.5])
    assert abs(study.effective_rank(10 * s) - study.effective_rank(s)) < 1e-12   # scale free
    # between 1 and the rank, strictly inside for unequal values
    assert 1.0 < study.effective_rank(s) < 4.0
    # masses 1/4, 1/4, 1/2: entropy (3/2) ln 2, so 2^(3/2)
    p = np.array([1.0, 1.0, 2.0])
    assert abs(study.effective_rank(p) - 2 ** 1.5) < 1e-12


def test_effective_rank_of_identity_and_low_rank_matrices():
    rng = np.random.default_rng(0)
    assert abs(study.effective_rank(np.linalg.svd(np.eye(12), compute_uv=False)) - 12) < 1e-9
    a = rng.standard_normal((30, 3)) @ rng.standard_normal((3, 20))
    assert study.effective_rank(np.linalg.svd(a, compute_uv=False)) <= 3.0 + 1e-6


def test_sqnr_matches_the_oracle_definition():
    rng = np.random.default_rng(1)
    ref = rng.standard_normal((9, 33))
    y = ref + 1e-2 * rng.standard_normal((9, 33))
    y[4] = ref[4]                                                        # exact row: +inf
    assert np.allclose(study.sqnr_db(ref, y)[np.arange(9) != 4],
                       cmp.sqnr_db(ref, y)[np.arange(9) != 4], rtol=1e-12)
    assert np.isinf(study.sqnr_db(ref, y)[4])
