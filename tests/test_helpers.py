"""The parity helpers themselves: the localized bound must catch an error that a
whole-matrix relative Frobenius norm lets through."""
import numpy as np

from helpers import local_rel, rel_fro


def test_local_rel_catches_one_bad_tile():
    ref = np.random.default_rng(0).standard_normal((1024, 1024))
    got = ref.copy()
    got[256:512, 768:1024] *= 1.3                      # 30 % error in one 256 x 256 tile of 16
    assert rel_fro(got, ref) < 2e-2 * 4               # the global norm sees ~0.3 / 4
    assert local_rel(got, ref) > 0.29


def test_local_rel_catches_a_ragged_tail_row_and_zero_blocks():
    ref = np.random.default_rng(1).standard_normal((300, 70))
    got = ref.copy()
    got[299] += 0.05 * np.abs(ref[299]).max()           # last (ragged) row only
    assert local_rel(got, ref) > 0.02 and rel_fro(got, ref) < 0.01
    z = np.zeros((4, 8))
    assert local_rel(z, z) == 0.0
    bad = z.copy()
    bad[2, 3] = 1e-30                                  # a zero reference row must be matched exactly
    assert local_rel(bad, z) == np.inf


def test_local_rel_of_vectors_and_exact_results():
    v = np.arange(1.0, 9.0)
    assert local_rel(v, v) == 0.0
    assert abs(local_rel(v * (1 + 1e-3), v) - 1e-3) < 1e-12
