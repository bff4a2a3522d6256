"""Pins of the oracle's tolerance metric (the relative Frobenius error per
tensor used to compare the GPU path with the oracle).

Hand values, invariances that a slip (a missing square root, normalising by
the wrong tensor, summing over the wrong axes) would break, and agreement with
the per-tensor metric of the parity tests, which is written separately."""

import math

import numpy as np

from oracle import kvx_oracle as O
from tests import _parity as P


def test_hand_values():
    assert O.rel_fro([3.0, 4.0], [0.0, 0.0]) == 5.0          # absolute when ref is zero
    assert O.rel_fro([1.0, 1.0], [1.0, 0.0]) == 1.0
    assert O.rel_fro([2.0, 0.0], [1.0, 0.0]) == 1.0
    assert O.rel_fro([1.0, 2.0], [1.0, 2.0]) == 0.0
    # ||(1,1) - (0,2)|| / ||(0,2)|| = sqrt(2) / 2 (a missing square root gives 1/2)
    assert abs(O.rel_fro([1.0, 1.0], [0.0, 2.0]) - math.sqrt(2) / 2) < 1e-15
    # normalised by the reference, not by x: ||(0,3) - (0,1)|| / ||(0,1)|| = 2
    assert O.rel_fro([0.0, 3.0], [0.0, 1.0]) == 2.0


def test_matrix_is_frobenius_not_spectral():
    ref = np.eye(3)
    x = np.zeros((3, 3))
    # Frobenius: ||I||_F = sqrt(3); spectral norm would give 1
    assert abs(O.rel_fro(x + 2 * ref, ref) - 1.0) < 1e-15
    assert abs(O.rel_fro(x, 2 * ref) - 1.0) < 1e-15
    e = np.zeros((3, 3))
    e[0, 0] = 1.0
    assert abs(O.rel_fro(ref + e, ref) - 1 / math.sqrt(3)) < 1e-15


def test_invariances():
    rng = np.random.default_rng(11)
    ref = rng.standard_normal((4, 5, 6))
    x = ref + 1e-3 * rng.standard_normal(ref.shape)
    r = O.rel_fro(x, ref)
    assert abs(O.rel_fro(7.5 * x, 7.5 * ref) - r) < 1e-12 * r       # scale invariant
    perm = rng.permutation(ref.size)
    assert abs(O.rel_fro(x.ravel()[perm], ref.ravel()[perm]) - r) < 1e-12 * r
    assert abs(O.rel_fro(x.reshape(20, 6), ref.reshape(20, 6)) - r) < 1e-12 * r


def test_agrees_with_parity_metric_per_tensor():
    rng = np.random.default_rng(12)
    want = rng.standard_normal((3, 2, 4, 9, 8))             # [L, K|V, H, T, d]
    got = (want + 1e-2 * rng.standard_normal(want.shape)).astype(np.float32)
    err = P.rel_errors(got, want)
    assert err.shape == (3, 2, 4)
    for l in range(3):
        for kv in range(2):
            for h in range(4):
                e = O.rel_fro(got[l, kv, h], want[l, kv, h])
                assert abs(err[l, kv, h] - e) <= 1e-12 * e
    # a zero reference tensor falls back to the absolute error on both sides
    want[1, 0, 2] = 0.0
    err = P.rel_errors(got, want)
    assert abs(err[1, 0, 2] - O.rel_fro(got[1, 0, 2], want[1, 0, 2])) < 1e-12
