"""Pins for the oracle of log-linear Mamba-2 with matrix-valued level weights
(oracle/matrix_lambda.py, the 4D-tensor view of App. A).

  * the three forms (level-by-level quadratic, per-level recurrent, and brute force over explicit
    d_k x d_k entries M[t, s] with greedy buckets and products of alpha) agree;
  * Lambda_t^(l) = lambda_t^(l) I reduces to the scalar-weight oracle of Sec. 3.4 (itself pinned
    to the paper's worked example and special cases), in both the diagonal and the full layout;
  * orientation: Lambda_t^(l) = lambda_t^(l) P for a fixed non-symmetric permutation P equals
    the scalar model on the permuted queries q P (a transposed Lambda gives q P^T instead);
  * level isolation: Lambda nonzero at one level only equals the scalar model with one-hot
    weights on the queries transformed by that level's matrix;
  * linearity in Lambda, and sampled rows against the full output."""

import numpy as np
import pytest

from oracle import fenwick, mamba2
from oracle import matrix_lambda as ml


def _rand(seed, B, T, H, dk, dv):
    rng = np.random.default_rng(seed)
    L = fenwick.num_levels(T)
    q = rng.standard_normal((B, T, H, dk)) / np.sqrt(dk)
    k = rng.standard_normal((B, T, H, dk)) / np.sqrt(dk)
    v = rng.standard_normal((B, T, H, dv))
    la = -np.logaddexp(0, rng.standard_normal((B, T, H)))
    full = rng.standard_normal((B, T, H, L, dk, dk)) / np.sqrt(dk)
    diag = np.logaddexp(0, rng.standard_normal((B, T, H, L, dk)))
    lam = np.logaddexp(0, rng.standard_normal((B, T, H, L)))
    return q, k, v, la, full, diag, lam


def _rel(a, b):
    return np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300)


@pytest.mark.parametrize("T", [1, 2, 5, 8, 13, 16])
def test_forms_match_bruteforce(T):
    q, k, v, la, full, diag, _ = _rand(T, 1, T, 2, 3, 2)
    for Lam in (full, diag):
        ref = ml.bruteforce(q, k, v, la, Lam)
        assert _rel(ml.quadratic(q, k, v, la, Lam), ref) < 1e-12
        assert _rel(ml.recurrent(q, k, v, la, Lam), ref) < 1e-12


@pytest.mark.parametrize("T", [37, 64, 100])
def test_recurrent_matches_quadratic(T):
    q, k, v, la, full, diag, _ = _rand(100 + T, 2, T, 2, 4, 3)
    for Lam in (full, diag):
        assert _rel(ml.recurrent(q, k, v, la, Lam), ml.quadratic(q, k, v, la, Lam)) < 1e-12


@pytest.mark.parametrize("T", [9, 70])
def test_scaled_identity_is_the_scalar_model(T):
    q, k, v, la, _, _, lam = _rand(200 + T, 2, T, 3, 4, 3)
    ref = mamba2.quadratic(q, k, v, la, lam)
    diag = np.repeat(lam[..., None], q.shape[-1], axis=-1)
    assert _rel(ml.quadratic(q, k, v, la, diag), ref) < 1e-12
    assert _rel(ml.quadratic(q, k, v, la, ml.as_full(diag)), ref) < 1e-12


def test_orientation_is_query_times_lambda():
    T, dk = 40, 5
    q, k, v, la, _, _, lam = _rand(7, 1, T, 2, dk, 3)
    P = np.roll(np.eye(dk), 1, axis=1)  # a cyclic shift: P != P^T
    Lam = lam[..., None, None] * P
    got = ml.quadratic(q, k, v, la, Lam)
    assert _rel(got, mamba2.quadratic(q @ P, k, v, la, lam)) < 1e-12
    assert _rel(got, mamba2.quadratic(q @ P.T, k, v, la, lam)) > 1e-2


@pytest.mark.parametrize("level", [0, 1, 3, 5])
def test_single_level_isolation(level):
    T, dk = 48, 4
    q, k, v, la, full, _, _ = _rand(30 + level, 1, T, 2, dk, 3)
    L = full.shape[3]
    Lam = np.zeros_like(full)
    Lam[:, :, :, level] = full[:, :, :, level]
    onehot = np.zeros(full.shape[:4])
    onehot[..., level] = 1.0
    # per row t: q_t Lambda_t^(level), a row-dependent transform, so compare row by row
    qt = np.einsum('btha,bthac->bthc', q, full[:, :, :, level])
    got = ml.quadratic(q, k, v, la, Lam)
    ref = mamba2.quadratic(qt, k, v, la, onehot)
    assert L > level and _rel(got, ref) < 1e-12


def test_linear_in_lambda_and_sampled_rows():
    T = 60
    q, k, v, la, full, diag, _ = _rand(5, 1, T, 2, 3, 2)
    a = ml.quadratic(q, k, v, la, full)
    b = ml.quadratic(q, k, v, la, ml.as_full(diag))
    assert _rel(ml.quadratic(q, k, v, la, full + ml.as_full(diag)), a + b) < 1e-12
    rows = np.array([0, 1, 31, 32, 59])
    assert _rel(ml.quadratic(q, k, v, la, full, rows=rows), a[:, rows]) < 1e-13
    assert _rel(ml.level_queries(q, diag), q[:, :, :, None, :] * diag) < 1e-15
