"""Pins for the oracle's log-linear Mamba-2 and Gated DeltaNet forms.

Each check compares against something fixed by the paper or by mathematics, not against a
retyped copy of the same formula: the two forms of the method against each other and against
explicit-product brute force; the reductions the paper states (equal lambdas give the
underlying linear-attention model; alpha = 1 gives plain linear attention); and closed forms
of the delta rule (orthogonal keys, querying the key just written)."""

import numpy as np
import pytest

from oracle import fenwick, gdn, mamba2
from synthetic import WORKLOADS, generate


def _rand(seed, B, T, H, dk, dv, slow=False):
    rng = np.random.default_rng(seed)
    L = fenwick.num_levels(T)
    q = rng.standard_normal((B, T, H, dk)) / np.sqrt(dk)
    k = rng.standard_normal((B, T, H, dk)) / np.sqrt(dk)
    v = rng.standard_normal((B, T, H, dv))
    shift = -6.0 if slow else 0.0
    la = -np.logaddexp(0, rng.standard_normal((B, T, H)) + shift)
    lam = np.logaddexp(0, rng.standard_normal((B, T, H, L)))
    beta = 1 / (1 + np.exp(-rng.standard_normal((B, T, H))))
    return q, k, v, la, lam, beta


def _rel(a, b):
    return np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300)


# ---------------------------------------------------------------- log-linear Mamba-2

def test_mamba2_forms_agree_first_workload():
    w = WORKLOADS["ll_mamba2_f32_T64"]
    x = generate(w)
    a = mamba2.quadratic(x["q"], x["k"], x["v"], x["log_alpha"], x["lam"])
    b = mamba2.recurrent(x["q"], x["k"], x["v"], x["log_alpha"], x["lam"])
    assert _rel(a, b) < 1e-12


@pytest.mark.parametrize("T", [1, 2, 3, 7, 33, 100, 257])
@pytest.mark.parametrize("slow", [False, True])
def test_mamba2_quadratic_equals_recurrent(T, slow):
    q, k, v, la, lam, _ = _rand(T, 2, T, 3, 5, 4, slow)
    assert _rel(mamba2.quadratic(q, k, v, la, lam), mamba2.recurrent(q, k, v, la, lam)) < 1e-12


@pytest.mark.parametrize("T", [1, 2, 5, 8, 13, 16])
def test_mamba2_bruteforce(T):
    q, k, v, la, lam, _ = _rand(100 + T, 1, T, 2, 4, 3, slow=True)
    ref = mamba2.bruteforce(q, k, v, la, lam)
    assert _rel(mamba2.quadratic(q, k, v, la, lam), ref) < 1e-12
    assert _rel(mamba2.recurrent(q, k, v, la, lam), ref) < 1e-12


def test_mamba2_lambda_one_is_gated_linear_attention():
    q, k, v, la, lam, _ = _rand(7, 2, 150, 2, 6, 5)
    ones = np.ones_like(lam)
    ref = mamba2.gla_recurrent(q, k, v, la)
    assert _rel(mamba2.quadratic(q, k, v, la, ones), ref) < 1e-12
    assert _rel(mamba2.recurrent(q, k, v, la, ones), ref) < 1e-12


def test_mamba2_alpha_one_lambda_one_is_linear_attention():
    q, k, v, la, lam, _ = _rand(8, 1, 70, 2, 4, 4)
    zero = np.zeros_like(la)
    ones = np.ones_like(lam)
    ref = mamba2.linear_attention_parallel(q, k, v)
    assert _rel(mamba2.quadratic(q, k, v, zero, ones), ref) < 1e-12
    assert _rel(mamba2.recurrent(q, k, v, zero, ones), ref) < 1e-12


def test_mamba2_lambda_constant_over_levels_scales_rows():
    # Sec. 3.1: lambdas that agree across levels (lambda_t^(l) = c_t) collapse to linear
    # attention; here gated: O = diag(c) O_GLA.
    q, k, v, la, lam, _ = _rand(9, 1, 90, 2, 4, 3)
    c = np.abs(np.random.default_rng(1).standard_normal((1, 90, 2))) + 0.1
    lam_c = np.repeat(c[..., None], lam.shape[-1], axis=-1)
    ref = c[..., None] * mamba2.gla_recurrent(q, k, v, la)
    assert _rel(mamba2.quadratic(q, k, v, la, lam_c), ref) < 1e-12


def test_mamba2_levels_partition_the_output():
    # O is linear in lambda and each (t, s) pair has exactly one level: the outputs with
    # one-hot level weights sum to the output with all-ones weights.
    q, k, v, la, lam, _ = _rand(10, 1, 64, 1, 4, 4, slow=True)
    L = lam.shape[-1]
    tot = 0
    for lv in range(L):
        oh = np.zeros_like(lam)
        oh[..., lv] = 1.0
        tot = tot + mamba2.quadratic(q, k, v, la, oh)
    assert _rel(tot, mamba2.gla_recurrent(q, k, v, la)) < 1e-12


def test_mamba2_sampled_rows_equal_full():
    q, k, v, la, lam, _ = _rand(11, 2, 120, 2, 4, 4)
    rows = np.array([0, 5, 63, 64, 119])
    full = mamba2.quadratic(q, k, v, la, lam)
    part = mamba2.quadratic(q, k, v, la, lam, rows=rows)
    np.testing.assert_allclose(part, full[:, rows], rtol=0, atol=1e-13)


# ---------------------------------------------------------------- log-linear Gated DeltaNet

@pytest.mark.parametrize("T", [1, 2, 5, 16, 37, 64])
def test_gdn_quadratic_equals_recurrent(T):
    q, k, v, la, lam, beta = _rand(200 + T, 2, T, 2, 6, 5)
    k = k / np.linalg.norm(k, axis=-1, keepdims=True)
    a = gdn.quadratic(q, k, v, la, beta, lam)
    b = gdn.recurrent(q, k, v, la, beta, lam)
    assert _rel(a, b) < 1e-11


@pytest.mark.parametrize("T", [1, 3, 8, 16])
def test_gdn_bruteforce(T):
    q, k, v, la, lam, beta = _rand(300 + T, 1, T, 2, 4, 3, slow=True)
    k = k / np.linalg.norm(k, axis=-1, keepdims=True)
    ref = gdn.bruteforce(q, k, v, la, beta, lam)
    assert _rel(gdn.quadratic(q, k, v, la, beta, lam), ref) < 1e-11
    assert _rel(gdn.recurrent(q, k, v, la, beta, lam), ref) < 1e-11


def test_gdn_delta_sign_reading():
    # Table 1 prints (I - L) inside the inverse; Sec. 2 and Sec. 3.4 print (L - I).  Only
    # (L - I) matches the recurrence.  Build the (I - L) variant here and check it fails.
    q, k, v, la, lam, beta = _rand(31, 1, 12, 1, 4, 3)
    k = k / np.linalg.norm(k, axis=-1, keepdims=True)
    ref = gdn.bruteforce(q, k, v, la, beta, lam)
    q2, k2, b2 = q[0, :, 0], k[0, :, 0], beta[0, :, 0]
    T = 12
    W = np.eye(T) - b2[:, None] * np.tril(k2 @ k2.T, -1)
    A = ((q2 @ k2.T) * np.tril(np.ones((T, T)))) @ np.linalg.inv(W) * b2[None, :]
    P = A * mamba2.ss_mask(la[0, :, 0]) * mamba2.h_mask(lam[0, :, 0])
    wrong = P @ v[0, :, 0]
    assert _rel(wrong, ref[0, :, 0]) > 1e-3


def test_gdn_beta_zero_gives_zero():
    q, k, v, la, lam, beta = _rand(12, 1, 40, 2, 4, 4)
    z = np.zeros_like(beta)
    assert np.max(np.abs(gdn.quadratic(q, k, v, la, z, lam))) == 0.0
    assert np.max(np.abs(gdn.recurrent(q, k, v, la, z, lam))) == 0.0


def test_gdn_lambda_one_is_gated_deltanet():
    q, k, v, la, lam, beta = _rand(13, 2, 80, 2, 5, 4)
    k = k / np.linalg.norm(k, axis=-1, keepdims=True)
    ones = np.ones_like(lam)
    ref = gdn.gdn_recurrent(q, k, v, la, beta)
    assert _rel(gdn.quadratic(q, k, v, la, beta, ones), ref) < 1e-11
    assert _rel(gdn.recurrent(q, k, v, la, beta, ones), ref) < 1e-11


def test_gdn_orthonormal_keys_reduce_to_gla():
    # With mutually orthogonal unit keys, (I - beta_t k_t k_t^T) leaves every earlier
    # k_s untouched, so the delta rule adds beta_t v_t k_t^T exactly like gated linear
    # attention with values beta_t v_t; this holds level by level, so for any lambda.
    B, T, H, d = 1, 12, 2, 16
    rng = np.random.default_rng(14)
    q, _, v, la, lam, beta = _rand(14, B, T, H, d, 3)
    k = np.zeros((B, T, H, d))
    for h in range(H):
        Qm, _ = np.linalg.qr(rng.standard_normal((d, d)))
        k[0, :, h] = Qm[:T]
    ref = mamba2.quadratic(q, k, beta[..., None] * v, la, lam)
    assert _rel(gdn.quadratic(q, k, v, la, beta, lam), ref) < 1e-12
    assert _rel(gdn.recurrent(q, k, v, la, beta, lam), ref) < 1e-12


def test_gdn_query_of_written_key_returns_value():
    # Delta rule with beta = 1, alpha = 1: S_t k_t = S_{t-1}(k_t - k_t) + v_t = v_t for a unit
    # key, so querying with q_t = k_t returns v_t exactly (lambda = 1).
    q, k, v, la, lam, beta = _rand(15, 1, 30, 2, 8, 5)
    k = k / np.linalg.norm(k, axis=-1, keepdims=True)
    out = gdn.quadratic(k, k, v, np.zeros_like(la), np.ones_like(beta), np.ones_like(lam))
    np.testing.assert_allclose(out, v, rtol=0, atol=1e-10)
    out = gdn.recurrent(k, k, v, np.zeros_like(la), np.ones_like(beta), np.ones_like(lam))
    np.testing.assert_allclose(out, v, rtol=0, atol=1e-10)


def test_gdn_workload_prefix_forms_agree():
    w = WORKLOADS["ll_gdn_bf16_T8192"]
    x = generate(w.with_(B=1, H=2, T=128, dk=16, dv=16))
    a = gdn.quadratic(x["q"], x["k"], x["v"], x["log_alpha"], x["beta"], x["lam"])
    b = gdn.recurrent(x["q"], x["k"], x["v"], x["log_alpha"], x["beta"], x["lam"])
    assert _rel(a, b) < 1e-11
