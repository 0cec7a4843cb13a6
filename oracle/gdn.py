"""Log-linear Gated DeltaNet in float64: the definition and two independent ways to compute it.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Shapes as in oracle.mamba2, plus
    beta       [B, T, H]          delta-rule strength beta_t

Readings of the paper (listed with the other readings in the design notes):
  * The delta rule carries beta_t as in the Sec. 2 footnote on DeltaNet:
        S_t = alpha_t S_{t-1} (I - beta_t k_t k_t^T) + beta_t v_t k_t^T.
  * The parallel form of Sec. 3.4 uses (L - I) inside the inverse (as in Sec. 2's
    DeltaNet paragraph); Table 1's shorthand prints (I - L), which contradicts the
    recurrence.  With beta restored, the attention-like matrix is
        A = (Q K^T (.) L) (I + diag(beta) (K K^T (.) (L - I)))^{-1} diag(beta).
  * Per-level states (recurrent form): every level is right-multiplied by the same
    transition alpha_t (I - beta_t k_t k_t^T); merges follow Sec. 3.2.

Forms
-----
quadratic      O = (A (.) M^S (.) M^H) V                                  (Sec. 3.4)
recurrent      per-level states with the Sec. 3.2 merge rule, Eq. 3 output
bruteforce     o_t = sum_s lambda_t^(l) beta_s (k_s^T A_{s+1} ... A_t q_t) v_s with the
               transitions A_t = alpha_t (I - beta_t k_t k_t^T) multiplied out explicitly (T <= 16)
gdn_recurrent  plain Gated DeltaNet recurrence (what lambda == 1 must reduce to)
"""

import numpy as np
from scipy.linalg import solve_triangular

from . import fenwick
from .mamba2 import ss_mask, h_mask, _f64


def attention_matrix(q2, k2, beta1, rows=None):
    """A = (Q K^T (.) L)(I + diag(beta)(K K^T (.) (L - I)))^{-1} diag(beta) for one (b, h),
    restricted to `rows`.  The unit lower-triangular system is solved, never inverted."""
    T = k2.shape[0]
    rows = np.arange(T) if rows is None else np.asarray(rows)
    W = np.eye(T) + beta1[:, None] * np.tril(k2 @ k2.T, -1)
    Bm = (q2[rows] @ k2.T) * (np.arange(T)[None, :] <= rows[:, None])
    # X W = Bm  <=>  W^T X^T = Bm^T, W^T unit upper-triangular
    X = solve_triangular(W.T, Bm.T, lower=False, unit_diagonal=True).T
    return X * beta1[None, :]


def quadratic(q, k, v, log_alpha, beta, lam, rows=None):
    """Parallel form of log-linear Gated DeltaNet (Sec. 3.4): O = (A (.) M^S (.) M^H) V."""
    q, k, v, log_alpha, beta, lam = _f64(q, k, v, log_alpha, beta, lam)
    B, T, H, _ = q.shape
    rows = np.arange(T) if rows is None else np.asarray(rows)
    out = np.zeros((B, len(rows), H, v.shape[-1]))
    for b in range(B):
        for h in range(H):
            A = attention_matrix(q[b, :, h], k[b, :, h], beta[b, :, h], rows)
            P = A * ss_mask(log_alpha[b, :, h], rows) * h_mask(lam[b, :, h, :], rows)
            out[b, :, h, :] = P @ v[b, :, h, :]
    return out


def recurrent(q, k, v, log_alpha, beta, lam):
    """Per-level recurrent form (Eq. 3 output, Sec. 3.2 merges) with the gated delta rule:
    every carried or merged level state is right-multiplied by alpha_t (I - beta_t k_t k_t^T),
    then beta_t v_t k_t^T enters level 0."""
    q, k, v, log_alpha, beta, lam = _f64(q, k, v, log_alpha, beta, lam)
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    L = lam.shape[-1]
    if L < fenwick.num_levels(T):
        raise ValueError("lambda has fewer levels than the sequence needs")
    S = np.zeros((B, H, L, dv, dk))
    out = np.zeros((B, T, H, dv))
    for t in range(T):
        kt = k[:, t]                                    # [B, H, dk]
        bt = beta[:, t][:, :, None, None, None]
        if t > 0:
            p = fenwick.lssb(t)
            merged = S[:, :, :p + 1].sum(axis=2)
            S[:, :, 1:p + 1] = 0.0
            S[:, :, p + 1] = merged
            Sk = S @ kt[:, :, None, :, None]                # [B, H, L, dv, 1]
            S = S - bt * Sk * kt[:, :, None, None, :]
            S *= np.exp(log_alpha[:, t, :])[:, :, None, None, None]
        S[:, :, 0] = beta[:, t][:, :, None, None] * v[:, t, :, :, None] * kt[:, :, None, :]
        Sq = S @ q[:, t, :, None, :, None]
        out[:, t] = np.einsum('bhl,bhlp->bhp', lam[:, t], Sq[..., 0])
    return out


def bruteforce(q, k, v, log_alpha, beta, lam):
    """Explicit loops for T <= 16 with dense transition matrices multiplied in time order."""
    q, k, v, log_alpha, beta, lam = _f64(q, k, v, log_alpha, beta, lam)
    B, T, H, dk = q.shape
    if T > 16:
        raise ValueError("bruteforce is for T <= 16")
    out = np.zeros((B, T, H, v.shape[-1]))
    I = np.eye(dk)
    for b in range(B):
        for h in range(H):
            A = [float(np.exp(log_alpha[b, t, h])) * (I - beta[b, t, h] * np.outer(k[b, t, h], k[b, t, h]))
                 for t in range(T)]
            for t in range(T):
                bk = fenwick.buckets(t)
                for s in range(t + 1):
                    level = [lv for lv, members in bk.items() if s in members]
                    assert len(level) == 1
                    prod = I.copy()
                    for kk in range(s + 1, t + 1):
                        prod = prod @ A[kk]
                    w = lam[b, t, h, level[0]] * beta[b, s, h] * float(k[b, s, h] @ prod @ q[b, t, h])
                    out[b, t, h] += w * v[b, s, h]
    return out


def gdn_recurrent(q, k, v, log_alpha, beta):
    """Gated DeltaNet, S_t = alpha_t S_{t-1} (I - beta_t k_t k_t^T) + beta_t v_t k_t^T,
    o_t = S_t q_t (Sec. 2).  Log-linear GDN with all lambda equal to 1 reduces to this."""
    q, k, v, log_alpha, beta = _f64(q, k, v, log_alpha, beta)
    B, T, H, dk = q.shape
    S = np.zeros((B, H, v.shape[-1], dk))
    out = np.zeros((B, T, H, v.shape[-1]))
    for t in range(T):
        kt = k[:, t]
        Sk = (S @ kt[..., None])                         # [B, H, dv, 1]
        S = np.exp(log_alpha[:, t])[:, :, None, None] * (S - beta[:, t][:, :, None, None] * Sk * kt[:, :, None, :])
        S = S + beta[:, t][:, :, None, None] * v[:, t, :, :, None] * kt[:, :, None, :]
        out[:, t] = (S @ q[:, t, :, :, None])[..., 0]
    return out
