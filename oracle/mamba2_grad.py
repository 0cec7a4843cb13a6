"""Gradients of log-linear Mamba-2 in float64, from the definition by the chain rule.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The forward pass is the quadratic masked form of Sec. 3.4 (Eq. 2 for M^S, Eq. 4 for M^H):

    O = (A (.) M) V,   A = Q K^T,   M = M^S (.) M^H,
    M^S[t, s] = exp(cum_t - cum_s)  (cum = cumulative sum of log alpha),
    M^H[t, s] = lambda_t^(l(t, s)),  both zero above the diagonal.

With G = dO V^T (the upstream gradient against every value) and Z = A (.) M (.) G, the
chain rule gives, per (b, h):

    dQ = (M (.) G) K          dK = (M (.) G)^T Q          dV = (M (.) A)^T dO
    dlambda_t^(l) = sum over s with l(t, s) = l of  M^S[t, s] A[t, s] G[t, s]
    dcum_t = sum_s Z[t, s] - sum_t' Z[t', t]   (cum_t enters row t with +, column t with -)
    dlog_alpha_tau = sum_{t >= tau} dcum_t      (cum_t = sum of log alpha up to t)

The paper states none of these (it only notes that its backward pass needs the lambda
gradients as well); they follow from the forward definition alone.  The tests pin them to
central finite differences of `mamba2.quadratic` and to invariants of the forward map.

Shapes as in `mamba2`: q, k [B, T, H, d_k]; v, do [B, T, H, d_v]; log_alpha [B, T, H];
lam [B, T, H, L].  All results are float64 in the layout of the matching input.
"""

import numpy as np

from . import fenwick
from .mamba2 import ss_mask, h_mask


def _f64(*xs):
    return [np.asarray(x, dtype=np.float64) for x in xs]


def quadratic_grad(q, k, v, log_alpha, lam, do):
    """(dq, dk, dv, dlog_alpha, dlam): the gradient of sum(O * do) with respect to every
    input of the quadratic form, O = (Q K^T (.) M^S (.) M^H) V."""
    q, k, v, log_alpha, lam, do = _f64(q, k, v, log_alpha, lam, do)
    B, T, H, _ = q.shape
    L = lam.shape[-1]
    dq, dk, dv = np.zeros_like(q), np.zeros_like(k), np.zeros_like(v)
    dla, dlam = np.zeros_like(log_alpha), np.zeros_like(lam)
    lev = fenwick.level_matrix(T)
    for b in range(B):
        for h in range(H):
            A = q[b, :, h] @ k[b, :, h].T
            MS = ss_mask(log_alpha[b, :, h])
            M = MS * h_mask(lam[b, :, h])
            G = do[b, :, h] @ v[b, :, h].T
            dq[b, :, h] = (M * G) @ k[b, :, h]
            dk[b, :, h] = (M * G).T @ q[b, :, h]
            dv[b, :, h] = (M * A).T @ do[b, :, h]
            Z = M * A * G
            dcum = Z.sum(axis=1) - Z.sum(axis=0)
            dla[b, :, h] = np.cumsum(dcum[::-1])[::-1]
            Y = MS * A * G
            for l in range(L):
                dlam[b, :, h, l] = np.where(lev == l, Y, 0.0).sum(axis=1)
    return dq, dk, dv, dla, dlam


def grad_rows(q, k, v, log_alpha, lam, do, rows):
    """Query-side gradients at the positions `rows` only: (dq [B, R, H, d_k],
    dlam [B, R, H, L]).  Row t needs the prefix 0..t, as in the forward."""
    q, k, v, log_alpha, lam, do = _f64(q, k, v, log_alpha, lam, do)
    B, T, H, _ = q.shape
    rows = np.asarray(rows)
    L = lam.shape[-1]
    dq = np.zeros((B, len(rows), H, q.shape[-1]))
    dlam = np.zeros((B, len(rows), H, L))
    for b in range(B):
        for h in range(H):
            A = q[b, rows, h] @ k[b, :, h].T
            MS = ss_mask(log_alpha[b, :, h], rows)
            M = MS * h_mask(lam[b, :, h], rows)
            G = do[b, rows, h] @ v[b, :, h].T
            dq[b, :, h] = (M * G) @ k[b, :, h]
            Y = MS * A * G
            for r, t in enumerate(rows):
                lv = fenwick.level_row(int(t))
                np.add.at(dlam[b, r, h], lv, Y[r, :t + 1])
    return dq, dlam


def grad_cols(q, k, v, log_alpha, lam, do, cols):
    """Key-side gradients at the positions `cols` only: (dk [B, S, H, d_k], dv [B, S, H, d_v]).
    Column s needs every query t >= s; the levels l(t, s) come from the footnote's greedy
    buckets of each t (`fenwick.level_col`)."""
    q, k, v, log_alpha, lam, do = _f64(q, k, v, log_alpha, lam, do)
    B, T, H, _ = q.shape
    cols = np.asarray(cols)
    dk = np.zeros((B, len(cols), H, k.shape[-1]))
    dv = np.zeros((B, len(cols), H, v.shape[-1]))
    for c, s in enumerate(cols):
        s = int(s)
        lv = fenwick.level_col(s, T)  # l(t, s) for t = s .. T-1
        ts = np.arange(s, T)
        for b in range(B):
            for h in range(H):
                cum = np.cumsum(log_alpha[b, :, h])
                m = np.exp(cum[ts] - cum[s]) * lam[b, ts, h, lv]
                a = q[b, ts, h] @ k[b, s, h]
                g = do[b, ts, h] @ v[b, s, h]
                dk[b, c, h] = (m * g) @ q[b, ts, h]
                dv[b, c, h] = (m * a) @ do[b, ts, h]
    return dk, dv


def dcum_at(q, k, v, log_alpha, lam, do, pos):
    """dcum_t = q_t . dq_t - k_t . dk_t at the positions `pos` ([B, P, H]).  It equals
    dlog_alpha_t - dlog_alpha_{t+1} (dlog_alpha_T = 0), so it checks the gate gradient at
    sampled positions without the full suffix sum."""
    q, k = _f64(q, k)
    pos = np.asarray(pos)
    dq, _ = grad_rows(q, k, v, log_alpha, lam, do, pos)
    dk, _ = grad_cols(q, k, v, log_alpha, lam, do, pos)
    return (np.einsum('bphd,bphd->bph', q[:, pos], dq) - np.einsum('bphd,bphd->bph', k[:, pos], dk))
