"""Log-linear Mamba-2 with matrix-valued level weights (the 4D-tensor view, App. A), in float64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

App. A writes the attention score of a pair as P[t, s] = q_t M[t, s] k_s^T with a d_k x d_k
matrix per pair (q_t, k_s row vectors).  For Mamba-2, M[t, s] is the product of the scalar gates
times the identity; the log-linear form puts a level- and data-dependent matrix in front of it,
M[t, s] = Lambda_t^(l) * prod_{r=s+1..t} alpha_r * I with l = l(t, s), so that

    O_t = sum_{s <= t} prod(alpha) * (q_t Lambda_t^(l(t,s)) . k_s) * v_s.

The scalar weights of Sec. 3.4 are the case Lambda_t^(l) = lambda_t^(l) I.

Shapes: q, k [B, T, H, d_k]; v [B, T, H, d_v]; log_alpha [B, T, H]; Lam either
    [B, T, H, L, d_k, d_k]   full matrices, Lam[..., a, c] = (Lambda_t^(l))_{a c}, or
    [B, T, H, L, d_k]        diagonals, Lambda_t^(l) = diag(Lam[b, t, h, l, :]).
L = fenwick.num_levels(T).  Outputs are [B, T, H, d_v] float64.

Forms
-----
quadratic   for each level l: the scores of the pairs at level l, computed with the level's
            transformed queries q_t Lambda_t^(l), times the Eq. 2 decay mask; their sum times V.
recurrent   the per-level Fenwick states of Sec. 3.2 (gated as in the scalar case) read out
            with the level's transformed query: o_t = sum_l S_t^(l) (q_t Lambda_t^(l))^T.
bruteforce  T <= 16: explicit loops over pairs, buckets from the footnote's greedy sequence and
            every M[t, s] built as an explicit d_k x d_k matrix product Lambda_t^(l) (prod alpha I).
"""

import numpy as np

from . import fenwick


def as_full(lam_diag):
    """Full matrices [..., d_k, d_k] with the given diagonals [..., d_k]."""
    lam_diag = np.asarray(lam_diag, dtype=np.float64)
    d = lam_diag.shape[-1]
    return lam_diag[..., :, None] * np.eye(d)


def _is_diag(Lam, dk):
    if Lam.ndim == 5 and Lam.shape[-1] == dk:
        return True
    if Lam.ndim == 6 and Lam.shape[-2:] == (dk, dk):
        return False
    raise ValueError("Lam must be [B, T, H, L, d_k] (diagonal) or [B, T, H, L, d_k, d_k] (full)")


def _full(Lam, dk):
    Lam = np.asarray(Lam, dtype=np.float64)
    return as_full(Lam) if _is_diag(Lam, dk) else Lam


def _times_lambda(qv, lam, diag):
    """q Lambda for row vectors qv [..., d_k] and matching weights lam ([..., d_k] diagonals, applied
    as the elementwise product that q diag(lam) is, or [..., d_k, d_k] matrices)."""
    lam = np.asarray(lam, dtype=np.float64)
    return qv * lam if diag else np.einsum('...a,...ac->...c', qv, lam)


def level_queries(q, Lam):
    """q_t Lambda_t^(l) for every (b, t, h, l): [B, T, H, L, d_k]."""
    q = np.asarray(q, dtype=np.float64)
    return _times_lambda(q[:, :, :, None, :], Lam, _is_diag(np.asarray(Lam), q.shape[-1]))


def quadratic(q, k, v, log_alpha, Lam, rows=None):
    """The definition, level by level; with `rows` only those output rows ([B, len(rows), H, d_v])."""
    q, k, v, log_alpha = (np.asarray(x, dtype=np.float64) for x in (q, k, v, log_alpha))
    B, T, H, dk = q.shape
    Lam = np.asarray(Lam)
    diag = _is_diag(Lam, dk)
    if Lam.shape[3] < fenwick.num_levels(T):
        raise ValueError("Lam has fewer levels than the sequence needs")
    rows = np.arange(T) if rows is None else np.asarray(rows)
    lev = np.full((len(rows), T), -1, dtype=np.int64)        # l(t, s), -1 above the diagonal
    for r, t in enumerate(rows):
        lev[r, :t + 1] = fenwick.level_row(int(t))
    cum = np.cumsum(log_alpha, axis=1)                       # [B, T, H]
    out = np.zeros((B, len(rows), H, v.shape[-1]))
    for b in range(B):
        for h in range(H):
            diff = cum[b, rows, h][:, None] - cum[b, :, h][None, :]
            decay = np.zeros_like(diff)
            decay[lev >= 0] = np.exp(diff[lev >= 0])              # Eq. 2 mask, causal pairs only
            for l in range(int(lev.max()) + 1):
                sel = lev == l
                if not sel.any():
                    continue
                ql = _times_lambda(q[b, rows, h], Lam[b, rows, h, l], diag)   # q_t Lambda_t^(l)
                scores = (ql @ k[b, :, h].T) * decay * sel
                out[b, :, h] += scores @ v[b, :, h]
    return out


def recurrent(q, k, v, log_alpha, Lam):
    """Per-level Fenwick states (merge rule of Sec. 3.2, every carried or merged state times
    alpha_t, the new token entering level 0 undecayed), each read out with its level's
    transformed query."""
    q, k, v, log_alpha = (np.asarray(x, dtype=np.float64) for x in (q, k, v, log_alpha))
    B, T, H, dk = q.shape
    Lam = np.asarray(Lam)
    diag = _is_diag(Lam, dk)
    L = Lam.shape[3]
    if L < fenwick.num_levels(T):
        raise ValueError("Lam has fewer levels than the sequence needs")
    S = np.zeros((B, H, L, v.shape[-1], dk))
    out = np.zeros((B, T, H, v.shape[-1]))
    for t in range(T):
        if t > 0:
            p = fenwick.lssb(t)
            merged = S[:, :, :p + 1].sum(axis=2)
            S[:, :, 1:p + 1] = 0.0
            S[:, :, p + 1] = merged
            S *= np.exp(log_alpha[:, t, :])[:, :, None, None, None]
        S[:, :, 0] = v[:, t, :, :, None] * k[:, t, :, None, :]
        ql = _times_lambda(q[:, t, :, None, :], Lam[:, t], diag)    # [B, H, L, d_k]
        out[:, t] = np.einsum('bhlpc,bhlc->bhp', S, ql)
    return out


def bruteforce(q, k, v, log_alpha, Lam):
    """Pure-Python loops for T <= 16 over the 4D tensor's entries M[t, s] (d_k x d_k each)."""
    q, k, v, log_alpha = (np.asarray(x, dtype=np.float64) for x in (q, k, v, log_alpha))
    B, T, H, dk = q.shape
    if T > 16:
        raise ValueError("bruteforce is for T <= 16")
    F = _full(Lam, dk)
    out = np.zeros((B, T, H, v.shape[-1]))
    eye = np.eye(dk)
    for b in range(B):
        for h in range(H):
            for t in range(T):
                bk = fenwick.buckets(t)
                for s in range(t + 1):
                    level = [lv for lv, members in bk.items() if s in members]
                    assert len(level) == 1
                    C = eye.copy()
                    for r in range(s + 1, t + 1):
                        C = (float(np.exp(log_alpha[b, r, h])) * eye) @ C
                    Mts = F[b, t, h, level[0]] @ C
                    out[b, t, h] += float(q[b, t, h] @ Mts @ k[b, s, h]) * v[b, s, h]
    return out
