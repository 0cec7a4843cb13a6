"""Log-linear Mamba-2 in float64: the definition and two independent ways to compute it.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Shapes (the layout of the paper's PyTorch listing, App. C):
    q, k       [B, T, H, d_k]     queries, keys
    v          [B, T, H, d_v]     values
    log_alpha  [B, T, H]          log of the scalar forget gate alpha_t in (0, 1]
    lam        [B, T, H, L]       level weights lambda_t^(l) >= 0, L = fenwick.num_levels(T)
Outputs are [B, T, H, d_v] float64.

Forms
-----
quadratic      O = (Q K^T  (.) M^S (.) M^H) V                    Sec. 3.4 (log-linear Mamba-2),
               with M^S from Eq. 2 and M^H from Eq. 4.  This is the definition; the chunked
               GPU algorithm of Sec. 3.3 reaches the same result up to rounding order.
recurrent      per-level Fenwick states, Eq. 3 output and the Sec. 3.2 merge recurrence,
               with every carried or merged state multiplied by alpha_t.
bruteforce     explicit loops, buckets from the footnote's greedy sequence and decays as
               explicit products of alpha (no cumulative sums), for T <= 16.
gla_recurrent  gated linear attention / Mamba-2, S_t = alpha_t S_{t-1} + v_t k_t^T (Eq. 2).
linear_attention_parallel  O = (Q K^T (.) L) V with L lower-triangular ones (Sec. 2).
"""

import numpy as np

from . import fenwick


def _f64(*xs):
    return [np.asarray(x, dtype=np.float64) for x in xs]


def ss_mask(log_alpha_1d: np.ndarray, rows=None) -> np.ndarray:
    """Eq. 2 mask M^S[t, s] = prod_{k=s+1..t} alpha_k for s <= t, else 0, for one (b, h).

    The product is formed as exp of a difference of float64 prefix sums of log alpha;
    `rows` restricts the output to the given t (all s < T columns are returned)."""
    la = np.asarray(log_alpha_1d, dtype=np.float64)
    T = la.shape[0]
    cum = np.cumsum(la)
    rows = np.arange(T) if rows is None else np.asarray(rows)
    diff = cum[rows][:, None] - cum[None, :]
    causal = np.arange(T)[None, :] <= rows[:, None]
    out = np.zeros((len(rows), T))
    out[causal] = np.exp(diff[causal])
    return out


def h_mask(lam_2d: np.ndarray, rows=None) -> np.ndarray:
    """Eq. 4 mask M^H[t, s] = lambda_t^(l(t, s)) for s <= t, else 0, for one (b, h).

    lam_2d is [T, L]; l(t, s) comes from the footnote's greedy buckets."""
    lam_2d = np.asarray(lam_2d, dtype=np.float64)
    T = lam_2d.shape[0]
    rows = np.arange(T) if rows is None else np.asarray(rows)
    out = np.zeros((len(rows), T))
    for r, t in enumerate(rows):
        lev = fenwick.level_row(int(t))
        out[r, :t + 1] = lam_2d[t, lev]
    return out


def quadratic(q, k, v, log_alpha, lam, rows=None):
    """O = (Q K^T (.) M^S (.) M^H) V, the parallel form of log-linear Mamba-2 (Sec. 3.4).

    With `rows` given, returns only those output rows ([B, len(rows), H, d_v]); because
    the masks are causal, row t needs only the prefix 0..t."""
    q, k, v, log_alpha, lam = _f64(q, k, v, log_alpha, lam)
    B, T, H, _ = q.shape
    rows = np.arange(T) if rows is None else np.asarray(rows)
    out = np.zeros((B, len(rows), H, v.shape[-1]))
    for b in range(B):
        for h in range(H):
            A = q[b, rows, h, :] @ k[b, :, h, :].T
            P = A * ss_mask(log_alpha[b, :, h], rows) * h_mask(lam[b, :, h, :], rows)
            out[b, :, h, :] = P @ v[b, :, h, :]
    return out


def recurrent(q, k, v, log_alpha, lam):
    """Per-level recurrent form: Eq. 3 output with the Sec. 3.2 state recurrence, gated.

    States S^(l) (d_v x d_k, one per level, vectorised over B and H) evolve as
      t = 0   : S^(0) = v_0 k_0^T, all other levels 0;
      t >= 1  : with p = lssb(t), level p+1 takes the sum of levels 0..p of step t-1,
                levels 1..p are emptied, higher levels carry over; every carried or merged
                state is multiplied by alpha_t; then S^(0) = v_t k_t^T (enters undecayed).
      output  : o_t = sum_l lambda_t^(l) S_t^(l) q_t.
    """
    q, k, v, log_alpha, lam = _f64(q, k, v, log_alpha, lam)
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    L = lam.shape[-1]
    if L < fenwick.num_levels(T):
        raise ValueError("lambda has fewer levels than the sequence needs")
    S = np.zeros((B, H, L, dv, dk))
    out = np.zeros((B, T, H, dv))
    for t in range(T):
        if t > 0:
            p = fenwick.lssb(t)
            merged = S[:, :, :p + 1].sum(axis=2)
            S[:, :, 1:p + 1] = 0.0
            S[:, :, p + 1] = merged
            S *= np.exp(log_alpha[:, t, :])[:, :, None, None, None]
        S[:, :, 0] = v[:, t, :, :, None] * k[:, t, :, None, :]
        Sq = S @ q[:, t, :, None, :, None]  # [B, H, L, dv, 1]
        out[:, t] = np.einsum('bhl,bhlp->bhp', lam[:, t], Sq[..., 0])
    return out


def bruteforce(q, k, v, log_alpha, lam):
    """Pure-Python loops for T <= 16: o_t = sum_{s<=t} lambda_t^(l) prod(alpha) (q_t.k_s) v_s,
    with l found by searching the footnote's greedy buckets of t for s and the decay
    formed as an explicit product of alpha_k = exp(log alpha_k), k = s+1..t."""
    q, k, v, log_alpha, lam = _f64(q, k, v, log_alpha, lam)
    B, T, H, _ = q.shape
    if T > 16:
        raise ValueError("bruteforce is for T <= 16")
    out = np.zeros((B, T, H, v.shape[-1]))
    for b in range(B):
        for h in range(H):
            for t in range(T):
                bk = fenwick.buckets(t)
                for s in range(t + 1):
                    level = [lv for lv, members in bk.items() if s in members]
                    assert len(level) == 1
                    decay = 1.0
                    for kk in range(s + 1, t + 1):
                        decay *= float(np.exp(log_alpha[b, kk, h]))
                    w = lam[b, t, h, level[0]] * decay * float(q[b, t, h] @ k[b, s, h])
                    out[b, t, h] += w * v[b, s, h]
    return out


def gla_recurrent(q, k, v, log_alpha):
    """Gated linear attention (Mamba-2) recurrence, Eq. 2: S_t = alpha_t S_{t-1} + v_t k_t^T,
    o_t = S_t q_t.  Log-linear Mamba-2 with all lambda equal to 1 must reduce to this."""
    q, k, v, log_alpha = _f64(q, k, v, log_alpha)
    B, T, H, dk = q.shape
    S = np.zeros((B, H, v.shape[-1], dk))
    out = np.zeros((B, T, H, v.shape[-1]))
    for t in range(T):
        S = S * np.exp(log_alpha[:, t, :])[:, :, None, None] + v[:, t, :, :, None] * k[:, t, :, None, :]
        out[:, t] = (S @ q[:, t, :, :, None])[..., 0]
    return out


def linear_attention_parallel(q, k, v):
    """Linear attention parallel form of Sec. 2: O = (Q K^T (.) L) V with L the
    lower-triangular matrix of ones (s <= t)."""
    q, k, v = _f64(q, k, v)
    B, T, H, _ = q.shape
    Lmask = np.tril(np.ones((T, T)))
    out = np.zeros((B, T, H, v.shape[-1]))
    for b in range(B):
        for h in range(H):
            out[b, :, h] = ((q[b, :, h] @ k[b, :, h].T) * Lmask) @ v[b, :, h]
    return out
