"""Pins for the oracle's log-linear Mamba-2 gradients (oracle/mamba2_grad.py).

The gradients are written out from the chain rule; these checks tie them to things that do
not share that derivation:
  * central finite differences of the explicit-product brute-force forward (loops over the
    footnote's greedy buckets, decays as products of alpha) and of the per-level recurrent
    form (Sec. 3.2), for every input: q, k, v, log alpha and lambda;
  * invariants of the forward map: O is linear in each of q, k, v and in lambda_t, so
    sum q.dq = sum k.dk = sum v.dv = sum dO.O and sum_l lambda_t^(l) dlambda_t^(l) = dO_t.O_t;
    shifting every cumulative log-gate by one constant changes nothing, so the gradient of the
    first gate is zero;
  * the sampled row/column forms against the full one."""

import numpy as np
import pytest

from oracle import fenwick, mamba2, mamba2_grad


def _rand(seed, B, T, H, dk, dv, slow=False):
    rng = np.random.default_rng(seed)
    L = fenwick.num_levels(T)
    q = rng.standard_normal((B, T, H, dk)) / np.sqrt(dk)
    k = rng.standard_normal((B, T, H, dk)) / np.sqrt(dk)
    v = rng.standard_normal((B, T, H, dv))
    la = -np.logaddexp(0, rng.standard_normal((B, T, H)) + (-4.0 if slow else 0.0))
    lam = np.logaddexp(0, rng.standard_normal((B, T, H, L)))
    do = rng.standard_normal((B, T, H, dv))
    return q, k, v, la, lam, do


def _rel(a, b):
    return np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300)


NAMES = ["q", "k", "v", "log_alpha", "lam"]


def _fd_check(forward, args, do, grads, n_entries, seed, eps=1e-6, tol=1e-7):
    """Central differences of sum(forward(*args) * do) at n_entries random entries of every
    input, against the analytic gradients."""
    rng = np.random.default_rng(seed)
    for idx, (name, g) in enumerate(zip(NAMES, grads)):
        x = args[idx]
        flat = rng.choice(x.size, size=min(n_entries, x.size), replace=False)
        scale = max(np.max(np.abs(g)), 1e-12)
        for f in flat:
            pos = np.unravel_index(f, x.shape)
            xp, xm = x.copy(), x.copy()
            xp[pos] += eps
            xm[pos] -= eps
            ap, am = list(args), list(args)
            ap[idx], am[idx] = xp, xm
            num = (np.sum(forward(*ap) * do) - np.sum(forward(*am) * do)) / (2 * eps)
            assert abs(num - g[pos]) <= tol * scale + 1e-9 * abs(num), (name, pos, num, g[pos])


@pytest.mark.parametrize("T", [1, 2, 5, 8, 13, 16])
def test_grad_matches_finite_differences_of_bruteforce(T):
    q, k, v, la, lam, do = _rand(10 + T, 1, T, 2, 3, 2)
    grads = mamba2_grad.quadratic_grad(q, k, v, la, lam, do)
    _fd_check(mamba2.bruteforce, [q, k, v, la, lam], do, grads, n_entries=12, seed=T)


@pytest.mark.parametrize("T,slow", [(37, False), (64, True)])
def test_grad_matches_finite_differences_of_recurrent(T, slow):
    q, k, v, la, lam, do = _rand(50 + T, 1, T, 2, 4, 3, slow)
    grads = mamba2_grad.quadratic_grad(q, k, v, la, lam, do)
    _fd_check(mamba2.recurrent, [q, k, v, la, lam], do, grads, n_entries=8, seed=T)


@pytest.mark.parametrize("T", [100, 129])
def test_grad_invariants(T):
    q, k, v, la, lam, do = _rand(T, 2, T, 3, 5, 4)
    dq, dk, dv, dla, dlam = mamba2_grad.quadratic_grad(q, k, v, la, lam, do)
    o = mamba2.quadratic(q, k, v, la, lam)
    total = np.sum(o * do)
    for x, dx in ((q, dq), (k, dk), (v, dv)):
        assert abs(np.sum(x * dx) - total) < 1e-11 * max(abs(total), 1.0)
    # linear in lambda_t: sum_l lambda dlambda = dO_t . O_t for every (b, t, h)
    per_row = np.einsum('bthl,bthl->bth', lam, dlam)
    assert _rel(per_row, np.einsum('bthd,bthd->bth', do, o)) < 1e-12
    # the first gate only shifts every cumulative sum by the same amount
    assert np.max(np.abs(dla[:, 0])) < 1e-11 * np.max(np.abs(dla))
    # levels no pair reaches get no gradient: row t reaches levels 0..bit_length(t) at most
    for t in range(T):
        top = int(fenwick.level_row(t).max())
        assert np.all(dlam[:, t, :, top + 1:] == 0.0)


def test_sampled_forms_match_full():
    T = 70
    q, k, v, la, lam, do = _rand(3, 2, T, 2, 4, 3)
    dq, dk, dv, dla, dlam = mamba2_grad.quadratic_grad(q, k, v, la, lam, do)
    pos = np.array([0, 1, 17, 31, 32, 63, 69])
    rq, rl = mamba2_grad.grad_rows(q, k, v, la, lam, do, pos)
    assert _rel(rq, dq[:, pos]) < 1e-12
    assert _rel(rl, dlam[:, pos]) < 1e-12
    ck, cv = mamba2_grad.grad_cols(q, k, v, la, lam, do, pos)
    assert _rel(ck, dk[:, pos]) < 1e-12
    assert _rel(cv, dv[:, pos]) < 1e-12
    dc = mamba2_grad.dcum_at(q, k, v, la, lam, do, pos)
    nxt = np.concatenate([dla[:, 1:], np.zeros_like(dla[:, :1])], axis=1)
    assert _rel(dc, (dla - nxt)[:, pos]) < 1e-10


def test_level_col_matches_level_matrix():
    T = 200
    m = fenwick.level_matrix(T)
    for s in (0, 1, 7, 64, 127, 199):
        assert np.array_equal(fenwick.level_col(s, T), m[s:, s])
