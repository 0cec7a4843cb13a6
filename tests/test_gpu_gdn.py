"""GPU parity of ll_gdn_fwd (log-linear Gated DeltaNet) against the float64 oracle, through the
C ABI.  bf16 inputs with fp32 accumulation: normalised max-abs error <= 2e-2."""

import numpy as np
import pytest

from oracle import gdn
from synthetic import WORKLOADS, generate
from tests.gpu_util import rel_err, run_gdn

pytestmark = pytest.mark.gpu

TOL = 2e-2


@pytest.fixture(scope="module", autouse=True)
def _device():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2506_04761_amd  # noqa: F401


def _ref(x, rows=None):
    return gdn.quadratic(x["q"], x["k"], x["v"], x["log_alpha"], x["beta"], x["lam"], rows=rows)


BASE = WORKLOADS["ll_gdn_bf16_T8192"]


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("chunks", [1, 2, 3, 5, 8, 16])
def test_parity_chunk_counts(d, chunks):
    x = generate(BASE.with_(B=1, H=2, T=64 * chunks, dk=d, dv=d, seed=50 + chunks))
    err = rel_err(run_gdn(x, 64), _ref(x))
    print(f"GDN d={d} chunks={chunks}: rel err {err:.3e}")
    assert err <= TOL, err


@pytest.mark.parametrize("dist", ["gdn_slow", "gdn_nodecay"])
def test_parity_stress_gates(dist):
    x = generate(BASE.with_(B=1, H=2, T=1024, dist=dist, seed=61))
    err = rel_err(run_gdn(x, 64), _ref(x))
    print(f"GDN gates {dist}: rel err {err:.3e}")
    assert err <= TOL, err


def test_each_level_alone():
    x = generate(BASE.with_(B=1, H=1, T=1024, dist="gdn_slow", seed=62))
    for lv in range(x["lam"].shape[-1]):
        y = dict(x)
        lam = np.zeros_like(x["lam"])
        lam[..., lv] = x["lam"][..., lv]
        y["lam"] = lam
        err = rel_err(run_gdn(y, 64), _ref(y))
        assert err <= TOL, (lv, err)


def test_lambda_null_is_gated_deltanet():
    x = generate(BASE.with_(B=2, H=2, T=1024, dist="gdn_slow", seed=63))
    ref = gdn.gdn_recurrent(x["q"], x["k"], x["v"], x["log_alpha"], x["beta"])
    assert rel_err(run_gdn(x, 64, with_lambda=False), ref) <= TOL
    y = dict(x)
    y["lam"] = np.ones_like(x["lam"])
    assert rel_err(run_gdn(y, 64), ref) <= TOL


def test_beta_zero_gives_zero():
    x = generate(BASE.with_(B=1, H=2, T=512, seed=64))
    x["beta"] = np.zeros_like(x["beta"])
    assert np.max(np.abs(run_gdn(x, 64))) == 0.0


def test_parity_full_size_sampled():
    x = generate(BASE)
    got = run_gdn(x, BASE.C)
    rng = np.random.default_rng(65)
    worst = 0.0
    for b, h in ((0, 0), (1, 15)):
        rows = np.unique(np.concatenate([[0, 63, 64, BASE.T - 1], rng.integers(0, BASE.T, 12)]))
        xs = {n: x[n][b:b + 1, :, h:h + 1] for n in ("q", "k", "v", "log_alpha", "beta", "lam")}
        worst = max(worst, rel_err(got[b:b + 1, rows, h:h + 1], _ref(xs, rows)))
    print(f"GDN T=8192 sampled rel err {worst:.3e}")
    assert worst <= TOL


@pytest.mark.parametrize("d,chunks", [(64, 600), (128, 300)])
def test_parity_upper_level_slots(d, chunks):
    """More than 256 chunks (chunk levels above 8): the scan instance with eight level slots per
    wave runs (600 chunks: levels up to 10; 300 chunks: up to 9).  Every output row of one head
    against the oracle's per-level recurrent form (the quadratic form's T x T solve is too large at
    this length); slow decay keeps the high levels large."""
    w = BASE.with_(B=1, H=2, T=64 * chunks, dk=d, dv=d, dist="gdn_slow", seed=67 + d)
    x = generate(w)
    got = run_gdn(x, 64)
    xs = {n: x[n][:, :, 1:2] for n in ("q", "k", "v", "log_alpha", "beta", "lam")}
    ref = gdn.recurrent(xs["q"], xs["k"], xs["v"], xs["log_alpha"], xs["beta"], xs["lam"])
    err = rel_err(got[:, :, 1:2], ref)
    print(f"GDN d={d} T={w.T} rel err {err:.3e}", flush=True)
    assert err <= TOL, err


def test_parity_full_size_every_row_two_heads():
    """Every output row of two heads of the T = 8192, 2 x 16-head workload (the launch
    configuration the benchmark times) against the oracle's per-level recurrent form."""
    from tests.oracle_pool import recurrent_heads
    x = generate(BASE)
    got = run_gdn(x, BASE.C)
    heads = [(0, 0), (1, 15)]
    refs = recurrent_heads("gdn", x, heads, ("q", "k", "v", "log_alpha", "beta", "lam"))
    for (b, h), ref in zip(heads, refs):
        err = rel_err(got[b:b + 1, :, h:h + 1], ref)
        print(f"GDN T=8192 (b, h) = ({b}, {h}): every row rel err {err:.3e}", flush=True)
        assert err <= TOL, (b, h, err)


@pytest.mark.parametrize("dist,chunks", [("gdn", 128), ("gdn_nodecay", 260)])
def test_lambda_null_long(dist, chunks):
    """lambda == NULL (Gated DeltaNet's single running state, carried across every chunk) over
    128 chunks with the workload's gates and 260 chunks with alpha = 1, every row against the
    oracle's plain gated delta-rule recurrence."""
    x = generate(BASE.with_(B=1, H=2, T=64 * chunks, dist=dist, seed=68 + chunks))
    ref = gdn.gdn_recurrent(x["q"], x["k"], x["v"], x["log_alpha"], x["beta"])
    err = rel_err(run_gdn(x, 64, with_lambda=False), ref)
    print(f"GDN lambda=NULL {dist} chunks={chunks}: rel err {err:.3e}", flush=True)
    assert err <= TOL, err


def test_deterministic():
    import torch
    import paper_2506_04761_amd as ll
    from tests.gpu_util import device_inputs
    x = generate(BASE.with_(B=1, H=4, T=2048, seed=66))
    d = device_inputs(x, "bf16")
    outs = []
    for _ in range(2):
        o = torch.full((1, 2048, 4, 128), float("nan"), dtype=torch.bfloat16, device="cuda")
        ll.ll_gdn_fwd(d["q"], d["k"], d["v"], d["log_alpha"], d["beta"], d["lam"], 64, out=o)
        torch.cuda.synchronize()
        assert not torch.isnan(o).any()
        outs.append(o.clone())
    assert torch.equal(outs[0], outs[1])
