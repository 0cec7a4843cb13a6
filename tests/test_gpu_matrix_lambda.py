"""GPU parity of ll_mamba2_fwd_matrix_lambda (matrix-valued level weights, the 4D-tensor view of
App. A) against the float64 oracle (oracle/matrix_lambda.py), through the C ABI.

The bar is the forward's: normalised max-abs error max|O_gpu - O_ref| / max|O_ref| at most 1e-4 for
fp32 storage and 2e-2 for bf16 (inputs rounded to bf16; the oracle receives the same rounded
values, and Lambda in float32, both upcast to float64).  Cases: both layouts of Lambda (diagonal
and full d_k x d_k), every compiled kernel shape, several tiles with a ragged last tile, the
scaled identity (which must match the scalar-weight oracle), sampled rows of the T = 8192
workload the benchmark times, and a NaN-filled determinism check."""

import numpy as np
import pytest

from oracle import mamba2
from oracle import matrix_lambda as ml
from synthetic import WORKLOADS, generate, level_weight_matrices
from tests.gpu_util import rel_err, to_dev

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-4, "bf16": 2e-2}


@pytest.fixture(scope="module", autouse=True)
def _device():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2506_04761_amd  # noqa: F401  (fails loudly if the library is missing)


def run_ml(x, Lam, dtype, C):
    import torch
    import paper_2506_04761_amd as ll
    o = ll.ll_mamba2_fwd_matrix_lambda(to_dev(x["q"], dtype), to_dev(x["k"], dtype), to_dev(x["v"], dtype),
                                       to_dev(x["log_alpha"]), to_dev(Lam), C)
    torch.cuda.synchronize()
    return o.float().cpu().numpy().astype(np.float64)


def _case(dtype, C, dk, dv, T, H, seed, dist="unit"):
    return WORKLOADS["ll_mamba2_bf16_T65536"].with_(dtype=dtype, B=1, H=H, T=T, dk=dk, dv=dv, C=C, seed=seed,
                                                      dist=dist)


@pytest.mark.parametrize("form", ["diag", "full"])
@pytest.mark.parametrize("dtype,C,dk,dv,T", [
    ("f32", 16, 16, 16, 16 * 13),      # tiles of 64 rows: 3 full tiles and a quarter of one
    ("f32", 64, 64, 64, 64 * 5),       # tiles of 128 rows, ragged last tile
    ("bf16", 64, 64, 64, 64 * 7),
    ("bf16", 64, 128, 64, 64 * 5),
    ("bf16", 64, 128, 128, 64 * 5),
])
def test_parity_small(form, dtype, C, dk, dv, T):
    w = _case(dtype, C, dk, dv, T, 2, seed=300 + T % 89 + dk)
    x = generate(w)
    Lam = level_weight_matrices(w, form)
    ref = ml.quadratic(x["q"], x["k"], x["v"], x["log_alpha"], Lam)
    e = rel_err(run_ml(x, Lam, dtype, C), ref)
    print(f"{form} {dtype} C={C} {dk}x{dv} T={T}: {e:.2e}", flush=True)
    assert e <= TOL[dtype]


@pytest.mark.parametrize("chunks", [1, 2, 3, 33])
def test_parity_diag_bf16_levels(chunks):
    # up to 17 tiles: tile levels 1-5, the reduced (block-tree) summaries included
    w = _case("bf16", 64, 128, 128, 64 * chunks, 2, seed=410 + chunks)
    x = generate(w)
    Lam = level_weight_matrices(w, "diag")
    ref = ml.quadratic(x["q"], x["k"], x["v"], x["log_alpha"], Lam)
    e = rel_err(run_ml(x, Lam, "bf16", 64), ref)
    print(f"diag bf16 chunks={chunks}: {e:.2e}", flush=True)
    assert e <= TOL["bf16"]


@pytest.mark.parametrize("dist", ["slow", "nodecay"])
def test_parity_full_gate_regimes(dist):
    # slow decay and alpha = 1 keep every level's terms large
    w = _case("bf16", 64, 64, 64, 64 * 9, 1, seed=77, dist=dist)
    x = generate(w)
    Lam = level_weight_matrices(w, "full")
    ref = ml.quadratic(x["q"], x["k"], x["v"], x["log_alpha"], Lam)
    e = rel_err(run_ml(x, Lam, "bf16", 64), ref)
    print(f"full bf16 {dist}: {e:.2e}", flush=True)
    assert e <= TOL["bf16"]


@pytest.mark.parametrize("dtype,C,dk,dv", [("f32", 16, 16, 16), ("bf16", 64, 128, 128)])
def test_scaled_identity_is_the_scalar_model(dtype, C, dk, dv):
    """Lambda_t^(l) = lambda_t^(l) I (diagonal layout) against the scalar-weight oracle."""
    w = _case(dtype, C, dk, dv, 64 * 11, 2, seed=91)
    x = generate(w)
    Lam = np.ascontiguousarray(np.repeat(x["lam"][..., None], dk, axis=-1))
    ref = mamba2.quadratic(x["q"], x["k"], x["v"], x["log_alpha"], x["lam"])
    e = rel_err(run_ml(x, Lam, dtype, C), ref)
    print(f"lambda I {dtype}: {e:.2e}", flush=True)
    assert e <= TOL[dtype]


def test_workload_sampled_rows():
    """The T = 8192, 16-head diagonal workload in the benchmark's launch configuration: sampled
    rows of two heads against the oracle (whole rows need only the causal prefix)."""
    w = WORKLOADS["ll_mamba2_diag_lambda_bf16_T8192"]
    x = generate(w)
    Lam = level_weight_matrices(w, "diag")
    got = run_ml(x, Lam, w.dtype, w.C)
    rows = np.array([0, 1, 127, 128, 4095, 5000, 8191])
    heads = [0, 9]
    xs = {n: x[n][:, :, heads] for n in ("q", "k", "v", "log_alpha")}
    ref = ml.quadratic(xs["q"], xs["k"], xs["v"], xs["log_alpha"], Lam[:, :, heads], rows=rows)
    e = rel_err(got[:, rows][:, :, heads], ref)
    print(f"T=8192 diag sampled rows: {e:.2e}", flush=True)
    assert e <= TOL["bf16"]
    assert np.all(np.isfinite(got))


def test_deterministic_and_writes_every_output():
    import torch
    import paper_2506_04761_amd as ll
    w = _case("bf16", 64, 128, 128, 64 * 13, 2, seed=5)
    x = generate(w)
    args = [to_dev(x[n], "bf16") for n in ("q", "k", "v")] + [to_dev(x["log_alpha"])]
    outs = []
    for form in ("diag", "full", "diag"):
        Lam = to_dev(level_weight_matrices(w, form))
        ws = ll.ll_mamba2_matrix_lambda_workspace(args[0], args[2], w.C)
        ws.fill_(255)  # NaN bit patterns
        o = torch.full_like(args[2], float("nan"))
        ll.ll_mamba2_fwd_matrix_lambda(*args, Lam, w.C, out=o, workspace=ws)
        torch.cuda.synchronize()
        assert not torch.isnan(o).any(), form
        outs.append(o.clone())
    assert torch.equal(outs[0], outs[2])


@pytest.mark.parametrize("dtype,C,dk,dv", [("f32", 16, 16, 16), ("bf16", 64, 128, 128)])
def test_diagonal_equals_its_full_expansion(dtype, C, dk, dv):
    """Diagonal weights (scaled in the tile kernel's registers) against the same matrices passed in
    full (level queries formed beforehand): both round q_t (.) diag once to the storage type and the
    full product adds exact zeros, so the outputs agree bit for bit."""
    import torch
    import paper_2506_04761_amd as ll
    w = _case(dtype, C, dk, dv, 64 * 9, 2, seed=17)
    x = generate(w)
    diag = level_weight_matrices(w, "diag")
    full = np.ascontiguousarray(ml.as_full(diag).astype(np.float32))
    args = [to_dev(x[n], dtype) for n in ("q", "k", "v")] + [to_dev(x["log_alpha"])]
    a = ll.ll_mamba2_fwd_matrix_lambda(*args, to_dev(diag), C)
    b = ll.ll_mamba2_fwd_matrix_lambda(*args, to_dev(full), C)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
