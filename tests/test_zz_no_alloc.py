"""The allocation-free forward, ll_mamba2_fwd_noalloc, against ll_mamba2_fwd through the C ABI.

Both run the same kernels on the same inputs: one in the library's static per-GPU scratch, the
other in a workspace the caller allocates.  The outputs must therefore agree bit for bit, which
is stronger than the oracle tolerance (the oracle parity of ll_mamba2_fwd itself is covered by
the ll_mamba2_fwd parity tests; the smaller input of each case is also checked against the
oracle here).  Each case makes two calls in a row, the second on a smaller input and on another
stream, so that the second call works in the scratch the first one left behind."""

import numpy as np
import pytest

from oracle import mamba2
from synthetic import WORKLOADS, generate
from tests.gpu_util import device_inputs, rel_err

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-4, "bf16": 2e-2}

# (dtype, C, d_k, d_v, with lambda, (B, T, H) of the first call, (B, T, H) of the second)
CASES = [
    ("bf16", 64, 128, 128, True, (1, 8192, 4), (1, 2176, 2)),   # single-pass kernels
    ("bf16", 64, 128, 64, True, (2, 4096, 4), (1, 1216, 3)),    # single-pass kernels, d_v = 64
    ("bf16", 64, 128, 128, False, (1, 8192, 4), (2, 704, 2)),   # lambda = NULL: single pass, unit weights
    ("f32", 16, 16, 16, True, (2, 1024, 3), (1, 80, 1)),        # fp32 three-kernel path
    ("f32", 16, 16, 16, False, (2, 1024, 3), (1, 80, 1)),       # fp32 lambda = NULL: running-scan path
]


@pytest.fixture(scope="module", autouse=True)
def _device():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2506_04761_amd  # noqa: F401  (fails loudly if the library is missing)


def _inputs(dtype, C, dk, dv, shape, seed):
    B, T, H = shape
    base = WORKLOADS["ll_mamba2_f32_T64" if dtype == "f32" else "ll_mamba2_bf16_T65536"]
    return generate(base.with_(B=B, T=T, H=H, dk=dk, dv=dv, seed=seed))


def _run(fn, d, lam, C, stream=None):
    import torch
    out = torch.full_like(d["v"], float("nan"))
    if stream is None:
        fn(d["q"], d["k"], d["v"], d["log_alpha"], lam, C, out=out)
    else:
        with torch.cuda.stream(stream):
            fn(d["q"], d["k"], d["v"], d["log_alpha"], lam, C, out=out, stream=stream)
    return out


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"{c[0]}_C{c[1]}_{c[2]}x{c[3]}_{'lam' if c[4] else 'null'}")
def test_noalloc_matches_workspace_entry_point(case):
    import torch
    import paper_2506_04761_amd as ll
    dtype, C, dk, dv, with_lam, big, small = case
    xs = [_inputs(dtype, C, dk, dv, big, 71), _inputs(dtype, C, dk, dv, small, 72)]
    ds = [device_inputs(x, dtype) for x in xs]
    lams = [d["lam"] if with_lam else None for d in ds]
    side = torch.cuda.Stream()
    print(f"noalloc {case}", flush=True)
    got = [_run(ll.ll_mamba2_fwd_noalloc, ds[0], lams[0], C)]
    torch.cuda.synchronize()
    got.append(_run(ll.ll_mamba2_fwd_noalloc, ds[1], lams[1], C, stream=side))
    side.synchronize()
    want = [_run(ll.ll_mamba2_fwd, d, lam, C) for d, lam in zip(ds, lams)]
    torch.cuda.synchronize()
    for i in range(2):
        assert torch.equal(got[i], want[i]), f"call {i}: max diff {(got[i].float() - want[i].float()).abs().max()}"
    x = xs[1]
    lam64 = x["lam"] if with_lam else np.ones_like(x["lam"])
    ref = mamba2.quadratic(x["q"], x["k"], x["v"], x["log_alpha"], lam64)
    err = rel_err(got[1].float().cpu().numpy().astype(np.float64), ref)
    print(f"second call rel err vs oracle {err:.3e}")
    assert err <= TOL[dtype]


def test_noalloc_rejects_a_workspace_beyond_its_scratch():
    import torch
    import paper_2506_04761_amd as ll
    B, T, H, d = 1, 16384, 16, 128
    assert ll.ll_workspace_size(ll.LL_MAMBA2, ll.LL_BF16, B, T, H, d, d, 64, 1) > ll.LL_NOALLOC_SCRATCH_BYTES
    q = torch.zeros((B, T, H, d), dtype=torch.bfloat16, device="cuda")
    la = torch.zeros((B, T, H), dtype=torch.float32, device="cuda")
    lam = torch.zeros((B, T, H, ll.ll_num_levels(T)), dtype=torch.float32, device="cuda")
    out = torch.full_like(q, 7.0)
    with pytest.raises(ll.LLError) as e:
        ll.ll_mamba2_fwd_noalloc(q, q, q, la, lam, 64, out=out)
    assert e.value.status == ll._lib.LL_ERR_SCRATCH
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())  # nothing was enqueued
