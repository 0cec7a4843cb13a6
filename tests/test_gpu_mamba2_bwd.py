"""GPU parity of ll_mamba2_bwd against the float64 oracle's gradients, through the C ABI.

Every gradient (dq, dk, dv, dlog_alpha, dlambda) is compared on its own, by the normalised
max-abs error max|g_gpu - g_ref| / max|g_ref| that the forward uses: at most 1e-4 for fp32
storage and 2e-2 for bf16 storage (inputs and dO rounded to bf16; the oracle receives the same
rounded values in float64).  Cases span several tiles, ragged tails, every tile level up to the
reduced ones (groups of >= 16 tiles), and the full T = 65536 workload on sampled rows and
columns (dlog_alpha there through its differences, which the oracle computes per position)."""

import numpy as np
import pytest

from oracle import mamba2_grad
from synthetic import WORKLOADS, generate, upstream_grad
from tests.gpu_util import rel_err, to_dev

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-4, "bf16": 2e-2}
NAMES = ("dq", "dk", "dv", "dlog_alpha", "dlambda")


@pytest.fixture(scope="module", autouse=True)
def _device():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2506_04761_amd  # noqa: F401  (fails loudly if the library is missing)


def run_bwd(x, do, dtype, C):
    import torch
    import paper_2506_04761_amd as ll
    args = [to_dev(x[n], dtype) for n in ("q", "k", "v")]
    args += [to_dev(x["log_alpha"]), to_dev(x["lam"]), to_dev(do, dtype)]
    grads = ll.ll_mamba2_bwd(*args, C)
    torch.cuda.synchronize()
    return [g.float().cpu().numpy().astype(np.float64) for g in grads]


def _check_all(w, x, do, label):
    got = run_bwd(x, do, w.dtype, w.C)
    ref = mamba2_grad.quadratic_grad(x["q"], x["k"], x["v"], x["log_alpha"], x["lam"], do)
    errs = {n: rel_err(g, r) for n, g, r in zip(NAMES, got, ref)}
    print(label, " ".join(f"{n} {e:.2e}" for n, e in errs.items()), flush=True)
    for n, e in errs.items():
        assert e <= TOL[w.dtype], (label, n, e)


@pytest.mark.parametrize("name", ["ll_mamba2_f32_T64", "ll_mamba2_bf16_T2048"])
def test_bwd_parity_small_workloads(name):
    w = WORKLOADS[name]
    _check_all(w, generate(w), upstream_grad(w), name)


@pytest.mark.parametrize("T", [16, 64 * 19, 64 * 37])
def test_bwd_parity_f32_chunk16(T):
    # fp32, C = 16 (tiles of 64 rows): 1216 tokens = 19 tiles (tile levels 1..5, a partial
    # last region); 2368 tokens = 37 tiles
    w = WORKLOADS["ll_mamba2_f32_T64"].with_(B=1, H=2, T=T, seed=60 + T % 97)
    _check_all(w, generate(w), upstream_grad(w), f"f32 C=16 T={T}")


def test_bwd_parity_f32_chunk64():
    w = WORKLOADS["ll_mamba2_f32_T64"].with_(B=1, H=2, T=64 * 23, dk=64, dv=64, C=64, seed=71)
    _check_all(w, generate(w), upstream_grad(w), "f32 C=64 T=1472")


@pytest.mark.parametrize("chunks", [1, 2, 3, 7, 33, 66])
@pytest.mark.parametrize("dk,dv", [(128, 64), (128, 128), (64, 64)])
def test_bwd_parity_bf16_ragged(chunks, dk, dv):
    w = WORKLOADS["ll_mamba2_bf16_T65536"].with_(B=1, H=2, T=64 * chunks, dk=dk, dv=dv, seed=80 + chunks)
    _check_all(w, generate(w), upstream_grad(w), f"bf16 {dk}x{dv} chunks={chunks}")


@pytest.mark.parametrize("dist", ["slow", "nodecay", "shifted"])
def test_bwd_parity_gate_regimes(dist):
    # slow decay and alpha = 1 keep every level's terms large; "shifted" is the second reading
    # of the input distribution (v ~ N(0, 1), log alpha = -softplus(x + 2))
    w = WORKLOADS["ll_mamba2_bf16_T65536"].with_(B=2, H=1, T=64 * 40, dist=dist, seed=90)
    _check_all(w, generate(w), upstream_grad(w), f"bf16 {dist}")


def test_bwd_full_size_sampled():
    """The T = 65536, 16-head workload in the launch configuration the benchmark times: sampled
    query rows (dq, dlambda), key columns (dk, dv) and positions of dlog_alpha's differences
    (dlog_alpha_t - dlog_alpha_{t+1} = q_t . dq_t - k_t . dk_t), for two heads."""
    w = WORKLOADS["ll_mamba2_bwd_bf16_T65536"]
    x = generate(w)
    do = upstream_grad(w)
    dq, dk, dv, dla, dlam = run_bwd(x, do, w.dtype, w.C)
    pos = np.array([0, 1, 127, 128, 4095, 4096, 32767, 40000, 65535])
    heads = [0, 11]
    xs = {n: x[n][:, :, heads] for n in x}
    do_s = do[:, :, heads]
    rq, rl = mamba2_grad.grad_rows(xs["q"], xs["k"], xs["v"], xs["log_alpha"], xs["lam"], do_s, pos)
    ck, cv = mamba2_grad.grad_cols(xs["q"], xs["k"], xs["v"], xs["log_alpha"], xs["lam"], do_s, pos)
    dc = mamba2_grad.dcum_at(xs["q"], xs["k"], xs["v"], xs["log_alpha"], xs["lam"], do_s, pos)
    nxt = np.concatenate([dla[:, 1:], np.zeros_like(dla[:, :1])], axis=1)
    diffs = (dla - nxt)[:, pos][:, :, heads]
    errs = {"dq": rel_err(dq[:, pos][:, :, heads], rq), "dlambda": rel_err(dlam[:, pos][:, :, heads], rl),
            "dk": rel_err(dk[:, pos][:, :, heads], ck), "dv": rel_err(dv[:, pos][:, :, heads], cv),
            "dlog_alpha differences": rel_err(diffs, dc)}
    print("T=65536 sampled", " ".join(f"{n} {e:.2e}" for n, e in errs.items()), flush=True)
    for n, e in errs.items():
        assert e <= TOL["bf16"], (n, e)
    # the first gate only shifts every cumulative sum: its gradient vanishes
    assert np.max(np.abs(dla[:, 0])) <= TOL["bf16"] * np.max(np.abs(dla))
    # Every position: dlog_alpha_t - dlog_alpha_{t+1} = q_t . dq_t - k_t . dk_t (dlog_alpha_T = 0), so
    # these T differences pin the kernels' reverse cumulative sum (tile sums included) at full
    # length.  The right side is formed in float64 from the returned bf16 dq and dk, whose rounding
    # (at most 2^-8 of each element) bounds the gap by 2^-8 a_t, a_t = sum_d |q dq| + |k dk|; the
    # test allows twice that plus a float32 margin.  (A reverse cumulative sum of the right side
    # itself would add up T of those rounding errors.)
    qf, kf = (x[n].astype(np.float64) for n in ("q", "k"))
    per_pos = np.einsum("bthd,bthd->bth", qf, dq) - np.einsum("bthd,bthd->bth", kf, dk)
    a_t = np.einsum("bthd,bthd->bth", np.abs(qf), np.abs(dq)) + np.einsum("bthd,bthd->bth", np.abs(kf), np.abs(dk))
    gap = np.abs((dla - nxt) - per_pos) / (2.0 ** -7 * a_t + 1e-6 * np.max(np.abs(dla)))
    print(f"T=65536 dlog_alpha differences at every position: worst gap / bound {gap.max():.3f}", flush=True)
    assert gap.max() <= 1.0, (np.unravel_index(np.argmax(gap), gap.shape), gap.max())
    assert np.all(np.isfinite(dq)) and np.all(np.isfinite(dk)) and np.all(np.isfinite(dv))


def _bwd_case(dtype, C, T, dk, dv, seed=97):
    w = WORKLOADS["ll_mamba2_bf16_T65536"].with_(dtype=dtype, C=C, B=1, H=2, T=T, dk=dk, dv=dv, seed=seed)
    x = generate(w)
    do = upstream_grad(w)
    args = [to_dev(x[n], dtype) for n in ("q", "k", "v")]
    args += [to_dev(x["log_alpha"]), to_dev(x["lam"]), to_dev(do, dtype)]
    return w, args


# Gradients from the single-pass forward's summaries against ll_mamba2_bwd's own (the same group
# summaries, each a bf16 rounding of fp32 sums formed in another order)
REUSE_TOL = 1e-2


def _check_reused(dtype, got, ref, label):
    import torch
    for n, a, b in zip(NAMES, got, ref):
        if dtype == "f32":
            assert torch.equal(a, b), (label, n)
        else:
            e = rel_err(a.float().cpu().numpy().astype(np.float64), b.float().cpu().numpy().astype(np.float64))
            print(label, n, f"{e:.2e}", flush=True)
            assert e <= REUSE_TOL, (label, n, e)


@pytest.mark.parametrize("dtype,C,T,dk,dv", [("bf16", 64, 64 * 66, 128, 128), ("bf16", 64, 64 * 19, 128, 64),
                                             ("bf16", 64, 64 * 21, 64, 64), ("f32", 16, 16 * 70, 16, 16)])
def test_bwd_after_fwd_reuses_the_forward_summaries(dtype, C, T, dk, dv):
    """ll_mamba2_bwd_after_fwd on the workspace a forward just filled.  After the three-kernel
    forward (fp32 here) it runs ll_mamba2_bwd's kernels on the summaries ll_mamba2_bwd would form:
    bit for bit equal.  After the single-pass forward (bf16, C = 64) it reads the nodes that forward
    published (also in the backward's order, with the tiles' gates): close to ll_mamba2_bwd's
    gradients and within the bar of the oracle's."""
    import torch
    import paper_2506_04761_amd as ll
    w, args = _bwd_case(dtype, C, T, dk, dv)
    ref = [g.clone() for g in ll.ll_mamba2_bwd(*args, w.C)]
    ws = ll.ll_mamba2_bwd_workspace(args[0], args[2], w.C)
    ws.fill_(255)  # stale bytes: everything the backward reads must come from the forward
    ll.ll_mamba2_fwd(*args[:5], w.C, workspace=ws)
    got = ll.ll_mamba2_bwd_after_fwd(*args, w.C, ws)
    torch.cuda.synchronize()
    _check_reused(dtype, got, ref, f"{dtype} T={T} d=({dk},{dv}) vs ll_mamba2_bwd")
    if dtype == "bf16":
        x = generate(w)
        do = upstream_grad(w)
        oref = mamba2_grad.quadratic_grad(x["q"], x["k"], x["v"], x["log_alpha"], x["lam"], do)
        for n, g, r in zip(NAMES, got, oref):
            e = rel_err(g.float().cpu().numpy().astype(np.float64), r)
            print(f"reused T={T} d=({dk},{dv}) vs oracle", n, f"{e:.2e}", flush=True)
            assert e <= TOL["bf16"], (n, e)


@pytest.mark.parametrize("dtype,C,T,dk,dv", [("f32", 16, 16 * 70, 16, 16), ("bf16", 64, 64 * 19, 128, 128)])
def test_bwd_after_fwd_detects_a_workspace_of_other_inputs(dtype, C, T, dk, dv):
    """The summaries in the workspace belong to the forward of other inputs (another k tensor), or a
    lambda = NULL forward overwrote them, or (single-pass path) a forward given only a forward-sized
    part of the buffer did: every gradient comes back NaN, not silently wrong; a forward on the right
    inputs makes the reuse valid again."""
    import torch
    import paper_2506_04761_amd as ll

    def all_nan(label):
        got = ll.ll_mamba2_bwd_after_fwd(*args, w.C, ws)
        torch.cuda.synchronize()
        for n, g in zip(NAMES, got):
            assert torch.isnan(g).all(), (label, n)

    w, args = _bwd_case(dtype, C, T, dk, dv, seed=5)
    _, other = _bwd_case(dtype, C, T, dk, dv, seed=6)
    ws = ll.ll_mamba2_bwd_workspace(args[0], args[2], w.C)
    ll.ll_mamba2_fwd(*other[:5], w.C, workspace=ws)
    all_nan("other inputs")
    ll.ll_mamba2_fwd(*args[:4], None, w.C, workspace=ws)  # lambda = NULL: no summaries left
    all_nan("lambda = NULL forward")
    if dtype == "bf16":
        ll.ll_mamba2_fwd(*args[:5], w.C, workspace=ws)
        need = ll.ll_workspace_size(ll.LL_MAMBA2, ll.LL_BF16, w.B, w.T, w.H, w.dk, w.dv, w.C, 1)
        ll.ll_mamba2_fwd(*args[:5], w.C, workspace=ws[:need])  # a forward-sized workspace: no summaries left
        all_nan("forward-sized workspace")
    ref = [g.clone() for g in ll.ll_mamba2_bwd(*args, w.C)]
    ll.ll_mamba2_fwd(*args[:5], w.C, workspace=ws)
    got = ll.ll_mamba2_bwd_after_fwd(*args, w.C, ws)
    torch.cuda.synchronize()
    _check_reused(dtype, got, ref, "valid again")


@pytest.mark.parametrize("dtype,C,dk,dv,H,Hqk,T", [
    ("bf16", 64, 128, 128, 8, 1, 2048),
    ("bf16", 64, 128, 64, 8, 2, 64 * 19),
    ("bf16", 64, 64, 64, 6, 3, 512),
    ("f32", 16, 16, 16, 4, 2, 256),
])
def test_bwd_grouped_qk_heads(dtype, C, dk, dv, H, Hqk, T):
    """Shared query/key heads: the gradient of a shared q (k) is the sum over its group of heads of
    the per-head gradients of the same model with q and k repeated to every head (chain rule
    through the repetition); the oracle computes the latter and sums it."""
    import torch
    import paper_2506_04761_amd as ll
    from synthetic import shared_qk
    w = WORKLOADS["ll_mamba2_bf16_T65536"].with_(dtype=dtype, B=1, H=H, T=T, dk=dk, dv=dv, C=C, seed=41 + H,
                                                   qk_heads=Hqk)
    x = generate(w)
    q, k = shared_qk(x, w)
    do = upstream_grad(w)
    G = H // Hqk
    qr, kr = np.repeat(q, G, axis=2), np.repeat(k, G, axis=2)
    ref = mamba2_grad.quadratic_grad(qr, kr, x["v"], x["log_alpha"], x["lam"], do)
    ref = [ref[0].reshape(1, T, Hqk, G, dk).sum(axis=3), ref[1].reshape(1, T, Hqk, G, dk).sum(axis=3)] + list(ref[2:])
    grads = ll.ll_mamba2_bwd(to_dev(q, dtype), to_dev(k, dtype), to_dev(x["v"], dtype), to_dev(x["log_alpha"]),
                             to_dev(x["lam"]), to_dev(do, dtype), C)
    torch.cuda.synchronize()
    got = [g.float().cpu().numpy().astype(np.float64) for g in grads]
    errs = {n: rel_err(g, r) for n, g, r in zip(NAMES, got, ref)}
    print(f"grouped H={H} H_qk={Hqk} T={T} {dtype}", " ".join(f"{n} {e:.2e}" for n, e in errs.items()), flush=True)
    for n, e in errs.items():
        assert e <= TOL[dtype], (n, e)


def test_bwd_maximum_length_sampled():
    """The longest sequence the library takes (2^20 - 64 tokens: 8192 tiles, a ragged last tile,
    21 levels, key-side groups of up to 4096 tiles), alpha = 1: sampled rows, columns and dcum
    positions of one head against the oracle."""
    w = WORKLOADS["ll_mamba2_bf16_T65536"].with_(B=1, H=2, T=(1 << 20) - 64, dist="nodecay", seed=124)
    x = generate(w)
    do = upstream_grad(w)
    dq, dk, dv, dla, dlam = run_bwd(x, do, w.dtype, w.C)
    rows = np.array([0, 128, 524288, 777777, w.T - 1])
    cols = np.array([5, 600001, w.T - 1])
    xs = {n: x[n][:, :, 1:2] for n in x}
    do_s = do[:, :, 1:2]
    rq, rl = mamba2_grad.grad_rows(xs["q"], xs["k"], xs["v"], xs["log_alpha"], xs["lam"], do_s, rows)
    ck, cv = mamba2_grad.grad_cols(xs["q"], xs["k"], xs["v"], xs["log_alpha"], xs["lam"], do_s, cols)
    errs = {"dq": rel_err(dq[:, rows, 1:2], rq), "dlambda": rel_err(dlam[:, rows, 1:2], rl),
            "dk": rel_err(dk[:, cols, 1:2], ck), "dv": rel_err(dv[:, cols, 1:2], cv)}
    print(f"T={w.T} sampled", " ".join(f"{n} {e:.2e}" for n, e in errs.items()), flush=True)
    for n, e in errs.items():
        assert e <= TOL["bf16"], (n, e)
    assert np.all(np.isfinite(dla)) and np.max(np.abs(dla[:, 0])) <= TOL["bf16"] * np.max(np.abs(dla))


@pytest.mark.parametrize("Hqk", [2, 1])
def test_autograd_function_matches_the_entry_points(Hqk):
    """log_linear_mamba2 under torch.autograd: the output equals ll_mamba2_fwd(_grouped) and the
    gradients of sum(O * dO) equal the entry points' (that forward, then ll_mamba2_bwd_after_fwd in
    the same backward-sized workspace), bit for bit."""
    import torch
    import paper_2506_04761_amd as ll
    from synthetic import shared_qk
    w = WORKLOADS["ll_mamba2_bf16_T65536"].with_(B=1, H=2, T=64 * 21, dk=128, dv=64, seed=61,
                                                   qk_heads=Hqk if Hqk < 2 else 0)
    x = generate(w)
    if w.qk_heads:
        x["q"], x["k"] = shared_qk(x, w)
    do = to_dev(upstream_grad(w), "bf16")
    leaves = [to_dev(x[n], "bf16").requires_grad_() for n in ("q", "k", "v")]
    leaves += [to_dev(x["log_alpha"]).requires_grad_(), to_dev(x["lam"]).requires_grad_()]
    o = ll.log_linear_mamba2(*leaves, w.C)
    (o.float() * do.float()).sum().backward()
    plain = [t.detach() for t in leaves]
    fwd = ll.ll_mamba2_fwd_grouped if w.qk_heads else ll.ll_mamba2_fwd
    assert torch.equal(o.detach(), fwd(*plain, w.C))
    ws = ll.ll_mamba2_bwd_workspace(plain[0], plain[2], w.C)
    fwd(*plain, w.C, workspace=ws)
    ref = ll.ll_mamba2_bwd_after_fwd(*plain, do, w.C, ws)
    torch.cuda.synchronize()
    for n, t, r in zip(NAMES, leaves, ref):
        assert torch.equal(t.grad, r), n


@pytest.mark.parametrize("dtype,C", [("bf16", 64), ("f32", 16)])
def test_autograd_backward_twice_with_retain_graph(dtype, C):
    """Two backward passes through one graph (retain_graph=True): both give the entry points'
    gradients (ll_mamba2_fwd, then ll_mamba2_bwd_after_fwd; the forward's workspace stays with the
    graph and the backward leaves its summaries as they were)."""
    import torch
    import paper_2506_04761_amd as ll
    w, args = _bwd_case(dtype, C, 16 * 72, 128 if dtype == "bf16" else 16, 64 if dtype == "bf16" else 16, seed=71)
    leaves = [t.clone().requires_grad_() for t in args[:5]]
    do = args[5]
    o = ll.log_linear_mamba2(*leaves, w.C)
    ws = ll.ll_mamba2_bwd_workspace(args[0], args[2], w.C)
    ll.ll_mamba2_fwd(*args[:5], w.C, workspace=ws)
    ref = ll.ll_mamba2_bwd_after_fwd(*args, w.C, ws)
    for rep in range(2):
        grads = torch.autograd.grad(o, leaves, grad_outputs=do, retain_graph=True)
        torch.cuda.synchronize()
        for n, g, r in zip(NAMES, grads, ref):
            assert torch.equal(g, r), (rep, n)


@pytest.mark.parametrize("dtype,C,dk,dv,H,Hqk,T", [
    ("bf16", 64, 128, 128, 2, 2, 64 * 67),
    ("bf16", 64, 128, 64, 4, 1, 64 * 19),
    ("f32", 16, 16, 16, 2, 2, 64 * 19 - 16),
])
def test_bwd_deterministic_and_writes_every_output(dtype, C, dk, dv, H, Hqk, T):
    """Two backward calls on the same inputs are equal bit for bit (no order-dependent
    accumulation), and every gradient element is written: the gradients and the workspace start
    as NaN bit patterns, so an element left unwritten, or computed from workspace bytes no kernel
    wrote, shows up as NaN."""
    import torch
    import paper_2506_04761_amd as ll
    from synthetic import shared_qk
    w = WORKLOADS["ll_mamba2_bf16_T65536"].with_(dtype=dtype, B=1, H=H, T=T, dk=dk, dv=dv, C=C, seed=131,
                                                   qk_heads=Hqk if Hqk < H else 0)
    x = generate(w)
    if w.qk_heads:
        x["q"], x["k"] = shared_qk(x, w)
    args = [to_dev(x[n], dtype) for n in ("q", "k", "v")]
    args += [to_dev(x["log_alpha"]), to_dev(x["lam"]), to_dev(upstream_grad(w), dtype)]
    outs = []
    for _ in range(2):
        ws = ll.ll_mamba2_bwd_workspace(args[0], args[2], C)
        ws.fill_(255)
        grads = tuple(torch.full_like(t, float("nan")) for t in (args[0], args[1], args[2], args[3], args[4]))
        ll.ll_mamba2_bwd(*args, C, grads=grads, workspace=ws)
        torch.cuda.synchronize()
        for n, g in zip(NAMES, grads):
            assert not torch.isnan(g).any(), n
        outs.append([g.clone() for g in grads])
    for n, a, b in zip(NAMES, *outs):
        assert torch.equal(a, b), n
