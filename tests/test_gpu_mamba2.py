"""GPU parity of ll_mamba2_fwd against the float64 oracle, through the C ABI.

Tolerances (normalised max-abs error max|O_gpu - O_ref| / max|O_ref|): 1e-4 for the fp32
path, 2e-2 for bf16 inputs with fp32 accumulation.  The oracle receives the same rounded
inputs, upcast to float64.  The level assignment must be bit-exact."""

import numpy as np
import pytest

from oracle import fenwick, mamba2
from synthetic import WORKLOADS, generate
from tests.gpu_util import rel_err, run_mamba2, run_mamba2_grouped

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-4, "bf16": 2e-2}


@pytest.fixture(scope="module", autouse=True)
def _device():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2506_04761_amd  # noqa: F401  (fails loudly if the library is missing)


def _oracle_full(x):
    return mamba2.quadratic(x["q"], x["k"], x["v"], x["log_alpha"], x["lam"])


# ------------------------------------------------------------------ level map (bit-exact)

@pytest.mark.parametrize("C", [8, 16, 64])
def test_level_map_bit_exact(C):
    import paper_2506_04761_amd as ll
    Ts = sorted({t for t in list(range(1, 65)) + [128, 192, 1024, 4096] if t % C == 0})
    for T in Ts:
        got = ll.ll_debug_level_map(T, C).cpu().numpy().astype(np.int64)
        np.testing.assert_array_equal(got, fenwick.level_matrix(T), err_msg=f"T={T} C={C}")


# ------------------------------------------------------------------ whole-output parity

@pytest.mark.parametrize("name", ["ll_mamba2_f32_T64", "ll_mamba2_bf16_T2048"])
def test_parity_small_workloads(name):
    w = WORKLOADS[name]
    x = generate(w)
    got = run_mamba2(x, w.dtype, w.C)
    err = rel_err(got, _oracle_full(x))
    print(f"{name}: rel err {err:.3e}")
    assert err <= TOL[w.dtype]


@pytest.mark.parametrize("chunks", [1, 2, 3, 5, 7, 16, 33])
@pytest.mark.parametrize("dk,dv", [(128, 64), (128, 128), (64, 64)])
def test_parity_ragged_chunk_counts(chunks, dk, dv):
    w = WORKLOADS["ll_mamba2_bf16_T65536"].with_(B=2, H=2, T=64 * chunks, dk=dk, dv=dv, seed=40 + chunks)
    x = generate(w)
    err = rel_err(run_mamba2(x, "bf16", 64), _oracle_full(x))
    print(f"bf16 {dk}x{dv} chunks={chunks}: rel err {err:.3e}")
    assert err <= TOL["bf16"], err


@pytest.mark.parametrize("chunks", [5, 7])
def test_parity_many_heads_short_blocks(chunks):
    # more (b, h) blocks of 4 tiles than block_state has persistent workgroups, every one of
    # them short (fewer than 4 tiles): the step pipeline crosses block boundaries with gaps
    w = WORKLOADS["ll_mamba2_bf16_T65536"].with_(B=2, H=160, T=64 * chunks, dk=64, dv=64, seed=60 + chunks)
    x = generate(w)
    for with_lambda in (True, False):
        lam = x["lam"] if with_lambda else np.ones_like(x["lam"])
        ref = mamba2.quadratic(x["q"], x["k"], x["v"], x["log_alpha"], lam)
        err = rel_err(run_mamba2(x, "bf16", 64, with_lambda=with_lambda), ref)
        print(f"B=2 H=160 T={w.T} lambda={with_lambda}: rel err {err:.3e}")
        assert err <= TOL["bf16"], err


@pytest.mark.parametrize("dk,dv", [(128, 128), (128, 64)])
def test_parity_uneven_head_blocks(dk, dv):
    # 69 (batch, head) pairs: the single-pass kernel's eight XCD queues take blocks of 9 and 8
    # consecutive pairs (blocks from 64 pairs on); 9 chunks give 5 tiles, the last one half full
    w = WORKLOADS["ll_mamba2_bf16_T65536"].with_(B=3, H=23, T=64 * 9, dk=dk, dv=dv, seed=77 + dv)
    x = generate(w)
    for with_lambda in (True, False):
        lam = x["lam"] if with_lambda else np.ones_like(x["lam"])
        ref = mamba2.quadratic(x["q"], x["k"], x["v"], x["log_alpha"], lam)
        err = rel_err(run_mamba2(x, "bf16", 64, with_lambda=with_lambda), ref)
        print(f"B=3 H=23 {dk}x{dv} T={w.T} lambda={with_lambda}: rel err {err:.3e}")
        assert err <= TOL["bf16"], err


@pytest.mark.parametrize("T", [16, 48, 256, 1024])
def test_parity_fp32_small_chunk(T):
    w = WORKLOADS["ll_mamba2_f32_T64"].with_(B=2, H=3, T=T, seed=T)
    x = generate(w)
    err = rel_err(run_mamba2(x, "f32", 16), _oracle_full(x))
    print(f"f32 C=16 T={T}: rel err {err:.3e}")
    assert err <= TOL["f32"], err


@pytest.mark.parametrize("T", [64, 320, 1024])
def test_parity_fp32_c64(T):
    w = WORKLOADS["ll_mamba2_f32_T64"].with_(B=1, H=2, T=T, dk=64, dv=64, C=64, seed=7 + T)
    x = generate(w)
    err = rel_err(run_mamba2(x, "f32", 64), _oracle_full(x))
    print(f"f32 C=64 T={T}: rel err {err:.3e}")
    assert err <= TOL["f32"], err


@pytest.mark.parametrize("dist", ["slow", "nodecay", "shifted"])
def test_parity_stress_gates(dist):
    # slow decay: every level carries a sizeable share of |O|; alpha = 1: no decay at all
    w = WORKLOADS["ll_mamba2_bf16_T65536"].with_(B=1, H=2, T=2048, dist=dist, seed=11)
    x = generate(w)
    err = rel_err(run_mamba2(x, "bf16", 64), _oracle_full(x))
    print(f"bf16 gates {dist}: rel err {err:.3e}")
    assert err <= TOL["bf16"], err


# ------------------------------------------------------------------ query/key heads shared in groups

@pytest.mark.parametrize("dtype,C,dk,dv,H,Hqk,T", [
    ("bf16", 64, 128, 128, 8, 1, 2048),   # multi-value form: one query/key head for all heads
    ("bf16", 64, 128, 64, 8, 2, 64 * 19),  # grouped, ragged tile count
    ("bf16", 64, 64, 64, 6, 3, 512),
    ("f32", 16, 16, 16, 4, 2, 256),
])
def test_parity_grouped_qk_heads(dtype, C, dk, dv, H, Hqk, T):
    """Sharing q, k across each group of H / H_qk heads equals the per-head computation with the
    group's q, k repeated to every head of the group (head h uses query/key head h // group)."""
    w = WORKLOADS["ll_mamba2_bf16_T65536"].with_(dtype=dtype, B=2, H=H, T=T, dk=dk, dv=dv, C=C, seed=80 + H + Hqk)
    x = generate(w)
    G = H // Hqk
    q, k = np.ascontiguousarray(x["q"][:, :, ::G]), np.ascontiguousarray(x["k"][:, :, ::G])
    qr, kr = np.repeat(q, G, axis=2), np.repeat(k, G, axis=2)
    for with_lambda in (True, False):
        lam = x["lam"] if with_lambda else np.ones_like(x["lam"])
        ref = mamba2.quadratic(qr, kr, x["v"], x["log_alpha"], lam)
        err = rel_err(run_mamba2_grouped(x, q, k, dtype, C, with_lambda=with_lambda), ref)
        print(f"H={H} H_qk={Hqk} T={T} {dtype} lambda={with_lambda}: rel err {err:.3e}")
        assert err <= TOL[dtype], err


# ------------------------------------------------------------------ one level at a time

@pytest.mark.parametrize("dtype,C,dk,dv,T", [("bf16", 64, 128, 128, 4096), ("f32", 16, 16, 16, 1024)])
def test_each_level_alone(dtype, C, dk, dv, T):
    """O is linear in lambda: a one-hot lambda isolates one level's contribution, normalised by
    its own maximum (whole-output parity cannot see the small top levels)."""
    w = WORKLOADS["ll_mamba2_bf16_T65536"].with_(dtype=dtype, B=1, H=2, T=T, dk=dk, dv=dv, C=C,
                                                   dist="slow", seed=21)
    x = generate(w)
    L = x["lam"].shape[-1]
    for lv in range(L):
        y = dict(x)
        lam = np.zeros_like(x["lam"])
        lam[..., lv] = x["lam"][..., lv]
        y["lam"] = lam
        err = rel_err(run_mamba2(y, dtype, C), _oracle_full(y))
        assert err <= TOL[dtype], (lv, err)


# ------------------------------------------------------------------ lambda == NULL (Mamba-2)

@pytest.mark.parametrize("dtype,C,dk,dv,T", [("bf16", 64, 128, 64, 2048), ("f32", 16, 16, 16, 512)])
def test_lambda_null_is_mamba2(dtype, C, dk, dv, T):
    w = WORKLOADS["ll_mamba2_bf16_T8192"].with_(dtype=dtype, B=2, H=2, T=T, dk=dk, dv=dv, C=C, seed=31)
    x = generate(w)
    ref = mamba2.gla_recurrent(x["q"], x["k"], x["v"], x["log_alpha"])
    got_null = run_mamba2(x, dtype, C, with_lambda=False)
    assert rel_err(got_null, ref) <= TOL[dtype]
    y = dict(x)
    y["lam"] = np.ones_like(x["lam"])
    got_ones = run_mamba2(y, dtype, C)
    assert rel_err(got_ones, ref) <= TOL[dtype]


@pytest.mark.parametrize("dist", ["slow", "nodecay"])
@pytest.mark.parametrize("dk,dv,T", [(128, 128, 64 * 37), (128, 64, 64 * 52), (64, 64, 64 * 21)])
def test_lambda_null_slow_decay_many_tiles(dist, dk, dv, T):
    """lambda == NULL sums a tile's source nodes into one state before its product pass; with slow or
    no decay every source group carries a sizeable share of |O|, so a wrong weight or node shows."""
    w = WORKLOADS["ll_mamba2_bf16_T65536"].with_(B=1, H=2, T=T, dk=dk, dv=dv, dist=dist, seed=43)
    x = generate(w)
    ref = mamba2.gla_recurrent(x["q"], x["k"], x["v"], x["log_alpha"])
    got = run_mamba2(x, "bf16", 64, with_lambda=False)
    err = rel_err(got, ref)
    print(f"lambda=NULL {dist} {dk}x{dv} T={T}: rel err {err:.3e}")
    assert err <= TOL["bf16"], err


# ------------------------------------------------------------------ full-size workloads, sampled rows

def _sampled_parity(name, rows_per_head=24, heads=((0, 0), (0, 5))):
    w = WORKLOADS[name]
    x = generate(w)
    got = run_mamba2(x, w.dtype, w.C)
    rng = np.random.default_rng(99)
    worst = 0.0
    for b, h in heads:
        rows = np.unique(np.concatenate([[0, w.C - 1, w.C, w.T - 1],
                                         rng.integers(0, w.T, rows_per_head)]))
        xs = {n: x[n][b:b + 1, :, h:h + 1] for n in ("q", "k", "v", "log_alpha", "lam")}
        ref = mamba2.quadratic(xs["q"], xs["k"], xs["v"], xs["log_alpha"], xs["lam"], rows=rows)
        worst = max(worst, rel_err(got[b:b + 1, rows, h:h + 1], ref))
    print(f"{name}: sampled rel err {worst:.3e}")
    return worst


def test_parity_T8192_full_size_sampled():
    assert _sampled_parity("ll_mamba2_bf16_T8192", heads=((0, 0), (3, 31), (2, 17))) <= TOL["bf16"]


def test_parity_T65536_full_size_sampled():
    assert _sampled_parity("ll_mamba2_bf16_T65536", heads=((0, 0), (0, 15))) <= TOL["bf16"]


def test_parity_T65536_every_row_four_heads():
    """Every output row of four of the 16 heads (the first and the last among them) of the
    T = 65536 workload, in the launch configuration the benchmark times, against the oracle's
    per-level recurrent form (one worker process per head)."""
    from tests.oracle_pool import recurrent_heads
    w = WORKLOADS["ll_mamba2_bf16_T65536"]
    x = generate(w)
    got = run_mamba2(x, w.dtype, w.C)
    heads = [(0, 0), (0, 5), (0, 10), (0, 15)]
    refs = recurrent_heads("mamba2", x, heads, ("q", "k", "v", "log_alpha", "lam"))
    for (b, h), ref in zip(heads, refs):
        err = rel_err(got[b:b + 1, :, h:h + 1], ref)
        print(f"T=65536 head {h}: every row rel err {err:.3e}", flush=True)
        assert err <= TOL["bf16"], (h, err)


@pytest.mark.parametrize("lv", [12, 13, 14, 15, 16])
def test_each_top_level_alone_T65536(lv):
    """One-hot lambda at one of the top token levels 12..16 of T = 65536 (inter-tile levels 5..9
    of the tiles of 128 tokens), with alpha = 1 so that the far levels carry full weight; sampled
    rows (half of them with bit lv - 1 set, i.e. with keys at that level) against the
    row-restricted quadratic form."""
    w = WORKLOADS["ll_mamba2_bf16_T65536"].with_(B=1, H=2, dist="nodecay", seed=130 + lv)
    x = generate(w)
    lam = np.zeros_like(x["lam"])
    lam[..., lv] = x["lam"][..., lv]
    y = dict(x, lam=lam)
    got = run_mamba2(y, w.dtype, w.C)
    rng = np.random.default_rng(lv)
    r = rng.integers(0, w.T, 24)
    rows = np.unique(np.concatenate([r | (1 << (lv - 1)), r & ~(1 << (lv - 1)), [w.T - 1, (1 << (lv - 1))]]))
    ref = mamba2.quadratic(y["q"], y["k"], y["v"], y["log_alpha"], y["lam"], rows=rows)
    assert np.max(np.abs(ref)) > 0
    err = rel_err(got[:, rows], ref)
    print(f"level {lv} alone at T=65536: rel err {err:.3e}", flush=True)
    assert err <= TOL["bf16"], err


def test_parity_T8192_other_reading_of_distribution():
    # The large workloads say "same distributions as config 1"; the other possible reading
    # (the second workload's gates and unscaled values) must pass too.
    w = WORKLOADS["ll_mamba2_bf16_T8192"].with_(B=1, H=2, dist="shifted", seed=33)
    x = generate(w)
    err = rel_err(run_mamba2(x, "bf16", 64), _oracle_full(x))
    assert err <= TOL["bf16"], err


# ------------------------------------------------------------------ hygiene

def test_deterministic_and_writes_every_output():
    import torch
    import paper_2506_04761_amd as ll
    from tests.gpu_util import device_inputs
    w = WORKLOADS["ll_mamba2_bf16_T2048"]
    x = generate(w)
    d = device_inputs(x, "bf16")
    need = ll.ll_workspace_size(ll.LL_MAMBA2, ll.LL_BF16, w.B, w.T, w.H, w.dk, w.dv, w.C, 1)
    outs = []
    for _ in range(2):
        ws = torch.full((need,), 0xFF, dtype=torch.uint8, device="cuda")  # NaN bit patterns
        o = torch.full((w.B, w.T, w.H, w.dv), float("nan"), dtype=torch.bfloat16, device="cuda")
        ll.ll_mamba2_fwd(d["q"], d["k"], d["v"], d["log_alpha"], d["lam"], w.C, out=o, workspace=ws)
        torch.cuda.synchronize()
        assert not torch.isnan(o).any()
        outs.append(o.clone())
    assert torch.equal(outs[0], outs[1])


def test_workspace_reuse_alternating_inputs():
    """Two different inputs run in turn through one workspace and one output buffer: every run
    must reproduce, bit for bit, its result on a fresh workspace (summaries left by the other
    input must never be read), and that result must match the oracle on sampled rows."""
    import torch
    import paper_2506_04761_amd as ll
    from tests.gpu_util import device_inputs
    base = WORKLOADS["ll_mamba2_bf16_T65536"].with_(B=2, H=16, T=16384)
    xs = [generate(base.with_(seed=s)) for s in (71, 72)]
    ds = [device_inputs(x, "bf16") for x in xs]
    need = ll.ll_workspace_size(ll.LL_MAMBA2, ll.LL_BF16, base.B, base.T, base.H, base.dk, base.dv, base.C, 1)
    o = torch.empty((base.B, base.T, base.H, base.dv), dtype=torch.bfloat16, device="cuda")

    def run(d, ws):
        ll.ll_mamba2_fwd(d["q"], d["k"], d["v"], d["log_alpha"], d["lam"], base.C, out=o, workspace=ws)
        torch.cuda.synchronize()
        return o.clone()

    fresh = [run(d, torch.zeros(need, dtype=torch.uint8, device="cuda")) for d in ds]
    ws = torch.zeros(need, dtype=torch.uint8, device="cuda")
    for it in range(6):
        got = run(ds[it % 2], ws)
        assert torch.equal(got, fresh[it % 2]), f"run {it}"
    rows = np.array([0, 127, 128, 4095, 8191, 8192, 12345, base.T - 1])
    for x, f in zip(xs, fresh):
        got = f.float().cpu().numpy().astype(np.float64)
        for b, h in ((0, 0), (1, 15)):
            xh = {n: x[n][b:b + 1, :, h:h + 1] for n in ("q", "k", "v", "log_alpha", "lam")}
            ref = mamba2.quadratic(xh["q"], xh["k"], xh["v"], xh["log_alpha"], xh["lam"], rows=rows)
            assert rel_err(got[b:b + 1, rows, h:h + 1], ref) <= TOL["bf16"]


def test_parity_maximum_length_sampled():
    """The longest sequence the library takes (8192 tiles of 128 rows; here 2^20 - 64 tokens, a
    ragged last tile, 21 levels, the deepest block tree), with alpha = 1 so that every level's
    terms stay large: sampled rows of two heads against the quadratic form."""
    w = WORKLOADS["ll_mamba2_bf16_T65536"].with_(B=1, H=2, T=(1 << 20) - 64, dist="nodecay", seed=123)
    x = generate(w)
    got = run_mamba2(x, w.dtype, w.C)
    rows = np.array([0, 127, 128, 65535, 65536, 524287, 524288, 777777, w.T - 65, w.T - 1])
    worst = 0.0
    for h in (0, 1):
        xs = {n: x[n][:, :, h:h + 1] for n in ("q", "k", "v", "log_alpha", "lam")}
        ref = mamba2.quadratic(xs["q"], xs["k"], xs["v"], xs["log_alpha"], xs["lam"], rows=rows)
        worst = max(worst, rel_err(got[:, rows, h:h + 1], ref))
    print(f"T={w.T}: sampled rel err {worst:.3e}")
    assert worst <= TOL["bf16"]
