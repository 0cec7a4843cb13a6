"""Workload table and the seeded input generator.

Draw order (numpy PCG64 `default_rng(seed)`, float32 standard normals, each a full array
in [B, T, H, ...] row-major order): q, k, v, the log-gate pre-activation x_a, the level
weight pre-activation x_l, and (delta-rule workloads only) the beta pre-activation x_b.
Workloads whose query/key heads are shared (qk_heads > 0) take q, k of the first head of each
group of H / qk_heads heads (see shared_qk).

Transforms by distribution name:
  "unit"     q, k ~ N/sqrt(d_k), v ~ N/sqrt(d_v), log alpha = -softplus(x_a),     lambda = softplus(x_l)
  "shifted"  q, k ~ N/sqrt(d_k), v ~ N(0,1),      log alpha = -softplus(x_a + 2), lambda = softplus(x_l)
  "gdn"      q ~ N/sqrt(d_k), k = x/|x| per (b,t,h), v ~ N(0,1), beta = sigmoid(x_b),
             log alpha = -softplus(x_a + 2), lambda = softplus(x_l)
  "slow"     as "unit" but log alpha = -softplus(x_a - 6) (about -0.0025: every level matters)
  "nodecay"  as "unit" but log alpha = 0 (alpha = 1)
  "gdn_slow", "gdn_nodecay"  as "gdn" with the "slow" / "nodecay" gates
q, k, v are then rounded to the storage dtype (bf16 round-to-nearest-even via torch on the
CPU, or kept float32); log alpha, lambda and beta are always float32.
"""

from dataclasses import dataclass, replace
import math

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    variant: str      # "mamba2", "gdn", "mamba2_bwd" (backward pass), "decode" or "gdn_decode" (decoding),
                      # "mamba2_diag_lambda" (matrix-valued level weights, diagonal)
    dtype: str        # "f32" or "bf16": storage dtype of q, k, v and o
    B: int
    H: int
    T: int
    dk: int
    dv: int
    C: int
    seed: int
    dist: str
    qk_heads: int = 0  # query/key heads shared by groups of heads (0: one per head)

    @property
    def levels(self) -> int:
        # ceil(log2 T) + 1, the level count of lambda's last axis
        return 1 if self.T == 1 else (self.T - 1).bit_length() + 1

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


WORKLOADS = {
    w.name: w for w in [
        Workload("ll_mamba2_f32_T64", "mamba2", "f32", 1, 1, 64, 16, 16, 16, 0, "unit"),
        Workload("ll_mamba2_bf16_T2048", "mamba2", "bf16", 2, 8, 2048, 64, 64, 64, 2, "shifted"),
        Workload("ll_mamba2_bf16_T8192", "mamba2", "bf16", 4, 32, 8192, 128, 64, 64, 3, "unit"),
        Workload("ll_mamba2_bf16_T65536", "mamba2", "bf16", 1, 16, 65536, 128, 128, 64, 4, "unit"),
        Workload("ll_gdn_bf16_T8192", "gdn", "bf16", 2, 16, 8192, 128, 128, 64, 5, "gdn"),
        # the shape of the paper's kernel benchmark (B = 2, 48 heads, head dim 64, state dim 128,
        # chunk 64, one query/key head for all heads), at T = 16384
        Workload("ll_mamba2_mva_bf16_T16384", "mamba2", "bf16", 2, 48, 16384, 128, 64, 64, 6, "unit", 1),
        # decoding: 64 sequences x 16 heads fed one token per step up to position 8191 (the token
        # inputs are the T = 1024 draw, cycled)
        # backward pass at the shared-head benchmark shape (one q/k head for all 48 heads)
        Workload("ll_mamba2_mva_bwd_bf16_T16384", "mamba2_bwd", "bf16", 2, 48, 16384, 128, 64, 64, 6, "unit", 1),
        # backward pass over the same inputs as the T = 65536 forward workload
        Workload("ll_mamba2_bwd_bf16_T65536", "mamba2_bwd", "bf16", 1, 16, 65536, 128, 128, 64, 4, "unit"),
        Workload("ll_gdn_decode_bf16_T8192", "gdn_decode", "bf16", 64, 16, 8192, 128, 128, 64, 8, "gdn"),
        Workload("ll_mamba2_decode_bf16_T8192", "decode", "bf16", 64, 16, 8192, 128, 128, 64, 7, "unit"),
        # matrix-valued level weights (diagonal Lambda_t^(l), see level_weight_matrices)
        Workload("ll_mamba2_diag_lambda_bf16_T8192", "mamba2_diag_lambda", "bf16", 1, 16, 8192, 128, 128, 64, 9,
                 "unit"),
    ]
}


def _softplus(x):
    return np.logaddexp(0.0, x)


def to_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round float values to the storage dtype and return them as float32 numpy
    (bf16 values are exactly representable in float32)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    if dtype == "f32":
        return x
    if dtype == "bf16":
        import torch
        return torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    raise ValueError(dtype)


def shared_qk(x: dict, w: Workload):
    """q, k of a workload with shared query/key heads: those of the first head of each group."""
    G = w.H // w.qk_heads
    return np.ascontiguousarray(x["q"][:, :, ::G]), np.ascontiguousarray(x["k"][:, :, ::G])


def generate(w: Workload, T: int = None, heads=None):
    """Inputs for workload w as a dict of float32 numpy arrays.

    `T` optionally truncates the sequence (a prefix is an exact sub-problem because the
    method is causal); `heads` optionally keeps a subset of heads.  Both are applied after
    drawing, so a truncated draw is a prefix of the full one."""
    rng = np.random.default_rng(w.seed)
    B, TT, H, dk, dv = w.B, w.T, w.H, w.dk, w.dv
    L = w.levels
    q = rng.standard_normal((B, TT, H, dk), dtype=np.float32)
    k = rng.standard_normal((B, TT, H, dk), dtype=np.float32)
    v = rng.standard_normal((B, TT, H, dv), dtype=np.float32)
    xa = rng.standard_normal((B, TT, H), dtype=np.float32)
    xl = rng.standard_normal((B, TT, H, L), dtype=np.float32)
    xb = rng.standard_normal((B, TT, H), dtype=np.float32) if w.variant in ("gdn", "gdn_decode") else None

    q = q / np.float32(math.sqrt(dk))
    if w.dist.startswith("gdn"):
        k = k / np.linalg.norm(k.astype(np.float64), axis=-1, keepdims=True).astype(np.float32)
    else:
        k = k / np.float32(math.sqrt(dk))
    if w.dist in ("unit", "slow", "nodecay"):
        v = v / np.float32(math.sqrt(dv))
    shift = {"unit": 0.0, "shifted": 2.0, "gdn": 2.0, "slow": -6.0, "nodecay": None,
             "gdn_slow": -6.0, "gdn_nodecay": None}[w.dist]
    if shift is None:
        log_alpha = np.zeros((B, TT, H), dtype=np.float32)
    else:
        log_alpha = (-_softplus(xa.astype(np.float64) + shift)).astype(np.float32)
    lam = _softplus(xl.astype(np.float64)).astype(np.float32)
    out = dict(q=to_storage(q, w.dtype), k=to_storage(k, w.dtype), v=to_storage(v, w.dtype),
               log_alpha=log_alpha, lam=lam)
    if xb is not None:
        out["beta"] = (1.0 / (1.0 + np.exp(-xb.astype(np.float64)))).astype(np.float32)
    if T is not None or heads is not None:
        T = TT if T is None else T
        hs = slice(None) if heads is None else heads
        Lt = 1 if T == 1 else (T - 1).bit_length() + 1
        for key in out:
            a = out[key][:, :T][:, :, hs]
            if key == "lam":
                a = a[..., :Lt]
            out[key] = np.ascontiguousarray(a)
    return out


def upstream_grad(w: Workload, T: int = None, heads=None):
    """The upstream gradient dO [B, T, H, d_v] for a backward pass over workload w: standard
    normals from their own stream (PCG64 seeded with seed + 1000), rounded to the storage dtype.
    `T` and `heads` select a prefix and a subset of heads of the full draw, as in generate."""
    rng = np.random.default_rng(w.seed + 1000)
    do = to_storage(rng.standard_normal((w.B, w.T, w.H, w.dv), dtype=np.float32), w.dtype)
    if T is not None or heads is not None:
        do = np.ascontiguousarray(do[:, :w.T if T is None else T][:, :, slice(None) if heads is None else heads])
    return do


def level_weight_matrices(w: Workload, form: str, T: int = None, heads=None) -> np.ndarray:
    """Matrix-valued level weights Lambda_t^(l) for workload w, float32.  Drawn from their own
    stream, torch's CPU generator seeded w.seed + 2000 (these arrays are large; the other inputs
    do not change), standard normals in row-major order, then:
      "diag"  [B, T, H, L, d_k]        softplus(x), the distribution of the scalar weights;
      "full"  [B, T, H, L, d_k, d_k]   x / sqrt(d_k), plus softplus(y) on the diagonal from a
                                       second draw y [B, T, H, L, d_k] (a perturbed positive
                                       diagonal).
    `T` and `heads` select a prefix and a subset of heads of the full draw, as in generate()."""
    import torch
    g = torch.Generator().manual_seed(w.seed + 2000)
    B, TT, H, dk, L = w.B, w.T, w.H, w.dk, w.levels
    zero = torch.zeros((), dtype=torch.float32)
    if form == "diag":
        lam = torch.logaddexp(zero, torch.randn((B, TT, H, L, dk), generator=g, dtype=torch.float32))
    elif form == "full":
        lam = torch.randn((B, TT, H, L, dk, dk), generator=g, dtype=torch.float32) / math.sqrt(dk)
        d = torch.logaddexp(zero, torch.randn((B, TT, H, L, dk), generator=g, dtype=torch.float32))
        lam.diagonal(dim1=-2, dim2=-1).add_(d)
    else:
        raise ValueError(form)
    lam = lam.numpy()
    if T is not None or heads is not None:
        T = TT if T is None else T
        Lt = 1 if T == 1 else (T - 1).bit_length() + 1
        lam = lam[:, :T][:, :, slice(None) if heads is None else heads][:, :, :, :Lt]
    return np.ascontiguousarray(lam)
