"""Helpers for the GPU parity tests: move the seeded inputs to the device, run the library
through its Python binding (which calls the C ABI), and measure the normalised error
max|O_gpu - O_ref| / max|O_ref| used throughout."""

import numpy as np


def torch_dtype(name):
    import torch
    return {"f32": torch.float32, "bf16": torch.bfloat16}[name]


def to_dev(x, dtype="f32"):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to("cuda").to(torch_dtype(dtype)).contiguous()


def device_inputs(inp, dtype):
    d = {n: to_dev(inp[n], dtype) for n in ("q", "k", "v")}
    for n in ("log_alpha", "lam", "beta"):
        if n in inp:
            d[n] = to_dev(inp[n], "f32")
    return d


def run_mamba2(inp, dtype, C, with_lambda=True, out=None, workspace=None):
    import torch
    import paper_2506_04761_amd as ll
    d = device_inputs(inp, dtype)
    o = ll.ll_mamba2_fwd(d["q"], d["k"], d["v"], d["log_alpha"], d["lam"] if with_lambda else None, C,
                         out=out, workspace=workspace)
    torch.cuda.synchronize()
    return o.float().cpu().numpy().astype(np.float64)


def run_mamba2_grouped(inp, q, k, dtype, C, with_lambda=True):
    """ll_mamba2_fwd_grouped with the given shared q, k ([B, T, H_qk, d_k]) and the rest of `inp`."""
    import torch
    import paper_2506_04761_amd as ll
    d = device_inputs(inp, dtype)
    o = ll.ll_mamba2_fwd_grouped(to_dev(q, dtype), to_dev(k, dtype), d["v"], d["log_alpha"],
                                 d["lam"] if with_lambda else None, C)
    torch.cuda.synchronize()
    return o.float().cpu().numpy().astype(np.float64)


def rel_err(got, ref):
    return float(np.max(np.abs(got - ref)) / max(float(np.max(np.abs(ref))), 1e-30))


def run_gdn(inp, C, with_lambda=True, out=None, workspace=None):
    import torch
    import paper_2506_04761_amd as ll
    d = device_inputs(inp, "bf16")
    o = ll.ll_gdn_fwd(d["q"], d["k"], d["v"], d["log_alpha"], d["beta"], d["lam"] if with_lambda else None, C,
                      out=out, workspace=workspace)
    torch.cuda.synchronize()
    return o.float().cpu().numpy().astype(np.float64)
