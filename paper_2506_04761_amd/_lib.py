"""ctypes binding of libloglinear.so (the C ABI declared in include/libloglinear.h).

Argument marshalling only: tensors are passed as raw device pointers plus sizes, and every step
of the computation runs in the library's HIP kernels.  PyTorch supplies device memory and the
current stream.  If the shared library is missing this module raises at import: there is no
fallback implementation.
"""

import ctypes
import os

# PyTorch ships its own HIP runtime under the same soname as ROCm's (libamdhip64.so.7).  Load it
# first so this library binds to the runtime that owns torch's device memory and streams.
import torch  # noqa: F401

HERE = os.path.dirname(os.path.abspath(__file__))
# LIBLOGLINEAR_PATH selects another build of the same sources (the host-sanitized one of
# build.py --asan); by default the in-tree library is loaded.
LIB_PATH = os.environ.get("LIBLOGLINEAR_PATH") or os.path.join(HERE, "libloglinear.so")

LL_OK, LL_ERR_NULL_ARG, LL_ERR_BAD_SHAPE, LL_ERR_UNSUPPORTED, LL_ERR_WORKSPACE, LL_ERR_HIP, LL_ERR_SCRATCH = range(7)
LL_NOALLOC_SCRATCH_BYTES = 64 << 20
LL_F32, LL_BF16 = 0, 1
LL_MAMBA2, LL_GDN, LL_MAMBA2_BWD = 0, 1, 2
LL_LAMBDA_DIAG, LL_LAMBDA_FULL = 0, 1

if not os.path.exists(LIB_PATH):
    raise ImportError(
        f"{LIB_PATH} is missing: build it with `python paper_2506_04761_amd/build.py` "
        "(libloglinear has no non-HIP implementation)")

lib = ctypes.CDLL(LIB_PATH)

_i64, _i32, _vp, _sz = ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p, ctypes.c_size_t

lib.ll_num_levels.argtypes = [_i64]
lib.ll_num_levels.restype = _i32
lib.ll_supported.argtypes = [_i32, _i32, _i64, _i64, _i64]
lib.ll_supported.restype = _i32
lib.ll_workspace_size.argtypes = [_i32, _i32, _i64, _i64, _i64, _i64, _i64, _i64, _i32]
lib.ll_workspace_size.restype = _sz
lib.ll_mamba2_fwd.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp, _i64, _i64, _i64, _i64, _i64, _i64, _i32, _vp, _sz, _vp]
lib.ll_mamba2_fwd.restype = _i32
lib.ll_mamba2_fwd_noalloc.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp, _i64, _i64, _i64, _i64, _i64, _i64, _i32, _vp]
lib.ll_mamba2_fwd_noalloc.restype = _i32
lib.ll_mamba2_fwd_grouped.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp, _i64, _i64, _i64, _i64, _i64, _i64, _i64, _i32,
                                       _vp, _sz, _vp]
lib.ll_mamba2_fwd_grouped.restype = _i32
lib.ll_decode_state_bytes.argtypes = [_i64, _i64, _i64, _i64, _i32]
lib.ll_decode_state_bytes.restype = _sz
lib.ll_mamba2_decode_init.argtypes = [_vp, _sz, _i64, _i64, _i64, _i64, _i32, _i32, _vp]
lib.ll_mamba2_decode_init.restype = _i32
lib.ll_mamba2_decode_step.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _i64, _i64, _i64, _i64, _i64, _i32,
                                      _i32, _vp]
lib.ll_mamba2_decode_step.restype = _i32
lib.ll_gdn_decode_init.argtypes = [_vp, _sz, _i64, _i64, _i64, _i64, _i32, _i32, _vp]
lib.ll_gdn_decode_init.restype = _i32
lib.ll_gdn_decode_step.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _i64, _i64, _i64, _i64, _i64, _i32,
                                   _i32, _vp]
lib.ll_gdn_decode_step.restype = _i32
lib.ll_mamba2_fwd_staged.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp, _i64, _i64, _i64, _i64, _i64, _i64, _i64, _i32,
                                      _vp, _sz, _vp, ctypes.POINTER(_vp)]
lib.ll_mamba2_fwd_staged.restype = _i32
lib.ll_mamba2_matrix_lambda_workspace_size.argtypes = [_i32, _i32, _i64, _i64, _i64, _i64, _i64, _i64]
lib.ll_mamba2_matrix_lambda_workspace_size.restype = _sz
lib.ll_mamba2_fwd_matrix_lambda.argtypes = [_vp, _vp, _vp, _vp, _vp, _i32, _vp, _i64, _i64, _i64, _i64, _i64, _i64,
                                            _i32, _vp, _sz, _vp]
lib.ll_mamba2_fwd_matrix_lambda.restype = _i32
lib.ll_mamba2_fwd_matrix_lambda_staged.argtypes = [_vp, _vp, _vp, _vp, _vp, _i32, _vp, _i64, _i64, _i64, _i64, _i64,
                                                   _i64, _i32, _vp, _sz, _vp, ctypes.POINTER(_vp)]
lib.ll_mamba2_fwd_matrix_lambda_staged.restype = _i32
lib.ll_gdn_fwd.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _i64, _i64, _i64, _i64, _i64, _i64, _i32, _vp, _sz, _vp]
lib.ll_gdn_fwd.restype = _i32
lib.ll_gdn_fwd_staged.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _i64, _i64, _i64, _i64, _i64, _i64, _i32, _vp, _sz,
                                   _vp, ctypes.POINTER(_vp)]
lib.ll_gdn_fwd_staged.restype = _i32
lib.ll_mamba2_bwd.argtypes = [_vp] * 11 + [_i64] * 6 + [_i32, _vp, _sz, _vp]
lib.ll_mamba2_bwd.restype = _i32
lib.ll_mamba2_bwd_after_fwd.argtypes = [_vp] * 11 + [_i64] * 7 + [_i32, _vp, _sz, _vp]
lib.ll_mamba2_bwd_grouped.argtypes = [_vp] * 11 + [_i64] * 7 + [_i32, _vp, _sz, _vp]
lib.ll_mamba2_bwd_grouped.restype = _i32
lib.ll_mamba2_bwd_workspace_size.argtypes = [_i32] + [_i64] * 7
lib.ll_mamba2_bwd_workspace_size.restype = _sz
lib.ll_mamba2_bwd_after_fwd.restype = _i32
lib.ll_mamba2_bwd_staged.argtypes = [_vp] * 11 + [_i64] * 7 + [_i32, _vp, _sz, _vp, _vp]
lib.ll_mamba2_bwd_staged.restype = _i32
lib.ll_debug_level_map.argtypes = [_i64, _i64, _vp, _vp]
lib.ll_debug_level_map.restype = _i32
lib.ll_status_string.argtypes = [_i32]
lib.ll_status_string.restype = ctypes.c_char_p


class LLError(RuntimeError):
    def __init__(self, status: int):
        self.status = status
        super().__init__(lib.ll_status_string(status).decode())


def ll_num_levels(T: int) -> int:
    return lib.ll_num_levels(T)


def ll_supported(variant: int, dtype: int, C: int, d_k: int, d_v: int) -> bool:
    return bool(lib.ll_supported(variant, dtype, C, d_k, d_v))


def ll_workspace_size(variant, dtype, B, T, H, d_k, d_v, C, has_lambda) -> int:
    return lib.ll_workspace_size(variant, dtype, B, T, H, d_k, d_v, C, int(bool(has_lambda)))


def ll_status_string(status: int) -> str:
    return lib.ll_status_string(status).decode()


# ----------------------------------------------------------------------- torch-facing wrappers

def _torch():
    import torch
    return torch


def _dtype_code(t):
    torch = _torch()
    if t.dtype == torch.float32:
        return LL_F32
    if t.dtype == torch.bfloat16:
        return LL_BF16
    raise TypeError(f"unsupported dtype {t.dtype}; q, k, v must be float32 or bfloat16")


def _check(t, name, dtype=None, shape=None):
    torch = _torch()
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _prepare(variant, q, k, v, log_alpha, beta, lam, C, out, workspace, grouped=False):
    torch = _torch()
    B, T, Hqk, dk = q.shape
    H = v.shape[2] if grouped else Hqk
    dv = v.shape[-1]
    _check(q, "q")
    _check(k, "k", q.dtype, (B, T, Hqk, dk))
    _check(v, "v", q.dtype, (B, T, H, dv))
    _check(log_alpha, "log_alpha", torch.float32, (B, T, H))
    if beta is not None:
        _check(beta, "beta", torch.float32, (B, T, H))
    L = ll_num_levels(T)
    if lam is not None:
        _check(lam, "lambda", torch.float32, (B, T, H, L))
    code = _dtype_code(q)
    if out is None:
        out = torch.empty((B, T, H, dv), dtype=q.dtype, device=q.device)
    _check(out, "out", q.dtype, (B, T, H, dv))
    need = ll_workspace_size(variant, code, B, T, H, dk, dv, C, lam is not None)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=q.device)
    _check(workspace, "workspace", torch.uint8)
    return (B, T, H, dk, dv, code), out, workspace


def ll_mamba2_fwd(q, k, v, log_alpha, lam, C, out=None, workspace=None, stream=None):
    """Log-linear Mamba-2 forward on device tensors laid out [B, T, H, d]; `lam` may be None
    (all level weights 1, i.e. Mamba-2).  Returns `out`.  Work is enqueued on `stream`
    (default: torch's current stream) and is not synchronised."""
    (B, T, H, dk, dv, code), out, ws = _prepare(LL_MAMBA2, q, k, v, log_alpha, None, lam, C, out, workspace)
    st = lib.ll_mamba2_fwd(_ptr(q), _ptr(k), _ptr(v), _ptr(log_alpha), _ptr(lam), _ptr(out),
                           B, T, H, dk, dv, C, code, _ptr(ws), ws.numel(), _stream(stream))
    if st != LL_OK:
        raise LLError(st)
    return out


def ll_mamba2_fwd_noalloc(q, k, v, log_alpha, lam, C, out, stream=None):
    """ll_mamba2_fwd through the entry point that allocates nothing: the library works in its
    static per-GPU scratch, so calls on one GPU must be ordered.  `out` is caller-allocated.
    Returns `out`; raises LLError (LL_ERR_SCRATCH beyond LL_NOALLOC_SCRATCH_BYTES)."""
    torch = _torch()
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    _check(q, "q")
    _check(k, "k", q.dtype, (B, T, H, dk))
    _check(v, "v", q.dtype, (B, T, H, dv))
    _check(log_alpha, "log_alpha", torch.float32, (B, T, H))
    if lam is not None:
        _check(lam, "lambda", torch.float32, (B, T, H, ll_num_levels(T)))
    _check(out, "out", q.dtype, (B, T, H, dv))
    st = lib.ll_mamba2_fwd_noalloc(_ptr(q), _ptr(k), _ptr(v), _ptr(log_alpha), _ptr(lam), _ptr(out),
                                   B, T, H, dk, dv, C, _dtype_code(q), _stream(stream))
    if st != LL_OK:
        raise LLError(st)
    return out


def _ml_call(q, k, v, log_alpha, Lam, C, out, workspace, stream, handles):
    torch = _torch()
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    _check(q, "q")
    _check(k, "k", q.dtype, (B, T, H, dk))
    _check(v, "v", q.dtype, (B, T, H, dv))
    _check(log_alpha, "log_alpha", torch.float32, (B, T, H))
    L = ll_num_levels(T)
    if Lam.dim() == 5:
        form = LL_LAMBDA_DIAG
        _check(Lam, "Lambda", torch.float32, (B, T, H, L, dk))
    else:
        form = LL_LAMBDA_FULL
        _check(Lam, "Lambda", torch.float32, (B, T, H, L, dk, dk))
    code = _dtype_code(q)
    if out is None:
        out = torch.empty((B, T, H, dv), dtype=q.dtype, device=q.device)
    _check(out, "out", q.dtype, (B, T, H, dv))
    if workspace is None:
        workspace = ll_mamba2_matrix_lambda_workspace(q, v, C, full=form == LL_LAMBDA_FULL)
    _check(workspace, "workspace", torch.uint8)
    args = [_ptr(q), _ptr(k), _ptr(v), _ptr(log_alpha), _ptr(Lam), form, _ptr(out), B, T, H, dk, dv, C, code,
            _ptr(workspace), workspace.numel(), _stream(stream)]
    st = (lib.ll_mamba2_fwd_matrix_lambda(*args) if handles is None
          else lib.ll_mamba2_fwd_matrix_lambda_staged(*args, handles))
    if st != LL_OK:
        raise LLError(st)
    return out


def ll_mamba2_matrix_lambda_workspace(q, v, C, full=True):
    """A workspace for ll_mamba2_fwd_matrix_lambda shaped for q [B, T, H, d_k] and v [B, T, H, d_v]
    (full=True: for full matrices, which also serves diagonal ones)."""
    torch = _torch()
    B, T, H, dk = q.shape
    form = LL_LAMBDA_FULL if full else LL_LAMBDA_DIAG
    need = lib.ll_mamba2_matrix_lambda_workspace_size(form, _dtype_code(q), B, T, H, dk, v.shape[-1], C)
    return torch.empty(max(need, 1), dtype=torch.uint8, device=q.device)


def ll_mamba2_fwd_matrix_lambda(q, k, v, log_alpha, Lam, C, out=None, workspace=None, stream=None):
    """Log-linear Mamba-2 with matrix-valued level weights (the 4D-tensor view of App. A):
    O_t = sum_{s<=t} prod(alpha) (q_t Lambda_t^(l(t,s)) . k_s) v_s.  `Lam` is float32, either
    [B, T, H, L, d_k] (diagonal matrices) or [B, T, H, L, d_k, d_k] (full matrices).  Returns `out`;
    enqueued on `stream` (default: torch's current stream), not synchronised."""
    return _ml_call(q, k, v, log_alpha, Lam, C, out, workspace, stream, None)


def ll_mamba2_fwd_matrix_lambda_staged(q, k, v, log_alpha, Lam, C, events, out=None, workspace=None, stream=None):
    """As ll_mamba2_fwd_matrix_lambda, and records the five torch.cuda.Event objects in `events` around
    the four stages (level queries, tile states, scan, tile outputs)."""
    handles, s = _event_handles(events, 5, stream)
    return _ml_call(q, k, v, log_alpha, Lam, C, out, workspace, s, handles)


def ll_mamba2_fwd_grouped(q, k, v, log_alpha, lam, C, out=None, workspace=None, stream=None):
    """As ll_mamba2_fwd with query/key heads shared by groups of heads: q, k are [B, T, H_qk, d_k]
    and v, log_alpha, lam, out have H heads (H a multiple of H_qk; head h uses query/key head
    h // (H // H_qk)).  Returns `out`."""
    (B, T, H, dk, dv, code), out, ws = _prepare(LL_MAMBA2, q, k, v, log_alpha, None, lam, C, out, workspace,
                                                grouped=True)
    st = lib.ll_mamba2_fwd_grouped(_ptr(q), _ptr(k), _ptr(v), _ptr(log_alpha), _ptr(lam), _ptr(out),
                                   B, T, H, q.shape[2], dk, dv, C, code, _ptr(ws), ws.numel(), _stream(stream))
    if st != LL_OK:
        raise LLError(st)
    return out


def ll_decode_state_bytes(B, H, dk, dv, L):
    return int(lib.ll_decode_state_bytes(B, H, dk, dv, L))


def ll_mamba2_decode_init(state, B, H, dk, dv, L, dtype, stream=None):
    """Resets `state` (a uint8 device tensor of ll_decode_state_bytes(...) bytes) to the empty
    sequence; `dtype` is the torch dtype of the per-token q, k, v, o."""
    code = LL_BF16 if dtype == _torch().bfloat16 else LL_F32
    st = lib.ll_mamba2_decode_init(_ptr(state), state.numel(), B, H, dk, dv, L, code, _stream(stream))
    if st != LL_OK:
        raise LLError(st)


def ll_mamba2_decode_step(q, k, v, log_alpha, lam, state, t, L, out=None, stream=None):
    """Feeds token t: q, k [B, H, d_k], v [B, H, d_v], log_alpha [B, H], lam [B, H, L] or None;
    returns o [B, H, d_v].  `state` is the uint8 device tensor set up by ll_mamba2_decode_init."""
    torch = _torch()
    B, H, dk = q.shape
    dv = v.shape[-1]
    _check(q, "q")
    _check(k, "k", q.dtype, (B, H, dk))
    _check(v, "v", q.dtype, (B, H, dv))
    _check(log_alpha, "log_alpha", torch.float32, (B, H))
    if lam is not None:
        _check(lam, "lambda", torch.float32, (B, H, L))
    _check(state, "state", torch.uint8)
    if out is None:
        out = torch.empty((B, H, dv), dtype=q.dtype, device=q.device)
    _check(out, "out", q.dtype, (B, H, dv))
    st = lib.ll_mamba2_decode_step(_ptr(q), _ptr(k), _ptr(v), _ptr(log_alpha), _ptr(lam), _ptr(out), _ptr(state),
                                   state.numel(), t, B, H, dk, dv, L, _dtype_code(q), _stream(stream))
    if st != LL_OK:
        raise LLError(st)
    return out


def ll_gdn_decode_init(state, B, H, dk, dv, L, dtype, stream=None):
    """Resets `state` for log-linear Gated DeltaNet decoding (same buffer as the Mamba-2 calls)."""
    code = LL_BF16 if dtype == _torch().bfloat16 else LL_F32
    st = lib.ll_gdn_decode_init(_ptr(state), state.numel(), B, H, dk, dv, L, code, _stream(stream))
    if st != LL_OK:
        raise LLError(st)


def ll_gdn_decode_step(q, k, v, log_alpha, beta, lam, state, t, L, out=None, stream=None):
    """Feeds token t to log-linear Gated DeltaNet decoding: as ll_mamba2_decode_step plus
    beta [B, H] (float32, required)."""
    torch = _torch()
    B, H, dk = q.shape
    dv = v.shape[-1]
    _check(q, "q")
    _check(k, "k", q.dtype, (B, H, dk))
    _check(v, "v", q.dtype, (B, H, dv))
    _check(log_alpha, "log_alpha", torch.float32, (B, H))
    _check(beta, "beta", torch.float32, (B, H))
    if lam is not None:
        _check(lam, "lambda", torch.float32, (B, H, L))
    _check(state, "state", torch.uint8)
    if out is None:
        out = torch.empty((B, H, dv), dtype=q.dtype, device=q.device)
    _check(out, "out", q.dtype, (B, H, dv))
    st = lib.ll_gdn_decode_step(_ptr(q), _ptr(k), _ptr(v), _ptr(log_alpha), _ptr(beta), _ptr(lam), _ptr(out),
                                _ptr(state), state.numel(), t, B, H, dk, dv, L, _dtype_code(q), _stream(stream))
    if st != LL_OK:
        raise LLError(st)
    return out


def _event_handles(events, n, stream):
    """HIP event handles of `n` torch.cuda.Event objects (created with enable_timing=True)."""
    torch = _torch()
    if len(events) != n:
        raise ValueError(f"events must hold {n} torch.cuda.Event objects")
    s = torch.cuda.current_stream() if stream is None else stream
    for e in events:
        if e.cuda_event == 0:  # torch creates the HIP event on its first record
            e.record(s)
    return (_vp * n)(*[e.cuda_event for e in events]), s


def ll_mamba2_fwd_staged(q, k, v, log_alpha, lam, C, events, out=None, workspace=None, stream=None):
    """As ll_mamba2_fwd (ll_mamba2_fwd_grouped when q, k have fewer heads than v), and records
    the four torch.cuda.Event objects in `events` (created with enable_timing=True) on the stream
    around the three kernel stages: events[i] before stage i and events[3] after the last.  The
    stages are the tile totals, their block sums and the tile kernel on the single-pass path (bf16,
    C = 64), and the tile states, the scan (summary tree, or running states for lam=None) and the
    tile outputs on the three-kernel path.
    Asynchronous; read the durations with events[i].elapsed_time(events[i + 1]) after
    synchronising."""
    handles, s = _event_handles(events, 4, stream)
    (B, T, H, dk, dv, code), out, ws = _prepare(LL_MAMBA2, q, k, v, log_alpha, None, lam, C, out, workspace,
                                                grouped=True)
    st = lib.ll_mamba2_fwd_staged(_ptr(q), _ptr(k), _ptr(v), _ptr(log_alpha), _ptr(lam), _ptr(out),
                                  B, T, H, q.shape[2], dk, dv, C, code, _ptr(ws), ws.numel(), _stream(s), handles)
    if st != LL_OK:
        raise LLError(st)
    return out


def _bwd_call(q, k, v, log_alpha, lam, d_o, C, grads, workspace, stream, handles, after_fwd=False):
    torch = _torch()
    B, T, Hqk, dk = q.shape
    H, dv = v.shape[2], v.shape[-1]
    _check(q, "q")
    _check(k, "k", q.dtype, (B, T, Hqk, dk))
    _check(v, "v", q.dtype, (B, T, H, dv))
    _check(d_o, "d_o", q.dtype, (B, T, H, dv))
    _check(log_alpha, "log_alpha", torch.float32, (B, T, H))
    L = ll_num_levels(T)
    _check(lam, "lambda", torch.float32, (B, T, H, L))
    code = _dtype_code(q)
    if grads is None:
        dev = q.device
        grads = (torch.empty_like(q), torch.empty_like(k), torch.empty_like(v),
                 torch.empty((B, T, H), dtype=torch.float32, device=dev),
                 torch.empty((B, T, H, L), dtype=torch.float32, device=dev))
    dq, dk_, dv_, dla, dlam = grads
    _check(dq, "dq", q.dtype, q.shape)
    _check(dk_, "dk", q.dtype, k.shape)
    _check(dv_, "dv", q.dtype, v.shape)
    _check(dla, "dlog_alpha", torch.float32, (B, T, H))
    _check(dlam, "dlambda", torch.float32, (B, T, H, L))
    if workspace is None:
        if after_fwd:
            raise ValueError("ll_mamba2_bwd_after_fwd needs the workspace its forward ran in")
        need = lib.ll_mamba2_bwd_workspace_size(code, B, T, H, Hqk, dk, dv, C)
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=q.device)
    _check(workspace, "workspace", torch.uint8)
    args = [_ptr(x) for x in (q, k, v, log_alpha, lam, d_o, dq, dk_, dv_, dla, dlam)]
    tail = [dk, dv, C, code, _ptr(workspace), workspace.numel(), _stream(stream)]
    if after_fwd:
        st = lib.ll_mamba2_bwd_after_fwd(*args, B, T, H, Hqk, *tail)
    elif handles is not None:
        st = lib.ll_mamba2_bwd_staged(*args, B, T, H, Hqk, *tail, handles)
    elif Hqk == H:
        st = lib.ll_mamba2_bwd(*args, B, T, H, *tail)
    else:
        st = lib.ll_mamba2_bwd_grouped(*args, B, T, H, Hqk, *tail)
    if st != LL_OK:
        raise LLError(st)
    return grads


def ll_mamba2_bwd(q, k, v, log_alpha, lam, d_o, C, grads=None, workspace=None, stream=None):
    """Gradients of sum(O * d_o) for the log-linear Mamba-2 forward O on the same inputs:
    returns (dq, dk, dv, dlog_alpha, dlambda) (dq, dk, dv in the dtype of q; the others float32),
    written into `grads` when given.  `lam` is required.  When q and k have fewer heads than v
    (shared query/key heads, as in ll_mamba2_fwd_grouped) this calls ll_mamba2_bwd_grouped and dq,
    dk have q's shape.  Enqueued on `stream` (default: torch's current stream), not synchronised."""
    return _bwd_call(q, k, v, log_alpha, lam, d_o, C, grads, workspace, stream, None)


def ll_mamba2_bwd_workspace(q, v, C):
    """A workspace for the backward shaped for q [B, T, H_qk, d_k] and v [B, T, H, d_v] (also usable
    by the forward, which then leaves there the level summaries ll_mamba2_bwd_after_fwd reuses)."""
    torch = _torch()
    B, T, Hqk, dk = q.shape
    need = lib.ll_mamba2_bwd_workspace_size(_dtype_code(q), B, T, v.shape[2], Hqk, dk, v.shape[-1], C)
    return torch.empty(max(need, 1), dtype=torch.uint8, device=q.device)


def ll_mamba2_bwd_after_fwd(q, k, v, log_alpha, lam, d_o, C, workspace, grads=None, stream=None):
    """As ll_mamba2_bwd, reusing the level summaries that ll_mamba2_fwd left in `workspace` (a
    ll_mamba2_bwd_workspace) for the same inputs; see include/libloglinear.h for the contract."""
    return _bwd_call(q, k, v, log_alpha, lam, d_o, C, grads, workspace, stream, None, after_fwd=True)


def ll_mamba2_bwd_staged(q, k, v, log_alpha, lam, d_o, C, events, grads=None, workspace=None, stream=None):
    """As ll_mamba2_bwd, and records the five torch.cuda.Event objects in `events` around the four
    stages (forward summaries, key-side summaries, dq and dlambda, dk dv and dlog_alpha)."""
    handles, s = _event_handles(events, 5, stream)
    return _bwd_call(q, k, v, log_alpha, lam, d_o, C, grads, workspace, s, handles)


def ll_gdn_fwd(q, k, v, log_alpha, beta, lam, C, out=None, workspace=None, stream=None):
    """Log-linear Gated DeltaNet forward; as ll_mamba2_fwd plus `beta` [B, T, H] float32."""
    (B, T, H, dk, dv, code), out, ws = _prepare(LL_GDN, q, k, v, log_alpha, beta, lam, C, out, workspace)
    st = lib.ll_gdn_fwd(_ptr(q), _ptr(k), _ptr(v), _ptr(log_alpha), _ptr(beta), _ptr(lam), _ptr(out),
                        B, T, H, dk, dv, C, code, _ptr(ws), ws.numel(), _stream(stream))
    if st != LL_OK:
        raise LLError(st)
    return out


def ll_gdn_fwd_staged(q, k, v, log_alpha, beta, lam, C, events, out=None, workspace=None, stream=None):
    """As ll_gdn_fwd, recording three torch.cuda.Event objects around its two kernel stages
    (per-chunk WY kernel; block tree and read-out); see ll_mamba2_fwd_staged."""
    handles, s = _event_handles(events, 3, stream)
    (B, T, H, dk, dv, code), out, ws = _prepare(LL_GDN, q, k, v, log_alpha, beta, lam, C, out, workspace)
    st = lib.ll_gdn_fwd_staged(_ptr(q), _ptr(k), _ptr(v), _ptr(log_alpha), _ptr(beta), _ptr(lam), _ptr(out),
                               B, T, H, dk, dv, C, code, _ptr(ws), ws.numel(), _stream(s), handles)
    if st != LL_OK:
        raise LLError(st)
    return out


def ll_debug_level_map(T, C, stream=None):
    """The level map the kernels use, as a [T, T] int8 device tensor (-1 above the diagonal)."""
    torch = _torch()
    out = torch.empty((T, T), dtype=torch.int8, device="cuda")
    st = lib.ll_debug_level_map(T, C, _ptr(out), _stream(stream))
    if st != LL_OK:
        raise LLError(st)
    return out


# ----------------------------------------------------------------------- autograd

def _autograd_function():
    torch = _torch()

    class LogLinearMamba2(torch.autograd.Function):
        """O = log-linear Mamba-2 attention of (q, k, v, log_alpha, lam) as a differentiable op: the
        forward runs ll_mamba2_fwd (ll_mamba2_fwd_grouped when q, k have fewer heads than v) in a
        backward-sized workspace kept with the graph, and the backward runs ll_mamba2_bwd_after_fwd
        on it (the forward's level summaries are reused where the forward leaves them, and the
        reuse is checked on the device).  Memory held until the graph is freed:
        ll_mamba2_bwd_workspace_size(...) bytes plus the saved inputs."""

        @staticmethod
        def forward(ctx, q, k, v, log_alpha, lam, C):
            q, k, v, log_alpha, lam = (x.contiguous() for x in (q, k, v, log_alpha, lam))
            ws = ll_mamba2_bwd_workspace(q, v, C)
            fwd = ll_mamba2_fwd_grouped if q.shape[2] != v.shape[2] else ll_mamba2_fwd
            o = fwd(q, k, v, log_alpha, lam, C, workspace=ws)
            ctx.save_for_backward(q, k, v, log_alpha, lam)
            ctx.ws, ctx.C = ws, C
            return o

        @staticmethod
        def backward(ctx, d_o):
            q, k, v, log_alpha, lam = ctx.saved_tensors
            # the workspace stays with ctx (freed with the graph): a second backward through the
            # same graph (retain_graph=True) reuses it as well
            grads = ll_mamba2_bwd_after_fwd(q, k, v, log_alpha, lam, d_o.contiguous(), ctx.C, ctx.ws)
            return (*grads, None)

    return LogLinearMamba2


_LLM2 = None


def log_linear_mamba2(q, k, v, log_alpha, lam, C):
    """Differentiable log-linear Mamba-2 attention (see LogLinearMamba2): returns O [B, T, H, d_v];
    gradients flow to q, k, v, log_alpha and lam.  lam is required (pass ones for Mamba-2)."""
    global _LLM2
    if _LLM2 is None:
        _LLM2 = _autograd_function()
    return _LLM2.apply(q, k, v, log_alpha, lam, C)
