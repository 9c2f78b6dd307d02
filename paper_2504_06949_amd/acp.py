"""ctypes binding of libacp.so, the HIP library behind include/acp.h.

Argument marshalling only: every step of the computation runs in the library's
kernels.  The functions named like the C entry points take raw device
addresses; the tensor-level helpers below them (boundary, forward, backward,
plan_views) allocate outputs with PyTorch and pass its current HIP stream.
There is no fallback: if the library is missing, every call raises.
"""
from __future__ import annotations

import ctypes
import os
import re

import torch

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libacp.so")
HEADER = os.path.join(os.path.dirname(PKG), "include", "acp.h")

ACP_F32, ACP_BF16 = 0, 1
ACP_OK, ACP_EINVAL, ACP_EUNSUPPORTED, ACP_EWORKSPACE, ACP_EHIP = 0, 1, 2, 3, 4

FLAG_POSITIVE_GATE = 1
FLAG_NONFINITE_GATE = 2
FLAG_INEXACT_CUMSUM = 4
FLAG_NONFINITE_NORM = 8
FLAG_KEPT_KEY_EVICTED = 16


class AcpError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(msg)
        self.status = status


class PlanLayout(ctypes.Structure):
    _fields_ = [(n, ctypes.c_size_t) for n in
                ("c", "bound_u", "delta", "row_start", "col_end", "kept", "flags", "sched_q",
                 "sched_k", "total")]


class DecodeLayout(ctypes.Structure):
    _fields_ = [(n, ctypes.c_size_t) for n in
                ("k_cache", "v_cache", "c", "cum", "delta", "pointer", "flags", "total")]


K_NAMES = ("rownorm", "plan", "fwd", "dsum", "dq", "dkdv", "dlogf", "decode_init", "decode",
           "project", "schedule", "gate")


class KernelTimes(ctypes.Structure):
    _fields_ = [("launches", ctypes.c_int64 * len(K_NAMES)),
                ("ms", ctypes.c_double * len(K_NAMES))]


_lib = None
_i, _d, _p, _sz = ctypes.c_int, ctypes.c_double, ctypes.c_void_p, ctypes.c_size_t
_i64 = ctypes.c_int64

_SIGS = {
    "acp_workspace_size": [_i, _i, _i, _i, _i, ctypes.POINTER(_sz)],
    "acp_plan_offsets": [_i, _i, _i, _i, _i, ctypes.POINTER(PlanLayout)],
    "acp_boundary": [_p, _p, _p, _i, _i, _i, _i, _i, _d, _p, _p, _p, _p, _p, _p, _p, _p, _sz, _p],
    "acp_boundary_qknorm": [_p, _p, _p, _i, _i, _i, _i, _i, _d, _p, _p, _p, _p, _p, _p, _p,
                            _p, _sz, _p],
    "fox_attn_fwd": [_p, _p, _p, _p, _i, _i, _i, _i, _i, _d, _p, _p, _p, _sz, _p],
    "fox_attn_fwd_qknorm": [_p, _p, _p, _p, _p, _p, _i, _i, _i, _i, _i, _d, _p, _p, _p, _sz,
                            _p],
    "fox_attn_bwd": [_p, _p, _p, _p, _p, _i, _i, _i, _i, _i, _p, _p, _p, _p, _p, _sz, _p],
    "fox_attn_fwd_noalloc": [_p, _p, _p, _p, _i, _i, _i, _i, _i, _d, _p, _p, _p],
    "acp_gate_project": [_p, _p, _p, _i, _i, _i, _i, _i, _p, _p, _sz, _p],
    "fox_attn_fwd_gated": [_p, _p, _p, _i, _i, _i, _i, _i, _d, _p, _p, _p, _sz, _p],
    "acp_noalloc_scratch_bytes": [],
    "acp_qk_project": [_p, _p, _p, _i, _i, _i, _i, _i, _i, _p, _p, _p, _sz, _p],
    "fox_attn_fwd_projected": [_p, _p, _p, _p, _i, _i, _i, _i, _i, _d, _p, _p, _p, _sz, _p],
    "acp_decode_state_size": [_i, _i, _i, _i, _i, ctypes.POINTER(_sz)],
    "acp_decode_offsets": [_i, _i, _i, _i, _i, ctypes.POINTER(DecodeLayout)],
    "acp_decode_init": [_p, _p, _p, _p, _p, _i, _i, _i, _i, _i, _i, _d, _i64, _p, _sz, _p],
    "fox_attn_decode": [_p, _p, _p, _p, _i, _i, _i, _i, _i, _i, _i64, _p, _p, _p, _sz, _p],
    "acp_timing_enable": [_i],
    "acp_timing_reset": [],
    "acp_timing_read": [ctypes.POINTER(KernelTimes)],
    "acp_status_string": [_i],
    "acp_last_error": [],
}


def lib() -> ctypes.CDLL:
    """Open libacp.so once; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise AcpError(-1, f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2504_06949_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name, args in _SIGS.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = (ctypes.c_char_p if name in ("acp_status_string", "acp_last_error")
                          else _sz if name == "acp_noalloc_scratch_bytes" else _i)
        _lib = L
    return _lib


def header_functions() -> list:
    """Names of the functions include/acp.h declares."""
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return re.findall(r"^\s*(?:const\s+)?\w+\*?\s+\*?(\w+)\s*\(", text, flags=re.M)


def acp_status_string(status: int) -> str:
    return lib().acp_status_string(status).decode()


def acp_last_error() -> str:
    return lib().acp_last_error().decode()


def _check(status: int):
    if status != ACP_OK:
        raise AcpError(status, f"{acp_status_string(status)}: {acp_last_error()}")


# ---- the C entry points, raw addresses ---------------------------------------

def acp_workspace_size(B, H, L, d, dt) -> int:
    out = _sz(0)
    _check(lib().acp_workspace_size(B, H, L, d, dt, ctypes.byref(out)))
    return out.value


def acp_plan_offsets(B, H, L, d, dt) -> PlanLayout:
    out = PlanLayout()
    _check(lib().acp_plan_offsets(B, H, L, d, dt, ctypes.byref(out)))
    return out


def acp_boundary(Q, K, log_f, dt, B, H, L, d, eps, c, bound_u, delta, row_start, col_end,
                 kept, flags, ws, ws_bytes, stream) -> int:
    return lib().acp_boundary(Q, K, log_f, dt, B, H, L, d, eps, c, bound_u, delta, row_start,
                              col_end, kept, flags, ws, ws_bytes, stream)


def acp_boundary_qknorm(log_f, gamma_q, gamma_k, dt, B, H, L, d, eps, c, bound_u, delta,
                        row_start, col_end, kept, flags, ws, ws_bytes, stream) -> int:
    return lib().acp_boundary_qknorm(log_f, gamma_q, gamma_k, dt, B, H, L, d, eps, c, bound_u,
                                     delta, row_start, col_end, kept, flags, ws, ws_bytes,
                                     stream)


def fox_attn_fwd(Q, K, V, log_f, dt, B, H, L, d, eps, O, lse, ws, ws_bytes, stream) -> int:
    return lib().fox_attn_fwd(Q, K, V, log_f, dt, B, H, L, d, eps, O, lse, ws, ws_bytes, stream)


def fox_attn_fwd_noalloc(Q, K, V, log_f, dt, B, H, L, d, eps, O, lse, stream) -> int:
    return lib().fox_attn_fwd_noalloc(Q, K, V, log_f, dt, B, H, L, d, eps, O, lse, stream)


def acp_gate_project(X, w_f, b_f, B, L, d_model, H, d, log_f, ws, ws_bytes, stream) -> int:
    return lib().acp_gate_project(X, w_f, b_f, B, L, d_model, H, d, log_f, ws, ws_bytes, stream)


def fox_attn_fwd_gated(Q, K, V, dt, B, H, L, d, eps, O, lse, ws, ws_bytes, stream) -> int:
    return lib().fox_attn_fwd_gated(Q, K, V, dt, B, H, L, d, eps, O, lse, ws, ws_bytes, stream)


def acp_noalloc_scratch_bytes() -> int:
    return lib().acp_noalloc_scratch_bytes()


def fox_attn_fwd_qknorm(Q, K, V, log_f, gamma_q, gamma_k, dt, B, H, L, d, eps, O, lse, ws,
                        ws_bytes, stream) -> int:
    return lib().fox_attn_fwd_qknorm(Q, K, V, log_f, gamma_q, gamma_k, dt, B, H, L, d, eps, O,
                                     lse, ws, ws_bytes, stream)


def fox_attn_bwd(Q, K, V, O, dO, dt, B, H, L, d, dQ, dK, dV, dlog_f, ws, ws_bytes,
                 stream) -> int:
    return lib().fox_attn_bwd(Q, K, V, O, dO, dt, B, H, L, d, dQ, dK, dV, dlog_f, ws,
                              ws_bytes, stream)


def acp_qk_project(X, Wq, Wk, dt, B, L, d_model, H, d, Q, K, ws, ws_bytes, stream) -> int:
    return lib().acp_qk_project(X, Wq, Wk, dt, B, L, d_model, H, d, Q, K, ws, ws_bytes, stream)


def fox_attn_fwd_projected(Q, K, V, log_f, dt, B, H, L, d, eps, O, lse, ws, ws_bytes,
                           stream) -> int:
    return lib().fox_attn_fwd_projected(Q, K, V, log_f, dt, B, H, L, d, eps, O, lse, ws,
                                        ws_bytes, stream)


def acp_decode_state_size(B, H, C, d, dt) -> int:
    out = _sz(0)
    _check(lib().acp_decode_state_size(B, H, C, d, dt, ctypes.byref(out)))
    return out.value


def acp_decode_offsets(B, H, C, d, dt) -> DecodeLayout:
    out = DecodeLayout()
    _check(lib().acp_decode_offsets(B, H, C, d, dt, ctypes.byref(out)))
    return out


def acp_decode_init(K, V, log_f, gamma_q, gamma_k, dt, B, H, L0, C, d, eps, L_max, state,
                    state_bytes, stream) -> int:
    return lib().acp_decode_init(K, V, log_f, gamma_q, gamma_k, dt, B, H, L0, C, d, eps, L_max,
                                 state, state_bytes, stream)


def fox_attn_decode(q, k, v, log_f, dt, B, H, t, C, d, L_max, O, lse, state, state_bytes,
                    stream) -> int:
    return lib().fox_attn_decode(q, k, v, log_f, dt, B, H, t, C, d, L_max, O, lse, state,
                                 state_bytes, stream)


def acp_timing_enable(on: bool):
    _check(lib().acp_timing_enable(1 if on else 0))


def acp_timing_reset():
    _check(lib().acp_timing_reset())


def acp_timing_read() -> dict:
    """{kernel name: (launches, summed ms)} since the last reset (waits for the GPU)."""
    t = KernelTimes()
    _check(lib().acp_timing_read(ctypes.byref(t)))
    return {n: (int(t.launches[i]), float(t.ms[i])) for i, n in enumerate(K_NAMES)}


# ---- tensor-level helpers ------------------------------------------------------

def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return ACP_F32
    if t.dtype == torch.bfloat16:
        return ACP_BF16
    raise TypeError(f"unsupported dtype {t.dtype}; use float32 or bfloat16")


def _dev(*ts):
    for t in ts:
        if not t.is_cuda:
            raise ValueError("tensors must live on the GPU")
        if not t.is_contiguous():
            raise ValueError("tensors must be contiguous")
    return ts[0].device


def _stream(device) -> int:
    return torch.cuda.current_stream(device).cuda_stream


def _shape(q: torch.Tensor):
    if q.dim() != 4:
        raise ValueError("Q/K/V must be [B, H, L, d]")
    return tuple(int(s) for s in q.shape)


def workspace(q: torch.Tensor) -> torch.Tensor:
    B, H, L, d = _shape(q)
    n = acp_workspace_size(B, H, L, d, _dt(q))
    return torch.empty(n, dtype=torch.uint8, device=q.device)


def _plan_outputs(B, H, L, dev) -> dict:
    M = L // 64
    return {
        "c": torch.empty((B, H, L), dtype=torch.float32, device=dev),
        "bound_u": torch.empty((B, H), dtype=torch.float64, device=dev),
        "delta": torch.empty((B, H), dtype=torch.float64, device=dev),
        "row_start": torch.empty((B, H, M), dtype=torch.int32, device=dev),
        "col_end": torch.empty((B, H, M), dtype=torch.int32, device=dev),
        "kept": torch.empty((B, H), dtype=torch.int64, device=dev),
        "flags": torch.empty((B, H), dtype=torch.int32, device=dev),
    }


def boundary(q, k, log_f, eps: float, ws: torch.Tensor | None = None) -> dict:
    """Stage 1 of ACP; returns c, bound_u, delta, row_start, col_end, kept, flags."""
    dev = _dev(q, k, log_f)
    B, H, L, d = _shape(q)
    if k.shape != q.shape or k.dtype != q.dtype or tuple(log_f.shape) != (B, H, L) \
            or log_f.dtype != torch.float32:
        raise ValueError("shape/dtype mismatch")
    ws = workspace(q) if ws is None else ws
    out = _plan_outputs(B, H, L, dev)
    _check(acp_boundary(q.data_ptr(), k.data_ptr(), log_f.data_ptr(), _dt(q), B, H, L, d, eps,
                        out["c"].data_ptr(), out["bound_u"].data_ptr(), out["delta"].data_ptr(),
                        out["row_start"].data_ptr(), out["col_end"].data_ptr(),
                        out["kept"].data_ptr(), out["flags"].data_ptr(), ws.data_ptr(),
                        ws.numel(), _stream(dev)))
    return out


def _check_gammas(gamma_q, gamma_k, H: int):
    for name, t in (("gamma_q", gamma_q), ("gamma_k", gamma_k)):
        if tuple(t.shape) != (H,) or t.dtype != torch.float32:
            raise ValueError(name + " must be float32 [H]")


def boundary_qknorm(log_f, gamma_q, gamma_k, d: int, eps: float, dtype=torch.bfloat16,
                    ws: torch.Tensor | None = None) -> dict:
    """Stage 1 with U = gamma_q gamma_k sqrt(d) from QK-norm scales (no pass over Q, K)."""
    dev = _dev(log_f, gamma_q, gamma_k)
    if log_f.dim() != 3 or log_f.dtype != torch.float32:
        raise ValueError("log_f must be float32 [B, H, L]")
    B, H, L = (int(s) for s in log_f.shape)
    _check_gammas(gamma_q, gamma_k, H)
    dt = ACP_F32 if dtype == torch.float32 else ACP_BF16
    if ws is None:
        ws = torch.empty(acp_workspace_size(B, H, L, d, dt), dtype=torch.uint8, device=dev)
    out = _plan_outputs(B, H, L, dev)
    _check(acp_boundary_qknorm(log_f.data_ptr(), gamma_q.data_ptr(), gamma_k.data_ptr(), dt, B, H,
                               L, d, eps, out["c"].data_ptr(), out["bound_u"].data_ptr(),
                               out["delta"].data_ptr(), out["row_start"].data_ptr(),
                               out["col_end"].data_ptr(), out["kept"].data_ptr(),
                               out["flags"].data_ptr(), ws.data_ptr(), ws.numel(), _stream(dev)))
    return out


def forward_qknorm(q, k, v, log_f, gamma_q, gamma_k, eps: float,
                   ws: torch.Tensor | None = None, out=None):
    """forward() with stage 1 bounded by QK-norm scales; returns (O, lse, ws)."""
    dev = _dev(q, k, v, log_f, gamma_q, gamma_k)
    B, H, L, d = _shape(q)
    if k.shape != q.shape or v.shape != q.shape or k.dtype != q.dtype or v.dtype != q.dtype:
        raise ValueError("Q, K, V must share shape and dtype")
    if tuple(log_f.shape) != (B, H, L) or log_f.dtype != torch.float32:
        raise ValueError("log_f must be float32 [B, H, L]")
    _check_gammas(gamma_q, gamma_k, H)
    ws = workspace(q) if ws is None else ws
    if out is None:
        o = torch.empty_like(q)
        lse = torch.empty((B, H, L), dtype=torch.float32, device=dev)
    else:
        o, lse = out
    _check(fox_attn_fwd_qknorm(q.data_ptr(), k.data_ptr(), v.data_ptr(), log_f.data_ptr(),
                               gamma_q.data_ptr(), gamma_k.data_ptr(), _dt(q), B, H, L, d, eps,
                               o.data_ptr(), lse.data_ptr(), ws.data_ptr(), ws.numel(),
                               _stream(dev)))
    return o, lse, ws


def project_qk(x, wq, wk, B: int, H: int, d: int, ws: torch.Tensor | None = None, out=None):
    """Q = X Wq, K = X Wk (X [B*L, d_model], W [d_model, H*d], bf16) written as
    [B, H, L, d]; the workspace receives the row-norm maxima that
    forward_projected() then uses.  Returns (Q, K, ws)."""
    dev = _dev(x, wq, wk)
    if x.dim() != 2 or wq.dim() != 2 or wq.shape != wk.shape:
        raise ValueError("X must be [B*L, d_model] and Wq, Wk [d_model, H*d]")
    for t in (x, wq, wk):
        if t.dtype != torch.bfloat16:
            raise TypeError("the projection takes bfloat16 tensors")
    M, Dm = (int(s) for s in x.shape)
    if M % B != 0 or tuple(wq.shape) != (Dm, H * d):
        raise ValueError("shape mismatch")
    L = M // B
    if ws is None:
        ws = torch.empty(acp_workspace_size(B, H, L, d, ACP_BF16), dtype=torch.uint8, device=dev)
    if out is None:
        q = torch.empty((B, H, L, d), dtype=torch.bfloat16, device=dev)
        k = torch.empty_like(q)
    else:
        q, k = out
    _check(acp_qk_project(x.data_ptr(), wq.data_ptr(), wk.data_ptr(), ACP_BF16, B, L, Dm, H, d,
                          q.data_ptr(), k.data_ptr(), ws.data_ptr(), ws.numel(), _stream(dev)))
    return q, k, ws


def forward_projected(q, k, v, log_f, eps: float, ws: torch.Tensor, out=None):
    """forward() for Q, K made by project_qk() into `ws`: stage 1 reuses the
    norm maxima of the projection's epilogue.  Returns (O, lse, ws)."""
    dev = _dev(q, k, v, log_f)
    B, H, L, d = _shape(q)
    if k.shape != q.shape or v.shape != q.shape or k.dtype != q.dtype or v.dtype != q.dtype:
        raise ValueError("Q, K, V must share shape and dtype")
    if tuple(log_f.shape) != (B, H, L) or log_f.dtype != torch.float32:
        raise ValueError("log_f must be float32 [B, H, L]")
    if out is None:
        o = torch.empty_like(q)
        lse = torch.empty((B, H, L), dtype=torch.float32, device=dev)
    else:
        o, lse = out
    _check(fox_attn_fwd_projected(q.data_ptr(), k.data_ptr(), v.data_ptr(), log_f.data_ptr(),
                                  _dt(q), B, H, L, d, eps, o.data_ptr(), lse.data_ptr(),
                                  ws.data_ptr(), ws.numel(), _stream(dev)))
    return o, lse, ws


def forward(q, k, v, log_f, eps: float, ws: torch.Tensor | None = None, out=None):
    """Returns (O, lse, ws); ws carries the plan and state the backward needs."""
    dev = _dev(q, k, v, log_f)
    B, H, L, d = _shape(q)
    if k.shape != q.shape or v.shape != q.shape or k.dtype != q.dtype or v.dtype != q.dtype:
        raise ValueError("Q, K, V must share shape and dtype")
    if tuple(log_f.shape) != (B, H, L) or log_f.dtype != torch.float32:
        raise ValueError("log_f must be float32 [B, H, L]")
    ws = workspace(q) if ws is None else ws
    if out is None:
        o = torch.empty_like(q)
        lse = torch.empty((B, H, L), dtype=torch.float32, device=dev)
    else:
        o, lse = out
    _check(fox_attn_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), log_f.data_ptr(), _dt(q),
                        B, H, L, d, eps, o.data_ptr(), lse.data_ptr(), ws.data_ptr(), ws.numel(),
                        _stream(dev)))
    return o, lse, ws


def gate_project(x, w_f, b_f, B: int, H: int, d: int, ws: torch.Tensor | None = None,
                 log_f: torch.Tensor | None = None, dtype=torch.bfloat16):
    """log f [B, H, L] of the gate projection of X [B*L, d_model] (bf16) with w_f
    [d_model, H] (bf16) and b_f [H] (float32); the workspace receives c and the
    gate checks that forward_gated() then uses.  Returns (log_f, ws)."""
    dev = _dev(x, w_f, b_f)
    if x.dim() != 2 or w_f.dim() != 2 or w_f.shape[0] != x.shape[1] or w_f.shape[1] != H:
        raise ValueError("X must be [B*L, d_model] and w_f [d_model, H]")
    if x.dtype != torch.bfloat16 or w_f.dtype != torch.bfloat16 or b_f.dtype != torch.float32:
        raise TypeError("X and w_f must be bfloat16, b_f float32")
    if tuple(b_f.shape) != (H,):
        raise ValueError("b_f must be [H]")
    M, Dm = (int(t) for t in x.shape)
    if M % B != 0:
        raise ValueError("shape mismatch")
    L = M // B
    if ws is None:
        ws = torch.empty(acp_workspace_size(B, H, L, d, _dt_of(dtype)), dtype=torch.uint8,
                         device=dev)
    if log_f is None:
        log_f = torch.empty((B, H, L), dtype=torch.float32, device=dev)
    _check(acp_gate_project(x.data_ptr(), w_f.data_ptr(), b_f.data_ptr(), B, L, Dm, H, d,
                            log_f.data_ptr(), ws.data_ptr(), ws.numel(), _stream(dev)))
    return log_f, ws


def forward_gated(q, k, v, eps: float, ws: torch.Tensor, out=None):
    """forward() for the gates gate_project() left in `ws`: stage 1 reads c from
    there instead of scanning log f.  Returns (O, lse, ws)."""
    dev = _dev(q, k, v)
    B, H, L, d = _shape(q)
    if k.shape != q.shape or v.shape != q.shape or k.dtype != q.dtype or v.dtype != q.dtype:
        raise ValueError("Q, K, V must share shape and dtype")
    if out is None:
        o = torch.empty_like(q)
        lse = torch.empty((B, H, L), dtype=torch.float32, device=dev)
    else:
        o, lse = out
    _check(fox_attn_fwd_gated(q.data_ptr(), k.data_ptr(), v.data_ptr(), _dt(q), B, H, L, d, eps,
                              o.data_ptr(), lse.data_ptr(), ws.data_ptr(), ws.numel(),
                              _stream(dev)))
    return o, lse, ws


def _dt_of(dtype) -> int:
    return ACP_F32 if dtype == torch.float32 else ACP_BF16


def backward(q, k, v, o, do, ws: torch.Tensor, out=None):
    """Returns (dQ, dK, dV, dlog_f) for the forward that produced `o` and filled `ws`."""
    dev = _dev(q, k, v, o, do)
    B, H, L, d = _shape(q)
    for name, t in (("O", o), ("dO", do)):
        if t.shape != q.shape or t.dtype != q.dtype:
            raise ValueError(name + " must match Q")
    if out is None:
        dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
        dlf = torch.empty((B, H, L), dtype=torch.float32, device=dev)
    else:
        dq, dk, dv, dlf = out
    _check(fox_attn_bwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), do.data_ptr(), _dt(q),
                        B, H, L, d, dq.data_ptr(), dk.data_ptr(), dv.data_ptr(), dlf.data_ptr(),
                        ws.data_ptr(), ws.numel(), _stream(dev)))
    return dq, dk, dv, dlf


class _FoxAttention(torch.autograd.Function):
    """Autograd node over forward() and backward(): the forward's workspace (its
    plan, and the state the backward reads) is saved with Q, K, V and O."""

    @staticmethod
    def forward(ctx, q, k, v, log_f, eps):
        q, k, v, log_f = (t.contiguous() for t in (q, k, v, log_f))
        o, lse, ws = forward(q, k, v, log_f, eps)
        ctx.save_for_backward(q, k, v, o, ws)
        ctx.mark_non_differentiable(lse)
        return o, lse

    @staticmethod
    def backward(ctx, do, _dlse):
        q, k, v, o, ws = ctx.saved_tensors
        dq, dk, dv, dlf = backward(q, k, v, o, do.to(q.dtype).contiguous(), ws)
        return dq, dk, dv, dlf, None


def fox_attention(q, k, v, log_f, eps: float):
    """Differentiable FoX attention with ACP: (O, lse) of forward(), with gradients
    for Q, K, V and log f from backward() when autograd asks for them.  lse carries
    no gradient.  Inputs need not be contiguous (they are copied if not)."""
    return _FoxAttention.apply(q, k, v, log_f, eps)


def plan_views(ws: torch.Tensor, B: int, H: int, L: int, d: int, dtype) -> dict:
    """Views into a workspace of the plan that fox_attn_fwd wrote."""
    dt = ACP_F32 if dtype == torch.float32 else ACP_BF16
    lay = acp_plan_offsets(B, H, L, d, dt)
    M = L // 64
    nb = (L + 127) // 128

    def view(off, n, t):
        nbytes = n * torch.empty((), dtype=t).element_size()
        return ws[off:off + nbytes].view(t)

    return {
        "c": view(lay.c, B * H * L, torch.float32).view(B, H, L),
        "bound_u": view(lay.bound_u, B * H, torch.float64).view(B, H),
        "delta": view(lay.delta, B * H, torch.float64).view(B, H),
        "row_start": view(lay.row_start, B * H * M, torch.int32).view(B, H, M),
        "col_end": view(lay.col_end, B * H * M, torch.int32).view(B, H, M),
        "kept": view(lay.kept, B * H, torch.int64).view(B, H),
        "flags": view(lay.flags, B * H, torch.int32).view(B, H),
        "sched_q": view(lay.sched_q, B * H * nb, torch.int32),
        "sched_k": view(lay.sched_k, B * H * nb, torch.int32),
    }


class Decoder:
    """Decoding state of acp_decode_init / fox_attn_decode for B x H heads: a ring
    cache of C positions per head plus the per-head pointer, delta and flags, in
    one device buffer.  Tracks the next position t on the host."""

    def __init__(self, B: int, H: int, C: int, d: int, dtype=torch.bfloat16, device="cuda"):
        self.B, self.H, self.C, self.d, self.dtype = B, H, C, d, dtype
        self.dt = ACP_F32 if dtype == torch.float32 else ACP_BF16
        n = acp_decode_state_size(B, H, C, d, self.dt)
        self.state = torch.empty(n, dtype=torch.uint8, device=device)
        self.t = None
        self.L_max = None

    def init(self, k, v, log_f, gamma_q, gamma_k, eps: float, L_max: int):
        """Build the state from a prompt: k, v [B, H, L0, d], log_f [B, H, L0]."""
        dev = _dev(k, v, log_f, gamma_q, gamma_k, self.state)
        B, H, L0, d = _shape(k)
        if (B, H, d) != (self.B, self.H, self.d) or v.shape != k.shape:
            raise ValueError("prompt K/V shape does not match the decoder")
        if k.dtype != self.dtype or v.dtype != self.dtype:
            raise ValueError("prompt K/V dtype does not match the decoder")
        if tuple(log_f.shape) != (B, H, L0) or log_f.dtype != torch.float32:
            raise ValueError("log_f must be float32 [B, H, L0]")
        _check_gammas(gamma_q, gamma_k, H)
        _check(acp_decode_init(k.data_ptr(), v.data_ptr(), log_f.data_ptr(), gamma_q.data_ptr(),
                               gamma_k.data_ptr(), self.dt, B, H, L0, self.C, d, eps, L_max,
                               self.state.data_ptr(), self.state.numel(), _stream(dev)))
        self.t, self.L_max = L0, L_max
        return self

    def step(self, q, k, v, log_f, out=None):
        """Append token t (k, v [B, H, d], log_f [B, H]) and attend with q [B, H, d];
        returns (O [B, H, d], lse [B, H])."""
        if self.t is None:
            raise RuntimeError("call init() first")
        dev = _dev(q, k, v, log_f, self.state)
        for name, x in (("q", q), ("k", k), ("v", v)):
            if tuple(x.shape) != (self.B, self.H, self.d) or x.dtype != self.dtype:
                raise ValueError(name + " must be [B, H, d] of the decoder's dtype")
        if tuple(log_f.shape) != (self.B, self.H) or log_f.dtype != torch.float32:
            raise ValueError("log_f must be float32 [B, H]")
        if out is None:
            o = torch.empty_like(q)
            lse = torch.empty((self.B, self.H), dtype=torch.float32, device=dev)
        else:
            o, lse = out
        _check(fox_attn_decode(q.data_ptr(), k.data_ptr(), v.data_ptr(), log_f.data_ptr(),
                               self.dt, self.B, self.H, self.t, self.C, self.d, self.L_max,
                               o.data_ptr(), lse.data_ptr(), self.state.data_ptr(),
                               self.state.numel(), _stream(dev)))
        self.t += 1
        return o, lse

    def current_pointer(self) -> torch.Tensor:
        """[B, H] pointer of the latest position (a view into the state)."""
        return self.views()["pointer"][(self.t - 1) % 2]

    def current_cum(self) -> torch.Tensor:
        """[B, H, 2] running sum after the latest position as a double-double
        pair (hi, lo): the value is hi + lo exactly (a view)."""
        return self.views()["cum"][(self.t - 1) % 2]

    def views(self) -> dict:
        """Views of the state: k_cache, v_cache [B,H,C,d], c [B,H,C], delta and
        flags [B,H]; pointer [2,B,H] and cum [2,B,H,2] (pairs hi, lo), the values
        after position p being copy p % 2 (current_pointer() and current_cum() pick
        the latest)."""
        lay = acp_decode_offsets(self.B, self.H, self.C, self.d, self.dt)
        B, H, C, d = self.B, self.H, self.C, self.d

        def view(off, n, t):
            nbytes = n * torch.empty((), dtype=t).element_size()
            return self.state[off:off + nbytes].view(t)

        return {
            "k_cache": view(lay.k_cache, B * H * C * d, self.dtype).view(B, H, C, d),
            "v_cache": view(lay.v_cache, B * H * C * d, self.dtype).view(B, H, C, d),
            "c": view(lay.c, B * H * C, torch.float32).view(B, H, C),
            "cum": view(lay.cum, 4 * B * H, torch.float64).view(2, B, H, 2),
            "delta": view(lay.delta, B * H, torch.float64).view(B, H),
            "pointer": view(lay.pointer, 2 * B * H, torch.int32).view(2, B, H),
            "flags": view(lay.flags, B * H, torch.int32).view(B, H),
        }
