"""The C ABI on the CPU: the library loads, exports what include/acp.h declares,
and rejects bad arguments on the host before launching anything."""
import ctypes
import math

import pytest

from paper_2504_06949_amd import acp
from tests._helpers import ensure_built


@pytest.fixture(scope="module", autouse=True)
def _lib():
    ensure_built()


def test_every_declared_symbol_is_exported():
    names = acp.header_functions()
    assert set(names) == {"acp_workspace_size", "acp_plan_offsets", "acp_boundary",
                          "acp_boundary_qknorm", "fox_attn_fwd", "fox_attn_fwd_qknorm",
                          "fox_attn_bwd", "acp_qk_project", "fox_attn_fwd_projected",
                          "acp_decode_state_size", "acp_decode_offsets",
                          "acp_decode_init", "fox_attn_decode",
                          "acp_timing_enable", "acp_timing_reset",
                          "acp_timing_read", "acp_status_string", "acp_last_error",
                          "acp_noalloc_scratch_bytes", "fox_attn_fwd_noalloc",
                          "acp_gate_project", "fox_attn_fwd_gated"}
    lib = ctypes.CDLL(acp.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings():
    assert acp.acp_status_string(acp.ACP_OK) == "ok"
    for s in (acp.ACP_EINVAL, acp.ACP_EUNSUPPORTED, acp.ACP_EWORKSPACE, acp.ACP_EHIP):
        assert acp.acp_status_string(s) not in ("ok", "unknown status")
    assert acp.acp_status_string(99) == "unknown status"


def test_workspace_size_and_layout():
    n = acp.acp_workspace_size(8, 12, 4096, 64, acp.ACP_BF16)
    lay = acp.acp_plan_offsets(8, 12, 4096, 64, acp.ACP_BF16)
    assert lay.total == n
    offs = [lay.c, lay.bound_u, lay.delta, lay.row_start, lay.col_end, lay.kept,
            lay.flags, lay.sched_q, lay.sched_k]
    assert all(o % 256 == 0 for o in offs)
    assert offs == sorted(offs) and len(set(offs)) == len(offs)
    BHL = 8 * 12 * 4096
    assert lay.bound_u - lay.c >= 4 * BHL
    # the two workgroup schedules: one int32 per (head, 128-row block)
    assert lay.sched_k - lay.sched_q >= 4 * 8 * 12 * 32
    assert lay.total - lay.sched_k >= 4 * 8 * 12 * 32
    # five float32 rows per position (c, L_i, Delta', row and column sums of dS)
    # dominate, and nothing scales with the head dim
    assert n >= 5 * 4 * BHL
    assert acp.acp_workspace_size(8, 12, 4096, 128, acp.ACP_BF16) == n


@pytest.mark.parametrize("args,status", [
    ((0, 1, 64, 64), acp.ACP_EINVAL),
    ((1, -2, 64, 64), acp.ACP_EINVAL),
    ((1, 1, 64, 96), acp.ACP_EUNSUPPORTED),
    ((1, 1, 100, 64), acp.ACP_EUNSUPPORTED),
    ((1, 1, 64 * 2049, 64), acp.ACP_EUNSUPPORTED),
    ((256, 256, 64, 64), acp.ACP_EUNSUPPORTED),
])
def test_shape_validation(args, status):
    with pytest.raises(acp.AcpError) as e:
        acp.acp_workspace_size(*args, acp.ACP_BF16)
    assert e.value.status == status


def _fwd(**kw):
    a = dict(Q=16, K=16, V=16, log_f=16, dt=acp.ACP_BF16, B=1, H=1, L=64, d=64, eps=1e-4,
             O=16, lse=16, ws=16, ws_bytes=1 << 40, stream=None)
    a.update(kw)
    return acp.fox_attn_fwd(*a.values())


@pytest.mark.parametrize("kw,status", [
    (dict(Q=0), acp.ACP_EINVAL),
    (dict(V=8), acp.ACP_EINVAL),              # misaligned
    (dict(lse=0), acp.ACP_EINVAL),
    (dict(eps=-1e-3), acp.ACP_EINVAL),
    (dict(eps=1.0), acp.ACP_EINVAL),
    (dict(eps=math.nan), acp.ACP_EINVAL),
    (dict(eps=math.inf), acp.ACP_EINVAL),
    (dict(dt=7), acp.ACP_EINVAL),
    (dict(d=32), acp.ACP_EUNSUPPORTED),
    (dict(L=96), acp.ACP_EUNSUPPORTED),
    (dict(ws_bytes=1000), acp.ACP_EWORKSPACE),
    (dict(ws=0), acp.ACP_EINVAL),
])
def test_forward_rejects_before_launch(kw, status):
    assert _fwd(**kw) == status
    assert acp.acp_last_error() != ""


def test_qknorm_entries_reject_before_launch():
    st = acp.acp_boundary_qknorm(16, 0, 16, acp.ACP_BF16, 1, 1, 64, 64, 0.5, 16, 16, 16, 16, 16,
                                 16, 16, 16, 1 << 40, None)
    assert st == acp.ACP_EINVAL and "gamma_q" in acp.acp_last_error()
    st = acp.acp_boundary_qknorm(16, 16, 16, acp.ACP_BF16, 1, 1, 64, 64, 1.5, 16, 16, 16, 16, 16,
                                 16, 16, 16, 1 << 40, None)
    assert st == acp.ACP_EINVAL and "eps" in acp.acp_last_error()
    st = acp.fox_attn_fwd_qknorm(16, 16, 16, 16, 16, 8, acp.ACP_BF16, 1, 1, 64, 64, 0.5, 16, 16,
                                 16, 1 << 40, None)
    assert st == acp.ACP_EINVAL and "gamma_k" in acp.acp_last_error()
    st = acp.fox_attn_fwd_qknorm(16, 16, 16, 16, 16, 16, acp.ACP_BF16, 1, 1, 64, 64, 0.5, 16, 16,
                                 16, 8, None)
    assert st == acp.ACP_EWORKSPACE


def test_backward_and_boundary_reject_before_launch():
    st = acp.fox_attn_bwd(16, 16, 16, 16, 0, acp.ACP_BF16, 1, 1, 64, 64, 16, 16, 16, 16, 16,
                          1 << 40, None)
    assert st == acp.ACP_EINVAL and "dO" in acp.acp_last_error()
    st = acp.fox_attn_bwd(16, 16, 16, 0, 16, acp.ACP_BF16, 1, 1, 64, 64, 16, 16, 16, 16, 16,
                          1 << 40, None)
    assert st == acp.ACP_EINVAL and "O" in acp.acp_last_error()
    st = acp.fox_attn_bwd(16, 16, 16, 16, 16, acp.ACP_BF16, 1, 1, 64, 64, 16, 16, 16, 16, 16, 8,
                          None)
    assert st == acp.ACP_EWORKSPACE
    st = acp.acp_boundary(16, 16, 16, acp.ACP_F32, 1, 1, 64, 64, 0.5, 16, 16, 16, 16, 16, 0, 16,
                          16, 1 << 40, None)
    assert st == acp.ACP_EINVAL and "kept" in acp.acp_last_error()
    st = acp.acp_boundary(16, 16, 16, acp.ACP_F32, 1, 1, 64, 64, 1.5, 16, 16, 16, 16, 16, 16,
                          16, 16, 1 << 40, None)
    assert st == acp.ACP_EINVAL


def test_tensor_helpers_refuse_cpu_tensors():
    import torch
    q = torch.zeros(1, 1, 64, 64)
    with pytest.raises(ValueError):
        acp.forward(q, q, q, torch.zeros(1, 1, 64), 1e-4)
    with pytest.raises(ValueError):
        acp.fox_attention(q.requires_grad_(True), q, q, torch.zeros(1, 1, 64), 1e-4)


def test_timing_state_without_launches():
    acp.acp_timing_reset()
    t = acp.acp_timing_read()
    assert set(t) == set(acp.K_NAMES) and all(v == (0, 0.0) for v in t.values())
    acp.acp_timing_enable(True)
    acp.acp_timing_enable(False)


def test_decode_state_layout():
    n = acp.acp_decode_state_size(2, 3, 256, 64, acp.ACP_BF16)
    lay = acp.acp_decode_offsets(2, 3, 256, 64, acp.ACP_BF16)
    offs = [getattr(lay, f) for f, _ in acp.DecodeLayout._fields_]
    assert all(o % 256 == 0 for o in offs) and offs == sorted(offs) and lay.total == n
    assert lay.v_cache - lay.k_cache >= 2 * 3 * 256 * 64 * 2
    assert acp.acp_decode_state_size(2, 3, 256, 64, acp.ACP_F32) > n
    with pytest.raises(acp.AcpError):
        acp.acp_decode_state_size(2, 3, 100, 64, acp.ACP_BF16)   # C not a multiple of 64


def test_decode_entries_reject_before_launch():
    big = 1 << 40
    # init: K, V, log_f, gamma_q, gamma_k, dt, B, H, L0, C, d, eps, L_max, state, bytes, stream
    st = acp.acp_decode_init(16, 16, 16, 16, 16, acp.ACP_BF16, 1, 1, 100, 128, 64, 0.5, 64, 16,
                             big, None)
    assert st == acp.ACP_EINVAL and "L_max" in acp.acp_last_error()        # L0 > L_max
    st = acp.acp_decode_init(16, 16, 16, 0, 16, acp.ACP_BF16, 1, 1, 100, 128, 64, 0.5, 1000, 16,
                             big, None)
    assert st == acp.ACP_EINVAL and "gamma_q" in acp.acp_last_error()
    st = acp.acp_decode_init(16, 16, 16, 16, 16, acp.ACP_BF16, 1, 1, 100, 96, 64, 0.5, 1000, 16,
                             big, None)
    assert st == acp.ACP_EUNSUPPORTED
    st = acp.acp_decode_init(16, 16, 16, 16, 16, acp.ACP_BF16, 1, 1, 100, 128, 64, 1.0, 1000, 16,
                             big, None)
    assert st == acp.ACP_EINVAL and "eps" in acp.acp_last_error()
    st = acp.acp_decode_init(16, 16, 16, 16, 16, acp.ACP_BF16, 1, 1, 100, 128, 64, 0.5, 1000, 16,
                             8, None)
    assert st == acp.ACP_EWORKSPACE
    # step: q, k, v, log_f, dt, B, H, t, C, d, L_max, O, lse, state, bytes, stream
    st = acp.fox_attn_decode(16, 16, 16, 16, acp.ACP_BF16, 1, 1, 1000, 128, 64, 1000, 16, 16, 16,
                             big, None)
    assert st == acp.ACP_EINVAL and "t=1000" in acp.acp_last_error()       # t >= L_max
    st = acp.fox_attn_decode(16, 16, 16, 16, acp.ACP_BF16, 1, 1, 0, 128, 64, 1000, 16, 16, 16,
                             big, None)
    assert st == acp.ACP_EINVAL
    st = acp.fox_attn_decode(16, 16, 16, 16, acp.ACP_BF16, 1, 1, 10, 128, 64, 1000, 16, 0, 16,
                             big, None)
    assert st == acp.ACP_EINVAL and "lse" in acp.acp_last_error()
    st = acp.fox_attn_decode(16, 16, 24, 16, acp.ACP_BF16, 1, 1, 10, 128, 64, 1000, 16, 16, 16,
                             big, None)
    assert st == acp.ACP_EINVAL and "aligned" in acp.acp_last_error()
    st = acp.fox_attn_decode(16, 16, 16, 16, acp.ACP_BF16, 1, 1, 10, 128, 64, 1000, 16, 16, 16,
                             8, None)
    assert st == acp.ACP_EWORKSPACE


def test_projection_rejects_before_launch():
    big = 1 << 40
    # X, Wq, Wk, dt, B, L, d_model, H, d, Q, K, ws, bytes, stream
    st = acp.acp_qk_project(16, 16, 16, acp.ACP_F32, 1, 128, 64, 2, 64, 16, 16, 16, big, None)
    assert st == acp.ACP_EUNSUPPORTED and "bfloat16" in acp.acp_last_error()
    st = acp.acp_qk_project(16, 16, 16, acp.ACP_BF16, 1, 192, 64, 2, 64, 16, 16, 16, big, None)
    assert st == acp.ACP_EUNSUPPORTED and "128" in acp.acp_last_error()      # L % 128
    st = acp.acp_qk_project(16, 16, 16, acp.ACP_BF16, 1, 128, 96, 2, 64, 16, 16, 16, big, None)
    assert st == acp.ACP_EUNSUPPORTED and "d_model" in acp.acp_last_error()
    st = acp.acp_qk_project(16, 16, 16, acp.ACP_BF16, 1, 128, 64, 1, 64, 16, 16, 16, big, None)
    assert st == acp.ACP_EUNSUPPORTED and "H*d" in acp.acp_last_error()
    st = acp.acp_qk_project(16, 0, 16, acp.ACP_BF16, 1, 128, 64, 2, 64, 16, 16, 16, big, None)
    assert st == acp.ACP_EINVAL and "Wq" in acp.acp_last_error()
    st = acp.acp_qk_project(16, 16, 16, acp.ACP_BF16, 1, 128, 64, 2, 64, 16, 16, 16, 8, None)
    assert st == acp.ACP_EWORKSPACE
    st = acp.fox_attn_fwd_projected(16, 16, 16, 16, acp.ACP_BF16, 1, 1, 64, 64, 0.5, 16, 16, 16,
                                    8, None)
    assert st == acp.ACP_EWORKSPACE


def test_noalloc_forward_rejects_shapes_beyond_its_fixed_scratch():
    """fox_attn_fwd_noalloc checks the shapes against its fixed scratch array
    (32 MiB) before it touches the GPU or any pointer."""
    size = acp.acp_noalloc_scratch_bytes()
    assert size == 32 << 20
    B, H, L, d = 1, 64, 32768, 64
    assert acp.acp_workspace_size(B, H, L, d, acp.ACP_BF16) > size
    st = acp.fox_attn_fwd_noalloc(16, 16, 16, 16, acp.ACP_BF16, B, H, L, d, 1e-4, 16, 16, None)
    assert st == acp.ACP_EWORKSPACE
    assert "fox_attn_fwd_noalloc" in acp.acp_last_error()
    st = acp.fox_attn_fwd_noalloc(16, 16, 16, 16, acp.ACP_BF16, 1, 1, 100, 64, 1e-4, 16, 16, None)
    assert st == acp.ACP_EUNSUPPORTED


@pytest.mark.parametrize("kw,status", [
    (dict(X=0), acp.ACP_EINVAL),
    (dict(w_f=8), acp.ACP_EINVAL),                 # misaligned
    (dict(b_f=0), acp.ACP_EINVAL),
    (dict(d_model=96), acp.ACP_EUNSUPPORTED),
    (dict(H=65), acp.ACP_EUNSUPPORTED),
    (dict(d_model=8200), acp.ACP_EUNSUPPORTED),
    (dict(L=100), acp.ACP_EUNSUPPORTED),
    (dict(ws_bytes=16), acp.ACP_EWORKSPACE),
    (dict(d_model=4096), acp.ACP_EUNSUPPORTED),     # weight copy beyond B*H*L*4 bytes
])
def test_gate_project_rejects_bad_arguments(kw, status):
    a = dict(X=16, w_f=16, b_f=16, B=1, L=64, d_model=64, H=2, d=64, log_f=16, ws=16,
             ws_bytes=1 << 40, stream=None)
    a.update(kw)
    assert acp.acp_gate_project(*a.values()) == status
    if kw.get("d_model") == 4096:
        assert "too large for these shapes" in acp.acp_last_error()
