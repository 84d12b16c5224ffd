"""libcas: multi-cartridge prefix attention on MI355X (gfx950).

A thin binding over the C ABI in include/cas.h. Every step of the attention
runs in the HIP library; this module only marshals torch tensors (device
memory and streams) into the C structures. There is no fallback: if libcas.so
is missing, or a call fails, an exception is raised.
"""
from __future__ import annotations

import ctypes
import dataclasses
from typing import List, Optional, Sequence, Tuple

from . import _lib
from ._lib import load  # noqa: F401

__all__ = ["Segment", "Problem", "CasError", "load", "prefix_attn_fwd", "prefix_attn_bwd",
           "workspace_size", "plan_info", "set_tuning", "get_tuning", "cartridge_stage",
           "timing_enable", "timing_reset", "timing_read"]


class CasError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{status_string(status)}: {message}")
        self.status = status
        self.message = message


def status_string(s: int) -> str:
    return load().cas_status_string(s).decode()


def _check(status: int) -> None:
    if status != _lib.CAS_OK:
        raise CasError(status, load().cas_last_error_message().decode())


@dataclasses.dataclass
class Segment:
    """One cartridge block seen by one batch row: k and v are [len, Hkv, d]
    views (any token / head strides, unit channel stride); dk, dv receive the
    gradient (same strides) or are None."""
    k: object
    v: object
    dk: Optional[object] = None
    dv: Optional[object] = None


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.bfloat16:
        return _lib.CAS_DTYPE_BF16
    if t.dtype == torch.float32:
        return _lib.CAS_DTYPE_FP32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


class Problem:
    """Host-side segment table (cas_problem_t) built from torch tensors.

    With ``q_offsets`` (batch+1 token offsets) the rows are packed samples of
    different lengths on one token axis and ``q_len`` must be 0."""

    def __init__(self, dtype_code: int, batch: int, q_len: int, num_kv_heads: int,
                 group_size: int, head_dim: int, softmax_scale: float,
                 rows: Sequence[Sequence[Segment]], q_offsets: Optional[Sequence[int]] = None):
        if len(rows) != batch:
            raise ValueError("rows must have one segment list per batch row")
        self._qoffs = None
        if q_offsets is not None:
            if len(q_offsets) != batch + 1:
                raise ValueError("q_offsets must have batch+1 entries")
            self._qoffs = (ctypes.c_int32 * (batch + 1))(*[int(x) for x in q_offsets])
        n = sum(len(r) for r in rows)
        self._segs = (_lib.Segment * max(n, 1))()
        self._offs = (ctypes.c_int32 * (batch + 1))()
        i = 0
        for b, row in enumerate(rows):
            self._offs[b] = i
            for s in row:
                k, v = s.k, s.v
                if k.dim() != 3 or k.shape != v.shape or k.stride() != v.stride():
                    raise ValueError("segment k and v must be [len, Hkv, d] with equal strides")
                for gt in (s.dk, s.dv):
                    if gt is not None and (gt.shape != k.shape or gt.stride() != k.stride()):
                        raise ValueError("segment dk/dv must match k's shape and strides")
                if k.shape[0] > 0 and k.stride(2) != 1:
                    raise ValueError("segment channel stride must be 1")
                e = self._segs[i]
                e.k, e.v, e.dk, e.dv = _ptr(k), _ptr(v), _ptr(s.dk), _ptr(s.dv)
                e.len = int(k.shape[0])
                e.stride_tok = int(k.stride(0))
                e.stride_head = int(k.stride(1))
                i += 1
        self._offs[batch] = i
        qo = (ctypes.cast(self._qoffs, ctypes.POINTER(ctypes.c_int32)) if self._qoffs is not None
              else ctypes.POINTER(ctypes.c_int32)())
        self.c = _lib.Problem(dtype_code, batch, q_len, num_kv_heads, group_size, head_dim,
                              float(softmax_scale),
                              ctypes.cast(self._segs, ctypes.POINTER(_lib.Segment)),
                              ctypes.cast(self._offs, ctypes.POINTER(ctypes.c_int32)), qo)

    @classmethod
    def from_tensors(cls, q, rows, num_kv_heads: int, group_size: int, softmax_scale: float,
                     q_offsets: Optional[Sequence[int]] = None):
        if q_offsets is None:
            B, Sq, Hq, D = q.shape
        else:
            T, Hq, D = q.shape
            B, Sq = len(q_offsets) - 1, 0
            if int(q_offsets[-1]) != T:
                raise ValueError("q_offsets[-1] must equal the packed token count")
        if Hq != num_kv_heads * group_size:
            raise ValueError("q heads must equal num_kv_heads * group_size")
        return cls(_dtype_code(q), B, Sq, num_kv_heads, group_size, D, softmax_scale, rows, q_offsets)


def workspace_size(problem: Problem, backward: bool) -> int:
    n = ctypes.c_size_t(0)
    _check(load().cas_prefix_attn_workspace_size(ctypes.byref(problem.c), int(backward), ctypes.byref(n)))
    return n.value


def plan_info(problem: Problem) -> dict:
    info = _lib.PlanInfo()
    _check(load().cas_plan_info(ctypes.byref(problem.c), ctypes.byref(info)))
    return {f: getattr(info, f) for f, _ in _lib.PlanInfo._fields_}


def set_tuning(fwd_splits: int = 0, dq_splits: int = 0) -> None:
    t = _lib.Tuning(fwd_splits, dq_splits)
    _check(load().cas_set_tuning(ctypes.byref(t)))


def get_tuning() -> dict:
    t = _lib.Tuning()
    _check(load().cas_get_tuning(ctypes.byref(t)))
    return {"fwd_splits": t.fwd_splits, "dq_splits": t.dq_splits}


def _stream_handle(device, stream) -> int:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream(device)
    return s.cuda_stream


def _workspace(nbytes: int, device):
    import torch
    return torch.empty(max(nbytes, 1), dtype=torch.uint8, device=device)


def prefix_attn_fwd(q, k_self, v_self, rows: Sequence[Sequence[Segment]], num_kv_heads: int,
                    group_size: int, softmax_scale: float, o=None, lse=None, need_lse: bool = True,
                    stream=None, workspace=None,
                    q_offsets: Optional[Sequence[int]] = None) -> Tuple[object, Optional[object]]:
    """O [B, Sq, Hq, d] and LSE [B, Hq, Sq] (fp32) over [row's segments || causal self].

    With ``q_offsets`` the rows are packed samples: q, k_self and v_self are
    [T, H, d], O is [T, Hq, d] and LSE is [Hq, T]."""
    import torch
    prob = Problem.from_tensors(q, rows, num_kv_heads, group_size, softmax_scale, q_offsets)
    if o is None:
        o = torch.empty_like(q)
    if lse is None and need_lse:
        if q_offsets is None:
            B, Sq, Hq, _ = q.shape
            lse = torch.empty((B, Hq, Sq), dtype=torch.float32, device=q.device)
        else:
            T, Hq, _ = q.shape
            lse = torch.empty((Hq, T), dtype=torch.float32, device=q.device)
    ws_n = workspace_size(prob, False)
    ws = workspace if workspace is not None and workspace.numel() >= ws_n else _workspace(ws_n, q.device)
    _check(load().cas_prefix_attn_fwd(ctypes.byref(prob.c), q.data_ptr(), k_self.data_ptr(),
                                      v_self.data_ptr(), o.data_ptr(), _ptr(lse), ws.data_ptr(),
                                      ws.numel(), _stream_handle(q.device, stream)))
    return o, lse


def prefix_attn_bwd(q, k_self, v_self, rows: Sequence[Sequence[Segment]], num_kv_heads: int,
                    group_size: int, softmax_scale: float, o, lse, d_o, dq=None, dk_self=None,
                    dv_self=None, want_dq: bool = True, want_self: bool = True, stream=None,
                    workspace=None, q_offsets: Optional[Sequence[int]] = None):
    """Returns (dq, dk_self, dv_self); segment gradients go to each Segment's dk/dv.
    ``q_offsets`` as for prefix_attn_fwd."""
    import torch
    prob = Problem.from_tensors(q, rows, num_kv_heads, group_size, softmax_scale, q_offsets)
    if dq is None and want_dq:
        dq = torch.empty_like(q)
    if want_self:
        if dk_self is None:
            dk_self = torch.empty_like(k_self)
        if dv_self is None:
            dv_self = torch.empty_like(v_self)
    ws_n = workspace_size(prob, True)
    ws = workspace if workspace is not None and workspace.numel() >= ws_n else _workspace(ws_n, q.device)
    _check(load().cas_prefix_attn_bwd(ctypes.byref(prob.c), q.data_ptr(), k_self.data_ptr(),
                                      v_self.data_ptr(), o.data_ptr(), lse.data_ptr(), d_o.data_ptr(),
                                      _ptr(dq), _ptr(dk_self), _ptr(dv_self), ws.data_ptr(),
                                      ws.numel(), _stream_handle(q.device, stream)))
    return dq, dk_self, dv_self


def cartridge_stage(copies: Sequence[Tuple[object, object]], side_stream, done_event=None) -> None:
    """Host (pinned) -> device copies of (host_tensor, device_tensor) pairs on side_stream,
    recording done_event (a torch.cuda.Event) after the last one."""
    arr = (_lib.StageCopy * max(len(copies), 1))()
    for i, (h, d) in enumerate(copies):
        nb = h.numel() * h.element_size()
        if d.numel() * d.element_size() < nb:
            raise ValueError("destination smaller than source")
        arr[i].host_src, arr[i].dev_dst, arr[i].bytes = h.data_ptr(), d.data_ptr(), nb
    ev = None
    if done_event is not None:
        if hasattr(done_event, "cuda_event"):
            if not done_event.cuda_event:
                done_event.record(side_stream)   # torch creates its event lazily
            ev = done_event.cuda_event
        else:
            ev = int(done_event)
    _check(load().cas_cartridge_stage(ctypes.cast(arr, ctypes.POINTER(_lib.StageCopy)), len(copies),
                                      side_stream.cuda_stream, ev))


def timing_enable(on: bool = True) -> None:
    _check(load().cas_timing_enable(int(on)))


def timing_reset() -> None:
    _check(load().cas_timing_reset())


def timing_read() -> dict:
    """{kernel name: (launches, total ms)} since the last reset."""
    cap = 32
    arr = (_lib.KernelTime * cap)()
    n = ctypes.c_int32(0)
    _check(load().cas_timing_read(arr, cap, ctypes.byref(n)))
    return {arr[i].name.decode(): (arr[i].launches, arr[i].total_ms) for i in range(min(n.value, cap))}
