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

__all__ = ["Segment", "Problem", "CasError", "load", "prefix_attn_fwd", "prefix_attn_fwd_noalloc",
           "prefix_attn_bwd",
           "workspace_size", "plan_info", "set_tuning", "get_tuning", "cartridge_stage",
           "timing_enable", "timing_reset", "timing_read", "AdamCartridge", "adam_lr_scale",
           "cartridge_adam", "DecodeProblem", "paged_decode_fwd", "plan_rotation", "CartridgePool"]


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
    """Launch-plan knobs (0 = automatic): key-axis splits of the forward and
    of the dQ pass."""
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


def prefix_attn_fwd_noalloc(q, k_self, v_self, rows: Sequence[Sequence[Segment]], num_kv_heads: int,
                            group_size: int, softmax_scale: float, o, lse, stream=None,
                            q_offsets: Optional[Sequence[int]] = None) -> None:
    """The forward through cas_prefix_attn_fwd_noalloc: writes the caller's
    ``o`` (and ``lse`` unless None) using the library's static device scratch
    instead of a workspace; nothing is allocated."""
    prob = Problem.from_tensors(q, rows, num_kv_heads, group_size, softmax_scale, q_offsets)
    _check(load().cas_prefix_attn_fwd_noalloc(ctypes.byref(prob.c), q.data_ptr(), k_self.data_ptr(),
                                              v_self.data_ptr(), o.data_ptr(), _ptr(lse),
                                              _stream_handle(q.device, stream)))


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


@dataclasses.dataclass
class AdamCartridge:
    """One cartridge for the optimizer step: bf16 k, v ([len, Hkv, d] views, any
    token/head strides) with their gradients dk, dv (same strides), fp32
    moments m1_k, m2_k, m1_v, m2_v (contiguous [len, Hkv, d]), the optimizer
    steps it has received and its frozen leading tokens."""
    k: object
    v: object
    dk: object
    dv: object
    m1_k: object
    m2_k: object
    m1_v: object
    m2_v: object
    step: int = 0
    frozen_tokens: int = 1


def adam_lr_scale(step: int, warmup_steps: int = 20, warmup_buckets: int = 4) -> float:
    """The bucketed per-cartridge warmup factor (cas_adam_lr_scale)."""
    return float(load().cas_adam_lr_scale(int(step), int(warmup_steps), int(warmup_buckets)))


def _adam_array(carts: Sequence[AdamCartridge]):
    arr = (_lib.AdamCartridge * max(len(carts), 1))()
    for i, c in enumerate(carts):
        if c.k.dim() != 3 or c.k.shape != c.v.shape or c.k.stride() != c.v.stride():
            raise ValueError("k and v must be [len, Hkv, d] views with equal strides")
        for t in (c.dk, c.dv):
            if t.shape != c.k.shape or t.stride() != c.k.stride():
                raise ValueError("dk and dv must match k's shape and strides")
        for t in (c.m1_k, c.m2_k, c.m1_v, c.m2_v):
            if t.shape != c.k.shape or not t.is_contiguous():
                raise ValueError("moments must be contiguous with k's shape")
        e = arr[i]
        e.k, e.v, e.dk, e.dv = c.k.data_ptr(), c.v.data_ptr(), c.dk.data_ptr(), c.dv.data_ptr()
        e.m1_k, e.m2_k, e.m1_v, e.m2_v = (c.m1_k.data_ptr(), c.m2_k.data_ptr(), c.m1_v.data_ptr(),
                                          c.m2_v.data_ptr())
        e.len, e.stride_tok, e.stride_head = int(c.k.shape[0]), int(c.k.stride(0)), int(c.k.stride(1))
        e.step, e.frozen_tokens = int(c.step), int(c.frozen_tokens)
    return arr


def cartridge_adam(carts: Sequence[AdamCartridge], lr: float, beta1: float = 0.9, beta2: float = 0.999,
                   eps: float = 1e-8, warmup_steps: int = 20, warmup_buckets: int = 4, stream=None,
                   workspace=None) -> None:
    """One fused Adam step over every cartridge's K and V (cas_cartridge_adam).
    The caller increments each cartridge's step afterwards."""
    if not carts:
        return
    arr = _adam_array(carts)
    Hkv, D = int(carts[0].k.shape[1]), int(carts[0].k.shape[2])
    n = ctypes.c_size_t(0)
    P = ctypes.POINTER(_lib.AdamCartridge)
    _check(load().cas_cartridge_adam_workspace_size(ctypes.cast(arr, P), len(carts), Hkv, D, ctypes.byref(n)))
    dev = carts[0].k.device
    ws = workspace if workspace is not None and workspace.numel() >= n.value else _workspace(n.value, dev)
    cfg = _lib.AdamConfig(lr, beta1, beta2, eps, warmup_steps, warmup_buckets)
    _check(load().cas_cartridge_adam(ctypes.cast(arr, P), len(carts), Hkv, D, ctypes.byref(cfg), ws.data_ptr(),
                                     ws.numel(), _stream_handle(dev, stream)))


class DecodeProblem:
    """Host tables of a paged decode call (cas_decode_problem_t): per request its
    query count, key count and page list (pages of [page_size, Hkv, d])."""

    def __init__(self, q_counts: Sequence[int], kv_lens: Sequence[int], page_lists: Sequence[Sequence[int]],
                 num_pages: int, page_size: int, num_kv_heads: int, group_size: int, head_dim: int,
                 softmax_scale: float):
        B = len(q_counts)
        if len(kv_lens) != B or len(page_lists) != B:
            raise ValueError("one query count, kv_len and page list per request")
        qo = [0]
        for n in q_counts:
            qo.append(qo[-1] + int(n))
        po = [0]
        for pl in page_lists:
            po.append(po[-1] + len(pl))
        ids = [int(x) for pl in page_lists for x in pl]
        self.Tq = qo[-1]
        self._qo = (ctypes.c_int32 * (B + 1))(*qo)
        self._kv = (ctypes.c_int32 * max(B, 1))(*[int(x) for x in kv_lens])
        self._po = (ctypes.c_int32 * (B + 1))(*po)
        self._ids = (ctypes.c_int32 * max(len(ids), 1))(*ids)
        I = ctypes.POINTER(ctypes.c_int32)
        self.c = _lib.DecodeProblem(B, num_kv_heads, group_size, head_dim, float(softmax_scale), page_size,
                                    int(num_pages), ctypes.cast(self._qo, I), ctypes.cast(self._kv, I),
                                    ctypes.cast(self._po, I), ctypes.cast(self._ids, I))


def paged_decode_fwd(q, k_pages, v_pages, q_counts: Sequence[int], kv_lens: Sequence[int],
                     page_lists: Sequence[Sequence[int]], num_kv_heads: int, group_size: int,
                     softmax_scale: float, o=None, lse=None, need_lse: bool = True, stream=None,
                     workspace=None, problem: Optional[DecodeProblem] = None):
    """Attention of each request's last q_counts[b] positions (q: [Tq, Hq, d]
    packed by request) over its kv_lens[b] keys held in the pages page_lists[b]
    of the pools k_pages, v_pages ([num_pages, page_size, Hkv, d] bf16).
    Returns O [Tq, Hq, d] and LSE [Hq, Tq] (fp32). A DecodeProblem built once
    from the same tables may be passed as ``problem`` to skip rebuilding them."""
    import torch
    num_pages, page_size, Hkv, D = k_pages.shape
    prob = problem if problem is not None else DecodeProblem(q_counts, kv_lens, page_lists, num_pages, page_size,
                                                             Hkv, group_size, D, softmax_scale)
    if o is None:
        o = torch.empty_like(q)
    if lse is None and need_lse:
        lse = torch.empty((q.shape[1], q.shape[0]), dtype=torch.float32, device=q.device)
    n = ctypes.c_size_t(0)
    _check(load().cas_paged_decode_workspace_size(ctypes.byref(prob.c), ctypes.byref(n)))
    ws = workspace if workspace is not None and workspace.numel() >= n.value else _workspace(n.value, q.device)
    _check(load().cas_paged_decode_fwd(ctypes.byref(prob.c), q.data_ptr(), k_pages.data_ptr(), v_pages.data_ptr(),
                                       o.data_ptr(), _ptr(lse), ws.data_ptr(), ws.numel(),
                                       _stream_handle(q.device, stream)))
    return o, lse


def plan_rotation(steps: Sequence[int], active: Sequence[bool], budget: int, swap_fraction: float):
    """The budget manager's rotation choice (cas_pool_plan_rotation): (evict, admit)."""
    n = len(steps)
    st = (ctypes.c_int32 * n)(*[int(x) for x in steps])
    ac = (ctypes.c_uint8 * n)(*[1 if a else 0 for a in active])
    ev = (ctypes.c_int32 * n)()
    ad = (ctypes.c_int32 * n)()
    m = ctypes.c_int32(0)
    _check(load().cas_pool_plan_rotation(st, ac, n, int(budget), float(swap_fraction), ev, ad, ctypes.byref(m)))
    return list(ev[:m.value]), list(ad[:m.value])


class _DevArray:
    """A device buffer of the pool seen by torch (__cuda_array_interface__)."""

    def __init__(self, ptr: int, shape, typestr: str):
        self.__cuda_array_interface__ = {"shape": tuple(shape), "typestr": typestr, "data": (int(ptr), False),
                                         "version": 2, "strides": None}


class CartridgePool:
    """Budget manager (cas_pool_*): pinned host copies of every cartridge's
    K/V, B active device slots and prefetched rotations. The Adam moments of
    offloaded cartridges stay in pinned host memory, or with ``moment_dir``
    in a file in that directory (the NVMe tier)."""

    def __init__(self, lens: Sequence[int], num_kv_heads: int, head_dim: int, budget: int, rotate_every: int,
                 swap_fraction: float, frozen_tokens: int = 1, moment_dir: Optional[str] = None):
        self.lens = [int(x) for x in lens]
        self.Hkv, self.D = num_kv_heads, head_dim
        self._lens = (ctypes.c_int64 * len(lens))(*self.lens)
        cfg = _lib.PoolConfig(len(lens), ctypes.cast(self._lens, ctypes.POINTER(ctypes.c_int64)), num_kv_heads,
                              head_dim, budget, rotate_every, swap_fraction, frozen_tokens,
                              None if moment_dir is None else str(moment_dir).encode())
        h = ctypes.c_void_p()
        _check(load().cas_pool_create(ctypes.byref(cfg), ctypes.byref(h)))
        self.h = h

    def close(self):
        if self.h:
            _check(load().cas_pool_destroy(self.h))
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def host(self, cart: int) -> dict:
        """Cartridge `cart` on the host: numpy views of its pinned k and v (bf16
        bits as int16; writable), a copy of its moments m1_k, m2_k, m1_v, m2_v
        (float32, from whichever tier holds them), and its step count."""
        import numpy as np
        v = _lib.AdamCartridge()
        _check(load().cas_pool_host_cartridge(self.h, int(cart), ctypes.byref(v)))
        L, shp = int(v.len), (int(v.len), self.Hkv, self.D)
        n = L * self.Hkv * self.D
        out = {}
        for name in ("k", "v"):
            out[name] = np.ctypeslib.as_array(ctypes.cast(getattr(v, name), ctypes.POINTER(ctypes.c_int16)),
                                              (n,)).reshape(shp)
        m = np.empty(4 * n, dtype=np.float32)
        _check(load().cas_pool_read_moments(self.h, int(cart), m.ctypes.data_as(ctypes.POINTER(ctypes.c_float))))
        for i, name in enumerate(("m1_k", "m2_k", "m1_v", "m2_v")):
            out[name] = m[i * n:(i + 1) * n].reshape(shp)
        out["step"] = int(v.step)
        return out

    def load(self, stream=None):
        import torch
        _check(load().cas_pool_load(self.h, _stream_handle(torch.device("cuda"), stream)))

    def active(self):
        """[(cartridge id, AdamCartridge of torch views over its device slot)]."""
        import torch
        cap = 1 << 12
        ids = (ctypes.c_int32 * cap)()
        views = (_lib.AdamCartridge * cap)()
        n = ctypes.c_int32(0)
        _check(load().cas_pool_active(self.h, ids, views, cap, ctypes.byref(n)))
        out = []
        for i in range(n.value):
            v = views[i]
            shp = (int(v.len), self.Hkv, self.D)
            t = {}
            for name in ("k", "v", "dk", "dv"):
                t[name] = torch.as_tensor(_DevArray(getattr(v, name), shp, "<i2"), device="cuda").view(torch.bfloat16)
            for name in ("m1_k", "m2_k", "m1_v", "m2_v"):
                t[name] = torch.as_tensor(_DevArray(getattr(v, name), shp, "<f4"), device="cuda")
            out.append((int(ids[i]), AdamCartridge(**t, step=int(v.step), frozen_tokens=int(v.frozen_tokens))))
        return out

    def end_step(self, stream=None):
        import torch
        _check(load().cas_pool_end_step(self.h, _stream_handle(torch.device("cuda"), stream)))

    def flush(self, stream=None):
        import torch
        _check(load().cas_pool_flush(self.h, _stream_handle(torch.device("cuda"), stream)))


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
