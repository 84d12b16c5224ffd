"""Helpers for the GPU parity tests: device copies of seeded workloads in the
requested cartridge layouts, calls through the C ABI, and error metrics.

The expected values always come from the fp64 oracle on the same input bits.
"""
from __future__ import annotations

import numpy as np

import casgen
import oracle

# Tolerances: max |gpu - oracle| / max |oracle| per tensor (per cartridge for
# dK/dV), and absolute error on the natural-log LSE.
TOL = {"fp32": 1e-5, "bf16": 2e-2}
LSE_TOL = {"fp32": 1e-5, "bf16": 1e-3}


def torch():
    import torch as t
    return t


def dev(arr: np.ndarray, dtype: str):
    t = torch()
    if dtype == "bf16":
        return t.from_numpy(np.ascontiguousarray(arr).view(np.int16)).view(t.bfloat16).cuda()
    return t.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).cuda()


def host(x) -> np.ndarray:
    return x.detach().float().cpu().numpy().astype(np.float64)


WIDE_STRIDE = 1 << 21   # elements between tokens of the "wide" layout (4 MiB in bf16)


def alloc_like_layout(L: int, Hkv: int, D: int, layout: str, dtype, fill=float("nan")):
    """A [L, Hkv, D] view with the requested storage: token-major, padded
    token stride, head-major, or "wide" (a token stride of 2^21 elements, so
    a segment of a thousand tokens spans several GiB)."""
    t = torch()
    if layout == "tok":
        x = t.full((L, Hkv, D), fill, dtype=dtype, device="cuda")
        return x, x
    if layout in ("padded", "wide"):
        row = Hkv * D + 64 if layout == "padded" else WIDE_STRIDE
        base = t.full((L, row), fill, dtype=dtype, device="cuda")
        return base[:, : Hkv * D].view(L, Hkv, D), base
    if layout == "head":
        base = t.full((Hkv, L, D), fill, dtype=dtype, device="cuda")
        return base.permute(1, 0, 2), base
    raise ValueError(layout)


class GpuCase:
    """Device tensors for one workload plus the float inputs the oracle reads."""

    def __init__(self, wl: casgen.Workload, tensors=None, grads: bool = True, layouts=None):
        import paper_2606_04557_amd as cas
        t = torch()
        self.wl = wl
        self.T = tensors if tensors is not None else casgen.make_tensors(wl)
        dt = wl.dtype
        self.tdtype = t.bfloat16 if dt == "bf16" else t.float32
        self.q = dev(self.T["q"], dt)
        self.k_self = dev(self.T["k_self"], dt)
        self.v_self = dev(self.T["v_self"], dt)
        self.d_o = dev(self.T["d_o"], dt) if "d_o" in self.T else None
        used = sorted({c for r in wl.rows for c in r})
        lay = layouts or wl.layouts or ["tok"] * len(wl.cart_lens)
        self.k, self.v, self.dk, self.dv, self.bases = {}, {}, {}, {}, {}
        Hkv, D = wl.num_kv_heads, wl.head_dim
        for c in used:
            L = wl.cart_lens[c]
            self.k[c], _ = alloc_like_layout(L, Hkv, D, lay[c], self.tdtype)
            self.k[c].copy_(dev(self.T["cart_k"][c], dt))
            self.v[c], _ = alloc_like_layout(L, Hkv, D, lay[c], self.tdtype)
            self.v[c].copy_(dev(self.T["cart_v"][c], dt))
            if grads:
                self.dk[c], self.bases[("dk", c)] = alloc_like_layout(L, Hkv, D, lay[c], self.tdtype)
                self.dv[c], self.bases[("dv", c)] = alloc_like_layout(L, Hkv, D, lay[c], self.tdtype)
        self.rows = [[cas.Segment(self.k[c], self.v[c], self.dk.get(c), self.dv.get(c)) for c in r]
                     for r in wl.rows]

    # -- library calls ---------------------------------------------------------
    def _layout_kw(self, kw):
        if self.wl.packed:
            kw = dict(kw)
            kw.setdefault("q_offsets", self.wl.q_offsets)
        return kw

    def fwd(self, **kw):
        import paper_2606_04557_amd as cas
        wl = self.wl
        return cas.prefix_attn_fwd(self.q, self.k_self, self.v_self, self.rows, wl.num_kv_heads,
                                   wl.group_size, float(wl.scale), **self._layout_kw(kw))

    def bwd(self, o, lse, **kw):
        import paper_2606_04557_amd as cas
        wl = self.wl
        return cas.prefix_attn_bwd(self.q, self.k_self, self.v_self, self.rows, wl.num_kv_heads,
                                   wl.group_size, float(wl.scale), o, lse, self.d_o,
                                   **self._layout_kw(kw))

    # -- oracle inputs ---------------------------------------------------------
    def oracle_args(self):
        dt = self.wl.dtype
        T = self.T
        f = lambda a: None if a is None else casgen.to_float(a, dt)
        return (f(T["q"]), f(T["k_self"]), f(T["v_self"]), [f(a) for a in T["cart_k"]],
                [f(a) for a in T["cart_v"]], self.wl.rows, float(self.wl.scale), self.wl.group_size)

    def oracle_do(self):
        return casgen.to_float(self.T["d_o"], self.wl.dtype)


def rel_err(gpu: np.ndarray, ref: np.ndarray) -> float:
    if np.asarray(ref).size == 0:
        return 0.0
    den = float(np.abs(ref).max())
    num = float(np.abs(np.asarray(gpu, dtype=np.float64) - ref).max())
    if den == 0.0:
        return num
    return num / den


def full_oracle(case: GpuCase, backward: bool = True):
    args = case.oracle_args()
    if case.wl.packed:
        q, ks, vs, ck, cv, rows, scale, g = args
        qo = case.wl.q_offsets
        O, LSE = oracle.packed_forward(q, ks, vs, ck, cv, rows, qo, scale, g)
        if not backward:
            return O, LSE, None
        grads = oracle.packed_backward(q, ks, vs, ck, cv, rows, qo, scale, g, case.oracle_do(), O=O, LSE=LSE)
        return O, LSE, grads
    O, LSE = oracle.forward(*args)
    if not backward:
        return O, LSE, None
    grads = oracle.backward(*args, case.oracle_do(), O=O, LSE=LSE)
    return O, LSE, grads
