"""Host-side checks of libcas that need no GPU: the library loads, exports
every function include/cas.h declares, validates arguments before touching
the device, and plans launches (splits, alias folding, workspace sizes).

Device pointers here are fabricated addresses: every call either fails
validation (which happens before any HIP call) or is a pure planning query.
"""
import ctypes
import os
import re

import pytest

from paper_2606_04557_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    return _lib.load()


def test_exports_match_header(lib):
    hdr = open(os.path.join(ROOT, "include", "cas.h")).read()
    declared = sorted(set(re.findall(r"\b(cas_[a-z_0-9]+)\s*\(", hdr)))
    assert declared == sorted(_lib.EXPORTS)
    for name in declared:
        assert hasattr(lib, name), name
    assert lib.cas_abi_version() == _lib.ABI_VERSION == 4
    assert lib.cas_status_string(_lib.CAS_ERR_NOT_PINNED) == b"CAS_ERR_NOT_PINNED"


BASE = 1 << 32     # fabricated, 16-byte aligned device addresses


class Fake:
    """Builds a cas_problem_t over fabricated addresses."""

    def __init__(self, B=1, Sq=8, Hkv=2, g=2, D=64, dtype=_lib.CAS_DTYPE_BF16, scale=0.125,
                 rows=((16, 8),), grads=True):
        self.B, self.Sq, self.Hkv, self.g, self.D = B, Sq, Hkv, g, D
        es = 2 if dtype == _lib.CAS_DTYPE_BF16 else 4
        self.es = es
        self.next = BASE
        nent = sum(len(r) for r in rows)
        self.segs = (_lib.Segment * max(1, nent))()
        self.offs = (ctypes.c_int32 * (B + 1))()
        i = 0
        for b in range(B):
            self.offs[b] = i
            for L in rows[b]:
                s = self.segs[i]
                nbytes = max(1, L) * Hkv * D * es
                s.k, s.v = self.alloc(nbytes), self.alloc(nbytes)
                if grads:
                    s.dk, s.dv = self.alloc(nbytes), self.alloc(nbytes)
                s.len, s.stride_tok, s.stride_head = L, Hkv * D, D
                i += 1
        self.offs[B] = i
        self.p = _lib.Problem(dtype, B, Sq, Hkv, g, D, scale,
                              ctypes.cast(self.segs, ctypes.POINTER(_lib.Segment)),
                              ctypes.cast(self.offs, ctypes.POINTER(ctypes.c_int32)))
        qn = B * Sq * Hkv * g * D * es
        kvn = B * Sq * Hkv * D * es
        self.q, self.ks, self.vs, self.o, self.do = (self.alloc(qn), self.alloc(kvn), self.alloc(kvn),
                                                      self.alloc(qn), self.alloc(qn))
        self.lse = self.alloc(B * Hkv * g * Sq * 4)
        self.dq, self.dks, self.dvs = self.alloc(qn), self.alloc(kvn), self.alloc(kvn)
        self.ws = self.alloc(1 << 30)

    def alloc(self, n):
        a = self.next
        self.next += (n + 4095) // 4096 * 4096 + 4096
        return a

    def fwd(self, lib, ws_bytes=1 << 30, **over):
        a = dict(q=self.q, ks=self.ks, vs=self.vs, o=self.o, lse=self.lse, ws=self.ws)
        a.update(over)
        return lib.cas_prefix_attn_fwd(ctypes.byref(self.p), a["q"], a["ks"], a["vs"], a["o"], a["lse"],
                                       a["ws"], ws_bytes, None)

    def bwd(self, lib, ws_bytes=1 << 30, **over):
        a = dict(q=self.q, ks=self.ks, vs=self.vs, o=self.o, lse=self.lse, do=self.do, dq=self.dq,
                 dks=self.dks, dvs=self.dvs, ws=self.ws)
        a.update(over)
        return lib.cas_prefix_attn_bwd(ctypes.byref(self.p), a["q"], a["ks"], a["vs"], a["o"], a["lse"],
                                       a["do"], a["dq"], a["dks"], a["dvs"], a["ws"], ws_bytes, None)


def _msg(lib):
    return lib.cas_last_error_message().decode()


@pytest.mark.parametrize("field,value,code", [
    ("batch", 0, _lib.CAS_ERR_INVALID_ARGUMENT),
    ("q_len", 0, _lib.CAS_ERR_INVALID_ARGUMENT),
    ("num_kv_heads", -1, _lib.CAS_ERR_INVALID_ARGUMENT),
    ("group_size", 0, _lib.CAS_ERR_INVALID_ARGUMENT),
    ("head_dim", 96, _lib.CAS_ERR_UNSUPPORTED),
    ("softmax_scale", 0.0, _lib.CAS_ERR_INVALID_ARGUMENT),
    ("softmax_scale", float("inf"), _lib.CAS_ERR_INVALID_ARGUMENT),
    ("dtype", 7, _lib.CAS_ERR_INVALID_ARGUMENT),
])
def test_shape_validation(lib, field, value, code):
    f = Fake()
    setattr(f.p, field, value)
    assert f.fwd(lib) == code, _msg(lib)
    assert f.bwd(lib) == code
    n = ctypes.c_size_t(0)
    assert lib.cas_prefix_attn_workspace_size(ctypes.byref(f.p), 0, ctypes.byref(n)) == code


def test_segment_table_validation(lib):
    f = Fake(B=2, rows=((16, 8), (4,)))
    f.offs[1] = 3
    f.offs[2] = 2                                   # decreasing offsets
    assert f.fwd(lib) == _lib.CAS_ERR_INVALID_ARGUMENT
    f = Fake()
    f.offs[0] = 1
    assert f.fwd(lib) == _lib.CAS_ERR_INVALID_ARGUMENT
    f = Fake()
    f.segs[0].len = -1
    assert f.fwd(lib) == _lib.CAS_ERR_INVALID_ARGUMENT
    f = Fake()
    f.segs[1].k = None                              # len > 0 with NULL k
    assert f.fwd(lib) == _lib.CAS_ERR_INVALID_ARGUMENT
    f = Fake()
    f.segs[1].stride_tok = 0
    assert f.fwd(lib) == _lib.CAS_ERR_INVALID_ARGUMENT
    f = Fake()
    f.p.segments = None
    assert f.fwd(lib) == _lib.CAS_ERR_INVALID_ARGUMENT
    # A zero-length entry is skipped even with NULL pointers.
    f = Fake(rows=((16, 0, 8),))
    f.segs[1].k = f.segs[1].v = None
    n = ctypes.c_size_t(0)
    assert lib.cas_prefix_attn_workspace_size(ctypes.byref(f.p), 0, ctypes.byref(n)) == _lib.CAS_OK


def test_alignment_validation(lib):
    f = Fake()
    f.segs[0].k = f.segs[0].k + 8
    assert f.fwd(lib) == _lib.CAS_ERR_ALIGNMENT
    f = Fake()
    f.segs[0].stride_tok = f.Hkv * f.D + 4           # 8-byte token stride remainder in bf16
    assert f.fwd(lib) == _lib.CAS_ERR_ALIGNMENT
    f = Fake()
    assert f.fwd(lib, q=f.q + 2) == _lib.CAS_ERR_ALIGNMENT
    assert f.fwd(lib, lse=f.lse + 2) == _lib.CAS_ERR_ALIGNMENT
    assert f.bwd(lib, dq=f.dq + 4) == _lib.CAS_ERR_ALIGNMENT


def test_pointer_and_overlap_validation(lib):
    f = Fake()
    assert f.fwd(lib, q=None) == _lib.CAS_ERR_INVALID_ARGUMENT
    assert f.bwd(lib, lse=None) == _lib.CAS_ERR_INVALID_ARGUMENT
    # Output overlapping an input.
    assert f.fwd(lib, o=f.q + 16) == _lib.CAS_ERR_INVALID_ARGUMENT
    assert "overlaps" in _msg(lib)
    assert f.bwd(lib, dq=f.segs[0].k) == _lib.CAS_ERR_INVALID_ARGUMENT
    # Two outputs overlapping.
    assert f.bwd(lib, dks=f.dq) == _lib.CAS_ERR_INVALID_ARGUMENT
    # A cartridge gradient written into another cartridge's keys.
    f = Fake(rows=((16, 8),))
    f.segs[1].dk = f.segs[0].k
    assert f.bwd(lib) == _lib.CAS_ERR_INVALID_ARGUMENT


def test_alias_rules(lib):
    f = Fake(B=2, rows=((16,), (16,)))
    # Point row 1's entry at row 0's cartridge, including its gradients: allowed.
    for a in ("k", "v", "dk", "dv"):
        setattr(f.segs[1], a, getattr(f.segs[0], a))
    info = _lib.PlanInfo()
    assert lib.cas_plan_info(ctypes.byref(f.p), ctypes.byref(info)) == _lib.CAS_OK
    assert info.unique_segments == 1
    # Same k/v storage with a different gradient buffer: rejected.
    f.segs[1].dk = f.alloc(16 * f.Hkv * f.D * 2)
    assert f.bwd(lib) == _lib.CAS_ERR_INVALID_ARGUMENT
    assert "share dk/dv" in _msg(lib)


def test_gradient_layout_self_overlap(lib):
    f = Fake(rows=((16,),))
    f.segs[0].stride_head = 8                      # heads overlap within a token
    assert f.bwd(lib) == _lib.CAS_ERR_INVALID_ARGUMENT
    # Head-major storage is fine: [Hkv, len, D].
    f = Fake(rows=((16,),))
    f.segs[0].stride_tok, f.segs[0].stride_head = f.D, 16 * f.D
    n = ctypes.c_size_t(0)
    assert lib.cas_prefix_attn_workspace_size(ctypes.byref(f.p), 1, ctypes.byref(n)) == _lib.CAS_OK


def test_workspace_validation(lib):
    f = Fake()
    n = ctypes.c_size_t(0)
    assert lib.cas_prefix_attn_workspace_size(ctypes.byref(f.p), 1, ctypes.byref(n)) == _lib.CAS_OK
    assert n.value > 0
    assert f.bwd(lib, ws_bytes=n.value - 1) == _lib.CAS_ERR_WORKSPACE
    assert f.bwd(lib, ws=None) == _lib.CAS_ERR_WORKSPACE


def test_tuning_roundtrip(lib):
    t = _lib.Tuning(3, 5)
    assert lib.cas_set_tuning(ctypes.byref(t)) == _lib.CAS_OK
    r = _lib.Tuning()
    assert lib.cas_get_tuning(ctypes.byref(r)) == _lib.CAS_OK
    assert (r.fwd_splits, r.dq_splits) == (3, 5)
    f = Fake()
    info = _lib.PlanInfo()
    assert lib.cas_plan_info(ctypes.byref(f.p), ctypes.byref(info)) == _lib.CAS_OK
    assert (info.fwd_splits, info.dq_splits) == (3, 5)
    bad = _lib.Tuning(-1, 0)
    assert lib.cas_set_tuning(ctypes.byref(bad)) == _lib.CAS_ERR_INVALID_ARGUMENT
    z = _lib.Tuning(0, 0)
    assert lib.cas_set_tuning(ctypes.byref(z)) == _lib.CAS_OK


def test_plans_of_benchmark_shapes(lib):
    """Occupancy planning on the benchmark shapes (256-CU target)."""
    # 16 x 2048 cartridges, B=2, 32/8 heads, Sq=2048: 512 forward workgroups, no split.
    f = Fake(B=2, Sq=2048, Hkv=8, g=4, D=128, rows=((2048,) * 16, (2048,) * 16))
    info = _lib.PlanInfo()
    assert lib.cas_plan_info(ctypes.byref(f.p), ctypes.byref(info)) == _lib.CAS_OK
    assert info.fwd_splits == 1 and info.fwd_workgroups == 512
    assert info.unique_segments == 32
    assert info.total_key_tiles == 32 * 16 + 2 * 16
    assert info.max_prefix_len == 32768
    # B=1, Sq=512: only 64 base workgroups, so the key axis is split.
    f = Fake(B=1, Sq=512, Hkv=8, g=4, D=128, rows=((1000,) * 64,))
    assert lib.cas_plan_info(ctypes.byref(f.p), ctypes.byref(info)) == _lib.CAS_OK
    assert info.fwd_splits == 8 and info.fwd_workgroups == 512
    assert info.dq_splits == 8     # bf16 dQ also takes 256 rows per workgroup
    assert info.ws_fwd_bytes >= 8 * 512 * 32 * 128 * 4


def test_stage_validation_without_device(lib):
    assert lib.cas_cartridge_stage(None, -1, None, None) == _lib.CAS_ERR_INVALID_ARGUMENT
    assert lib.cas_cartridge_stage(None, 2, None, None) == _lib.CAS_ERR_INVALID_ARGUMENT
    arr = (_lib.StageCopy * 1)()
    arr[0].host_src, arr[0].dev_dst, arr[0].bytes = None, BASE, 64
    assert lib.cas_cartridge_stage(arr, 1, None, None) == _lib.CAS_ERR_INVALID_ARGUMENT
    # Zero copies is a no-op.
    assert lib.cas_cartridge_stage(None, 0, None, None) == _lib.CAS_OK


def _packed(f, offs):
    arr = (ctypes.c_int32 * len(offs))(*offs)
    f.keep = arr
    f.p.q_offsets = ctypes.cast(arr, ctypes.POINTER(ctypes.c_int32))
    f.p.q_len = 0


@pytest.mark.parametrize("offs,q_len,ok", [
    ((0, 5, 9), 0, True),
    ((0, 0, 9), 0, True),            # an empty sample
    ((0, 5, 9), 4, False),           # q_len must be 0 with q_offsets
    ((1, 5, 9), 0, False),           # q_offsets[0] != 0
    ((0, 6, 5), 0, False),           # decreasing
    ((0, 0, 0), 0, False),           # no query token at all
])
def test_packed_offsets_validation(lib, offs, q_len, ok):
    f = Fake(B=2, Sq=1, rows=((16,), (8,)))
    _packed(f, offs)
    f.p.q_len = q_len
    n = ctypes.c_size_t(0)
    st = lib.cas_prefix_attn_workspace_size(ctypes.byref(f.p), 1, ctypes.byref(n))
    if ok:
        assert st == _lib.CAS_OK, _msg(lib)
        assert n.value > 0
    else:
        assert st == _lib.CAS_ERR_INVALID_ARGUMENT, _msg(lib)
        assert f.fwd(lib) == _lib.CAS_ERR_INVALID_ARGUMENT


def test_packed_equal_lengths_plan_like_fixed(lib):
    """Equal-length packed samples plan exactly like the fixed-length batch."""
    for bwd in (0, 1):
        a = Fake(B=3, Sq=70, Hkv=2, g=4, D=128, rows=((40, 3), (129,), ()))
        b = Fake(B=3, Sq=70, Hkv=2, g=4, D=128, rows=((40, 3), (129,), ()))
        _packed(b, (0, 70, 140, 210))
        na, nb = ctypes.c_size_t(0), ctypes.c_size_t(0)
        assert lib.cas_prefix_attn_workspace_size(ctypes.byref(a.p), bwd, ctypes.byref(na)) == _lib.CAS_OK
        assert lib.cas_prefix_attn_workspace_size(ctypes.byref(b.p), bwd, ctypes.byref(nb)) == _lib.CAS_OK
        assert na.value == nb.value
    ia, ib = _lib.PlanInfo(), _lib.PlanInfo()
    assert lib.cas_plan_info(ctypes.byref(a.p), ctypes.byref(ia)) == _lib.CAS_OK
    assert lib.cas_plan_info(ctypes.byref(b.p), ctypes.byref(ib)) == _lib.CAS_OK
    for fld, _ in _lib.PlanInfo._fields_:
        assert getattr(ia, fld) == getattr(ib, fld), fld
    # Uneven samples: the dK/dV list holds each row's own self tiles.
    c = Fake(B=3, Sq=1, Hkv=2, g=4, D=128, rows=((40,), (), (7,)))
    _packed(c, (0, 300, 301, 301))
    ic = _lib.PlanInfo()
    assert lib.cas_plan_info(ctypes.byref(c.p), ctypes.byref(ic)) == _lib.CAS_OK
    assert ic.dkdv_workgroups == (1 + 1 + 3 + 1 + 0) * 2   # 2 cartridge tiles + self tiles 3, 1, 0


def _adam_cart(f, L=40, Hkv=2, D=64, step=0, frozen=1, stride_tok=None):
    c = _lib.AdamCartridge()
    st = stride_tok or Hkv * D
    nb = L * st * 2 + 4096
    c.k, c.v, c.dk, c.dv = f.alloc(nb), f.alloc(nb), f.alloc(nb), f.alloc(nb)
    mb = L * Hkv * D * 4
    c.m1_k, c.m2_k, c.m1_v, c.m2_v = f.alloc(mb), f.alloc(mb), f.alloc(mb), f.alloc(mb)
    c.len, c.stride_tok, c.stride_head, c.step, c.frozen_tokens = L, st, D, step, frozen
    return c


def test_adam_validation(lib):
    f = Fake()
    arr = (_lib.AdamCartridge * 3)(_adam_cart(f), _adam_cart(f, L=1), _adam_cart(f, L=17, frozen=0))
    P = ctypes.cast(arr, ctypes.POINTER(_lib.AdamCartridge))
    n = ctypes.c_size_t(0)
    assert lib.cas_cartridge_adam_workspace_size(P, 3, 2, 64, ctypes.byref(n)) == _lib.CAS_OK, _msg(lib)
    # 4 tensor records (80 bytes each, padded to 512), then 2 x ceil(39/16) + 0 (only the
    # frozen token) + 2 x ceil(17/16) = 10 chunk records of 8 bytes (padded to 256)
    assert n.value == 512 + 256
    cfg = _lib.AdamConfig(0.05, 0.9, 0.999, 1e-8, 20, 4)
    for bad in (dict(lr=-1.0), dict(beta1=1.0), dict(eps=0.0), dict(warmup_buckets=0), dict(lr=float("nan"))):
        c2 = _lib.AdamConfig(0.05, 0.9, 0.999, 1e-8, 20, 4)
        for k, v in bad.items():
            setattr(c2, k, v)
        assert lib.cas_cartridge_adam(P, 3, 2, 64, ctypes.byref(c2), f.ws, 1 << 20, None) == \
            _lib.CAS_ERR_INVALID_ARGUMENT, bad
    assert lib.cas_cartridge_adam(P, 3, 2, 96, ctypes.byref(cfg), f.ws, 1 << 20, None) == _lib.CAS_ERR_UNSUPPORTED
    arr[0].m2_k = arr[0].m1_k                                  # moments share a buffer
    assert lib.cas_cartridge_adam_workspace_size(P, 3, 2, 64, ctypes.byref(n)) == _lib.CAS_ERR_INVALID_ARGUMENT
    arr[0].m2_k = arr[2].k                                     # a moment over another cartridge's k
    assert lib.cas_cartridge_adam_workspace_size(P, 3, 2, 64, ctypes.byref(n)) == _lib.CAS_ERR_INVALID_ARGUMENT
    arr[0] = _adam_cart(f, stride_tok=2 * 64 + 4)              # stride not a multiple of 8 elements
    assert lib.cas_cartridge_adam_workspace_size(P, 3, 2, 64, ctypes.byref(n)) == _lib.CAS_ERR_ALIGNMENT
    arr[0] = _adam_cart(f, stride_tok=32)                      # tokens overlap each other
    assert lib.cas_cartridge_adam_workspace_size(P, 3, 2, 64, ctypes.byref(n)) == _lib.CAS_ERR_INVALID_ARGUMENT
    arr[0] = _adam_cart(f, step=-1)
    assert lib.cas_cartridge_adam_workspace_size(P, 3, 2, 64, ctypes.byref(n)) == _lib.CAS_ERR_INVALID_ARGUMENT
    assert lib.cas_cartridge_adam_workspace_size(P, 0, 2, 64, ctypes.byref(n)) == _lib.CAS_OK and n.value == 0


def _decode_problem(B=2, qc=(1, 2), kv=(20, 3), pages=((0, 1), (2,)), P=16, npages=4, Hkv=2, g=2, D=64):
    qo = [0]
    for n in qc:
        qo.append(qo[-1] + n)
    po = [0]
    for p in pages:
        po.append(po[-1] + len(p))
    ids = [x for p in pages for x in p]
    keep = [(ctypes.c_int32 * len(qo))(*qo), (ctypes.c_int32 * len(kv))(*kv), (ctypes.c_int32 * len(po))(*po),
            (ctypes.c_int32 * max(1, len(ids)))(*ids)]
    I = ctypes.POINTER(ctypes.c_int32)
    prob = _lib.DecodeProblem(B, Hkv, g, D, 0.125, P, npages, *[ctypes.cast(k, I) for k in keep])
    return prob, keep


@pytest.mark.parametrize("over,code", [
    (dict(), _lib.CAS_OK),
    (dict(P=24), _lib.CAS_ERR_UNSUPPORTED),
    (dict(D=96), _lib.CAS_ERR_UNSUPPORTED),
    (dict(pages=((0, 4), (2,))), _lib.CAS_ERR_INVALID_ARGUMENT),     # page id out of range
    (dict(pages=((0,), (2,))), _lib.CAS_ERR_INVALID_ARGUMENT),       # 20 keys need 2 pages of 16
    (dict(qc=(1, 4)), _lib.CAS_ERR_INVALID_ARGUMENT),                # 4 queries, 3 keys
    (dict(qc=(0, 2)), _lib.CAS_ERR_INVALID_ARGUMENT),                # a request without a query
])
def test_decode_validation(lib, over, code):
    prob, keep = _decode_problem(**over)
    n = ctypes.c_size_t(0)
    assert lib.cas_paged_decode_workspace_size(ctypes.byref(prob), ctypes.byref(n)) == code, _msg(lib)
    if code == _lib.CAS_OK:
        assert n.value > 0


def test_pool_config_validation(lib):
    lens = (ctypes.c_int64 * 3)(10, 20, 30)
    P = ctypes.POINTER(ctypes.c_int64)
    h = ctypes.c_void_p()
    for bad in (dict(budget=0), dict(budget=4), dict(rotate_every=0), dict(swap_fraction=1.5),
                dict(head_dim=96), dict(num_kv_heads=0)):
        cfg = _lib.PoolConfig(3, ctypes.cast(lens, P), 2, 64, 2, 10, 0.5, 1)
        for k, v in bad.items():
            setattr(cfg, k, v)
        st = lib.cas_pool_create(ctypes.byref(cfg), ctypes.byref(h))
        assert st in (_lib.CAS_ERR_INVALID_ARGUMENT, _lib.CAS_ERR_UNSUPPORTED), (bad, st)
        assert not h.value
    bad_lens = (ctypes.c_int64 * 3)(10, 0, 30)
    cfg = _lib.PoolConfig(3, ctypes.cast(bad_lens, P), 2, 64, 2, 10, 0.5, 1)
    assert lib.cas_pool_create(ctypes.byref(cfg), ctypes.byref(h)) == _lib.CAS_ERR_INVALID_ARGUMENT
    assert lib.cas_pool_active(None, None, None, 0, ctypes.byref(ctypes.c_int32())) == _lib.CAS_ERR_INVALID_ARGUMENT
    assert lib.cas_pool_destroy(None) == _lib.CAS_OK
    # The moment file tier: a directory that cannot hold the file is refused
    # (before any device call) with CAS_ERR_IO.
    cfg = _lib.PoolConfig(3, ctypes.cast(lens, P), 2, 64, 2, 10, 0.5, 1, b"/nonexistent/cas-moments")
    assert lib.cas_pool_create(ctypes.byref(cfg), ctypes.byref(h)) == _lib.CAS_ERR_IO
    assert "/nonexistent/cas-moments" in _msg(lib) and not h.value
    assert lib.cas_status_string(_lib.CAS_ERR_IO) == b"CAS_ERR_IO"
    buf = (ctypes.c_float * 4)()
    assert lib.cas_pool_read_moments(None, 0, buf) == _lib.CAS_ERR_INVALID_ARGUMENT


def test_noalloc_forward_validation(lib):
    """The no-allocation forward validates like the forward, before it touches
    the device: bad shapes, NULL or misaligned tensors, overlapping outputs,
    and launch tables larger than its fixed scratch are refused."""
    def call(f, **over):
        a = dict(q=f.q, ks=f.ks, vs=f.vs, o=f.o, lse=f.lse)
        a.update(over)
        return lib.cas_prefix_attn_fwd_noalloc(ctypes.byref(f.p), a["q"], a["ks"], a["vs"], a["o"],
                                               a["lse"], None)
    f = Fake()
    f.p.head_dim = 96
    assert call(f) == _lib.CAS_ERR_UNSUPPORTED
    f = Fake()
    assert call(f, q=None) == _lib.CAS_ERR_INVALID_ARGUMENT
    assert call(f, o=f.o + 8) == _lib.CAS_ERR_ALIGNMENT
    assert call(f, o=f.q) == _lib.CAS_ERR_INVALID_ARGUMENT
    assert call(f, lse=f.o) == _lib.CAS_ERR_INVALID_ARGUMENT
    # 2^25 prefix tokens: 2^19 tiles of 32 bytes = 16 MiB of tables alone.
    f = Fake(rows=((1 << 25,),), grads=False)
    assert call(f) == _lib.CAS_ERR_UNSUPPORTED
    assert "scratch" in _msg(lib)
