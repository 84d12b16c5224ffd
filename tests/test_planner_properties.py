"""Property tests of the launch planner on random segment tables (no GPU).

Random problems go through the pure planning queries (cas_plan_info,
cas_prefix_attn_workspace_size); their counts are checked against what the
segment table defines, computed independently here:
* distinct cartridges with a gradient after folding the entries that name
  the same storage (the same cartridge used by several rows, or twice in one
  row, is one tensor whose gradient is the sum over its uses);
* dK/dV key tiles of 128 tokens over those cartridges and every row's self
  keys, once per KV head;
* bf16 forward workgroups of 256 packed query rows per (row, KV head), times
  the key-axis splits;
* the longest row prefix;
* workspace sizes as both queries report them.
Device pointers are fabricated: nothing here touches a device.
"""
import ctypes

import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

from paper_2606_04557_amd import _lib

KEY_TILE = 128      # dK/dV keys per workgroup
ROWS_PER_WG = 256   # bf16 forward / dQ packed query rows per workgroup
BASE = 1 << 36


@pytest.fixture(scope="module")
def lib():
    return _lib.load()


def ceil_div(a, b):
    return -(-a // b)


@st.composite
def problems(draw):
    B = draw(st.integers(1, 5))
    Sq = draw(st.integers(1, 600))
    Hkv = draw(st.integers(1, 4))
    g = draw(st.sampled_from([1, 2, 3, 4, 5, 8]))
    D = draw(st.sampled_from([64, 128]))
    dtype = draw(st.sampled_from([_lib.CAS_DTYPE_BF16, _lib.CAS_DTYPE_FP32]))
    rows = []
    fresh = 0
    for _ in range(B):
        ents = []
        for _ in range(draw(st.integers(0, 5))):
            earlier = [e for r in rows for e in r] + ents
            if earlier and draw(st.booleans()) and draw(st.booleans()):
                ents.append(draw(st.sampled_from(earlier)))       # an alias of an earlier entry
            else:
                L = draw(st.sampled_from([0, 1, 63, 64, 65, 127, 128, 129, 255, 256, 700, 2049]))
                grad = draw(st.sampled_from([True, True, True, False]))
                ents.append(("c%d" % fresh, L, grad))
                fresh += 1
        rows.append(ents)
    return dict(B=B, Sq=Sq, Hkv=Hkv, g=g, D=D, dtype=dtype, rows=rows)


class Built:
    """cas_problem_t over fabricated, disjoint, 16-byte aligned addresses;
    entries with the same cartridge name share every pointer."""

    def __init__(self, pr):
        es = 2 if pr["dtype"] == _lib.CAS_DTYPE_BF16 else 4
        Hkv, D = pr["Hkv"], pr["D"]
        self.next = BASE
        bufs = {}
        nent = sum(len(r) for r in pr["rows"])
        self.segs = (_lib.Segment * max(1, nent))()
        self.offs = (ctypes.c_int32 * (pr["B"] + 1))()
        i = 0
        for b, r in enumerate(pr["rows"]):
            self.offs[b] = i
            for name, L, grad in r:
                if name not in bufs:
                    n = max(1, L) * Hkv * D * es
                    bufs[name] = (self.alloc(n), self.alloc(n),
                                  self.alloc(n) if grad else None, self.alloc(n) if grad else None)
                s = self.segs[i]
                s.k, s.v, s.dk, s.dv = bufs[name]
                s.len, s.stride_tok, s.stride_head = L, Hkv * D, D
                i += 1
        self.offs[pr["B"]] = i
        self.p = _lib.Problem(pr["dtype"], pr["B"], pr["Sq"], Hkv, pr["g"], D, D ** -0.5,
                              ctypes.cast(self.segs, ctypes.POINTER(_lib.Segment)),
                              ctypes.cast(self.offs, ctypes.POINTER(ctypes.c_int32)))

    def alloc(self, n):
        a = self.next
        self.next += (n + 4095) // 4096 * 4096 + 4096
        return a


@settings(max_examples=300, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(pr=problems())
def test_plan_counts_follow_the_segment_table(lib, pr):
    info = _lib.PlanInfo()
    prob = Built(pr)
    assert lib.cas_plan_info(ctypes.byref(prob.p), ctypes.byref(info)) == _lib.CAS_OK, \
        lib.cas_last_error_message().decode()

    # Distinct cartridges with a gradient, non-empty; their tiles; the self tiles.
    carts = {}
    for r in pr["rows"]:
        for name, L, grad in r:
            if L > 0 and grad:
                carts[name] = L
    assert info.unique_segments == len(carts)
    self_tiles = pr["B"] * ceil_div(pr["Sq"], KEY_TILE)
    tiles = sum(ceil_div(L, KEY_TILE) for L in carts.values()) + self_tiles
    assert info.total_key_tiles == tiles
    assert info.dkdv_workgroups == tiles * pr["Hkv"]

    # Longest prefix of a row (every entry counts, with or without gradient).
    assert info.max_prefix_len == max(sum(L for _, L, _ in r) for r in pr["rows"])

    # bf16: one forward workgroup per 256-row block of each (row, KV head), per split.
    assert 1 <= info.fwd_splits and 1 <= info.dq_splits
    if pr["dtype"] == _lib.CAS_DTYPE_BF16:
        blocks = pr["B"] * pr["Hkv"] * ceil_div(pr["Sq"] * pr["g"], ROWS_PER_WG)
        assert info.fwd_workgroups == blocks * info.fwd_splits

    # Both workspace queries agree with the plan.
    for bwd, ref in ((0, info.ws_fwd_bytes), (1, info.ws_bwd_bytes)):
        n = ctypes.c_size_t(0)
        assert lib.cas_prefix_attn_workspace_size(ctypes.byref(prob.p), bwd, ctypes.byref(n)) == _lib.CAS_OK
        assert n.value == ref and n.value > 0
