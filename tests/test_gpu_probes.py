"""GPU probes through the C ABI: integer-exact segment indexing and masking
(visible-count and needle probes), canary guard bands, determinism,
order invariance, concatenation equivalence, skipped gradients and error
paths. Expected values come from the definition of the operation (counts,
exact values of single keys) or from the fp64 oracle.
"""
import math

import numpy as np
import pytest

import casgen
from gpu_util import GpuCase, TOL, full_oracle, host, rel_err

pytestmark = pytest.mark.gpu

PROBE = dict(dtype="bf16", batch=2, q_len=150, num_q_heads=8, num_kv_heads=2, head_dim=128,
             cart_lens=[100, 1, 200, 64, 130], rows=[[0, 1, 2], [3, 4]],
             layouts=["tok", "padded", "head", "tok", "padded"])


def _torch():
    import torch
    return torch


def _probe_case(seed=301, **over):
    spec = dict(PROBE, **over)
    return GpuCase(casgen.custom("probe", seed=seed, cart_std=0.5, **spec))


@pytest.mark.parametrize("splits", [0, 4])
def test_visible_count(splits):
    """Q = 0 makes every visible score 0, so exp(LSE) is exactly the number of
    visible keys: the row's whole prefix plus self keys 0..t."""
    import paper_2606_04557_amd as cas
    case = _probe_case()
    case.q.zero_()
    try:
        cas.set_tuning(fwd_splits=splits)
        o, lse = case.fwd()
    finally:
        cas.set_tuning(0, 0)
    _torch().cuda.synchronize()
    wl = case.wl
    L = host(lse)
    for b in range(wl.batch):
        npre = wl.prefix_len(b)
        expected = npre + np.arange(wl.q_len) + 1
        got = np.rint(np.exp(L[b]))                         # [Hq, Sq]
        assert np.array_equal(got, np.broadcast_to(expected, got.shape)), b


def _needle_targets(wl):
    """(batch row, cartridge id or -1 for self, token) at segment starts and ends,
    64-key tile boundaries, ragged tails and around the causal diagonal."""
    out = []
    for b, row in enumerate(wl.rows):
        for c in row:
            L = wl.cart_lens[c]
            for j in sorted({0, L - 1, min(L - 1, 63), min(L - 1, 64), min(L - 1, 127), min(L - 1, 128)}):
                out.append((b, c, j))
        for j in (0, 63, 64, 100, wl.q_len - 1):
            out.append((b, -1, j))
    return out


@pytest.mark.parametrize("splits", [0, 3])
def test_needle(splits):
    """One key matches the queries with a score of 48^2 * scale ~ 204 and every other
    visible score is 0, so P is exactly 1 on that key and exactly 0 elsewhere: O equals
    the needle's value bitwise exactly for the rows that see it, and not otherwise. With
    dO in {0, 1}, dV of the needle is the exact integer count of rows that see it."""
    import paper_2606_04557_amd as cas
    torch = _torch()
    case = _probe_case(seed=302)
    wl = case.wl
    g, Hkv = wl.group_size, wl.num_kv_heads
    rng = np.random.default_rng(7)
    do_np = (rng.random((wl.batch, wl.q_len, wl.num_q_heads, wl.head_dim)) < 0.04).astype(np.float32)
    case.d_o = torch.from_numpy(do_np).to(torch.bfloat16).cuda()
    cas.set_tuning(fwd_splits=splits, dq_splits=splits)
    try:
        for (b, c, j) in _needle_targets(wl):
            case.q.zero_()
            case.q[b, :, :, 0] = 48.0
            case.k_self.zero_()
            for cc in case.k:
                case.k[cc].zero_()
            if c < 0:
                case.k_self[b, j, :, 0] = 48.0
                vstar = case.v_self[b, j]                       # [Hkv, D]
            else:
                case.k[c][j, :, 0] = 48.0
                vstar = case.v[c][j]
            o, lse = case.fwd()
            dq, dks, dvs = case.bwd(o, lse)
            torch.cuda.synchronize()
            for t in range(wl.q_len):
                visible = c >= 0 or j <= t
                for h in range(wl.num_q_heads):
                    same = torch.equal(o[b, t, h], vstar[h // g])
                    assert same == visible, (b, c, j, t, h)
            # dV of the needle: the number of (t, h) rows of its kv group that see it,
            # counted where dO = 1, channel by channel.
            dvn = dvs[b, j] if c < 0 else case.dv[c][j]
            for kv in range(Hkv):
                ts = np.arange(wl.q_len) if c >= 0 else np.arange(j, wl.q_len)
                exp = do_np[b][ts][:, kv * g:(kv + 1) * g].sum((0, 1))
                assert np.array_equal(host(dvn[kv]), exp), (b, c, j, kv)
    finally:
        cas.set_tuning(0, 0)


def _guarded(shape, dtype, guard=4096, fill=-7.25):
    torch = _torch()
    n = int(np.prod(shape))
    base = torch.full((n + 2 * guard,), fill, dtype=dtype, device="cuda")
    return base, base[guard:guard + n].view(*shape)


def test_canaries_and_determinism():
    """Guard bands around every output stay untouched, and two runs agree bitwise
    (no atomics anywhere, so every summation order is fixed)."""
    torch = _torch()
    case = _probe_case(seed=303)
    wl = case.wl
    B, Sq, Hq, Hkv, D = wl.batch, wl.q_len, wl.num_q_heads, wl.num_kv_heads, wl.head_dim
    bases = {}
    outs = {}
    for name, shape, dt in [("o", (B, Sq, Hq, D), torch.bfloat16), ("lse", (B, Hq, Sq), torch.float32),
                            ("dq", (B, Sq, Hq, D), torch.bfloat16), ("dks", (B, Sq, Hkv, D), torch.bfloat16),
                            ("dvs", (B, Sq, Hkv, D), torch.bfloat16)]:
        bases[name], outs[name] = _guarded(shape, dt)
    runs = []
    for _ in range(2):
        case.fwd(o=outs["o"], lse=outs["lse"])
        case.bwd(outs["o"], outs["lse"], dq=outs["dq"], dk_self=outs["dks"], dv_self=outs["dvs"])
        torch.cuda.synchronize()
        runs.append({k: v.clone() for k, v in outs.items()} |
                    {f"dk{c}": case.dk[c].clone() for c in case.dk} |
                    {f"dv{c}": case.dv[c].clone() for c in case.dv})
    for name, base in bases.items():
        g = 4096
        assert torch.all(base[:g] == -7.25) and torch.all(base[-g:] == -7.25), name
    for k in runs[0]:
        assert torch.equal(runs[0][k], runs[1][k]), k
    # and the results are right
    O, LSE, (rdq, *_rest) = full_oracle(case)
    assert rel_err(host(outs["o"]), O) <= TOL["bf16"]
    assert rel_err(host(outs["dq"]), rdq) <= TOL["bf16"]


@pytest.mark.parametrize("splits", [0, 4])
def test_score_spike_takes_exact_pass(splits):
    """A key late in a row whose scores sit far above everything the row saw
    first (more than 64 in log2 units) pushes the forward past its fixed
    softmax offset: the workgroup is recomputed by the exact online-softmax
    pass. O, LSE and all gradients must still match the oracle."""
    import paper_2606_04557_amd as cas
    wl = casgen.custom("probe", seed=305, cart_std=0.5, **PROBE)
    T = casgen.make_tensors(wl)
    q = casgen.to_float(T["q"], "bf16")
    # Row 0's last cartridge (id 2, 200 tokens): token 150 of every KV head is
    # aligned with query position 0 of that head's first query head, 60x its
    # unit direction, so those queries score about 60 |q| ~ 680 above zero.
    c, tok = wl.rows[0][-1], 150
    k = casgen.to_float(T["cart_k"][c], "bf16")
    for h in range(wl.num_kv_heads):
        qv = q[0, 0, h * wl.group_size]
        k[tok, h] = 60.0 * qv / np.linalg.norm(qv)
    T["cart_k"][c] = casgen.rng.f64_to_bf16_bits(k)
    spike = float(casgen.to_float(T["cart_k"][c], "bf16")[tok, 0] @ q[0, 0, 0]) * float(wl.scale)
    assert spike / math.log(2) > 64 + 20          # far beyond the margin
    case = GpuCase(wl, tensors=T)
    try:
        cas.set_tuning(fwd_splits=splits)
        o, lse = case.fwd()
    finally:
        cas.set_tuning(0, 0)
    dq, _, _ = case.bwd(o, lse)
    _torch().cuda.synchronize()
    O, LSE, (rdq, _, _, rdk, rdv) = full_oracle(case)
    assert rel_err(host(o), O) <= TOL["bf16"]
    assert float(np.abs(host(lse) - LSE).max()) <= 1e-3
    assert rel_err(host(dq), rdq) <= TOL["bf16"]
    for cc in case.dk:
        assert rel_err(host(case.dk[cc]), rdk[cc]) <= TOL["bf16"]
        assert rel_err(host(case.dv[cc]), rdv[cc]) <= TOL["bf16"]


def test_order_invariance_and_concatenation():
    """Reordering a row's cartridges, or joining them into one cartridge, leaves O, LSE
    and dQ unchanged up to rounding and moves each cartridge's gradient with it."""
    import paper_2606_04557_amd as cas
    torch = _torch()
    case = _probe_case(seed=304)
    wl = case.wl
    o, lse = case.fwd()
    dq, dks, dvs = case.bwd(o, lse)
    grads = {c: (case.dk[c].clone(), case.dv[c].clone()) for c in case.dk}
    torch.cuda.synchronize()
    # Reversed order.
    rows_rev = [list(reversed(r)) for r in case.rows]
    o2, lse2 = cas.prefix_attn_fwd(case.q, case.k_self, case.v_self, rows_rev, wl.num_kv_heads,
                                   wl.group_size, float(wl.scale))
    dq2, _, _ = cas.prefix_attn_bwd(case.q, case.k_self, case.v_self, rows_rev, wl.num_kv_heads,
                                    wl.group_size, float(wl.scale), o2, lse2, case.d_o)
    torch.cuda.synchronize()
    # Both orders are within the bf16 bar of the oracle, and of each other.
    tol = TOL["bf16"]
    O, LSE, (rdq, _, _, rdk, rdv) = full_oracle(case)
    for oo, qq in ((o, dq), (o2, dq2)):
        assert rel_err(host(oo), O) <= tol and rel_err(host(qq), rdq) <= tol
    assert rel_err(host(o2), host(o)) <= tol
    assert float((lse2 - lse).abs().max()) <= 1e-4
    assert rel_err(host(dq2), host(dq)) <= tol
    for c in case.dk:
        assert rel_err(host(case.dk[c]), rdk[c]) <= tol and rel_err(host(case.dv[c]), rdv[c]) <= tol
        assert rel_err(host(case.dk[c]), host(grads[c][0])) <= tol
        assert rel_err(host(case.dv[c]), host(grads[c][1])) <= tol
    # One joined cartridge per row.
    rows_cat, joined = [], []
    for b, row in enumerate(wl.rows):
        k = torch.cat([case.k[c] for c in row]).contiguous()
        v = torch.cat([case.v[c] for c in row]).contiguous()
        dk, dv = torch.empty_like(k), torch.empty_like(v)
        rows_cat.append([cas.Segment(k, v, dk, dv)])
        joined.append((row, dk, dv))
    o3, lse3 = cas.prefix_attn_fwd(case.q, case.k_self, case.v_self, rows_cat, wl.num_kv_heads,
                                   wl.group_size, float(wl.scale))
    cas.prefix_attn_bwd(case.q, case.k_self, case.v_self, rows_cat, wl.num_kv_heads, wl.group_size,
                        float(wl.scale), o3, lse3, case.d_o)
    torch.cuda.synchronize()
    assert rel_err(host(o3), O) <= tol and rel_err(host(o3), host(o)) <= tol
    assert float((lse3 - lse).abs().max()) <= 1e-4
    for row, dk, dv in joined:
        off = 0
        for c in row:
            L = wl.cart_lens[c]
            assert rel_err(host(dk[off:off + L]), rdk[c]) <= tol
            assert rel_err(host(dv[off:off + L]), rdv[c]) <= tol
            off += L


def test_skipped_gradients_are_untouched():
    """NULL segment gradients and a NULL dq are not written; the rest is unchanged."""
    import paper_2606_04557_amd as cas
    torch = _torch()
    case = _probe_case(seed=305)
    wl = case.wl
    o, lse = case.fwd()
    case.bwd(o, lse)
    torch.cuda.synchronize()
    ref = {c: (case.dk[c].clone(), case.dv[c].clone()) for c in case.dk}
    sentinel = torch.full_like(case.dk[0], 3.0)
    rows = []
    for r in wl.rows:
        row = []
        for c in r:
            if c == 0:
                row.append(cas.Segment(case.k[c], case.v[c], None, None))
            elif c == 3:
                row.append(cas.Segment(case.k[c], case.v[c], case.dk[c], None))
            else:
                row.append(cas.Segment(case.k[c], case.v[c], case.dk[c], case.dv[c]))
        rows.append(row)
    case.dv[3].fill_(5.0)
    for c in case.dk:
        if c not in (0, 3):
            case.dk[c].zero_()
            case.dv[c].zero_()
    dq, dks, dvs = cas.prefix_attn_bwd(case.q, case.k_self, case.v_self, rows, wl.num_kv_heads,
                                       wl.group_size, float(wl.scale), o, lse, case.d_o, want_dq=False)
    torch.cuda.synchronize()
    assert dq is None
    assert torch.all(case.dv[3] == 5.0)
    assert torch.equal(case.dk[3], ref[3][0])
    for c in case.dk:
        if c not in (0, 3):
            assert torch.equal(case.dk[c], ref[c][0]) and torch.equal(case.dv[c], ref[c][1])
    del sentinel


def test_errors_leave_outputs_untouched():
    """A too-small workspace and an output aliasing an input are rejected before
    anything is enqueued."""
    import ctypes
    import paper_2606_04557_amd as cas
    from paper_2606_04557_amd import _check
    torch = _torch()
    case = _probe_case(seed=306)
    wl = case.wl
    o = torch.full_like(case.q, 2.0)
    small = torch.empty(16, dtype=torch.uint8, device="cuda")
    prob = cas.Problem.from_tensors(case.q, case.rows, wl.num_kv_heads, wl.group_size, float(wl.scale))
    with pytest.raises(cas.CasError) as ei:
        _check(cas.load().cas_prefix_attn_fwd(ctypes.byref(prob.c), case.q.data_ptr(),
                                              case.k_self.data_ptr(), case.v_self.data_ptr(),
                                              o.data_ptr(), None, small.data_ptr(), 16,
                                              torch.cuda.current_stream().cuda_stream))
    assert "CAS_ERR_WORKSPACE" in str(ei.value)
    with pytest.raises(cas.CasError) as ei:
        cas.prefix_attn_fwd(case.q, case.k_self, case.v_self, case.rows, wl.num_kv_heads,
                            wl.group_size, float(wl.scale), o=case.q)
    assert "CAS_ERR_INVALID_ARGUMENT" in str(ei.value)
    torch.cuda.synchronize()
    assert torch.all(o == 2.0)
