"""Pins of the fp64 oracle against facts that do not come from the oracle.

Each test pins some part of the oracle's arithmetic to a closed form, an
invariant of softmax attention, an independent library routine (torch's fp64
attention with autograd), brute-force enumeration or central finite
differences, on tiny inputs (head_dim <= 8, <= 3 cartridges including
zero-length and single-token ones, q_len <= 5, group sizes 1 and 2).
"""
import itertools
import math

import numpy as np
import pytest

import oracle


def _problem(seed, B=2, Sq=4, Hq=2, Hkv=1, D=4, lens=(2, 0, 1), rows=((0, 1, 2), (2, 0))):
    r = np.random.default_rng(seed)
    q = r.standard_normal((B, Sq, Hq, D))
    ks = r.standard_normal((B, Sq, Hkv, D))
    vs = r.standard_normal((B, Sq, Hkv, D))
    ck = [r.standard_normal((L, Hkv, D)) for L in lens]
    cv = [r.standard_normal((L, Hkv, D)) for L in lens]
    do = r.standard_normal((B, Sq, Hq, D))
    return dict(q=q, k_self=ks, v_self=vs, cart_k=ck, cart_v=cv, rows=[list(x) for x in rows],
                scale=0.37, group_size=Hq // Hkv, d_o=do)


def _fwd(p, **over):
    a = dict(p, **over)
    return oracle.forward(a["q"], a["k_self"], a["v_self"], a["cart_k"], a["cart_v"], a["rows"],
                          a["scale"], a["group_size"])


def _bwd(p, **over):
    a = dict(p, **over)
    return oracle.backward(a["q"], a["k_self"], a["v_self"], a["cart_k"], a["cart_v"], a["rows"],
                           a["scale"], a["group_size"], a["d_o"])


PROBLEMS = [
    dict(seed=1),
    dict(seed=2, Hq=2, Hkv=2),                                        # g = 1
    dict(seed=3, Hq=4, Hkv=2, lens=(3, 1), rows=((0, 1), (1, 1, 0))),  # alias inside a row
    dict(seed=4, B=1, Sq=5, lens=(), rows=((),)),                     # no cartridges
    dict(seed=5, B=1, Sq=1, lens=(1,), rows=((0,),)),
]


@pytest.mark.parametrize("spec", PROBLEMS)
def test_p1_finite_differences(spec):
    """P1: the backward equals central differences of L = sum(dO * O) for every input element."""
    p = _problem(**spec)
    dq, dks, dvs, dck, dcv = _bwd(p)

    def loss(**over):
        O, _ = _fwd(p, **over)
        return float((p["d_o"] * O).sum())

    h = 1e-5

    def fd(name, arr, idx=None):
        out = np.zeros_like(arr)
        for ix in itertools.product(*[range(n) for n in arr.shape]):
            a1 = arr.copy(); a1[ix] += h
            a2 = arr.copy(); a2[ix] -= h
            if idx is None:
                out[ix] = (loss(**{name: a1}) - loss(**{name: a2})) / (2 * h)
            else:
                l1 = list(p[name]); l1[idx] = a1
                l2 = list(p[name]); l2[idx] = a2
                out[ix] = (loss(**{name: l1}) - loss(**{name: l2})) / (2 * h)
        return out

    def close(a, b):
        den = max(np.abs(b).max(), 1e-12)
        assert np.abs(a - b).max() / den <= 1e-7, (np.abs(a - b).max(), den)

    close(dq, fd("q", p["q"]))
    close(dks, fd("k_self", p["k_self"]))
    close(dvs, fd("v_self", p["v_self"]))
    for c in range(len(p["cart_k"])):
        if p["cart_k"][c].shape[0] == 0:
            continue
        close(dck[c], fd("cart_k", p["cart_k"][c], c))
        close(dcv[c], fd("cart_v", p["cart_v"][c], c))


def _visible_lists(p, b, t):
    """Brute-force enumeration of the keys (cartridge id or -1 for self, token) seen by
    query t of row b, in prefix order."""
    out = []
    for c in p["rows"][b]:
        for j in range(p["cart_k"][c].shape[0]):
            out.append((c, j))
    for j in range(t + 1):
        out.append((-1, j))
    return out


@pytest.mark.parametrize("spec", PROBLEMS)
def test_p2_equal_scores_closed_form(spec):
    """P2: with Q = 0 every visible score is 0, so O is the mean of the visible
    values, LSE = ln(n_visible) and dV_j = sum over rows seeing j of dO / n_visible."""
    p = _problem(**spec)
    p["q"] = np.zeros_like(p["q"])
    O, LSE = _fwd(p)
    dq, dks, dvs, dck, dcv = _bwd(p)
    B, Sq, Hq, D = p["q"].shape
    g = p["group_size"]
    exp_dv_self = np.zeros_like(p["v_self"])
    exp_dv_cart = [np.zeros_like(v) for v in p["cart_v"]]
    for b in range(B):
        for h in range(Hq):
            kv = h // g
            for t in range(Sq):
                keys = _visible_lists(p, b, t)
                n = len(keys)
                acc = np.zeros(D)
                for c, j in keys:
                    acc += (p["v_self"][b, j, kv] if c < 0 else p["cart_v"][c][j, kv])
                assert np.allclose(O[b, t, h], acc / n, rtol=0, atol=1e-13)
                assert abs(LSE[b, h, t] - math.log(n)) <= 1e-13
                for c, j in keys:
                    tgt = exp_dv_self[b, j, kv] if c < 0 else exp_dv_cart[c][j, kv]
                    tgt += p["d_o"][b, t, h] / n
    assert np.allclose(dvs, exp_dv_self, rtol=0, atol=1e-12)
    for c in range(len(p["cart_v"])):
        if dcv[c] is not None:
            assert np.allclose(dcv[c], exp_dv_cart[c], rtol=0, atol=1e-12)


def test_p2_equal_keys_zero_dq():
    """P2: when every visible key is the same vector the scores are equal, O is the mean
    of V and dQ vanishes (sum_j dS_j = 0 and all k_j equal)."""
    p = _problem(7)
    kvec = np.array([0.3, -1.2, 0.8, 2.0])
    p["k_self"] = np.broadcast_to(kvec, p["k_self"].shape).copy()
    p["cart_k"] = [np.broadcast_to(kvec, k.shape).copy() for k in p["cart_k"]]
    dq, *_ = _bwd(p)
    assert np.abs(dq).max() <= 1e-13


@pytest.mark.parametrize("spec", PROBLEMS[:3])
def test_p3_concat_equivalence(spec):
    """P3: a row's cartridges [A, B, C] give the same results as one cartridge A||B||C,
    and the joined cartridge's gradient is the per-cartridge gradients side by side."""
    p = _problem(**spec)
    O, LSE = _fwd(p)
    dq, dks, dvs, dck, dcv = _bwd(p)
    # Build a problem where each row has one joined cartridge of its own.
    ck2, cv2, rows2 = [], [], []
    for b, row in enumerate(p["rows"]):
        ck2.append(np.concatenate([p["cart_k"][c] for c in row] + [np.zeros((0,) + p["k_self"].shape[2:])]))
        cv2.append(np.concatenate([p["cart_v"][c] for c in row] + [np.zeros((0,) + p["v_self"].shape[2:])]))
        rows2.append([b])
    O2, LSE2 = _fwd(p, cart_k=ck2, cart_v=cv2, rows=rows2)
    dq2, dks2, dvs2, dck2, dcv2 = _bwd(p, cart_k=ck2, cart_v=cv2, rows=rows2)
    assert np.allclose(O, O2, rtol=0, atol=1e-13)
    assert np.allclose(LSE, LSE2, rtol=0, atol=1e-13)
    assert np.allclose(dq, dq2, rtol=0, atol=1e-13)
    assert np.allclose(dks, dks2, rtol=0, atol=1e-13)
    assert np.allclose(dvs, dvs2, rtol=0, atol=1e-13)
    # Summing the joined gradient back per cartridge reproduces the aliased sums.
    sk = [np.zeros_like(k) for k in p["cart_k"]]
    sv = [np.zeros_like(v) for v in p["cart_v"]]
    for b, row in enumerate(p["rows"]):
        off = 0
        for c in row:
            L = p["cart_k"][c].shape[0]
            sk[c] += dck2[b][off:off + L]
            sv[c] += dcv2[b][off:off + L]
            off += L
    for c in range(len(p["cart_k"])):
        if dck[c] is not None:
            assert np.allclose(dck[c], sk[c], rtol=0, atol=1e-13)
            assert np.allclose(dcv[c], sv[c], rtol=0, atol=1e-13)


def test_p4_permutation_invariance():
    """P4: reordering a row's cartridges leaves O, LSE and dQ unchanged and moves each
    cartridge's gradient with it (keys arrive post-RoPE, so order carries no position)."""
    p = _problem(11, B=1, Sq=5, Hq=4, Hkv=2, D=6, lens=(3, 1, 2), rows=((0, 1, 2),))
    base = _bwd(p)
    O, LSE = _fwd(p)
    for perm in itertools.permutations([0, 1, 2]):
        rows = [list(perm)]
        O2, LSE2 = _fwd(p, rows=rows)
        out = _bwd(p, rows=rows)
        assert np.abs(O - O2).max() <= 1e-13
        assert np.abs(LSE - LSE2).max() <= 1e-13
        assert np.abs(base[0] - out[0]).max() <= 1e-13
        for c in range(3):
            assert np.abs(base[3][c] - out[3][c]).max() <= 1e-13
            assert np.abs(base[4][c] - out[4][c]).max() <= 1e-13


@pytest.mark.parametrize("spec", PROBLEMS)
def test_p5_torch_fp64_reference(spec):
    """P5: equals torch's fp64 scaled-dot-product attention over the explicitly
    concatenated keys with a boolean visibility mask, differentiated by autograd."""
    torch = pytest.importorskip("torch")
    F = torch.nn.functional
    p = _problem(**spec)
    O, LSE = _fwd(p)
    dq, dks, dvs, dck, dcv = _bwd(p)
    B, Sq, Hq, D = p["q"].shape
    g = p["group_size"]
    tq = torch.tensor(p["q"], requires_grad=True)
    tks = torch.tensor(p["k_self"], requires_grad=True)
    tvs = torch.tensor(p["v_self"], requires_grad=True)
    tck = [torch.tensor(k, requires_grad=True) for k in p["cart_k"]]
    tcv = [torch.tensor(v, requires_grad=True) for v in p["cart_v"]]
    outs, lses = [], []
    for b in range(B):
        K = torch.cat([tck[c] for c in p["rows"][b]] + [tks[b]], dim=0)   # [N, Hkv, D]
        V = torch.cat([tcv[c] for c in p["rows"][b]] + [tvs[b]], dim=0)
        npre = K.shape[0] - Sq
        mask = torch.ones(Sq, K.shape[0], dtype=torch.bool)
        mask[:, npre:] = torch.tril(torch.ones(Sq, Sq, dtype=torch.bool))
        Kh = K.permute(1, 0, 2).repeat_interleave(g, dim=0)              # [Hq, N, D]
        Vh = V.permute(1, 0, 2).repeat_interleave(g, dim=0)
        Qh = tq[b].permute(1, 0, 2)                                      # [Hq, Sq, D]
        o = F.scaled_dot_product_attention(Qh, Kh, Vh, attn_mask=mask, scale=p["scale"])
        outs.append(o.permute(1, 0, 2))
        s = (Qh @ Kh.transpose(1, 2)) * p["scale"]
        lses.append(torch.logsumexp(s.masked_fill(~mask, float("-inf")), dim=-1))
    tO = torch.stack(outs)
    tO.backward(torch.tensor(p["d_o"]))
    assert np.abs(O - tO.detach().numpy()).max() <= 1e-12
    assert np.abs(LSE - torch.stack(lses).detach().numpy()).max() <= 1e-12
    assert np.abs(dq - tq.grad.numpy()).max() <= 1e-12
    assert np.abs(dks - tks.grad.numpy()).max() <= 1e-12
    assert np.abs(dvs - tvs.grad.numpy()).max() <= 1e-12
    for c in range(len(p["cart_k"])):
        if dck[c] is None or p["cart_k"][c].shape[0] == 0:
            continue
        assert np.abs(dck[c] - tck[c].grad.numpy()).max() <= 1e-12
        assert np.abs(dcv[c] - tcv[c].grad.numpy()).max() <= 1e-12


def test_p6_single_visible_key():
    """P6: one row, no cartridges, one query: the only visible key is the query's own,
    so O = v_0, dQ = 0, dK = 0 and dV = dO summed over the group's heads."""
    p = _problem(13, B=1, Sq=1, Hq=2, Hkv=1, D=5, lens=(), rows=((),))
    O, LSE = _fwd(p)
    dq, dks, dvs, _, _ = _bwd(p)
    assert np.array_equal(O[0, 0, 0], p["v_self"][0, 0, 0])
    assert np.array_equal(O[0, 0, 1], p["v_self"][0, 0, 0])
    # dQ and dK are P (dP - D) with P = 1 and dP = D up to summation order.
    assert np.abs(dq).max() <= 1e-14
    assert np.abs(dks).max() <= 1e-14
    assert np.allclose(dvs[0, 0, 0], p["d_o"][0, 0, 0] + p["d_o"][0, 0, 1], rtol=0, atol=1e-15)


def test_p7_gradient_bookkeeping():
    """P7: per (row, KV head) with no cartridge shared between rows, the dV rows sum to
    the sum of dO over the group's queries (sum_j P_j = 1) and the dK rows sum to zero
    (sum_j dS_j = 0)."""
    p = _problem(17, B=2, Sq=5, Hq=4, Hkv=2, D=3, lens=(2, 3, 1, 0), rows=((0, 1), (2, 3)))
    dq, dks, dvs, dck, dcv = _bwd(p)
    g = p["group_size"]
    for b in range(2):
        for kv in range(2):
            sv = dvs[b, :, kv].sum(0) + sum(dcv[c][:, kv].sum(0) for c in p["rows"][b])
            sk = dks[b, :, kv].sum(0) + sum(dck[c][:, kv].sum(0) for c in p["rows"][b])
            exp = p["d_o"][b, :, kv * g:(kv + 1) * g].sum((0, 1))
            assert np.abs(sv - exp).max() <= 1e-13
            assert np.abs(sk).max() <= 1e-13


def test_p8_key_shift_invariance():
    """P8: adding one vector c to every key leaves O and all gradients unchanged and
    shifts LSE by scale * q . c."""
    p = _problem(19, B=1, Sq=4, Hq=2, Hkv=1, D=4, lens=(3, 2), rows=((0, 1),))
    c = np.array([0.5, -0.25, 1.5, 0.75])
    O, LSE = _fwd(p)
    b1 = _bwd(p)
    ks2 = p["k_self"] + c
    ck2 = [k + c for k in p["cart_k"]]
    O2, LSE2 = _fwd(p, k_self=ks2, cart_k=ck2)
    b2 = _bwd(p, k_self=ks2, cart_k=ck2)
    assert np.abs(O - O2).max() <= 1e-12
    shift = p["scale"] * np.einsum("bthd,d->bht", p["q"], c)
    assert np.abs(LSE2 - LSE - shift).max() <= 1e-12
    for a, b in zip(b1[:3], b2[:3]):
        assert np.abs(a - b).max() <= 1e-12
    for a, b in zip(b1[3] + b1[4], b2[3] + b2[4]):
        assert np.abs(a - b).max() <= 1e-12


def test_p9_linearity_in_v():
    """P9: O is linear in the values: O(V1 + V2) = O(V1) + O(V2)."""
    p1 = _problem(23)
    p2 = _problem(29)
    O1, _ = _fwd(p1)
    O2, _ = _fwd(p1, v_self=p2["v_self"], cart_v=p2["cart_v"])
    O3, _ = _fwd(p1, v_self=p1["v_self"] + p2["v_self"],
                 cart_v=[a + b for a, b in zip(p1["cart_v"], p2["cart_v"])])
    assert np.abs(O1 + O2 - O3).max() <= 1e-13


def test_p10_visible_count_and_needle():
    """P10: with Q = 0, exp(LSE) is the exact number of visible keys; a single large
    matching score (needle) makes O equal that key's value exactly when it is visible."""
    p = _problem(31, B=2, Sq=5, Hq=2, Hkv=1, D=4, lens=(3, 0, 2), rows=((0, 1, 2), (2,)))
    p["q"] = np.zeros_like(p["q"])
    _, LSE = _fwd(p)
    for b in range(2):
        npre = sum(p["cart_k"][c].shape[0] for c in p["rows"][b])
        for t in range(5):
            assert round(math.exp(LSE[b, 0, t])) == npre + t + 1
    # Needles: every key component zero except one key per probe.
    scale = 1.0 / math.sqrt(128.0)
    for (b, key) in [(0, (0, 0)), (0, (2, 1)), (0, (-1, 0)), (0, (-1, 3)), (1, (2, 0)), (1, (-1, 4))]:
        q = np.zeros_like(p["q"]); q[b, :, :, 0] = 48.0
        ks = np.zeros_like(p["k_self"])
        ck = [np.zeros_like(k) for k in p["cart_k"]]
        c, j = key
        if c < 0:
            ks[b, j, 0, 0] = 48.0
            vstar = p["v_self"][b, j, 0]
        else:
            ck[c][j, 0, 0] = 48.0
            vstar = p["cart_v"][c][j, 0]
        O, _ = _fwd(p, q=q, k_self=ks, cart_k=ck, scale=scale)
        for t in range(5):
            visible = c >= 0 or j <= t
            hit = np.allclose(O[b, t, 0], vstar, rtol=0, atol=1e-12)
            assert hit == visible, (b, key, t)


def test_p11_brute_force_enumeration():
    """P11: scalar loops over the brute-force visible-key list (math.exp, no matrices)
    reproduce the oracle's O and LSE."""
    p = _problem(37, B=2, Sq=4, Hq=4, Hkv=2, D=3, lens=(2, 0, 1), rows=((0, 1, 2), (2, 0, 2)))
    O, LSE = _fwd(p)
    B, Sq, Hq, D = p["q"].shape
    g = p["group_size"]
    for b, h, t in itertools.product(range(B), range(Hq), range(Sq)):
        kv = h // g
        keys = _visible_lists(p, b, t)
        scores = []
        for c, j in keys:
            k = p["k_self"][b, j, kv] if c < 0 else p["cart_k"][c][j, kv]
            scores.append(p["scale"] * sum(p["q"][b, t, h, i] * k[i] for i in range(D)))
        m = max(scores)
        l = sum(math.exp(s - m) for s in scores)
        lse = m + math.log(l)
        o = [0.0] * D
        for (c, j), s in zip(keys, scores):
            v = p["v_self"][b, j, kv] if c < 0 else p["cart_v"][c][j, kv]
            w = math.exp(s - lse)
            for i in range(D):
                o[i] += w * v[i]
        assert abs(lse - LSE[b, h, t]) <= 1e-13
        assert np.abs(np.array(o) - O[b, t, h]).max() <= 1e-13


def test_sampled_paths_match_full():
    """The sampled row and key-column evaluations equal the full evaluation."""
    p = _problem(41, B=2, Sq=5, Hq=4, Hkv=2, D=3, lens=(2, 3, 1), rows=((0, 1, 0), (2, 1)))
    O, LSE = _fwd(p)
    dq, dks, dvs, dck, dcv = _bwd(p)
    args = (p["q"], p["k_self"], p["v_self"], p["cart_k"], p["cart_v"], p["rows"], p["scale"],
            p["group_size"])
    o, lse, dqs = oracle.rows_forward_backward(*args, b=1, h=3, t_idx=[0, 2, 4], d_o=p["d_o"])
    assert np.abs(o - O[1, [0, 2, 4], 3]).max() <= 1e-13
    assert np.abs(lse - LSE[1, 3, [0, 2, 4]]).max() <= 1e-13
    assert np.abs(dqs - dq[1, [0, 2, 4], 3]).max() <= 1e-13
    for cart, toks in [(0, [0, 1]), (1, [2, 0]), (2, [0]), (-1, [0, 3, 4]), (-2, [1])]:
        for kv in range(2):
            dk, dv = oracle.key_grads(*args, p["d_o"], kv=kv, cart=cart, tok_idx=toks)
            if cart >= 0:
                ek, ev = dck[cart][toks, kv], dcv[cart][toks, kv]
            else:
                ek, ev = dks[-cart - 1, toks, kv], dvs[-cart - 1, toks, kv]
            assert np.abs(dk - ek).max() <= 1e-13
            assert np.abs(dv - ev).max() <= 1e-13


def test_key_grads_many_matches_full():
    """key_grads_many against the full backward: several targets per call, one
    cartridge named by two targets, a cartridge referenced by every row and
    twice within one row, a cartridge used by one row only, zero-length and
    one-token cartridges, and self targets of every row, on each KV head."""
    p = _problem(43, B=3, Sq=5, Hq=4, Hkv=2, D=3, lens=(3, 2, 0, 1, 4),
                 rows=((0, 1, 0), (2, 0, 3), (4, 0, 1)))
    dq, dks, dvs, dck, dcv = _bwd(p)
    args = (p["q"], p["k_self"], p["v_self"], p["cart_k"], p["cart_v"], p["rows"], p["scale"],
            p["group_size"])
    targets = [(0, [2, 0, 1]), (1, [1]), (0, [1]), (3, [0]), (4, [3, 0, 2]), (2, []),
               (-1, [4, 0]), (-2, [0, 1, 2, 3, 4]), (-3, [2])]
    for kv in range(2):
        res = oracle.key_grads_many(*args, p["d_o"], kv=kv, targets=targets)
        assert len(res) == len(targets)
        for (cart, toks), (dk, dv) in zip(targets, res):
            if cart >= 0:
                ek, ev = dck[cart][toks, kv], dcv[cart][toks, kv]
            else:
                ek, ev = dks[-cart - 1, toks, kv], dvs[-cart - 1, toks, kv]
            assert dk.shape == ek.shape and dv.shape == ev.shape
            assert np.abs(dk - ek).max(initial=0) <= 1e-13, (kv, cart, toks)
            assert np.abs(dv - ev).max(initial=0) <= 1e-13, (kv, cart, toks)


def test_kv_head_restriction_matches_full():
    """forward/backward restricted to some KV heads equal the full evaluation
    on those heads' outputs and leave every other head at zero."""
    p = _problem(47, B=2, Sq=4, Hq=6, Hkv=3, D=3, lens=(2, 3), rows=((0, 1), (1, 0, 1)))
    O, LSE = _fwd(p)
    full = _bwd(p)
    args = (p["q"], p["k_self"], p["v_self"], p["cart_k"], p["cart_v"], p["rows"], p["scale"],
            p["group_size"])
    for sel in ([0], [2], [0, 2]):
        Or, Lr = oracle.forward(*args, kv_heads=sel)
        part = oracle.backward(*args, p["d_o"], kv_heads=sel)
        qh = [h for h in range(6) if h // 2 in sel]
        qo = [h for h in range(6) if h // 2 not in sel]
        ko = [k for k in range(3) if k not in sel]
        assert np.array_equal(Or[:, :, qh], O[:, :, qh]) and not Or[:, :, qo].any()
        assert np.array_equal(Lr[:, qh], LSE[:, qh]) and not Lr[:, qo].any()
        assert np.abs(part[0][:, :, qh] - full[0][:, :, qh]).max() <= 1e-13
        assert not part[0][:, :, qo].any()
        for i in (1, 2):
            assert np.abs(part[i][:, :, sel] - full[i][:, :, sel]).max() <= 1e-13
            assert not part[i][:, :, ko].any()
        for i in (3, 4):
            for c in range(2):
                assert np.abs(part[i][c][:, sel] - full[i][c][:, sel]).max() <= 1e-13
                assert not part[i][c][:, ko].any()


# ---------------------------------------------------------------------------
# Packed samples (one token axis, per-sample cartridges, block-diagonal self).
# ---------------------------------------------------------------------------

def _packed_problem(seed, q_lens=(3, 0, 2, 1), Hq=2, Hkv=1, D=4, lens=(2, 1, 3),
                    rows=((0, 1), (2,), (1, 1, 0), ())):
    r = np.random.default_rng(seed)
    T = sum(q_lens)
    qo = [0] + list(np.cumsum(q_lens))
    return dict(q=r.standard_normal((T, Hq, D)), k_self=r.standard_normal((T, Hkv, D)),
                v_self=r.standard_normal((T, Hkv, D)),
                cart_k=[r.standard_normal((L, Hkv, D)) for L in lens],
                cart_v=[r.standard_normal((L, Hkv, D)) for L in lens],
                rows=[list(x) for x in rows], q_offsets=qo, scale=0.41, group_size=Hq // Hkv,
                d_o=r.standard_normal((T, Hq, D)))


def _pfwd(p, **over):
    a = dict(p, **over)
    return oracle.packed_forward(a["q"], a["k_self"], a["v_self"], a["cart_k"], a["cart_v"], a["rows"],
                                 a["q_offsets"], a["scale"], a["group_size"])


def test_p12_packed_finite_differences():
    """P12: the packed backward equals central differences of sum(dO * O) for
    every input element, with a cartridge shared by two samples (and twice in
    one), an empty sample whose cartridge no one else uses, and a sample with
    no cartridge."""
    p = _packed_problem(12)
    dq, dks, dvs, dck, dcv = oracle.packed_backward(
        p["q"], p["k_self"], p["v_self"], p["cart_k"], p["cart_v"], p["rows"], p["q_offsets"],
        p["scale"], p["group_size"], p["d_o"])

    def loss(**over):
        O, _ = _pfwd(p, **over)
        return float((p["d_o"] * O).sum())

    h = 1e-5

    def fd(name, arr, idx=None):
        out = np.zeros_like(arr)
        for ix in itertools.product(*[range(n) for n in arr.shape]):
            a1 = arr.copy(); a1[ix] += h
            a2 = arr.copy(); a2[ix] -= h
            if idx is None:
                out[ix] = (loss(**{name: a1}) - loss(**{name: a2})) / (2 * h)
            else:
                l1 = list(p[name]); l1[idx] = a1
                l2 = list(p[name]); l2[idx] = a2
                out[ix] = (loss(**{name: l1}) - loss(**{name: l2})) / (2 * h)
        return out

    def close(a, b):
        den = max(np.abs(b).max(), 1e-12)
        assert np.abs(a - b).max() / den <= 1e-7, (np.abs(a - b).max(), den)

    close(dq, fd("q", p["q"]))
    close(dks, fd("k_self", p["k_self"]))
    close(dvs, fd("v_self", p["v_self"]))
    for c in range(len(p["cart_k"])):
        close(dck[c], fd("cart_k", p["cart_k"][c], c))
        close(dcv[c], fd("cart_v", p["cart_v"][c], c))
    # Cartridge 2 is seen only by the empty sample: no gradient at all.
    assert not dck[2].any() and not dcv[2].any()


def test_p13_packed_block_diagonal_and_fixed_layout():
    """P13: (a) a sample's outputs ignore every other sample's tokens
    (block-diagonal self); (b) equal-length packed samples are the
    fixed-length batch, with LSE laid out [Hq, T] instead of [B, Hq, Sq]."""
    p = _packed_problem(13, q_lens=(3, 2), rows=((0, 2), (1,)))
    O, LSE = _pfwd(p)
    q2, k2 = p["q"].copy(), p["k_self"].copy()
    q2[3:] += 5.0
    k2[3:] -= 3.0
    O2, LSE2 = _pfwd(p, q=q2, k_self=k2)
    assert np.array_equal(O[:3], O2[:3]) and np.array_equal(LSE[:, :3], LSE2[:, :3])
    assert not np.allclose(O[3:], O2[3:])
    f = _packed_problem(14, q_lens=(2, 2, 2), rows=((0,), (1, 0), ()))
    Of, LSEf = oracle.forward(f["q"].reshape(3, 2, 2, 4), f["k_self"].reshape(3, 2, 1, 4),
                              f["v_self"].reshape(3, 2, 1, 4), f["cart_k"], f["cart_v"], f["rows"],
                              f["scale"], f["group_size"])
    Op, LSEp = _pfwd(f)
    assert np.allclose(Op, Of.reshape(6, 2, 4), rtol=0, atol=1e-14)
    assert np.allclose(LSEp, LSEf.transpose(1, 0, 2).reshape(2, 6), rtol=0, atol=1e-14)


def test_packed_sampled_paths_match_full():
    """packed_rows_forward_backward at every (sample, head, position) and
    packed_key_grads_many for every cartridge (one shared by two samples and
    referenced twice by one, one seen only by an empty sample) and for the
    self keys of every sample, against packed_forward / packed_backward."""
    p = _packed_problem(15, q_lens=(3, 0, 2, 1), Hq=4, Hkv=2)
    args = (p["q"], p["k_self"], p["v_self"], p["cart_k"], p["cart_v"], p["rows"], p["q_offsets"],
            p["scale"], p["group_size"])
    O, LSE = oracle.packed_forward(*args)
    dq, dks, dvs, dck, dcv = oracle.packed_backward(*args, p["d_o"])
    qo = p["q_offsets"]
    for b in range(len(p["rows"])):
        n = qo[b + 1] - qo[b]
        for h in range(4):
            if n == 0:
                continue
            t_idx = list(range(n))[::-1]
            o, lse, d = oracle.packed_rows_forward_backward(*args, b, h, t_idx, p["d_o"])
            glob = [qo[b] + t for t in t_idx]
            assert np.abs(o - O[glob, h]).max() <= 1e-13
            assert np.abs(lse - LSE[h, glob]).max() <= 1e-13
            assert np.abs(d - dq[glob, h]).max() <= 1e-13
    targets = [(0, [1, 0]), (1, [0]), (2, [2, 0]), (0, [1]), (-1, [2, 0, 1]), (-3, [1, 0]),
               (-4, [0])]
    for kv in range(2):
        res = oracle.packed_key_grads_many(*args, p["d_o"], kv, targets)
        for (cart, toks), (dk, dv) in zip(targets, res):
            if cart >= 0:
                ek, ev = dck[cart][toks, kv], dcv[cart][toks, kv]
            else:
                glob = [qo[-cart - 1] + t for t in toks]
                ek, ev = dks[glob, kv], dvs[glob, kv]
            assert np.abs(dk - ek).max() <= 1e-13, (kv, cart, toks)
            assert np.abs(dv - ev).max() <= 1e-13, (kv, cart, toks)
    # Cartridge 2 belongs to the empty sample only: its gradient is exactly zero.
    assert not dck[2].any()


# ---------------------------------------------------------------------------
# Paged decode (requests over page lists; the last n keys are the new tokens).
# ---------------------------------------------------------------------------

def _paged_problem(seed, P=4, npages=9, Hq=4, Hkv=2, D=4, reqs=((9, 1), (4, 3), (12, 2))):
    r = np.random.default_rng(seed)
    kp = r.standard_normal((npages, P, Hkv, D))
    vp = r.standard_normal((npages, P, Hkv, D))
    kv_lens = [L for L, _ in reqs]
    q_counts = [n for _, n in reqs]
    pages = [list(r.permutation(npages)[: -(-L // P)]) for L in kv_lens]
    q = r.standard_normal((sum(q_counts), Hq, D))
    return q, kp, vp, q_counts, kv_lens, pages


def test_p14_paged_decode_equals_prefix_plus_self():
    """P14: each request equals the fixed-layout problem whose single cartridge
    is its first L - n gathered keys and whose self tokens are the last n."""
    q, kp, vp, qc, kl, pages = _paged_problem(14)
    O, LSE = oracle.paged_decode_forward(q, kp, vp, qc, kl, pages, 0.45, 2)
    q0 = 0
    for b, n in enumerate(qc):
        K = np.concatenate([kp[p] for p in pages[b]])[: kl[b]]
        V = np.concatenate([vp[p] for p in pages[b]])[: kl[b]]
        L = kl[b]
        Of, LSEf = oracle.forward(q[None, q0:q0 + n], K[None, L - n:], V[None, L - n:], [K[: L - n]],
                                  [V[: L - n]], [[0]], 0.45, 2)
        assert np.allclose(O[q0:q0 + n], Of[0], rtol=0, atol=1e-14)
        assert np.allclose(LSE[:, q0:q0 + n], LSEf[0], rtol=0, atol=1e-14)
        q0 += n


def test_p15_paged_decode_brute_force():
    """P15: scalar loops over the keys each query sees, with math.exp."""
    q, kp, vp, qc, kl, pages = _paged_problem(15, P=2, npages=7, reqs=((5, 2), (3, 1)))
    O, LSE = oracle.paged_decode_forward(q, kp, vp, qc, kl, pages, 0.8, 2)
    q0 = 0
    for b, n in enumerate(qc):
        keys = [(p, j) for p in pages[b] for j in range(kp.shape[1])][: kl[b]]
        for i in range(n):
            for h in range(q.shape[1]):
                kv = h // 2
                vis = keys[: kl[b] - n + i + 1]
                s = [0.8 * sum(q[q0 + i, h, d] * kp[p, j, kv, d] for d in range(q.shape[2])) for p, j in vis]
                m = max(s)
                z = sum(math.exp(x - m) for x in s)
                assert abs(LSE[h, q0 + i] - (m + math.log(z))) < 1e-12
                for d in range(q.shape[2]):
                    ref = sum(math.exp(x - m) / z * vp[p, j, kv, d] for x, (p, j) in zip(s, vis))
                    assert abs(O[q0 + i, h, d] - ref) < 1e-12
        q0 += n
