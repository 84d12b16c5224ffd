"""GPU parity: libcas (through the C ABI) against the fp64 oracle on the same
seeded input bits.

Bars: max |gpu - oracle| / max |oracle| <= 1e-5 for fp32 inputs and <= 2e-2
for bf16 inputs, per output tensor (per cartridge for dK/dV); LSE absolute
error <= 1e-5 (fp32) / 1e-3 (bf16). Small cases and the 4 x 1024-cartridge
configuration compare every element; the 16 x 2048 and ragged 64-cartridge
configurations compare two whole KV heads element by element, plus sampled
rows and tile-edge keys on the other heads and whole-tensor properties.
"""
import numpy as np
import pytest

import casgen
import oracle
from gpu_util import GpuCase, LSE_TOL, TOL, full_oracle, host, rel_err

pytestmark = pytest.mark.gpu


def _sync():
    import torch
    torch.cuda.synchronize()


def _check_full(case, label=""):
    import torch
    wl = case.wl
    o, lse = case.fwd()
    dq, dks, dvs = case.bwd(o, lse)
    _sync()
    O, LSE, (rdq, rdks, rdvs, rdck, rdcv) = full_oracle(case)
    tol = TOL[wl.dtype]
    errs = {
        "o": rel_err(host(o), O),
        "lse": float(np.abs(host(lse) - LSE).max()),
        "dq": rel_err(host(dq), rdq),
        "dk_self": rel_err(host(dks), rdks),
        "dv_self": rel_err(host(dvs), rdvs),
    }
    for c in case.dk:
        errs[f"dk[{c}]"] = rel_err(host(case.dk[c]), rdck[c])
        errs[f"dv[{c}]"] = rel_err(host(case.dv[c]), rdcv[c])
    print(label, {k: f"{v:.2e}" for k, v in errs.items()})
    for k, v in errs.items():
        lim = LSE_TOL[wl.dtype] if k == "lse" else tol
        assert v <= lim, (label, k, v, errs)
    # Padding between tokens of padded-stride gradients is never written.
    for (kind, c), base in case.bases.items():
        if base.dim() == 2 and base.shape[1] > wl.num_kv_heads * wl.head_dim:
            assert torch.isnan(base[:, wl.num_kv_heads * wl.head_dim:].float()).all(), (kind, c)
    return o, lse, (dq, dks, dvs)


def test_c1_fp32_full():
    """The tiny fp32 configuration, every output element."""
    _check_full(GpuCase(casgen.config(1)), "C1")


def test_c1_fp32_forced_splits():
    import paper_2606_04557_amd as cas
    try:
        cas.set_tuning(fwd_splits=3, dq_splits=2)
        _check_full(GpuCase(casgen.config(1)), "C1 split")
    finally:
        cas.set_tuning(0, 0)


SMALL = [
    # ragged cartridge tails, a zero-length and a one-token cartridge, mixed layouts, 2.3 q-blocks
    dict(name="ragged", dtype="bf16", batch=2, q_len=150, num_q_heads=8, num_kv_heads=2,
         head_dim=128, cart_lens=[100, 0, 1, 64, 130, 257], rows=[[0, 1, 2], [3, 4, 5]],
         layouts=["tok", "tok", "padded", "head", "padded", "head"]),
    dict(name="d64_g1", dtype="bf16", batch=1, q_len=70, num_q_heads=4, num_kv_heads=4,
         head_dim=64, cart_lens=[33, 64], rows=[[0, 1]]),
    dict(name="g3", dtype="bf16", batch=1, q_len=90, num_q_heads=6, num_kv_heads=2, head_dim=128,
         cart_lens=[200], rows=[[0]]),
    # one cartridge referenced by every row, twice in the last one
    dict(name="alias", dtype="bf16", batch=3, q_len=40, num_q_heads=4, num_kv_heads=1,
         head_dim=128, cart_lens=[70, 129], rows=[[0, 1], [1, 0], [0, 0]]),
    dict(name="no_prefix", dtype="bf16", batch=2, q_len=257, num_q_heads=4, num_kv_heads=2,
         head_dim=128, cart_lens=[], rows=[[], []]),
    # GQA groups of 8 and 16 (a 64-row block starts on a position boundary)
    # and of 5 (it does not), with d = 64 and 128
    dict(name="g8_d64", dtype="bf16", batch=1, q_len=100, num_q_heads=16, num_kv_heads=2,
         head_dim=64, cart_lens=[150, 77], rows=[[0, 1]], layouts=["padded", "head"]),
    dict(name="g16", dtype="bf16", batch=2, q_len=50, num_q_heads=16, num_kv_heads=1,
         head_dim=128, cart_lens=[300, 65], rows=[[0], [1, 0]]),
    dict(name="g5_d64", dtype="bf16", batch=1, q_len=45, num_q_heads=10, num_kv_heads=2,
         head_dim=64, cart_lens=[90, 40], rows=[[1, 0]]),
    # one query per row: a single 4-row block per (row, KV head) against a
    # long prefix (the planner splits the key axis), and rows with no prefix
    dict(name="q1_long", dtype="bf16", batch=2, q_len=1, num_q_heads=8, num_kv_heads=2, head_dim=128,
         cart_lens=[3000, 1, 70], rows=[[0], [1, 0, 2]], layouts=["head", "tok", "padded"]),
    dict(name="q1_nocart", dtype="bf16", batch=3, q_len=1, num_q_heads=4, num_kv_heads=1, head_dim=64,
         cart_lens=[], rows=[[], [], []]),
    # 16 KV heads: two per XCD in the XCD-affine dK/dV order
    dict(name="kv16", dtype="bf16", batch=2, q_len=70, num_q_heads=32, num_kv_heads=16,
         head_dim=64, cart_lens=[130, 64, 200], rows=[[0, 1], [2, 0]], layouts=["tok", "head", "padded"]),
    dict(name="fp32_d128", dtype="fp32", batch=1, q_len=33, num_q_heads=4, num_kv_heads=2,
         head_dim=128, cart_lens=[65, 3], rows=[[0, 1]]),
    dict(name="fp32_alias", dtype="fp32", batch=2, q_len=20, num_q_heads=2, num_kv_heads=1,
         head_dim=64, cart_lens=[31], rows=[[0], [0]]),
]


@pytest.mark.parametrize("spec", SMALL, ids=[s["name"] for s in SMALL])
def test_small_full(spec):
    spec = dict(spec)
    name = spec.pop("name")
    wl = casgen.custom(name, seed=100 + len(name), cart_std=0.5, **spec)
    _check_full(GpuCase(wl), name)


@pytest.mark.parametrize("spec", SMALL[:4], ids=[s["name"] for s in SMALL[:4]])
def test_small_forced_splits(spec):
    import paper_2606_04557_amd as cas
    spec = dict(spec)
    name = spec.pop("name")
    wl = casgen.custom(name, seed=200 + len(name), cart_std=0.5, **spec)
    try:
        cas.set_tuning(fwd_splits=5, dq_splits=3)
        _check_full(GpuCase(wl), name + " split")
    finally:
        cas.set_tuning(0, 0)


def test_wide_token_stride():
    """A 1,024-token cartridge stored with a token stride of 2^21 elements
    (4 MiB), so that its keys and gradients span 4 GiB: byte offsets within a
    segment pass 2^31 and 2^32 (the largest stride the library accepts is
    2^22 elements). It is used by both rows, once beside a compact one; every
    element is compared, with the automatic plan and with forced key-axis
    splits, and the 4 MiB gaps between gradient rows stay unwritten."""
    import paper_2606_04557_amd as cas
    import torch
    spec = dict(dtype="bf16", batch=2, q_len=40, num_q_heads=4, num_kv_heads=1, head_dim=64,
                cart_lens=[1024, 100], rows=[[0, 1], [1, 0]], layouts=["wide", "tok"])
    wl = casgen.custom("wide", seed=321, cart_std=0.5, **spec)
    case = GpuCase(wl)
    print("wide: K span %.2f GiB" % ((wl.cart_lens[0] - 1) * case.k[0].stride(0) * 2 / 2 ** 30))
    _check_full(case, "wide")
    del case
    torch.cuda.empty_cache()
    try:
        cas.set_tuning(fwd_splits=4, dq_splits=3)
        _check_full(GpuCase(wl), "wide split")
    finally:
        cas.set_tuning(0, 0)
    torch.cuda.empty_cache()


def test_large_launch_tables():
    """512 rows that each list the same 16 cartridges, in a rotated order:
    8,192 segment entries and 8,704 key tiles, about 600 KB of launch tables,
    which the table upload copies in several grid-stride passes. Every
    cartridge's gradient sums over all 512 rows. Every output element."""
    rows = [[(i + b) % 16 for i in range(16)] for b in range(512)]
    wl = casgen.custom("bigtables", "bf16", batch=512, q_len=16, num_q_heads=4, num_kv_heads=1,
                       head_dim=128, cart_lens=[64] * 16, rows=rows, seed=321, cart_std=0.5)
    _check_full(GpuCase(wl), "bigtables")


def _sampled_check(case, n_rows=24, key_targets=None, seed=0, forward_only=False, results=None):
    """Oracle evaluated on sampled query rows (O, LSE, dQ) and sampled keys (dK, dV)."""
    wl = case.wl
    if results is None:
        o, lse = case.fwd()
        grads = None
        if not forward_only:
            grads = case.bwd(o, lse)
        _sync()
    else:
        o, lse, grads = results
    args = case.oracle_args()
    d_o = None if forward_only else case.oracle_do()
    rng = np.random.default_rng(seed)
    B, Sq, Hq = wl.batch, wl.q_len, wl.num_q_heads
    picks = [(int(rng.integers(B)), int(rng.integers(Hq)), int(rng.integers(Sq))) for _ in range(n_rows)]
    picks += [(0, 0, 0), (B - 1, Hq - 1, Sq - 1), (0, Hq // 2, min(Sq - 1, 63)),
              (B - 1, 1, min(Sq - 1, 64))]
    go, glse = host(o), host(lse)
    gdq = host(grads[0]) if grads else None
    ro, rl, rq, vo, vl, vq = [], [], [], [], [], []
    for (b, h, t) in picks:
        oo, ll, dd = oracle.rows_forward_backward(*args, b=b, h=h, t_idx=[t], d_o=d_o)
        ro.append(oo[0]); rl.append(ll[0]); vo.append(go[b, t, h]); vl.append(glse[b, h, t])
        if grads:
            rq.append(dd[0]); vq.append(gdq[b, t, h])
    tol = TOL[wl.dtype]
    e_o = rel_err(np.array(vo), np.array(ro))
    e_l = float(np.abs(np.array(vl) - np.array(rl)).max())
    print(wl.name, "sampled O", f"{e_o:.2e}", "LSE", f"{e_l:.2e}")
    assert e_o <= tol and e_l <= LSE_TOL[wl.dtype]
    if grads:
        e_q = rel_err(np.array(vq), np.array(rq))
        print(wl.name, "sampled dQ", f"{e_q:.2e}")
        assert e_q <= tol
        for kv, targets in (key_targets or {}).items():
            res = oracle.key_grads_many(*args, d_o, kv=kv, targets=targets)
            for (cart, toks), (rk, rv) in zip(targets, res):
                if cart >= 0:
                    gk = host(case.dk[cart][toks, kv])
                    gv = host(case.dv[cart][toks, kv])
                else:
                    gk = host(grads[1][-cart - 1, toks, kv])
                    gv = host(grads[2][-cart - 1, toks, kv])
                ek, ev = rel_err(gk, rk), rel_err(gv, rv)
                print(wl.name, f"kv{kv} cart{cart} dK {ek:.2e} dV {ev:.2e}")
                assert ek <= tol and ev <= tol
    return o, lse, grads


def _check_heads(case, kv_heads):
    """Whole KV heads compared element by element: O, LSE and dQ of every query
    row of their GQA groups, and the self dK/dV and every cartridge's dK/dV at
    those heads (every token). Returns the library's results for further
    checks on the other heads."""
    import torch
    wl = case.wl
    o, lse = case.fwd()
    grads = case.bwd(o, lse)
    _sync()
    args = case.oracle_args()
    O, LSE = oracle.forward(*args, kv_heads=kv_heads)
    rdq, rdks, rdvs, rdck, rdcv = oracle.backward(*args, case.oracle_do(), O=O, LSE=LSE,
                                                  kv_heads=kv_heads)
    g = wl.group_size
    qh = [h for h in range(wl.num_q_heads) if h // g in kv_heads]
    kvi = torch.tensor(kv_heads, device=o.device)
    qhi = torch.tensor(qh, device=o.device)
    tol = TOL[wl.dtype]
    errs = {
        "o": rel_err(host(o.index_select(2, qhi)), O[:, :, qh]),
        "lse": float(np.abs(host(lse.index_select(1, qhi)) - LSE[:, qh]).max()),
        "dq": rel_err(host(grads[0].index_select(2, qhi)), rdq[:, :, qh]),
        "dk_self": rel_err(host(grads[1].index_select(2, kvi)), rdks[:, :, kv_heads]),
        "dv_self": rel_err(host(grads[2].index_select(2, kvi)), rdvs[:, :, kv_heads]),
    }
    for c in case.dk:
        errs[f"dk[{c}]"] = rel_err(host(case.dk[c].index_select(1, kvi)), rdck[c][:, kv_heads])
        errs[f"dv[{c}]"] = rel_err(host(case.dv[c].index_select(1, kvi)), rdcv[c][:, kv_heads])
    worst = max((v, k) for k, v in errs.items() if k != "lse")
    print(wl.name, f"kv heads {kv_heads} in full:", {k: f"{v:.2e}" for k, v in errs.items()
                                                    if k in ("o", "lse", "dq", "dk_self", "dv_self")},
          f"worst {worst[1]} {worst[0]:.2e} over {len(case.dk)} cartridges")
    for k, v in errs.items():
        lim = LSE_TOL[wl.dtype] if k == "lse" else tol
        assert v <= lim, (wl.name, k, v)
    return o, lse, grads


def _gradient_sums(case, grads):
    """Whole-tensor properties per (row, kv head) when no cartridge is shared
    between rows: (a) the dV of all visible keys sums to the dO of the group's
    query rows (each softmax row sums to one); (b) the dK of all visible keys
    sums to zero (each row of dS sums to zero), measured against the sum of
    |dK|."""
    wl = case.wl
    g = wl.group_size
    do = case.d_o.float()
    for b in range(wl.batch):
        tot = grads[2][b].float().sum(0)                      # [Hkv, D]
        tk = grads[1][b].float().sum(0)
        ak = grads[1][b].float().abs().sum(0)
        for c in wl.rows[b]:
            tot = tot + case.dv[c].float().sum(0)
            tk = tk + case.dk[c].float().sum(0)
            ak = ak + case.dk[c].float().abs().sum(0)
        exp = do[b].view(wl.q_len, wl.num_kv_heads, g, wl.head_dim).sum((0, 2))
        err = (tot - exp).abs().max().item() / exp.abs().max().item()
        errk = (tk.abs() / ak).max().item()
        print(wl.name, f"row {b} sum dV rel err {err:.2e}, |sum dK| / sum |dK| {errk:.2e}")
        assert err <= 2e-2
        assert errk <= 2e-3


def _edge_tokens(L):
    """Tile-edge tokens of a length-L key block (64-key tiles, 128-key dK/dV
    workgroups) plus the last one."""
    return sorted({t for t in (0, 1, 63, 64, 127, 128, L // 2, L - 2, L - 1) if 0 <= t < L})


def test_c2_full_size():
    """4 rows x 4 x 1024-token cartridges: every output element against the oracle."""
    case = GpuCase(casgen.config(2))
    _, _, grads = _check_full(case, "C2")
    _gradient_sums(case, grads)


def test_c3_full_size():
    """The headline 16 x 2048-cartridge configuration in the launch plan the
    bench times: KV heads 0 and 7 (the first and last XCD range of the
    forward and dQ order) in full; on every other head, sampled query rows and
    tile-edge keys of a cartridge of each row and of the self keys."""
    wl = casgen.config(3)
    case = GpuCase(wl)
    res = _check_heads(case, [0, 7])
    targets = {}
    for kv in range(1, 7):
        b = kv % 2
        c0, c1 = wl.rows[b][kv], wl.rows[b][15 - kv]
        targets[kv] = [(c0, _edge_tokens(2048)), (c1, [1000, 1024, 1535, 1536]),
                       (-b - 1, _edge_tokens(wl.q_len))]
    _sampled_check(case, n_rows=32, key_targets=targets, seed=3, results=res)
    _gradient_sums(case, res[2])


def test_c4_full_size():
    """64 cartridges of U[256, 4096] tokens in separate allocations with padded and
    head-major layouts; B = 1 forces key-axis splits in the forward and dQ.
    KV heads 2 and 6 in full; on every other head, tile-edge keys of two
    cartridges of each layout kind and of the self keys."""
    import paper_2606_04557_amd as cas
    wl = casgen.config(4)
    case = GpuCase(wl)
    prob = cas.Problem.from_tensors(case.q, case.rows, wl.num_kv_heads, wl.group_size, float(wl.scale))
    info = cas.plan_info(prob)
    assert info["fwd_splits"] > 1 and info["dq_splits"] > 1
    res = _check_heads(case, [2, 6])
    targets = {}
    for kv in (0, 1, 3, 4, 5, 7):
        picks = []
        for kind in ("tok", "padded", "head"):
            ids = [c for c in range(64) if wl.layouts[c] == kind]
            c = ids[(kv * 5) % len(ids)]
            picks.append((c, _edge_tokens(wl.cart_lens[c])))
        picks.append((-1, _edge_tokens(wl.q_len)))
        targets[kv] = picks
    _sampled_check(case, n_rows=32, key_targets=targets, seed=4, results=res)
    _gradient_sums(case, res[2])


def test_c5_forward_with_staging():
    """Retrieval-style inference mix: 64 requests each over 4 cartridges of a
    256-cartridge pool; the pool's second half is staged host -> HBM with
    cas_cartridge_stage on a side stream, and the forward waits on its events.
    Every O and LSE element is compared with the oracle."""
    import torch
    import paper_2606_04557_amd as cas
    wl = casgen.config(5)
    used = sorted({c for r in wl.rows for c in r})
    T = casgen.make_tensors(wl, carts=used)
    case = GpuCase(wl, tensors=T, grads=False)
    # Re-stage the second half from pinned host memory into the same device buffers.
    for c in used:
        if c >= 128:
            case.k[c].fill_(float("nan"))
            case.v[c].fill_(float("nan"))
    side = torch.cuda.Stream()
    events = []
    staged = [c for c in used if c >= 128]
    hosts = []
    for i in range(0, len(staged), 16):
        chunk = staged[i:i + 16]
        copies = []
        for c in chunk:
            for src, dst in ((T["cart_k"][c], case.k[c]), (T["cart_v"][c], case.v[c])):
                h = torch.from_numpy(src.view(np.int16)).view(torch.bfloat16).pin_memory()
                hosts.append(h)
                copies.append((h, dst))
        ev = torch.cuda.Event()
        torch.cuda.synchronize()
        cas.cartridge_stage(copies, side, ev)
        events.append(ev)
    for ev in events:
        torch.cuda.current_stream().wait_event(ev)
    o, lse = case.fwd()
    _sync()
    O, LSE, _ = full_oracle(case, backward=False)
    e_o, e_l = rel_err(host(o), O), float(np.abs(host(lse) - LSE).max())
    print("C5 every element: O", f"{e_o:.2e}", "LSE", f"{e_l:.2e}")
    assert e_o <= TOL["bf16"] and e_l <= LSE_TOL["bf16"]
    # A pageable source is refused before anything is enqueued.
    src = torch.zeros(1024, dtype=torch.bfloat16)
    dst = torch.zeros(1024, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(cas.CasError) as ei:
        cas.cartridge_stage([(src, dst)], side)
    assert "CAS_ERR_NOT_PINNED" in str(ei.value)


def test_stage_contiguous_and_scattered_copies():
    """cas_cartridge_stage moves runs of address-contiguous entries as one
    transfer: a list mixing such runs, gaps, zero-byte entries and a reversed
    order must still land every byte where its entry says."""
    import torch
    import paper_2606_04557_amd as cas
    n = 1 << 16
    host = torch.arange(8 * n, dtype=torch.int32).pin_memory()
    dev = torch.full((10 * n,), -1, dtype=torch.int32, device="cuda")
    pieces = [(0, 0), (1, 1), (2, 2),          # one contiguous run
              (3, 5), (4, 6),                  # a second run after a gap in the destination
              (6, 3), (5, 4),                  # reversed: two transfers
              (7, 9)]
    copies = [(host[s * n:(s + 1) * n], dev[d * n:(d + 1) * n]) for s, d in pieces]
    copies.insert(3, (host[:0], dev[:0]))      # a zero-byte entry inside the list
    side = torch.cuda.Stream()
    ev = torch.cuda.Event()
    torch.cuda.synchronize()
    cas.cartridge_stage(copies, side, ev)
    torch.cuda.current_stream().wait_event(ev)
    got = dev.cpu()
    want = torch.full((10 * n,), -1, dtype=torch.int32)
    for s, d in pieces:
        want[d * n:(d + 1) * n] = host[s * n:(s + 1) * n]
    assert torch.equal(got, want)
