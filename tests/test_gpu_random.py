"""GPU parity on seeded random problems: batch, query length (or, in the
packed layout, the samples' lengths), KV heads, GQA group, head_dim,
cartridge lengths, storage layouts, aliasing and dtype are drawn per case
(for the paged decode path: page size, heads, group, head_dim, the
cartridge pool and each request's cartridges, own tokens and queries),
and every output element is compared with the fp64 oracle
(bars as in test_gpu_parity: 2e-2 relative for bf16, 1e-5 for fp32; LSE
absolute 1e-3 / 1e-5). The draws are fixed by the case number, so a failing
case is reproducible by its id.
"""
import numpy as np
import pytest

import casgen
from gpu_util import GpuCase, LSE_TOL, TOL, full_oracle, host, rel_err

pytestmark = pytest.mark.gpu

N_CASES = 16


def draw_case(i):
    r = np.random.RandomState(1000 + i)
    dtype = "fp32" if i % 4 == 3 else "bf16"
    D = int(r.choice([64, 128]))
    Hkv = int(r.randint(1, 4))
    g = int(r.choice([1, 2, 3, 4, 5, 8]))
    B = int(r.randint(1, 4))
    q_len = int(r.choice([1, 7, 33, 64, 65, 100, 190]))
    n_carts = int(r.randint(0, 6))
    cart_lens = [int(r.choice([0, 1, 31, 64, 100, 128, 129, 257, 300])) for _ in range(n_carts)]
    layouts = [str(r.choice(["tok", "padded", "head"])) for _ in range(n_carts)]
    rows = []
    for _ in range(B):
        k = int(r.randint(0, 5)) if n_carts else 0
        rows.append([int(c) for c in r.randint(0, n_carts, size=k)] if k else [])
    return dict(name=f"rand{i}", dtype=dtype, batch=B, q_len=q_len, num_q_heads=Hkv * g,
                num_kv_heads=Hkv, head_dim=D, cart_lens=cart_lens, rows=rows, layouts=layouts)


@pytest.mark.parametrize("i", range(N_CASES), ids=[f"case{i}" for i in range(N_CASES)])
def test_random_problem(i):
    import torch
    spec = draw_case(i)
    name = spec.pop("name")
    wl = casgen.custom(name, seed=5000 + i, cart_std=0.5, **spec)
    case = GpuCase(wl)
    o, lse = case.fwd()
    dq, dks, dvs = case.bwd(o, lse)
    torch.cuda.synchronize()
    O, LSE, (rdq, rdks, rdvs, rdck, rdcv) = full_oracle(case)
    errs = {"o": rel_err(host(o), O), "lse": float(np.abs(host(lse) - LSE).max()),
            "dq": rel_err(host(dq), rdq), "dk_self": rel_err(host(dks), rdks),
            "dv_self": rel_err(host(dvs), rdvs)}
    for c in case.dk:
        errs[f"dk[{c}]"] = rel_err(host(case.dk[c]), rdck[c])
        errs[f"dv[{c}]"] = rel_err(host(case.dv[c]), rdcv[c])
    print(name, {k: spec[k] for k in ("dtype", "batch", "q_len", "num_kv_heads", "head_dim")},
          "g", wl.group_size, "carts", wl.cart_lens, "rows", wl.rows,
          {k: f"{v:.1e}" for k, v in errs.items()})
    for k, v in errs.items():
        lim = LSE_TOL[wl.dtype] if k == "lse" else TOL[wl.dtype]
        assert v <= lim, (name, k, v)


def draw_packed(i):
    """Packed samples (one token axis; samples of 0..300 tokens, some empty),
    each over a random subset of a shared cartridge pool."""
    r = np.random.RandomState(2000 + i)
    dtype = "fp32" if i % 4 == 3 else "bf16"
    D = int(r.choice([64, 128]))
    Hkv = int(r.randint(1, 3))
    g = int(r.choice([1, 2, 4, 5, 8]))
    n_s = int(r.randint(1, 7))
    q_lens = [int(r.choice([0, 1, 15, 64, 65, 130, 300])) for _ in range(n_s)]
    if sum(q_lens) == 0:
        q_lens[0] = 33
    n_carts = int(r.randint(1, 6))
    cart_lens = [int(r.choice([1, 31, 64, 100, 129, 257])) for _ in range(n_carts)]
    layouts = [str(r.choice(["tok", "padded", "head"])) for _ in range(n_carts)]
    rows = [[int(c) for c in r.randint(0, n_carts, size=int(r.randint(0, 4)))] for _ in range(n_s)]
    return dict(name=f"prand{i}", dtype=dtype, batch=n_s, q_len=0, q_lens=q_lens, num_q_heads=Hkv * g,
                num_kv_heads=Hkv, head_dim=D, cart_lens=cart_lens, rows=rows, layouts=layouts)


@pytest.mark.parametrize("i", range(8), ids=[f"packed{i}" for i in range(8)])
def test_random_packed_problem(i):
    from test_gpu_parity import _check_full
    spec = draw_packed(i)
    name = spec.pop("name")
    wl = casgen.custom(name, seed=6000 + i, cart_std=0.5, **spec)
    print(name, "q_lens", wl.q_lens, "g", wl.group_size, "d", wl.head_dim, "carts", wl.cart_lens, "rows", wl.rows)
    _check_full(GpuCase(wl), name)


def draw_decode(i):
    """Paged decode: page size, heads, group, head_dim, a cartridge pool, and
    requests over random (possibly repeated) cartridges with their own
    tokens and 1..12 queries."""
    r = np.random.RandomState(3000 + i)
    P = int(r.choice([16, 32, 64, 128]))
    Hkv = int(r.choice([1, 2, 4]))
    g = int(r.choice([1, 2, 4, 8]))
    D = int(r.choice([64, 128]))
    n_carts = int(r.randint(1, 6))
    cart_pages = int(r.randint(1, 7))
    reqs = []
    for _ in range(int(r.randint(1, 7))):
        carts = [int(c) for c in r.randint(0, n_carts, size=int(r.randint(0, 5)))]
        own = int(r.randint(1, 101))
        kv = len(carts) * cart_pages * P + own
        reqs.append((carts, own, int(r.randint(1, min(kv, 12) + 1))))
    return dict(P=P, Hkv=Hkv, g=g, D=D, n_carts=n_carts, cart_pages=cart_pages, reqs=reqs)


@pytest.mark.parametrize("i", range(8), ids=[f"decode{i}" for i in range(8)])
def test_random_decode_problem(i):
    from test_gpu_decode import _pool, _run
    c = draw_decode(i)
    print(f"decode{i}", c)
    kp, vp, kl, qc, pages = _pool(7000 + i, c["n_carts"], c["cart_pages"], c["P"], c["Hkv"], c["D"], c["reqs"],
                                  own_extra=int(i % 3))
    _run(kp, vp, kl, qc, pages, c["Hkv"], c["g"], c["D"], 7100 + i)
