"""GPU parity of the packed-sample layout (several samples of different lengths
on one token axis, each over its own cartridges, block-diagonal causal self;
paper: Section "Training with Multiple Cartridges", Eq. mixing, and the
hyperparameter table's 8,192-token packed sequences) against the fp64 oracle.

Bars as in test_gpu_parity: max |gpu - oracle| / max |oracle| <= 1e-5 (fp32)
or 2e-2 (bf16) per tensor, LSE absolute error <= 1e-5 / 1e-3.
"""
import pytest

import casgen
from gpu_util import GpuCase
from test_gpu_parity import _check_full

pytestmark = pytest.mark.gpu


def _sync():
    import torch
    torch.cuda.synchronize()


PACKED = [
    # empty samples (one whose only cartridge nobody else uses: its gradient is
    # zero), one-token and block-boundary lengths, a sample with no prefix, a
    # cartridge shared by several samples and referenced twice in one
    dict(name="pk_mixed", dtype="bf16", num_q_heads=8, num_kv_heads=2, head_dim=128,
         q_lens=[37, 0, 130, 64, 1, 65, 0], cart_lens=[100, 1, 257, 64, 33],
         rows=[[0, 1], [4], [3, 0], [], [1, 2, 3, 0], [0, 0], [2]],
         layouts=["tok", "padded", "head", "tok", "padded"]),
    # GQA group of 5: 64-row blocks do not start on a position boundary
    dict(name="pk_g5_d64", dtype="bf16", num_q_heads=10, num_kv_heads=2, head_dim=64,
         q_lens=[45, 3, 70], cart_lens=[90, 40], rows=[[1, 0], [0], [1]]),
    dict(name="pk_g16", dtype="bf16", num_q_heads=16, num_kv_heads=1, head_dim=128,
         q_lens=[50, 7, 129], cart_lens=[300, 65], rows=[[0], [0, 1], [1]]),
    dict(name="pk_fp32", dtype="fp32", num_q_heads=4, num_kv_heads=2, head_dim=64,
         q_lens=[20, 0, 33], cart_lens=[31, 17], rows=[[0], [1], [0, 1]]),
]


def _workload(spec, seed):
    spec = dict(spec)
    name = spec.pop("name")
    q_lens = spec.pop("q_lens")
    return casgen.custom(name, batch=len(q_lens), q_len=0, seed=seed, cart_std=0.5, q_lens=q_lens, **spec)


@pytest.mark.parametrize("spec", PACKED, ids=[s["name"] for s in PACKED])
def test_packed_small_full(spec):
    wl = _workload(spec, 300 + len(spec["name"]))
    _check_full(GpuCase(wl), wl.name)


def test_packed_forced_splits():
    import paper_2606_04557_amd as cas
    wl = _workload(PACKED[0], 400)
    try:
        cas.set_tuning(fwd_splits=5, dq_splits=3)
        _check_full(GpuCase(wl), wl.name + " split")
    finally:
        cas.set_tuning(0, 0)


def test_packed_equal_lengths_match_fixed_layout():
    """Packed samples of equal length are the fixed-length batch with another
    LSE layout: the same kernels must give bit-identical outputs."""
    import torch
    fixed = casgen.custom("fx", "bf16", batch=3, q_len=100, num_q_heads=8, num_kv_heads=2,
                          head_dim=128, cart_lens=[70, 129], rows=[[0, 1], [1], [0]], seed=77,
                          cart_std=0.5)
    a = GpuCase(fixed)
    o1, l1 = a.fwd()
    g1 = a.bwd(o1, l1)
    d1 = {c: (a.dk[c].clone(), a.dv[c].clone()) for c in a.dk}
    b = GpuCase(fixed)
    T = 3 * 100
    qo = [0, 100, 200, 300]
    flat = lambda x: x.reshape(T, *x.shape[2:])
    b.q, b.k_self, b.v_self, b.d_o = flat(b.q), flat(b.k_self), flat(b.v_self), flat(b.d_o)
    o2, l2 = b.fwd(q_offsets=qo)
    g2 = b.bwd(o2, l2, q_offsets=qo)
    _sync()
    assert torch.equal(o2, flat(o1))
    assert torch.equal(l2, l1.permute(1, 0, 2).reshape(8, T))
    for x, y in zip(g2, g1):
        assert torch.equal(x, flat(y))
    for c in d1:
        assert torch.equal(b.dk[c], d1[c][0]) and torch.equal(b.dv[c], d1[c][1])


def test_packed_8k_full():
    """The 8,192-token packed training layout (20-cartridge pool, target plus up
    to 10 distractors per sample): every output element against the oracle,
    and the whole-tensor identity that every query row's P sums to one, so the
    dV of all keys (each cartridge once, all self keys) adds up to the dO of
    every query row of the group."""
    wl = casgen.packed()
    case = GpuCase(wl)
    _, _, (dq, dks, dvs) = _check_full(case, "P8K")
    g = wl.group_size
    tot = dvs.float().sum(0)
    for c in case.dv:
        tot = tot + case.dv[c].float().sum(0)
    exp = case.d_o.float().view(-1, wl.num_kv_heads, g, wl.head_dim).sum((0, 2))
    err = (tot - exp).abs().max().item() / exp.abs().max().item()
    print("P8K sum dV rel err", f"{err:.2e}")
    assert err <= 2e-2
