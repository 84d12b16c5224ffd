"""The no-allocation forward (cas_prefix_attn_fwd_noalloc: static device
scratch, tables as kernel arguments) against the forward with a caller
workspace, on two calls in a row, the second with a smaller problem.

Bars as in the parity tests: max |a - b| / max |b| <= 2e-2 for bf16 and
LSE absolute error <= 1e-3 where the plans differ (the first problem splits
its key axis into more partials than the scratch holds, so the no-allocation
call uses fewer); bit-identical outputs where they agree.
"""
import pytest

import casgen
from gpu_util import GpuCase, LSE_TOL, TOL, host, rel_err

pytestmark = pytest.mark.gpu


def test_noalloc_forward_matches_workspace_forward():
    import torch
    import paper_2606_04557_amd as cas
    torch.cuda.synchronize()
    # B = 1 and 256 queries give 32 forward workgroups, so the planner splits
    # the 40K-token ragged prefix 16 ways: 67 MB of partials, more than the
    # 16 MiB scratch, which then holds 3 splits.
    lens = [1500 + 37 * i for i in range(20)]
    big = casgen.custom("noalloc_big", "bf16", batch=1, q_len=256, num_q_heads=32, num_kv_heads=8,
                        head_dim=128, cart_lens=lens, rows=[list(range(20))], seed=91, cart_std=0.5)
    small = casgen.custom("noalloc_small", "bf16", batch=2, q_len=100, num_q_heads=8, num_kv_heads=2,
                          head_dim=128, cart_lens=[70, 129, 1], rows=[[0, 1], [2, 0]], seed=92,
                          cart_std=0.5)
    a = GpuCase(big, grads=False)
    b = GpuCase(small, grads=False)
    pa = cas.Problem.from_tensors(a.q, a.rows, big.num_kv_heads, big.group_size, float(big.scale))
    assert cas.plan_info(pa)["fwd_splits"] > 3
    na_o, na_l = torch.full_like(a.q, float("nan")), torch.empty(1, 32, 256, device="cuda")
    nb_o, nb_l = torch.full_like(b.q, float("nan")), torch.empty(2, 8, 100, device="cuda")
    # Two no-allocation calls in a row on one stream, the second smaller.
    cas.prefix_attn_fwd_noalloc(a.q, a.k_self, a.v_self, a.rows, big.num_kv_heads, big.group_size,
                                float(big.scale), na_o, na_l)
    cas.prefix_attn_fwd_noalloc(b.q, b.k_self, b.v_self, b.rows, small.num_kv_heads, small.group_size,
                                float(small.scale), nb_o, nb_l)
    torch.cuda.synchronize()
    ra_o, ra_l = a.fwd()
    rb_o, rb_l = b.fwd()
    torch.cuda.synchronize()
    e_o = rel_err(host(na_o), host(ra_o))
    e_l = float((na_l - ra_l).abs().max())
    print("no-allocation forward, 3 vs", cas.plan_info(pa)["fwd_splits"], "splits: O", f"{e_o:.2e}",
          "LSE", f"{e_l:.2e}")
    assert e_o <= TOL["bf16"] and e_l <= LSE_TOL["bf16"]
    assert torch.equal(nb_o, rb_o) and torch.equal(nb_l, rb_l)
    # A third call, larger again, still matches (the scratch keeps no state).
    cas.prefix_attn_fwd_noalloc(a.q, a.k_self, a.v_self, a.rows, big.num_kv_heads, big.group_size,
                                float(big.scale), na_o, na_l)
    torch.cuda.synchronize()
    assert rel_err(host(na_o), host(ra_o)) == e_o
