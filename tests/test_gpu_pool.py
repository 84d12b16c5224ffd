"""GPU test of the budget manager (cas_pool_*): a small training loop through
the pool (rotations with prefetched admissions and copied-back evictions)
must leave every cartridge's host copy bit-identical to a host simulation of
the same policy (oracle/pool.py) and Adam step (oracle/adam.py), with the
moments of offloaded cartridges in pinned host memory or in a file."""
import numpy as np
import pytest

from casgen import rng
from oracle import adam, pool as pool_ref

pytestmark = pytest.mark.gpu

CFG = dict(lr=0.05, beta1=0.9, beta2=0.999, eps=1e-8, warmup_steps=4, warmup_buckets=2)


def _bits(key, shape, std):
    return rng.f64_to_bf16_bits(rng.normal(key, int(np.prod(shape)), std).reshape(shape)).view(np.int16)


def _f32(bits):
    return rng.bf16_bits_to_f32(bits.view(np.uint16)).astype(np.float32)


@pytest.mark.parametrize("phi,tier,B", [(0.67, "host", 3), (0.34, "host", 3), (0.67, "file", 3),
                                        (0.34, "file", 3), (0.0, "file", 3), (0.4, "file", 5)])
def test_pool_training_matches_reference(phi, tier, B, tmp_path):
    """tier "file": the moments of offloaded cartridges go through a file
    (written on eviction, read back on admission by the pool thread). With
    B = 5 and phi = 0.4 every rotation admits exactly the cartridges the
    previous one evicted (their moments are read right after being written)."""
    import torch
    import paper_2606_04557_amd as cas
    lens = [37, 64, 20, 100, 51, 16, 80]
    N, Hkv, D, R = len(lens), 2, 64, 2
    p = cas.CartridgePool(lens, Hkv, D, B, R, phi, frozen_tokens=1,
                          moment_dir=str(tmp_path) if tier == "file" else None)
    ref = {}
    for c, L in enumerate(lens):
        h = p.host(c)
        for i, name in enumerate(("k", "v")):
            h[name][...] = _bits(rng.stream_key(41, c, i), (L, Hkv, D), 0.5)
        ref[c] = dict(k=_f32(h["k"].copy()), v=_f32(h["v"].copy()),
                      **{m: np.zeros((L, Hkv, D), np.float32) for m in ("m1_k", "m2_k", "m1_v", "m2_v")})
    steps = [0] * N
    active = set(pool_ref.first_active(steps, B))
    p.load()
    for it in range(9):
        act = p.active()
        assert sorted(c for c, _ in act) == sorted(active), (it, act, active)
        for c, ac in act:
            assert ac.step == steps[c]
            for i, (g, name) in enumerate(((ac.dk, "k"), (ac.dv, "v"))):
                gb = _bits(rng.stream_key(42, it, c, i), tuple(g.shape), 1e-2)
                g.copy_(torch.from_numpy(gb).view(torch.bfloat16).cuda())
                x, m1, m2 = adam.adam_step(ref[c][name], _f32(gb), ref[c]["m1_" + name], ref[c]["m2_" + name],
                                           steps[c], frozen_tokens=1, **CFG)
                ref[c][name], ref[c]["m1_" + name], ref[c]["m2_" + name] = x, m1, m2
        cas.cartridge_adam([ac for _, ac in act], **CFG)
        p.end_step()
        for c in active:
            steps[c] += 1
        if (it + 1) % R == 0:
            ev, ad = pool_ref.plan_rotation(steps, [c in active for c in range(N)], B, phi)
            active = (active - set(ev)) | set(ad)
    p.flush()
    torch.cuda.synchronize()
    for c in range(N):
        h = p.host(c)
        for name in ("k", "v"):
            assert np.array_equal(_f32(h[name]).view(np.uint32), ref[c][name].view(np.uint32)), (c, name)
            for m in ("m1_", "m2_"):
                assert np.array_equal(h[m + name].view(np.uint32), ref[c][m + name].view(np.uint32)), (c, m + name)
        assert h["step"] == steps[c], (c, h["step"], steps[c])
    if phi > 0:
        assert sum(s > 0 for s in steps) > B      # rotation brought offloaded cartridges in
    p.close()
