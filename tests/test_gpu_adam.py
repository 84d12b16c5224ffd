"""GPU parity of the cartridge Adam step (cas_cartridge_adam) against the
fp32 reference in oracle/adam.py.

Both sides round once per operation in Algorithm 1's order (the library's
kernel is built without multiply-add contraction), so the bar is bit
equality of the new bf16 parameters and of both fp32 moments.
"""
import numpy as np
import pytest

from casgen import rng
from gpu_util import alloc_like_layout
from oracle import adam

pytestmark = pytest.mark.gpu

CFG = dict(lr=0.05, beta1=0.9, beta2=0.999, eps=1e-8, warmup_steps=20, warmup_buckets=4)


def _bf16_host(key, shape, std):
    bits = rng.f64_to_bf16_bits(rng.normal(key, int(np.prod(shape)), std).reshape(shape))
    return rng.bf16_bits_to_f32(bits).astype(np.float32)


def _to_dev_bf16(a, layout):
    import torch
    L, H, D = a.shape
    view, base = alloc_like_layout(L, H, D, layout, torch.bfloat16)
    view.copy_(torch.from_numpy(a).to(torch.bfloat16).cuda())
    return view, base


class Cart:
    """Host arrays and device tensors of one cartridge's optimizer state."""

    def __init__(self, seed, L, Hkv, D, layout, step, frozen):
        import torch
        self.step, self.frozen, self.layout = step, frozen, layout
        shp = (L, Hkv, D)
        self.h = {}
        for i, name in enumerate(("k", "v")):
            self.h[name] = _bf16_host(rng.stream_key(seed, 20 + i), shp, 0.5)
            self.h["d" + name] = _bf16_host(rng.stream_key(seed, 22 + i), shp, 1e-2)
            if step == 0:
                m1 = np.zeros(shp, np.float32)
                m2 = np.zeros(shp, np.float32)
            else:
                m1 = (rng.normal(rng.stream_key(seed, 24 + i), int(np.prod(shp)), 1e-3).reshape(shp)
                      .astype(np.float32))
                m2 = (np.abs(rng.normal(rng.stream_key(seed, 26 + i), int(np.prod(shp)), 1e-4))
                      .reshape(shp).astype(np.float32))
            self.h["m1_" + name], self.h["m2_" + name] = m1, m2
        self.d = {}
        self.bases = {}
        for name in ("k", "v", "dk", "dv"):
            self.d[name], self.bases[name] = _to_dev_bf16(self.h[name], layout)
        for name in ("m1_k", "m2_k", "m1_v", "m2_v"):
            self.d[name] = torch.from_numpy(self.h[name].copy()).cuda()

    def handle(self):
        import paper_2606_04557_amd as cas
        d = self.d
        return cas.AdamCartridge(d["k"], d["v"], d["dk"], d["dv"], d["m1_k"], d["m2_k"], d["m1_v"], d["m2_v"],
                                 step=self.step, frozen_tokens=self.frozen)

    def oracle_step(self):
        for name in ("k", "v"):
            x, m1, m2 = adam.adam_step(self.h[name], self.h["d" + name], self.h["m1_" + name],
                                       self.h["m2_" + name], self.step, frozen_tokens=self.frozen, **CFG)
            self.h[name], self.h["m1_" + name], self.h["m2_" + name] = x, m1, m2
        self.step += 1

    def check(self, label):
        import torch
        for name in ("k", "v"):
            got = self.d[name].float().cpu().numpy()
            assert np.array_equal(got.view(np.uint32), self.h[name].view(np.uint32)), (label, name)
            for m in ("m1_", "m2_"):
                g = self.d[m + name].cpu().numpy()
                assert np.array_equal(g.view(np.uint32), self.h[m + name].view(np.uint32)), (label, m + name)
        if self.layout == "padded":   # the padding between tokens is never written
            for name in ("k", "v"):
                base = self.bases[name]
                assert torch.isnan(base[:, self.d[name].shape[1] * self.d[name].shape[2]:].float()).all()


SPECS = [
    # (length, layout, optimizer steps received, frozen tokens)
    (37, "tok", 0, 1),
    (130, "padded", 3, 1),
    (1, "head", 0, 1),        # only the frozen token: untouched
    (17, "tok", 25, 0),
    (64, "head", 9, 2),
    (300, "tok", 5, 1),
]


@pytest.mark.parametrize("D", [128, 64])
def test_adam_bit_exact(D):
    import torch
    import paper_2606_04557_amd as cas
    carts = [Cart(500 + i, L, 8 if D == 128 else 2, D, lay, st, fr) for i, (L, lay, st, fr) in enumerate(SPECS)]
    cas.cartridge_adam([c.handle() for c in carts], **CFG)
    torch.cuda.synchronize()
    for i, c in enumerate(carts):
        c.oracle_step()
        c.check(f"D{D} cart{i}")


def test_adam_three_steps_with_rotation():
    """Three steps with fresh gradients; between them one cartridge leaves the
    call (rotated out) and comes back with its step count and moments."""
    import torch
    import paper_2606_04557_amd as cas
    carts = [Cart(600 + i, L, 8, 128, lay, st, fr) for i, (L, lay, st, fr) in enumerate(SPECS)]
    for it in range(3):
        active = [c for i, c in enumerate(carts) if not (it == 1 and i == 3)]
        if it > 0:
            for i, c in enumerate(active):
                for name in ("dk", "dv"):
                    c.h[name] = _bf16_host(rng.stream_key(700 + it, i, len(name)), c.h[name].shape, 1e-2)
                    c.d[name].copy_(torch.from_numpy(c.h[name]).to(torch.bfloat16).cuda())
        cas.cartridge_adam([c.handle() for c in active], **CFG)
        torch.cuda.synchronize()
        for c in active:
            c.oracle_step()
        for i, c in enumerate(carts):
            c.check(f"step {it} cart{i}")


def test_adam_rejects_bad_input_before_launch():
    import torch
    import paper_2606_04557_amd as cas
    c = Cart(800, 20, 8, 128, "tok", 2, 1)
    before = c.d["k"].clone()
    with pytest.raises(cas.CasError):
        cas.cartridge_adam([c.handle()], lr=-1.0)
    h = c.handle()
    h.m2_k = h.m1_k                       # two moments in one buffer
    with pytest.raises(cas.CasError):
        cas.cartridge_adam([h], **CFG)
    torch.cuda.synchronize()
    assert torch.equal(c.d["k"], before)
