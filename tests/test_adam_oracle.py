"""Pins of the cartridge Adam reference (oracle/adam.py) against facts that do
not come from it: torch's own Adam, the first-step closed form, the paper's
warmup formula at the bucket edges, exact bf16 rounding cases, and the
library's host-side warmup factor."""
import math

import numpy as np
import pytest

from oracle import adam


def test_a1_matches_torch_adam_over_steps():
    """A1: several steps of the fp32 reference (no bf16 rounding) against
    torch.optim.Adam on fp32 parameters (its operation order differs, so the
    bar is a few fp32 ulps)."""
    import torch
    r = np.random.default_rng(1)
    x0 = r.standard_normal((7, 3, 8)).astype(np.float32)
    grads = [r.standard_normal(x0.shape).astype(np.float32) * 0.01 for _ in range(5)]
    p = torch.nn.Parameter(torch.from_numpy(x0.copy()))
    # The same fp32 constants on both sides (torch takes them as doubles).
    f = lambda v: float(np.float32(v))
    opt = torch.optim.Adam([p], lr=f(0.05), betas=(f(0.9), f(0.999)), eps=f(1e-8))
    x, m1, m2 = x0.copy(), np.zeros_like(x0), np.zeros_like(x0)
    for s, g in enumerate(grads):
        p.grad = torch.from_numpy(g.copy())
        opt.step()
        x, m1, m2 = adam.adam_step(x, g, m1, m2, step=s, lr=0.05, warmup_steps=0, frozen_tokens=0,
                                   round_bf16=False)
        st = opt.state[p]
        ref1 = st["exp_avg"].numpy()   # terms of both signs cancel: absolute bar at the terms' scale
        np.testing.assert_allclose(m1, ref1, rtol=1e-6, atol=1e-6 * np.abs(ref1).max())
        np.testing.assert_allclose(m2, st["exp_avg_sq"].numpy(), rtol=1e-6, atol=1e-16)
        np.testing.assert_allclose(x, p.detach().numpy(), rtol=0, atol=2e-7 * (s + 1))


def test_a2_first_step_closed_form():
    """A2: from zero moments the first step moves every element by lr * g / (|g| + eps)
    (m1_hat = g and m2_hat = g^2 up to rounding), i.e. by about lr * sign(g)."""
    r = np.random.default_rng(2)
    x = r.standard_normal((5, 2, 8)).astype(np.float32)
    g = (r.standard_normal(x.shape) * 1e-2).astype(np.float32)
    nx, m1, m2 = adam.adam_step(x, g, 0, 0, step=0, lr=0.1, warmup_steps=0, frozen_tokens=0, round_bf16=False)
    exp = x - 0.1 * g / (np.abs(g) + 1e-8)
    np.testing.assert_allclose(nx, exp, rtol=0, atol=1e-6)
    # (the betas are fp32: 1 - beta2 = 1 - fl32(0.999) = 0.000999987...)
    np.testing.assert_allclose(m1, (1 - float(np.float32(0.9))) * g.astype(np.float64), rtol=1e-6)
    np.testing.assert_allclose(m2, (1 - float(np.float32(0.999))) * g.astype(np.float64) ** 2, rtol=1e-6)


def test_a3_warmup_buckets():
    """A3: the bucketed factor is one of N_b levels, never below the paper's
    min(1, s / W_c), less than one level above it, and 1 from s = W_c on."""
    for W, N in ((20, 4), (20, 1), (7, 3), (5, 8)):
        for s in range(0, 3 * W):
            f = adam.warmup_scale(s, W, N)
            exact = min(1.0, s / W)
            assert any(abs(f - k / N) < 1e-12 for k in range(1, N + 1))
            assert f >= exact - 1e-12 and (f - exact < 1.0 / N + 1e-12)
            if s >= W:
                assert f == 1.0
    assert [adam.warmup_scale(s, 20, 4) for s in (0, 1, 5, 6, 10, 11, 15, 16, 19, 20)] == \
        [0.25, 0.25, 0.25, 0.5, 0.5, 0.75, 0.75, 1.0, 1.0, 1.0]
    assert adam.warmup_scale(3, 0, 4) == 1.0


def test_a4_bf16_rounding_and_frozen_tokens():
    """A4: RNE to bf16 on hand-picked values (ties to even, carries into the
    exponent), and frozen tokens keep parameters and moments."""
    v = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -9, -(2.0 - 2 ** -9), 3.0e-39],
                 dtype=np.float32)
    want = np.array([1.0, 1.0, 1.0 + 2 ** -6, 1.0, -2.0, 3.0e-39], dtype=np.float32)
    got = adam.to_bf16(v)
    np.testing.assert_array_equal(got[:5], want[:5])
    assert (got[5].view(np.uint32) & 0xFFFF) == 0 and abs(got[5] - v[5]) < 2 ** -133
    r = np.random.default_rng(4)
    x = adam.to_bf16(r.standard_normal((4, 2, 8)).astype(np.float32))
    g = r.standard_normal(x.shape).astype(np.float32)
    m1 = r.standard_normal(x.shape).astype(np.float32)
    m2 = np.abs(r.standard_normal(x.shape)).astype(np.float32)
    nx, n1, n2 = adam.adam_step(x, g, m1, m2, step=7, lr=0.05, frozen_tokens=2)
    assert np.array_equal(nx[:2], x[:2]) and np.array_equal(n1[:2], m1[:2]) and np.array_equal(n2[:2], m2[:2])
    assert not np.array_equal(nx[2:], x[2:])
    # Bias correction uses the cartridge's own step: with beta = 0 it is 1 and
    # m1 = g exactly, so the step is lr * g / (|g| + eps).
    nx, n1, _ = adam.adam_step(x, g, m1, m2, step=3, lr=0.5, beta1=0.0, beta2=0.0, warmup_steps=0,
                               frozen_tokens=0, round_bf16=False)
    np.testing.assert_array_equal(n1, g)
    np.testing.assert_allclose(nx, x - 0.5 * g / (np.abs(g) + 1e-8), rtol=0, atol=1e-6)


def test_a5_library_warmup_factor_matches():
    """The library's host-side factor (cas_adam_lr_scale) equals the reference's."""
    import paper_2606_04557_amd as cas
    for W, N in ((20, 4), (20, 1), (7, 3), (0, 4)):
        for s in range(0, 50):
            assert cas.adam_lr_scale(s, W, N) == float(np.float32(adam.warmup_scale(s, W, N)))
    assert math.isnan(cas.adam_lr_scale(1, 20, 0))
