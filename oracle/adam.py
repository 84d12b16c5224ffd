"""Optimizer step of the trainable cartridges: reference for the tests.

TEST INFRASTRUCTURE ONLY. Nothing in the library's product path may import,
call or execute this module; only the tests and the bench's CPU-baseline leg
use it. It shares no code with the HIP library.

What is computed (paper: Section "Optimization Dynamics", paragraphs
"Optimizer" and "Per-cartridge LR warmup"; the hyperparameter table):
Adam on bf16 cartridge weights with fp32 state. Each cartridge ramps its own
learning rate: with s the number of steps it has been trained so far, its
rate is the global rate times min(1, s / W_c), quantised to N_b levels so a
step sees only a handful of distinct rates (W_c = 20; one frozen BOS token). Adam itself is Algorithm 1 of Kingma and Ba, "Adam: A
Method for Stochastic Optimization" (ICLR 2015):

    t  = s + 1
    m1 = beta1 m1 + (1 - beta1) g
    m2 = beta2 m2 + (1 - beta2) g^2
    m1_hat = m1 / (1 - beta1^t),  m2_hat = m2 / (1 - beta2^t)
    x  = x - lr m1_hat / (sqrt(m2_hat) + eps)

Precision: the paper fixes fp32 for the optimizer, so every operation above
runs in float32 (numpy, one rounding per operation, left to right), with
1 - beta^t evaluated in float64 and rounded once; the new parameter is then
rounded to bfloat16 (round to nearest even), the storage type of the weights.

Readings where the paper is silent: the N_b levels are 1/N_b, ..., 1 and the
warmup factor is rounded up to the next level (the first level also at
s = 0, so a newly loaded cartridge moves at once); bias correction counts the
cartridge's own steps (its moments start at zero when it is first trained);
the frozen tokens keep their parameters and moments untouched.
"""
from __future__ import annotations

import math

import numpy as np

F32 = np.float32


def warmup_scale(step: int, warmup_steps: int, buckets: int) -> float:
    """Bucketed per-cartridge warmup factor."""
    if warmup_steps <= 0:
        return 1.0
    exact = min(1.0, step / warmup_steps)
    level = max(1, math.ceil(buckets * exact - 1e-12))
    return min(level, buckets) / buckets


def one_minus_pow(beta: float, t: int) -> np.float32:
    """1 - beta^t in float64, rounded once to float32 (beta as stored in fp32)."""
    return F32(1.0 - float(F32(beta)) ** t)


def to_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 to the nearest bfloat16 (ties to even); returned as float32."""
    b = np.asarray(x, dtype=F32).view(np.uint32).astype(np.uint64)
    lsb = (b >> 16) & 1
    r = ((b + 0x7FFF + lsb) >> 16) << 16
    return r.astype(np.uint32).view(F32)


def adam_step(x, g, m1, m2, step: int, lr: float, beta1: float = 0.9, beta2: float = 0.999,
              eps: float = 1e-8, warmup_steps: int = 20, warmup_buckets: int = 4,
              frozen_tokens: int = 1, round_bf16: bool = True):
    """One step for one tensor [len, ...] (token axis first).

    x, g: parameter and gradient values (bf16 values as float32); m1, m2:
    float32 moments. Returns new (x, m1, m2); tokens below frozen_tokens are
    returned unchanged."""
    x = np.array(x, dtype=F32)
    g = np.asarray(g, dtype=F32)
    m1 = np.array(np.broadcast_to(np.asarray(m1, dtype=F32), x.shape))
    m2 = np.array(np.broadcast_to(np.asarray(m2, dtype=F32), x.shape))
    f = frozen_tokens
    t = step + 1
    b1, b2 = F32(beta1), F32(beta2)
    lr_c = F32(F32(lr) * F32(warmup_scale(step, warmup_steps, warmup_buckets)))
    a = b1 * m1[f:] + (F32(1) - b1) * g[f:]
    s = b2 * m2[f:] + (F32(1) - b2) * (g[f:] * g[f:])
    m1_hat = a / one_minus_pow(beta1, t)
    m2_hat = s / one_minus_pow(beta2, t)
    new = x[f:] - (lr_c * m1_hat) / (np.sqrt(m2_hat) + F32(eps))
    m1[f:] = a
    m2[f:] = s
    x[f:] = to_bf16(new) if round_bf16 else new
    return x, m1, m2
