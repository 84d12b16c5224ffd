"""Synthetic workloads for multi-cartridge prefix attention.

A workload is one attention layer: ``batch`` rows of ``q_len`` query tokens
with ``num_q_heads`` heads of size ``head_dim``, grouped onto
``num_kv_heads`` key/value heads, each row attending over a list of
cartridges (trainable KV prefixes) followed by its own causal self-KV.
Cartridges are stored once (``cart_lens``) and referenced by id from the
rows, so a cartridge referenced by several rows is one shared tensor.

Shapes follow the paper's setting: 8 KV heads of 128 channels with 32 query
heads, the 8B-class GQA layer whose bf16 KV footprint the paper quotes in its
cost analysis (Discussion section); cartridge lengths in the ranges of the
cartridge-size table (appendix on cartridge sizes); target-plus-distractor
mixes as in the mixed-visibility sampling (Eq. mixing); retrieval-style
selection of k cartridges from a pool (Inference section). The paper's QA
datasets and model weights are not used: seeded Gaussian tensors stand in.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional

import numpy as np

from . import rng


@dataclasses.dataclass
class Workload:
    name: str
    dtype: str                      # "bf16" or "fp32"
    batch: int
    q_len: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    cart_lens: List[int]            # one entry per distinct cartridge tensor
    rows: List[List[int]]           # per batch row: cartridge ids in prefix order
    seed: int
    q_std: float = 1.0
    cart_std: float = 1.0
    self_std: float = 1.0
    do_std: float = 1.0
    layouts: Optional[List[str]] = None   # per cartridge: "tok", "padded", "head"
    staged: Optional[List[int]] = None    # cartridge ids staged host -> HBM
    forward_only: bool = False
    description: str = ""
    q_lens: Optional[List[int]] = None    # packed samples: per-row query tokens (q_len is 0)

    @property
    def packed(self) -> bool:
        return self.q_lens is not None

    @property
    def row_lens(self) -> List[int]:
        return list(self.q_lens) if self.packed else [self.q_len] * self.batch

    @property
    def q_offsets(self) -> List[int]:
        return [0] + [int(x) for x in np.cumsum(self.row_lens)]

    @property
    def group_size(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    @property
    def scale(self) -> np.float32:
        return np.float32(1.0 / np.sqrt(self.head_dim))

    def prefix_len(self, b: int) -> int:
        return int(sum(self.cart_lens[c] for c in self.rows[b]))

    def visible_pairs(self) -> int:
        """Visible (query, key) pairs summed over query heads: each query
        sees its row's whole prefix plus self keys 0..t."""
        tot = 0
        for b, sq in enumerate(self.row_lens):
            tot += sq * self.prefix_len(b) + sq * (sq + 1) // 2
        return tot * self.num_q_heads

    def flops(self, per_pair: int) -> float:
        return float(per_pair) * self.head_dim * self.visible_pairs()


def _layouts_for(n: int, key: int) -> List[str]:
    """A quarter padded token stride, a quarter head-major, the rest plain."""
    u = rng.uniform(key, n)
    out = []
    for x in u:
        out.append("padded" if x < 0.25 else ("head" if x < 0.5 else "tok"))
    return out


def config(n: int) -> Workload:
    """The five benchmark configurations (1-based)."""
    if n == 1:
        return Workload(
            name="C1", dtype="fp32", batch=1, q_len=64, num_q_heads=4, num_kv_heads=2,
            head_dim=64, cart_lens=[128, 128], rows=[[0, 1]], seed=1,
            description="fp32 B=1 Hq=4 Hkv=2 d=64, 2x128 cartridges + 64 causal queries")
    if n == 2:
        ncart = 4
        return Workload(
            name="C2", dtype="bf16", batch=4, q_len=1024, num_q_heads=32, num_kv_heads=8,
            head_dim=128, cart_lens=[1024] * (4 * ncart),
            rows=[[b * ncart + i for i in range(ncart)] for b in range(4)], seed=2,
            cart_std=0.5,
            description="bf16 B=4 Hq=32 Hkv=8 d=128, 4x1024 cartridges (1 target + 3 "
                        "distractors) + 1024 causal queries")
    if n == 3:
        ncart = 16
        return Workload(
            name="C3", dtype="bf16", batch=2, q_len=2048, num_q_heads=32, num_kv_heads=8,
            head_dim=128, cart_lens=[2048] * (2 * ncart),
            rows=[[b * ncart + i for i in range(ncart)] for b in range(2)], seed=3,
            cart_std=0.5,
            description="bf16 B=2 Hq=32 Hkv=8 d=128, 16x2048 cartridges (32K prefix) + "
                        "2048 causal queries")
    if n == 4:
        lens = [int(x) for x in rng.randint(rng.stream_key(4, rng.TAG_LENGTHS), 64, 256, 4096)]
        return Workload(
            name="C4", dtype="bf16", batch=1, q_len=512, num_q_heads=32, num_kv_heads=8,
            head_dim=128, cart_lens=lens, rows=[list(range(64))], seed=4, cart_std=0.5,
            layouts=_layouts_for(64, rng.stream_key(4, rng.TAG_GAPS)),
            description="bf16 B=1 Hq=32 Hkv=8 d=128, 64 cartridges of U[256,4096] tokens "
                        "(non-contiguous, mixed layouts) + 512 causal queries")
    if n == 5:
        pool, nreq, k = 256, 64, 4
        rows = [rng.choose_distinct(rng.stream_key(5, rng.TAG_SELECT, r), pool, k)
                for r in range(nreq)]
        return Workload(
            name="C5", dtype="bf16", batch=nreq, q_len=64, num_q_heads=32, num_kv_heads=8,
            head_dim=128, cart_lens=[1024] * pool, rows=rows, seed=5, cart_std=0.5,
            staged=list(range(pool // 2, pool)), forward_only=True,
            description="bf16 forward: 64 requests x 64 causal queries, each over 4 of a "
                        "256 x 1024-token cartridge pool; second half staged host->HBM")
    raise ValueError(f"no config {n}")


def packed(seed: int = 6, total: int = 8192, pool: int = 20, k_max: int = 10,
           p_iso: float = 0.75) -> Workload:
    """Packed multi-sample training layout (paper: Section "Training with
    Multiple Cartridges", Eq. mixing, and the hyperparameter table: packed
    sequences of 8,192 tokens, a GPU pool of B = 20 cartridges, isolation
    probability 0.75, up to 10 distractors per example).

    Synthetic recipe (the paper fixes none of these lengths): cartridge
    lengths uniform on [256, 2048] in multiples of 16 (the page size); sample
    lengths uniform on [256, 2048], packed until ``total`` tokens (the last
    sample cut to fit); each sample draws a target from the pool and, with
    probability 1 - p_iso, k ~ U{1..k_max} distinct distractors, all in a
    shuffled order. bf16, 32 query heads, 8 KV heads, d = 128."""
    lens = [16 * int(x) for x in rng.randint(rng.stream_key(seed, rng.TAG_LENGTHS), pool, 16, 128)]
    q_lens: List[int] = []
    draws = rng.randint(rng.stream_key(seed, rng.TAG_LENGTHS, 1), 64, 256, 2048)
    for x in draws:
        room = total - sum(q_lens)
        if room <= 0:
            break
        q_lens.append(int(min(int(x), room)))
    assert sum(q_lens) == total
    rows = []
    for b in range(len(q_lens)):
        u = rng.uniform(rng.stream_key(seed, rng.TAG_SELECT, b), 3)
        target = int(np.floor(u[0] * pool))
        k = 0 if u[1] < p_iso else 1 + int(np.floor(u[2] * k_max))
        others = [c for c in range(pool) if c != target]
        pick = [others[i] for i in rng.choose_distinct(rng.stream_key(seed, rng.TAG_SELECT, b, 1),
                                                       pool - 1, k)]
        order = rng.choose_distinct(rng.stream_key(seed, rng.TAG_SELECT, b, 2), k + 1, k + 1)
        ids = [target] + pick
        rows.append([ids[i] for i in order])
    return Workload(
        name="P8K", dtype="bf16", batch=len(q_lens), q_len=0, num_q_heads=32, num_kv_heads=8,
        head_dim=128, cart_lens=lens, rows=rows, seed=seed, cart_std=0.5, q_lens=q_lens,
        description=f"bf16 packed training layout: {len(q_lens)} samples in {total} tokens, each over "
                    f"its own subset of a {pool}-cartridge pool (target + up to {k_max} distractors)")


def custom(name: str, dtype: str, batch: int, q_len: int, num_q_heads: int,
           num_kv_heads: int, head_dim: int, cart_lens: List[int],
           rows: List[List[int]], seed: int, **kw) -> Workload:
    return Workload(name=name, dtype=dtype, batch=batch, q_len=q_len,
                    num_q_heads=num_q_heads, num_kv_heads=num_kv_heads,
                    head_dim=head_dim, cart_lens=list(cart_lens),
                    rows=[list(r) for r in rows], seed=seed, **kw)


def _draw(key: int, shape, std: float, dtype: str) -> np.ndarray:
    n = int(np.prod(shape))
    x = rng.normal(key, n, std).reshape(shape)
    if dtype == "bf16":
        return rng.f64_to_bf16_bits(x)
    if dtype == "fp32":
        return rng.f64_to_f32(x)
    raise ValueError(dtype)


def make_tensors(wl: Workload, carts: Optional[List[int]] = None,
                 with_grad_out: bool = True) -> Dict[str, object]:
    """Seeded host tensors of ``wl``.

    bf16 tensors are returned as uint16 bit patterns, fp32 tensors as float32.
    ``carts`` restricts which cartridge tensors are drawn (others are None);
    each cartridge has its own substream, so the subset does not change the
    bits of the ones drawn.
    """
    B, Hq, Hkv, D = wl.batch, wl.num_q_heads, wl.num_kv_heads, wl.head_dim
    s = wl.seed
    lens = wl.row_lens
    # Fixed-length rows stack to [B, Sq, H, D]; packed samples concatenate to [T, H, D].
    join = np.concatenate if wl.packed else np.stack

    def per_row(tag, H, std):
        return join([_draw(rng.stream_key(s, tag, b), (lens[b], H, D), std, wl.dtype) for b in range(B)])

    out: Dict[str, object] = {}
    out["q"] = per_row(rng.TAG_Q, Hq, wl.q_std)
    out["k_self"] = per_row(rng.TAG_K_SELF, Hkv, wl.self_std)
    out["v_self"] = per_row(rng.TAG_V_SELF, Hkv, wl.self_std)
    if with_grad_out and not wl.forward_only:
        out["d_o"] = per_row(rng.TAG_DO, Hq, wl.do_std)
    want = range(len(wl.cart_lens)) if carts is None else carts
    ck: List[Optional[np.ndarray]] = [None] * len(wl.cart_lens)
    cv: List[Optional[np.ndarray]] = [None] * len(wl.cart_lens)
    for c in want:
        L = wl.cart_lens[c]
        ck[c] = _draw(rng.stream_key(s, rng.TAG_K_CART, c), (L, Hkv, D), wl.cart_std, wl.dtype)
        cv[c] = _draw(rng.stream_key(s, rng.TAG_V_CART, c), (L, Hkv, D), wl.cart_std, wl.dtype)
    out["cart_k"] = ck
    out["cart_v"] = cv
    return out


def to_float(x: np.ndarray, dtype: str) -> np.ndarray:
    """Exact float32 view of generated bits (bf16 widened, fp32 as is)."""
    if dtype == "bf16":
        return rng.bf16_bits_to_f32(x)
    return np.asarray(x, dtype=np.float32)
