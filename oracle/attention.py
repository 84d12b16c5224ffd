"""fp64 reference for multi-cartridge prefix attention (forward and backward).

TEST INFRASTRUCTURE ONLY. Nothing in the library's product path may import,
call or execute this module; only the tests, the smoke check and the bench's
CPU-baseline leg use it. It shares no code with the HIP library.

What is computed (paper, Section "Cartridges at Scale (CAS) Training",
Background paragraph; Section "Inference"; Limitations, "Cartridge KV
position"):

* A cartridge is a trainable KV prefix injected into an attention layer.
  Several cartridges are concatenated in order and placed before the query
  tokens; the query tokens then see each other under ordinary causal masking.
  So for batch row b, query head h and query position t, with key/value head
  kv = floor(h / group_size), the visible keys are every token of every
  cartridge of row b in order, then the row's own tokens 0..t.
* Softmax attention over the visible keys: scores s_j = scale * q . k_j,
  row log-sum-exp LSE = m + ln sum_j exp(s_j - m) with m = max_j s_j,
  probabilities P_j = exp(s_j - LSE), output O = sum_j P_j v_j.
* Only the cartridges' keys and values are trained and the model is frozen,
  so the backward returns dK/dV for each cartridge (plus dQ, and dK/dV of the
  self tokens, which flow into the frozen model below). Given dO:
  D = dO . O, dP_j = dO . v_j, dS_j = P_j (dP_j - D),
  dQ = scale * sum_j dS_j k_j, dK_j += scale * dS_j q, dV_j += P_j dO.
  A cartridge referenced several times (by several rows, or twice in one row)
  is one tensor, so its gradient is the sum over every reference.

Readings where the paper is silent: contiguous GQA groups (kv = h // g);
inclusive causal diagonal (j <= t); keys and queries arrive post-RoPE, so no
positional operation is applied here; LSE in natural log.

Everything runs in float64 with two-pass softmax (max, then sum), no tiling
and no online rescaling; matrix products use numpy's matmul as a primitive.
"""
from __future__ import annotations

from typing import List, Optional, Sequence

import numpy as np


def _f64(x) -> np.ndarray:
    return np.asarray(x, dtype=np.float64)


def visible_mask(n_prefix: int, q_len: int, t_idx: Sequence[int]) -> np.ndarray:
    """Boolean [len(t_idx), n_prefix + q_len]: prefix keys always visible,
    self key j visible to query t iff j <= t."""
    t = np.asarray(t_idx, dtype=np.int64)[:, None]
    j = np.arange(q_len, dtype=np.int64)[None, :]
    self_vis = j <= t
    pre = np.ones((t.shape[0], n_prefix), dtype=bool)
    return np.concatenate([pre, self_vis], axis=1)


def row_keys(cart_k: Sequence, cart_v: Sequence, row: Sequence[int], k_self_b, v_self_b,
             kv: int):
    """Concatenated key/value matrices [n_prefix + q_len, D] of one batch row
    and one KV head, in prefix order, plus the number of prefix tokens."""
    ks = [_f64(cart_k[c])[:, kv, :] for c in row]
    vs = [_f64(cart_v[c])[:, kv, :] for c in row]
    n_prefix = int(sum(k.shape[0] for k in ks))
    K = np.concatenate(ks + [_f64(k_self_b)[:, kv, :]], axis=0)
    V = np.concatenate(vs + [_f64(v_self_b)[:, kv, :]], axis=0)
    return K, V, n_prefix


def head_forward(qh: np.ndarray, K: np.ndarray, V: np.ndarray, n_prefix: int, q_len: int,
                 t_idx: Sequence[int], scale: float):
    """Forward for the query rows ``t_idx`` of one (row, head).

    Returns O [T, D], LSE [T] and the probability matrix P [T, N]."""
    mask = visible_mask(n_prefix, q_len, t_idx)
    S = float(scale) * (qh @ K.T)
    S = np.where(mask, S, -np.inf)
    m = S.max(axis=1)
    l = np.exp(S - m[:, None]).sum(axis=1)
    lse = m + np.log(l)
    P = np.exp(S - lse[:, None])          # exp(-inf) = 0 on hidden keys
    O = P @ V
    return O, lse, P


def head_backward(qh: np.ndarray, K: np.ndarray, V: np.ndarray, n_prefix: int, q_len: int,
                  t_idx: Sequence[int], scale: float, dOh: np.ndarray, Oh: np.ndarray,
                  lse: np.ndarray, key_cols: Optional[np.ndarray] = None):
    """Backward for the query rows ``t_idx`` of one (row, head).

    ``Oh`` and ``lse`` are this oracle's own forward results for those rows.
    Returns dQ [T, D] (only meaningful when ``key_cols`` is None) and the
    contributions of these rows to dK and dV over the key columns
    ``key_cols`` (all keys when None)."""
    mask = visible_mask(n_prefix, q_len, t_idx)
    if key_cols is not None:
        mask = mask[:, key_cols]
        K = K[key_cols]
        V = V[key_cols]
    S = float(scale) * (qh @ K.T)
    P = np.where(mask, np.exp(S - lse[:, None]), 0.0)
    Dr = (dOh * Oh).sum(axis=1)
    dP = dOh @ V.T
    dS = P * (dP - Dr[:, None])
    dQ = float(scale) * (dS @ K)
    dK = float(scale) * (dS.T @ qh)
    dV = P.T @ dOh
    return dQ, dK, dV


def forward(q, k_self, v_self, cart_k: Sequence, cart_v: Sequence, rows: Sequence[Sequence[int]],
            scale: float, group_size: int, kv_heads: Optional[Sequence[int]] = None):
    """O [B, Sq, Hq, D] and LSE [B, Hq, Sq] over [cartridges of the row || causal self].

    With ``kv_heads`` given, only the query heads of those KV heads' groups
    are evaluated (every other head's O and LSE stay zero)."""
    q = _f64(q)
    B, Sq, Hq, Dh = q.shape
    O = np.zeros((B, Sq, Hq, Dh))
    LSE = np.zeros((B, Hq, Sq))
    t_all = np.arange(Sq)
    for b in range(B):
        for h in range(Hq):
            kv = h // group_size
            if kv_heads is not None and kv not in kv_heads:
                continue
            K, V, npre = row_keys(cart_k, cart_v, rows[b], k_self[b], v_self[b], kv)
            o, lse, _ = head_forward(q[b, :, h, :], K, V, npre, Sq, t_all, scale)
            O[b, :, h, :] = o
            LSE[b, h, :] = lse
    return O, LSE


def backward(q, k_self, v_self, cart_k: Sequence, cart_v: Sequence, rows: Sequence[Sequence[int]],
             scale: float, group_size: int, d_o, O=None, LSE=None,
             kv_heads: Optional[Sequence[int]] = None):
    """Gradients of sum(dO * O).

    Returns dq, dk_self, dv_self, dcart_k, dcart_v; dcart_* hold one entry per
    cartridge tensor (None for cartridges no row references) and sum over all
    references of that cartridge.

    With ``kv_heads`` given, only those KV heads (and the query heads of
    their groups) are evaluated; every other head's gradients stay zero. The
    gradients of a KV head depend on its own group's queries only, so the
    evaluated heads are complete."""
    q = _f64(q)
    d_o = _f64(d_o)
    B, Sq, Hq, Dh = q.shape
    Hkv = np.asarray(k_self).shape[2]
    if O is None or LSE is None:
        O, LSE = forward(q, k_self, v_self, cart_k, cart_v, rows, scale, group_size, kv_heads)
    dq = np.zeros_like(q)
    dk_self = np.zeros((B, Sq, Hkv, Dh))
    dv_self = np.zeros((B, Sq, Hkv, Dh))
    dck: List[Optional[np.ndarray]] = [None] * len(cart_k)
    dcv: List[Optional[np.ndarray]] = [None] * len(cart_k)
    for b in range(B):
        for c in rows[b]:
            if dck[c] is None:
                shp = np.asarray(cart_k[c]).shape
                dck[c] = np.zeros(shp)
                dcv[c] = np.zeros(shp)
    t_all = np.arange(Sq)
    for b in range(B):
        for h in range(Hq):
            kv = h // group_size
            if kv_heads is not None and kv not in kv_heads:
                continue
            K, V, npre = row_keys(cart_k, cart_v, rows[b], k_self[b], v_self[b], kv)
            dQh, dK, dV = head_backward(q[b, :, h, :], K, V, npre, Sq, t_all, scale,
                                        d_o[b, :, h, :], O[b, :, h, :], LSE[b, h, :])
            dq[b, :, h, :] = dQh
            off = 0
            for c in rows[b]:
                L = np.asarray(cart_k[c]).shape[0]
                dck[c][:, kv, :] += dK[off:off + L]
                dcv[c][:, kv, :] += dV[off:off + L]
                off += L
            dk_self[b, :, kv, :] += dK[off:]
            dv_self[b, :, kv, :] += dV[off:]
    return dq, dk_self, dv_self, dck, dcv


# ---------------------------------------------------------------------------
# Sampled evaluation for large shapes: the same definitions, evaluated only on
# chosen query rows or chosen key columns.
# ---------------------------------------------------------------------------

def rows_forward_backward(q, k_self, v_self, cart_k, cart_v, rows, scale, group_size,
                          b: int, h: int, t_idx: Sequence[int], d_o=None):
    """O, LSE (and dQ when ``d_o`` is given) for query rows ``t_idx`` of (b, h)."""
    q = _f64(q)
    Sq = q.shape[1]
    kv = h // group_size
    K, V, npre = row_keys(cart_k, cart_v, rows[b], k_self[b], v_self[b], kv)
    t_idx = np.asarray(t_idx)
    o, lse, _ = head_forward(q[b, t_idx, h, :], K, V, npre, Sq, t_idx, scale)
    if d_o is None:
        return o, lse, None
    dQ, _, _ = head_backward(q[b, t_idx, h, :], K, V, npre, Sq, t_idx, scale,
                             _f64(d_o)[b, t_idx, h, :], o, lse)
    return o, lse, dQ


def key_grads(q, k_self, v_self, cart_k, cart_v, rows, scale, group_size, d_o, kv: int,
              cart: int, tok_idx: Sequence[int]):
    """dK, dV [len(tok_idx), D] for KV head ``kv`` at tokens ``tok_idx`` of
    cartridge ``cart`` (summed over every reference to it), or of the self
    keys of batch row ``-cart - 1`` when ``cart`` is negative.

    Each contributing (row, head) is evaluated with its full forward, since
    every query's LSE and O enter the gradient."""
    q = _f64(q)
    d_o = _f64(d_o)
    B, Sq, Hq, Dh = q.shape
    tok_idx = np.asarray(tok_idx, dtype=np.int64)
    dK = np.zeros((len(tok_idx), Dh))
    dV = np.zeros((len(tok_idx), Dh))
    t_all = np.arange(Sq)
    for b in range(B):
        if cart < 0:
            if b != -cart - 1:
                continue
            uses = [None]
        else:
            uses = []
            off = 0
            for c in rows[b]:
                if c == cart:
                    uses.append(off)
                off += np.asarray(cart_k[c]).shape[0]
            if not uses:
                continue
        for hh in range(group_size):
            h = kv * group_size + hh
            K, V, npre = row_keys(cart_k, cart_v, rows[b], k_self[b], v_self[b], kv)
            o, lse, _ = head_forward(q[b, :, h, :], K, V, npre, Sq, t_all, scale)
            for off in uses:
                cols = (npre + tok_idx) if off is None else (off + tok_idx)
                _, dk, dv = head_backward(q[b, :, h, :], K, V, npre, Sq, t_all, scale,
                                          d_o[b, :, h, :], o, lse, key_cols=cols)
                dK += dk
                dV += dv
    return dK, dV


def key_grads_many(q, k_self, v_self, cart_k, cart_v, rows, scale, group_size, d_o, kv: int,
                   targets):
    """``key_grads`` for several (cart, tok_idx) targets of one KV head, sharing
    each contributing (row, head) forward. Returns [(dK, dV), ...]."""
    q = _f64(q)
    d_o = _f64(d_o)
    B, Sq, Hq, Dh = q.shape
    out = [(np.zeros((len(t), Dh)), np.zeros((len(t), Dh))) for _, t in targets]
    t_all = np.arange(Sq)
    for b in range(B):
        cols_per_target = []
        for cart, toks in targets:
            toks = np.asarray(toks, dtype=np.int64)
            cols = []
            if cart < 0:
                if b == -cart - 1:
                    cols.append(None)
            else:
                off = 0
                for c in rows[b]:
                    if c == cart:
                        cols.append(off)
                    off += np.asarray(cart_k[c]).shape[0]
            cols_per_target.append((toks, cols))
        if not any(cols for _, cols in cols_per_target):
            continue
        K, V, npre = row_keys(cart_k, cart_v, rows[b], k_self[b], v_self[b], kv)
        for hh in range(group_size):
            h = kv * group_size + hh
            o, lse, _ = head_forward(q[b, :, h, :], K, V, npre, Sq, t_all, scale)
            for i, (toks, cols) in enumerate(cols_per_target):
                for off in cols:
                    kc = (npre + toks) if off is None else (off + toks)
                    _, dk, dv = head_backward(q[b, :, h, :], K, V, npre, Sq, t_all, scale,
                                              d_o[b, :, h, :], o, lse, key_cols=kc)
                    out[i][0][:] += dk
                    out[i][1][:] += dv
    return out


# ---------------------------------------------------------------------------
# Packed samples (paper: Section "Training with Multiple Cartridges" and Eq.
# mixing: every training example carries its own target and distractor
# cartridges). Several samples share one token axis; sample b owns tokens
# q_offsets[b] .. q_offsets[b+1]-1 and attends over its own cartridges, then
# causally over its own tokens only (block-diagonal self). Each sample is the
# single-row problem above; a cartridge that several samples reference gets
# the sum of their gradients.
# ---------------------------------------------------------------------------

def _sample(x, a: int, e: int):
    return _f64(x)[None, a:e]


def packed_forward(q, k_self, v_self, cart_k: Sequence, cart_v: Sequence,
                   rows: Sequence[Sequence[int]], q_offsets: Sequence[int], scale: float,
                   group_size: int):
    """O [T, Hq, D] and LSE [Hq, T] of packed samples (q [T, Hq, D], k_self and
    v_self [T, Hkv, D])."""
    q = _f64(q)
    T, Hq, Dh = q.shape
    O = np.zeros((T, Hq, Dh))
    LSE = np.zeros((Hq, T))
    for b in range(len(rows)):
        a, e = int(q_offsets[b]), int(q_offsets[b + 1])
        if e == a:
            continue
        o, lse = forward(q[None, a:e], _sample(k_self, a, e), _sample(v_self, a, e), cart_k, cart_v,
                         [rows[b]], scale, group_size)
        O[a:e] = o[0]
        LSE[:, a:e] = lse[0]
    return O, LSE


def packed_backward(q, k_self, v_self, cart_k: Sequence, cart_v: Sequence,
                    rows: Sequence[Sequence[int]], q_offsets: Sequence[int], scale: float,
                    group_size: int, d_o, O=None, LSE=None):
    """Gradients of sum(dO * O) for packed samples: dq [T, Hq, D], dk_self and
    dv_self [T, Hkv, D], and per-cartridge dK/dV summed over every sample (and
    every reference within a sample) that uses the cartridge."""
    q = _f64(q)
    d_o = _f64(d_o)
    T, Hq, Dh = q.shape
    Hkv = np.asarray(k_self).shape[1]
    if O is None or LSE is None:
        O, LSE = packed_forward(q, k_self, v_self, cart_k, cart_v, rows, q_offsets, scale, group_size)
    dq = np.zeros_like(q)
    dk_self = np.zeros((T, Hkv, Dh))
    dv_self = np.zeros((T, Hkv, Dh))
    dck: List[Optional[np.ndarray]] = [None] * len(cart_k)
    dcv: List[Optional[np.ndarray]] = [None] * len(cart_k)
    for b in range(len(rows)):
        a, e = int(q_offsets[b]), int(q_offsets[b + 1])
        for c in rows[b]:
            if dck[c] is None:
                shp = np.asarray(cart_k[c]).shape
                dck[c] = np.zeros(shp)
                dcv[c] = np.zeros(shp)
        if e == a:
            continue
        g = backward(q[None, a:e], _sample(k_self, a, e), _sample(v_self, a, e), cart_k, cart_v,
                     [rows[b]], scale, group_size, d_o[None, a:e], O=_f64(O)[None, a:e],
                     LSE=_f64(LSE)[None, :, a:e])
        dq[a:e] = g[0][0]
        dk_self[a:e] = g[1][0]
        dv_self[a:e] = g[2][0]
        for c in set(rows[b]):
            dck[c] += g[3][c]
            dcv[c] += g[4][c]
    return dq, dk_self, dv_self, dck, dcv


def packed_rows_forward_backward(q, k_self, v_self, cart_k, cart_v, rows, q_offsets, scale,
                                 group_size, b: int, h: int, t_idx: Sequence[int], d_o=None):
    """rows_forward_backward for sample b of packed samples (t_idx local to it)."""
    a, e = int(q_offsets[b]), int(q_offsets[b + 1])
    return rows_forward_backward(_sample(q, a, e), _sample(k_self, a, e), _sample(v_self, a, e),
                                 cart_k, cart_v, [rows[b]], scale, group_size, 0, h, t_idx,
                                 None if d_o is None else _sample(d_o, a, e))


def packed_key_grads_many(q, k_self, v_self, cart_k, cart_v, rows, q_offsets, scale, group_size,
                          d_o, kv: int, targets):
    """key_grads_many for packed samples: a target (cart, toks) with cart >= 0
    sums over every sample that references the cartridge; cart = -b-1 names
    the self keys of sample b (toks local to it)."""
    Dh = np.asarray(q).shape[2]
    out = [(np.zeros((len(t), Dh)), np.zeros((len(t), Dh))) for _, t in targets]
    for b in range(len(rows)):
        a, e = int(q_offsets[b]), int(q_offsets[b + 1])
        if e == a:
            continue
        local = []
        for i, (cart, toks) in enumerate(targets):
            if cart >= 0 and cart in rows[b]:
                local.append((i, (cart, toks)))
            elif cart < 0 and -cart - 1 == b:
                local.append((i, (-1, toks)))
        if not local:
            continue
        res = key_grads_many(_sample(q, a, e), _sample(k_self, a, e), _sample(v_self, a, e), cart_k,
                             cart_v, [rows[b]], scale, group_size, _sample(d_o, a, e), kv,
                             [t for _, t in local])
        for (i, _), (dk, dv) in zip(local, res):
            out[i][0][:] += dk
            out[i][1][:] += dv
    return out


# ---------------------------------------------------------------------------
# Short-query / decode attention over paged cartridges (paper: Section
# "Inference", paragraph "Cartridge RAG", appendix on cartridge sizes: the
# retrieved cartridges' KV caches, kept in 16-token pages, precede the
# prompt). Request b's keys are its pages in order, cut to kv_lens[b]; its
# n_b queries are the last n_b positions: query i sees keys 0 .. L - n + i.
# ---------------------------------------------------------------------------

def paged_keys(k_pages, v_pages, pages: Sequence[int], kv_len: int):
    """Keys and values [kv_len, Hkv, D] of one request, gathered from its pages."""
    K = np.concatenate([_f64(k_pages[p]) for p in pages], axis=0)[:kv_len]
    V = np.concatenate([_f64(v_pages[p]) for p in pages], axis=0)[:kv_len]
    return K, V


def paged_decode_forward(q, k_pages, v_pages, q_counts: Sequence[int], kv_lens: Sequence[int],
                         page_lists: Sequence[Sequence[int]], scale: float, group_size: int):
    """O [Tq, Hq, D] and LSE [Hq, Tq] (q packed by request, [Tq, Hq, D])."""
    q = _f64(q)
    Tq, Hq, Dh = q.shape
    O = np.zeros((Tq, Hq, Dh))
    LSE = np.zeros((Hq, Tq))
    q0 = 0
    for b, n in enumerate(q_counts):
        L = int(kv_lens[b])
        K, V = paged_keys(k_pages, v_pages, page_lists[b], L)
        for h in range(Hq):
            kv = h // group_size
            o, lse, _ = head_forward(q[q0:q0 + n, h, :], K[:, kv, :], V[:, kv, :], L - n, n,
                                     np.arange(n), scale)
            O[q0:q0 + n, h, :] = o
            LSE[h, q0:q0 + n] = lse
        q0 += n
    return O, LSE
