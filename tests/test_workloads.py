"""Synthetic-input generator and benchmark shapes."""
import numpy as np

import casgen
from casgen import rng


def test_counter_form_matches_sequential_splitmix():
    """The vectorised counter form equals the sequential SplitMix64 recurrence
    (state += gamma; output = mix(state))."""
    key = rng.stream_key(3, 1, 2)
    got = rng.raw_u64(key, 6)
    state = key
    for i in range(6):
        state = (state + 0x9E3779B97F4A7C15) & ((1 << 64) - 1)
        assert int(got[i]) == rng._mix_py(state)
    # An offset window is the same stream.
    assert np.array_equal(rng.raw_u64(key, 3, start=3), got[3:])


def test_normal_moments_and_rounding():
    x = rng.normal(rng.stream_key(9), 1 << 18, std=0.5)
    assert abs(x.mean()) < 5e-3 and abs(x.std() - 0.5) < 5e-3
    bits = rng.f64_to_bf16_bits(x)
    back = rng.bf16_bits_to_f32(bits).astype(np.float64)
    # RNE to bf16: relative error at most 2^-9.
    assert np.all(np.abs(back - x) <= np.abs(x) * 2.0 ** -8 + 1e-30)
    # Exactly representable values round-trip.
    v = np.array([1.0, -2.5, 0.15625, 3.0 * 2 ** -20], dtype=np.float32)
    assert np.array_equal(rng.bf16_bits_to_f32(rng.f32_to_bf16_bits(v)), v)
    # Ties go to even: 1 + 2^-8 lies halfway between 1 and 1 + 2^-7.
    t = np.array([1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8], dtype=np.float32)
    assert np.array_equal(rng.bf16_bits_to_f32(rng.f32_to_bf16_bits(t)),
                          np.array([1.0, 1.0 + 2.0 ** -6], dtype=np.float32))


def test_kv_footprint_matches_paper():
    """The 8B-class layer shape (8 KV heads x 128 channels, bf16) gives the
    paper's quoted KV-cache footprint of about 141 MiB per 1K tokens for the
    4B/8B models (Discussion, cost analysis), with the 36 decoder layers of the
    public Qwen3-8B configuration (a fact about the model, not printed in the paper)."""
    wl = casgen.config(3)
    per_token_per_layer = 2 * wl.num_kv_heads * wl.head_dim * 2
    assert per_token_per_layer == 4096
    mib = 1000 * 36 * per_token_per_layer / 2 ** 20
    assert abs(mib - 141) < 0.5


def test_config_shapes():
    c = [casgen.config(i) for i in range(1, 6)]
    assert [w.dtype for w in c] == ["fp32", "bf16", "bf16", "bf16", "bf16"]
    assert c[0].visible_pairs() == 73856
    assert c[1].visible_pairs() == 604045312
    assert c[2].visible_pairs() == 4429250560
    assert c[4].visible_pairs() == 541130752
    assert c[2].prefix_len(0) == 32768
    lens = c[3].cart_lens
    assert len(lens) == 64 and min(lens) >= 256 and max(lens) <= 4096
    sel = c[4].rows
    assert len(sel) == 64 and all(len(set(r)) == 4 for r in sel)
    assert all(0 <= x < 256 for r in sel for x in r)


def test_tensors_are_seeded_and_substreamed():
    wl = casgen.custom("t", "bf16", 2, 5, 4, 2, 64, [7, 3, 2], [[0, 1], [2, 1]], seed=11,
                       cart_std=0.5)
    a = casgen.make_tensors(wl)
    b = casgen.make_tensors(wl, carts=[1])
    assert a["q"].dtype == np.uint16 and a["q"].shape == (2, 5, 4, 64)
    assert np.array_equal(a["q"], b["q"])
    assert np.array_equal(a["cart_k"][1], b["cart_k"][1])
    assert b["cart_k"][0] is None
    assert not np.array_equal(a["cart_k"][1][:2], a["cart_v"][1][:2])


def test_packed_training_layout():
    """8,192 packed tokens; every sample sees its target and at most 10
    distractors, all distinct, from a 20-cartridge pool; cartridge lengths are
    multiples of 16."""
    w = casgen.packed()
    assert w.packed and w.q_len == 0 and sum(w.q_lens) == 8192 and w.q_offsets[-1] == 8192
    assert len(w.cart_lens) == 20 and all(L % 16 == 0 and 256 <= L <= 2048 for L in w.cart_lens)
    assert all(1 <= len(r) <= 11 and len(set(r)) == len(r) for r in w.rows)
    assert any(len(r) == 1 for r in w.rows) and any(len(r) > 1 for r in w.rows)
    T = casgen.make_tensors(w)
    assert T["q"].shape == (8192, 32, 128) and T["k_self"].shape == (8192, 8, 128)
    pairs = sum(L * w.prefix_len(b) + L * (L + 1) // 2 for b, L in enumerate(w.q_lens)) * 32
    assert w.visible_pairs() == pairs
