"""Pins of the oracle's elementary operations against library routines and
closed forms (CPU only)."""
import numpy as np
import pytest
import torch

from oracle.numerics import bf16, layer_norm, gelu, attention, rope, rope_tables, softmax
from oracle.philox import philox4x64, _mulhilo, to_uniform, uniforms


def test_bf16_matches_torch_rne():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 10 ** rng.uniform(-6, 6, 100000).astype(np.float32),
                        np.array([0.0, -0.0, 1.0, 1.00390625, 1.01171875, -2.5], np.float32)])
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    np.testing.assert_array_equal(bf16(x), ref)


def test_layer_norm_matches_torch():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((7, 96)) * 3 + 1.5
    g = rng.standard_normal(96)
    b = rng.standard_normal(96)
    ref = torch.nn.functional.layer_norm(torch.from_numpy(x), (96,), torch.from_numpy(g), torch.from_numpy(b), 1e-5).numpy()
    np.testing.assert_allclose(layer_norm(x, g, b, np.float64), ref, rtol=0, atol=1e-12)


def test_gelu_exact_erf():
    x = np.linspace(-8, 8, 2001)
    ref = torch.nn.functional.gelu(torch.from_numpy(x), approximate="none").numpy()
    np.testing.assert_allclose(gelu(x), ref, rtol=0, atol=1e-14)
    # closed forms: GELU(0) = 0, GELU(x) - GELU(-x) = x
    assert gelu(np.array([0.0]))[0] == 0.0
    np.testing.assert_allclose(gelu(x) - gelu(-x), x, atol=1e-14)


def test_attention_matches_sdpa_causal_and_full():
    rng = np.random.default_rng(2)
    R, T, H, hd = 5, 11, 3, 64
    q = rng.standard_normal((R, H, hd))
    k = rng.standard_normal((T, H, hd))
    v = rng.standard_normal((T, H, hd))
    pos = np.arange(T - R, T)
    allowed = np.arange(T)[None, :] <= pos[:, None]
    out = attention(q, k, v, allowed, np.float64)
    tq = torch.from_numpy(q).permute(1, 0, 2)
    tk = torch.from_numpy(k).permute(1, 0, 2)
    tv = torch.from_numpy(v).permute(1, 0, 2)
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=torch.from_numpy(allowed))
    np.testing.assert_allclose(out, ref.permute(1, 0, 2).reshape(R, H * hd).numpy(), atol=1e-12)
    full = attention(q, k, v, np.ones((R, T), bool), np.float64)
    ref2 = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv)
    np.testing.assert_allclose(full, ref2.permute(1, 0, 2).reshape(R, H * hd).numpy(), atol=1e-12)


def test_softmax_sums_to_one_and_shift_invariant():
    rng = np.random.default_rng(3)
    s = rng.standard_normal((4, 50)) * 30
    p = softmax(s)
    np.testing.assert_allclose(p.sum(-1), 1.0, atol=1e-12)
    np.testing.assert_allclose(softmax(s + 1234.5), p, atol=1e-12)


def test_rope_rotation_direction_pairing_and_norm():
    hd = 64
    # position 0 is the identity
    x = np.random.default_rng(4).standard_normal((3, 2, hd))
    np.testing.assert_allclose(rope(x, [0, 0, 0], np.float64), x, atol=0)
    # basis vector e_i at position p rotates into the plane (i, i+32) by +theta_i(p)
    c, s = rope_tables(np.array([5]), hd)
    for i in (0, 7, 31):
        e = np.zeros((1, 1, hd))
        e[0, 0, i] = 1.0
        y = rope(e, [5], np.float64)[0, 0]
        theta = np.float32(np.float32(5.0) * np.float32(10000.0 ** (-2 * i / 64)))
        assert abs(y[i] - np.cos(np.float64(theta))) < 1e-7
        assert abs(y[i + 32] - np.sin(np.float64(theta))) < 1e-7
        assert np.count_nonzero(np.abs(y) > 1e-12) <= 2
    # rotations preserve norms
    y = rope(x, [3, 77, 400], np.float64)
    np.testing.assert_allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-6)


def test_rope_relative_property():
    """<RoPE(q, m), RoPE(k, n)> depends only on m - n (up to fp32 phase rounding)."""
    rng = np.random.default_rng(5)
    q = rng.standard_normal((1, 1, 64))
    k = rng.standard_normal((1, 1, 64))
    base = (rope(q, [10], np.float64) * rope(k, [3], np.float64)).sum()
    for delta in (1, 50, 300):
        shifted = (rope(q, [10 + delta], np.float64) * rope(k, [3 + delta], np.float64)).sum()
        assert abs(shifted - base) < 1e-4 * np.linalg.norm(q) * np.linalg.norm(k)


def test_mulhilo_brute():
    rng = np.random.default_rng(6)
    a = rng.integers(0, 2 ** 63, 500, dtype=np.uint64) * np.uint64(2) + rng.integers(0, 2, 500, dtype=np.uint64)
    b = rng.integers(0, 2 ** 63, 500, dtype=np.uint64) * np.uint64(2) + np.uint64(1)
    hi, lo = _mulhilo(a, b)
    for x, y, h, l in zip(a, b, hi, lo):
        p = int(x) * int(y)
        assert p >> 64 == int(h) and p & (2 ** 64 - 1) == int(l)


@pytest.mark.parametrize("key", [(0, 0), (0x123456789ABCDEF0, 0x0FEDCBA987654321), (2 ** 64 - 1, 2 ** 64 - 1)])
def test_philox_matches_numpy_bit_generator(key):
    """numpy's Philox bit generator is Philox4x64-10; its raw output for counter c is
    produced after it increments the stored counter, so store c - 1."""
    key = np.array(key, dtype=np.uint64)
    for ctr0 in ([5, 7, 11, 13], [2 ** 64 - 3, 0, 2 ** 40, 1]):
        ctr = np.array(ctr0, dtype=np.uint64)
        bg = np.random.Philox(key=key)
        st = bg.state
        st["state"]["counter"] = ctr - np.array([1, 0, 0, 0], dtype=np.uint64)
        st["buffer_pos"] = 4
        bg.state = st
        raw = bg.random_raw(8)
        nxt = ctr.copy()
        nxt[0] = nxt[0] + np.uint64(1)
        if nxt[0] == 0:
            nxt[1] += np.uint64(1)
        mine = philox4x64(np.stack([ctr, nxt]), key)
        np.testing.assert_array_equal(raw, mine.reshape(-1))


def test_uniforms_in_open_interval_and_uniform():
    x = np.array([0, 2 ** 64 - 1, 2 ** 41 - 1, 2 ** 41], dtype=np.uint64)
    u = to_uniform(x)
    assert u[0] == np.float32(0.5 * 2 ** -23) and u[1] == np.float32(1 - 0.5 * 2 ** -23)
    assert u[2] == u[0] and u[3] == np.float32(1.5 * 2 ** -23)
    v = uniforms(9, 2, 3, 4, 5, 200000)
    assert v.dtype == np.float32 and v.min() > 0 and v.max() < 1
    hist, _ = np.histogram(v, bins=20, range=(0, 1))
    exp = len(v) / 20
    chi2 = ((hist - exp) ** 2 / exp).sum()
    assert chi2 < 50  # 19 dof, p ~ 1e-4
