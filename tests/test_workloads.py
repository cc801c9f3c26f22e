"""The seeded input generator: determinism, bf16 rounding and table shapes."""
import numpy as np

from workloads import (DENSE, FRAME_LOCAL, TOPK, WORKLOADS, bf16_bits_from_f32,
                       bf16_bits_to_f32, make_qkv, make_table)


def test_bf16_rounding_is_nearest_even():
    x = np.array([1.0, 1.00390625, 1.01171875, 1.0 + 2 ** -8 + 2 ** -20, -2.5, 3.0e38], np.float32)
    bits = bf16_bits_from_f32(x)
    # bf16 steps near 1 are 2^-7: 1+2^-8 ties to even (1.0), 1+3*2^-8 ties to
    # even (1+2^-6 = 0x3F82), anything above a tie rounds up
    assert list(bits) == [0x3F80, 0x3F80, 0x3F82, 0x3F81, 0xC020, 0x7F62]
    np.testing.assert_array_equal(bf16_bits_to_f32(bits)[:2], [1.0, 1.0])


def test_generation_is_deterministic_and_seeded():
    w = WORKLOADS["S4xT261-f32"]
    a = make_qkv(w, seed=3)
    b = make_qkv(w, seed=3)
    c = make_qkv(w, seed=4)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)
    assert not np.array_equal(a[0], c[0])
    assert a[0].shape == (16, 1044, 64) and a[0].dtype == np.float32


def test_special_keys_have_large_norm():
    w = WORKLOADS["S4xT261-f32"]
    _, k, _ = make_qkv(w, heads=[0])
    norms = np.linalg.norm(k[0], axis=1)
    special = (np.arange(w.tokens) % w.tokens_per_frame) < 5
    assert norms[special].mean() > 3 * norms[~special].mean()


def test_tables_follow_their_rules():
    t = make_table(WORKLOADS["S4xT261-f32"])
    assert sorted(p for p, _ in t) == [DENSE] * 4 + [FRAME_LOCAL] * 6 + [TOPK] * 6
    assert {k for p, k in t if p == TOPK} == {2}
    t = make_table(WORKLOADS["S8xT1374-bf16"])
    assert sorted(p for p, _ in t) == [DENSE] + [FRAME_LOCAL] * 6 + [TOPK] * 9
    assert {k for p, k in t if p == TOPK} == {13}
    t = make_table(WORKLOADS["S100xT1374-bf16"])
    assert sorted(p for p, _ in t) == [FRAME_LOCAL] * 6 + [TOPK] * 10
    assert {k for p, k in t if p == TOPK} == {159}
    t = make_table(WORKLOADS["S32xT1374-bf16"])
    assert {k for p, k in t if p == TOPK} <= {14, 35, 69, 138}
    w = WORKLOADS["S200xT1374-bf16-L24"]
    for layer in range(w.layers):
        t = make_table(w, layer)
        assert all(1 <= k <= w.nb for p, k in t if p == TOPK)
