"""Pins of the oracle's decode-time attention (section 8): special cases with closed-form
answers, invariances of softmax attention, the grouped-query head mapping, and agreement
with torch's scaled-dot-product attention on the CPU."""
import numpy as np
import pytest
import torch

from oracle import attention as oat


def test_equal_scores_average_the_values(rng):
    K = np.zeros((2, 7, 4))
    V = rng.standard_normal((2, 7, 4))
    Q = rng.standard_normal((2, 4))
    out = oat.attend(K, V, layer=0, n_heads=2, Q=Q, scale=0.5)
    np.testing.assert_allclose(out, V.mean(axis=1), rtol=1e-14)


def test_a_dominant_key_selects_its_value(rng):
    K = rng.standard_normal((1, 9, 8)) * 0.01
    K[0, 5] = 50.0 * np.ones(8)
    V = rng.standard_normal((1, 9, 8))
    out = oat.attend(K, V, 0, 1, np.ones((1, 8)), scale=1.0)
    np.testing.assert_allclose(out[0], V[0, 5], atol=1e-12)


def test_token_order_does_not_matter(rng):
    K, V = rng.standard_normal((3, 11, 6)), rng.standard_normal((3, 11, 6))
    Q = rng.standard_normal((3, 6))
    perm = rng.permutation(11)
    a = oat.attend(K, V, 0, 3, Q, 0.4)
    b = oat.attend(K[:, perm], V[:, perm], 0, 3, Q, 0.4)
    np.testing.assert_allclose(a, b, rtol=1e-12)


def test_grouped_query_heads_read_their_layer_and_group(rng):
    # 2 layers x 2 kv heads; layer 1, 6 query heads -> groups of 3 on slices 2 and 3
    K, V = rng.standard_normal((4, 5, 3)), rng.standard_normal((4, 5, 3))
    Q = rng.standard_normal((6, 3))
    out = oat.attend(K, V, layer=1, n_heads=2, Q=Q, scale=0.7)
    for j in range(6):
        s = 2 + j // 3
        w = np.exp(0.7 * K[s] @ Q[j])
        np.testing.assert_allclose(out[j], (w / w.sum()) @ V[s], rtol=1e-12)
    with pytest.raises(ValueError):
        oat.attend(K, V, 1, 2, Q[:5], 0.7)


def test_matches_torch_scaled_dot_product_attention(rng):
    H, rep, T, d = 4, 2, 33, 16
    K, V = rng.standard_normal((H, T, d)), rng.standard_normal((H, T, d))
    Q = rng.standard_normal((H * rep, d))
    out = oat.attend(K, V, 0, H, Q, 1.0 / np.sqrt(d))
    kt = torch.from_numpy(np.repeat(K, rep, axis=0))[None]       # [1, n_q, T, d]
    vt = torch.from_numpy(np.repeat(V, rep, axis=0))[None]
    qt = torch.from_numpy(Q)[None, :, None, :]                     # [1, n_q, 1, d]
    ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt)[0, :, 0].numpy()
    np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-12)
