"""Pins for the oracle's causal grouped-query attention: a library routine
(torch CPU float64 SDPA), closed forms and special cases."""
import numpy as np
import pytest
import torch

from oracle.attention import attend


def _rand(rng, *shape):
    return rng.standard_normal(shape)


def _torch_reference(q, k, v, q_pos, k_pos, scale, visible=None):
    n, Hq, D = q.shape
    Hkv = k.shape[1]
    group = Hq // Hkv
    mask = torch.from_numpy(k_pos[None, :] <= q_pos[:, None])
    if visible is not None:
        mask = mask & torch.from_numpy(visible)[None, :]
    qt = torch.from_numpy(q).permute(1, 0, 2)                              # [Hq][n][D]
    kt = torch.from_numpy(k).permute(1, 0, 2).repeat_interleave(group, 0)  # [Hq][R][D]
    vt = torch.from_numpy(v).permute(1, 0, 2).repeat_interleave(group, 0)
    o = torch.nn.functional.scaled_dot_product_attention(
        qt, kt.contiguous(), vt.contiguous(), attn_mask=mask, scale=scale)
    return o.permute(1, 0, 2).numpy()


@pytest.mark.parametrize("Hq,Hkv,D,R,n", [(4, 1, 64, 50, 7), (32, 8, 128, 300, 22),
                                          (8, 8, 32, 40, 5), (6, 2, 16, 9, 9)])
def test_matches_torch_sdpa_float64(Hq, Hkv, D, R, n):
    rng = np.random.default_rng(Hq * 1000 + R)
    q, k, v = _rand(rng, n, Hq, D), _rand(rng, R, Hkv, D), _rand(rng, R, Hkv, D)
    k_pos = np.sort(rng.choice(10 * R, R, replace=False))
    q_pos = k_pos[R - n:]
    scale = 1 / np.sqrt(D)
    got = attend(q, k, v, q_pos, k_pos, scale)
    want = _torch_reference(q, k, v, q_pos, k_pos, scale)
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-12)


def test_masked_keys_match_torch():
    rng = np.random.default_rng(7)
    q, k, v = _rand(rng, 4, 4, 16), _rand(rng, 30, 2, 16), _rand(rng, 30, 2, 16)
    k_pos = np.arange(30)
    q_pos = k_pos[26:]
    vis = rng.random(30) < 0.6
    vis[26:] = True
    got = attend(q, k, v, q_pos, k_pos, 0.3, visible=vis)
    want = _torch_reference(q, k, v, q_pos, k_pos, 0.3, visible=vis)
    np.testing.assert_allclose(got, want, atol=1e-12)


def test_zero_keys_give_mean_of_visible_values():
    rng = np.random.default_rng(8)
    R, n = 20, 5
    v = _rand(rng, R, 1, 8)
    o = attend(_rand(rng, n, 2, 8), np.zeros((R, 1, 8)), v, np.arange(R - n, R), np.arange(R), 1.0)
    for i in range(n):
        want = v[: R - n + i + 1, 0, :].mean(axis=0)
        np.testing.assert_allclose(o[i, 0], want, atol=1e-14)
        np.testing.assert_allclose(o[i, 1], want, atol=1e-14)


def test_single_visible_key_returns_its_value():
    rng = np.random.default_rng(9)
    v = _rand(rng, 6, 2, 8)
    o = attend(_rand(rng, 1, 4, 8), _rand(rng, 6, 2, 8), v, np.array([0]), np.arange(6), 0.5)
    np.testing.assert_allclose(o[0, 0], v[0, 0], atol=0)
    np.testing.assert_allclose(o[0, 3], v[0, 1], atol=0)


def test_group_mapping_is_contiguous():
    # query head h reads KV head h // (Hq/Hkv): give every KV head constant values
    rng = np.random.default_rng(10)
    v = np.zeros((5, 4, 8))
    for g in range(4):
        v[:, g, :] = g
    o = attend(_rand(rng, 2, 8, 8), _rand(rng, 5, 4, 8), v, np.array([3, 4]), np.arange(5), 1.0)
    for h in range(8):
        np.testing.assert_allclose(o[:, h, :], h // 2, atol=1e-15)


def test_decode_equals_last_row_of_chunk():
    rng = np.random.default_rng(11)
    q, k, v = _rand(rng, 6, 4, 16), _rand(rng, 40, 1, 16), _rand(rng, 40, 1, 16)
    pos = np.arange(40)
    chunk = attend(q, k, v, pos[34:], pos, 0.25)
    dec = attend(q[-1:], k, v, pos[39:], pos, 0.25)
    np.testing.assert_allclose(dec[0], chunk[-1], atol=1e-15)


def test_causal_rule_includes_self_and_uses_positions():
    # a key at the query's own position is visible; one position later is not
    k = np.zeros((3, 1, 4))
    v = np.array([[[1.0] * 4], [[2.0] * 4], [[100.0] * 4]])
    o = attend(np.ones((1, 1, 4)), k, v, np.array([11]), np.array([5, 11, 12]), 1.0)
    np.testing.assert_allclose(o[0, 0], 1.5)


def test_scale_enters_logits():
    # two keys with logits 0 and 1 (before scale): weights sigmoid-like closed form
    q = np.array([[[1.0, 0.0]]])
    k = np.array([[[0.0, 0.0]], [[1.0, 0.0]]])
    v = np.array([[[0.0, 0.0]], [[1.0, 0.0]]])
    for scale in (0.5, 2.0):
        o = attend(q, k, v, np.array([1]), np.array([0, 1]), scale)
        assert o[0, 0, 0] == pytest.approx(np.exp(scale) / (1 + np.exp(scale)), abs=1e-15)
