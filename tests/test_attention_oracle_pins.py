"""Pins of the decode-attention oracle (Sec. 2.1, Eq. 1) on the CPU."""
import numpy as np
import pytest
import torch

import oracle
import synth
from oracle import attention as oat
from oracle import decode_step as ods


def _rand(shape, tid, scale=1.0):
    return synth.normal(shape, oracle.F32, 5, tid, 0.0, scale).astype(np.float64)


def test_single_position_returns_the_value():
    q, K, V = _rand((2, 128), 1), _rand((2, 1, 128), 2), _rand((2, 1, 128), 3)
    assert np.array_equal(oat.attend(q, K, V, 64), V[:, 0, :])


def test_equal_keys_average_the_values():
    q, V = _rand((1, 128), 4), _rand((1, 9, 128), 5)
    K = np.repeat(_rand((1, 1, 128), 6), 9, axis=1)
    assert np.allclose(oat.attend(q, K, V, 128), V.mean(axis=1), rtol=0, atol=1e-12)


@pytest.mark.parametrize("D,n", [(64, 1), (64, 70), (128, 129), (128, 5)])
def test_matches_torch_sdpa_in_float64(D, n):
    B, heads = 3, 4
    H = heads * D
    q, K, V = _rand((B, H), 7), _rand((B, n, H), 8), _rand((B, n, H), 9)
    split = lambda t, L: torch.from_numpy(t.reshape(B, L, heads, D).transpose(0, 2, 1, 3).copy())
    ref = torch.nn.functional.scaled_dot_product_attention(split(q, 1), split(K, n), split(V, n))
    ref = ref.numpy().transpose(0, 2, 1, 3).reshape(B, H)
    assert np.allclose(oat.attend(q, K, V, D), ref, rtol=0, atol=1e-12)


def test_position_order_does_not_matter():
    q, K, V = _rand((2, 256), 10), _rand((2, 33, 256), 11), _rand((2, 33, 256), 12)
    perm = np.random.default_rng(0).permutation(33)
    assert np.allclose(oat.attend(q, K, V, 128), oat.attend(q, K[:, perm], V[:, perm], 128), rtol=0, atol=1e-12)


def test_dominant_score_selects_its_value():
    D = 64
    q = np.zeros((1, D))
    q[0, 0] = 1.0
    K = np.zeros((1, 5, D))
    K[0, 3, 0] = 400.0  # s_3 = 400 / 8 = 50: weight of the others ~ e^-50
    V = _rand((1, 5, D), 13)
    assert np.allclose(oat.attend(q, K, V, D), V[:, 3], rtol=0, atol=1e-18 + 1e-20 * np.abs(V).max())


def test_append_is_eq1_concat():
    c = _rand((2, 4, 8), 14)
    new = _rand((2, 8), 15)
    out = oat.append(c, new)
    assert out.shape == (2, 5, 8) and np.array_equal(out[:, :4], c) and np.array_equal(out[:, 4], new)
    assert np.array_equal(oat.append(None, new)[:, 0], new)


def _layers(L, H, F, dtype):
    shapes = {"qkv": (3 * H, H), "out": (H, H), "fc1": (F, H), "fc2": (H, F)}
    return [{name: (synth.normal((n, k), dtype, 0, 1000 + 8 * l + 2 * i, 0, 0.02),
                    synth.normal((n,), dtype, 0, 1001 + 8 * l + 2 * i, 0, 0.02))
             for i, (name, (n, k)) in enumerate(shapes.items())} for l in range(L)]


@pytest.mark.parametrize("dtype", [oracle.F16, oracle.BF16])
def test_empty_cache_step_equals_the_value_slice_step(dtype):
    """With no earlier positions the attention returns V exactly, so the step with a
    cache reduces bit for bit to the empty-cache reading of the decode step."""
    L, H, F = 2, 128, 256
    layers = _layers(L, H, F, dtype)
    x = synth.normal((2, H), dtype, 0, 10)
    want, _ = ods.decode_step(x, layers, H, dtype)
    got, _, kc, vc = oat.decode_step_kv(x, layers, H, dtype, [None] * L, [None] * L, 64)
    assert np.array_equal(got, want)
    assert all(k.shape == (2, 1, H) for k in kc)


def test_cache_grows_with_the_new_keys_and_values():
    dtype, L, H, F = oracle.F16, 1, 128, 256
    layers = _layers(L, H, F, dtype)
    kc = [synth.normal((1, 3, H), dtype, 0, 50)]
    vc = [synth.normal((1, 3, H), dtype, 0, 51)]
    x = synth.normal((1, H), dtype, 0, 11)
    _, trace, kc2, vc2 = oat.decode_step_kv(x, layers, H, dtype, kc, vc, 64)
    qkv = trace[0][3]
    assert np.array_equal(kc2[0][:, :3], kc[0]) and np.array_equal(kc2[0][:, 3], qkv[:, H:2 * H])
    assert np.array_equal(vc2[0][:, 3], qkv[:, 2 * H:])
