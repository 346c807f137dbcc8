"""Pins for the oracle's Qwen3-style layer math: closed forms, invariants, and
transformers' Qwen3 implementation run on the CPU with the same weights."""
import numpy as np
import pytest

from oracle import OracleModel, Precision
from oracle import model as om
from workloads import get, make_prompts, make_weights

from hf_reference import hf_logits, qwen3_from_weights


def test_rms_norm_hand_value():
    x = np.array([[3.0, 4.0]])
    out = om.rms_norm(x, np.array([1.0, 2.0]), 0.0)
    r = np.sqrt(12.5)
    np.testing.assert_allclose(out, [[3 / r, 8 / r]], rtol=1e-15)


def test_rms_norm_unit_mean_square():
    x = np.random.default_rng(0).standard_normal((5, 64)) * 7.0
    out = om.rms_norm(x, np.ones(64), 0.0)
    np.testing.assert_allclose(np.mean(out ** 2, axis=1), 1.0, rtol=1e-13)


def test_silu_and_sigmoid_identities():
    x = np.linspace(-8, 8, 101)
    np.testing.assert_allclose(om.silu(x) - om.silu(-x), x, atol=1e-13)
    np.testing.assert_allclose(om.sigmoid(x) + om.sigmoid(-x), 1.0, atol=1e-15)
    assert om.sigmoid(np.array([0.0]))[0] == 0.5
    np.testing.assert_allclose(om.sigmoid(np.log(3.0)), 0.75, rtol=1e-15)


def test_rope_position_zero_is_identity_and_rotation_preserves_norm():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((3, 2, 64))
    np.testing.assert_array_equal(om.apply_rope(x, np.zeros(3, int), 1e6), x)
    y = om.apply_rope(x, np.array([5, 700, 16000]), 1e6)
    # each (i, i + hd/2) pair is rotated, so its length is unchanged
    n_in = x[..., :32] ** 2 + x[..., 32:] ** 2
    n_out = y[..., :32] ** 2 + y[..., 32:] ** 2
    np.testing.assert_allclose(n_out, n_in, rtol=1e-12)


def test_rope_first_pair_rotates_by_position():
    # inv_freq_0 = 1, so the first pair turns by exactly `position` radians
    x = np.zeros((1, 1, 8))
    x[0, 0, 0] = 1.0
    y = om.apply_rope(x, np.array([3]), 1e6)
    np.testing.assert_allclose([y[0, 0, 0], y[0, 0, 4]], [np.cos(3.0), np.sin(3.0)], rtol=1e-15)


def test_rope_relative_position_property():
    rng = np.random.default_rng(2)
    q, k = rng.standard_normal((1, 1, 64)), rng.standard_normal((1, 1, 64))
    dots = [np.sum(om.apply_rope(q, np.array([p + 7]), 1e6) * om.apply_rope(k, np.array([p]), 1e6))
            for p in (0, 13, 250)]
    np.testing.assert_allclose(dots, dots[0], atol=1e-5)


def test_attention_special_cases():
    rng = np.random.default_rng(3)
    hq, hkv, hd, T = 4, 2, 8, 5
    v = rng.standard_normal((T, hkv, hd))
    k = rng.standard_normal((T, hkv, hd))
    # q = 0: uniform weights over visible keys -> mean of visible values of the head's kv group
    q = np.zeros((T, hq, hd))
    pos = np.arange(T)
    out = om.attention(q, k, v, pos, pos, causal=True)
    for i in range(T):
        for h in range(hq):
            np.testing.assert_allclose(out[i, h], v[: i + 1, h // 2].mean(axis=0), rtol=1e-13)
    out_nc = om.attention(q, k, v, pos, pos, causal=False)
    for h in range(hq):
        np.testing.assert_allclose(out_nc[0, h], v[:, h // 2].mean(axis=0), rtol=1e-13)
    # a dominant key selects its value
    q2 = np.zeros((1, hq, hd)); q2[0, :, 0] = 1.0
    k2 = np.zeros((T, hkv, hd)); k2[3, :, 0] = 200.0
    out2 = om.attention(q2, k2, v, np.array([10]), pos, causal=True)
    np.testing.assert_allclose(out2[0, 1], v[3, 0], atol=1e-12)
    np.testing.assert_allclose(out2[0, 2], v[3, 1], atol=1e-12)
    # two keys with scaled scores 0 and -1 (q . k / sqrt(hd) with hd = 4): weights
    # 1 / (1 + e^-1) and e^-1 / (1 + e^-1), unrounded
    q3 = np.zeros((1, 1, 4)); q3[0, 0, 0] = 2.0
    k3 = np.zeros((2, 1, 4)); k3[1, 0, 0] = -1.0
    v3 = rng.standard_normal((2, 1, 4))
    out3 = om.attention(q3, k3, v3, np.array([1]), np.array([0, 1]), causal=True)
    w = np.exp(-1.0)
    np.testing.assert_allclose(out3[0, 0], (v3[0, 0] + w * v3[1, 0]) / (1.0 + w), rtol=1e-14)


@pytest.fixture(scope="module")
def tiny():
    wl = get("tiny-f32", norm_init="perturbed")
    return wl, make_weights(wl), make_prompts(wl)[0]


def test_target_matches_transformers_qwen3(tiny):
    wl, W, prompt = tiny
    ref = hf_logits(qwen3_from_weights(wl, W), prompt)
    m = OracleModel(wl, W, prec=Precision.for_dtype("f64"))
    out = m.target_forward(m.new_state(prompt, 0), prompt, 0)
    # transformers evaluates RoPE cos/sin in float32; everything else agrees in float64
    np.testing.assert_allclose(out.logits, ref, atol=2e-6, rtol=0)


def test_incremental_decode_matches_full_forward(tiny):
    wl, W, prompt = tiny
    m = OracleModel(wl, W, prec=Precision.for_dtype("f64"))
    full = m.target_forward(m.new_state(prompt, 0), prompt, 0).logits
    st = m.new_state(prompt, 0)
    a = m.target_forward(st, prompt[:40], 0).logits
    b = m.target_forward(st, prompt[40:56], 40).logits
    c = m.target_forward(st, prompt[56:57], 56).logits
    np.testing.assert_allclose(np.concatenate([a, b, c]), full[:57], atol=1e-12, rtol=0)


@pytest.mark.parametrize("name", ["tiny-f32", "mini-bf16"])
def test_weight_cache_modes_are_bit_identical(name):
    """The float32 weight cache (used for the largest shapes) widens stored bf16 / fp32
    values exactly, so every result equals the float64-cache oracle bit for bit."""
    wl = get(name, norm_init="perturbed")
    W = make_weights(wl)
    prompt = make_prompts(wl)[0][:24]
    outs = []
    for cache in (True, "f32", False):
        m = OracleModel(wl, W, cache=cache)
        outs.append(m.target_forward(m.new_state(prompt, 0), prompt, 0).logits)
    np.testing.assert_array_equal(outs[0], outs[1])
    np.testing.assert_array_equal(outs[0], outs[2])
