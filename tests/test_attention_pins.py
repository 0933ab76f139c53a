"""Pins of the per-group attention oracle (CPU only).

Each check ties the oracle to something other than itself: a complex-number
form of the rotary embedding, torch's scaled-dot-product attention (a library
routine), closed forms for one token and for equal keys, causality under
perturbation of later tokens, and the cross-group average of identical groups.
"""
import numpy as np
import pytest
import torch

from oracle import attention_oracle as ao
from paper_2605_06206_amd import synth


def _rope_complex(v, S, hd, theta, scale):
    """Rotation as complex multiplication: pair i is the complex number
    v[i] + 1j*v[i+hd/2], multiplied by exp(1j * (s/scale) * theta^(-2i/hd))."""
    h = hd // 2
    z = v[:, :h] + 1j * v[:, h:]
    pos = np.arange(S)[:, None] / scale
    freq = np.array([theta ** (-2.0 * i / hd) for i in range(h)])[None, :]
    w = z * np.exp(1j * pos * freq)
    return np.concatenate([w.real, w.imag], axis=1)


@pytest.mark.parametrize("hd", [96, 128])
def test_rope_matches_complex_rotation_and_keeps_norms(hd):
    rng = np.random.default_rng(1)
    S = 37
    v = rng.standard_normal((S, hd))
    for theta, scale in ((10000.0, 1.0), (500000.0, 16.0)):
        cos, sin = ao.rope_angles(S, hd, theta, scale)
        r = ao.apply_rope(v, cos, sin)
        assert np.max(np.abs(r - _rope_complex(v, S, hd, theta, scale))) <= 1e-12
        # position 0 is the identity; every pair keeps its length
        assert np.max(np.abs(r[0] - v[0])) <= 1e-15
        h = hd // 2
        assert np.max(np.abs(r[:, :h] ** 2 + r[:, h:] ** 2 - v[:, :h] ** 2 - v[:, h:] ** 2)) <= 1e-12


@pytest.mark.parametrize("hd", [96, 128])
def test_rope_scores_depend_on_relative_position_only(hd):
    rng = np.random.default_rng(2)
    S = 40
    q0, k0 = rng.standard_normal(hd), rng.standard_normal(hd)
    cos, sin = ao.rope_angles(S, hd, 500000.0, 16.0)
    q = ao.apply_rope(np.tile(q0, (S, 1)), cos, sin)
    k = ao.apply_rope(np.tile(k0, (S, 1)), cos, sin)
    for m, n, dm in ((10, 3, 5), (30, 30, 7), (20, 2, 11)):
        assert abs(q[m] @ k[n] - q[m + dm] @ k[n + dm]) <= 1e-9


def _qkv_parts(S=23, d=32, nq=2, hd=128, seed=3):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((S, d))
    w_qkv = rng.standard_normal(((nq + 2) * hd, d)) * 0.1
    w_o = rng.standard_normal((d, nq * hd)) * 0.1
    return x, w_qkv, w_o


@pytest.mark.parametrize("nq,hd", [(3, 128), (1, 96)])
def test_attention_matches_torch_sdpa(nq, hd):
    """The core softmax attention against torch's causal SDPA in fp64 on the
    oracle's own rotated q, k and v (the key/value head repeated for every
    query head: grouped-query attention)."""
    S, d = 29, 32
    x, w_qkv, w_o = _qkv_parts(S, d, nq, hd, seed=4)
    out, parts = ao.group_attention(x, w_qkv, w_o, nq, hd, 500000.0, 16.0)
    q = torch.from_numpy(parts["q"]).permute(1, 0, 2)            # [nq, S, hd]
    k = torch.from_numpy(parts["k"])[None].expand(nq, S, hd)
    v = torch.from_numpy(parts["v"])[None].expand(nq, S, hd)
    o = torch.nn.functional.scaled_dot_product_attention(q, k, v, is_causal=True)
    o = o.permute(1, 0, 2).reshape(S, nq * hd).numpy()
    assert np.max(np.abs(o - parts["o"])) <= 1e-12
    assert np.max(np.abs(o @ w_o.T - out)) <= 1e-11


def test_one_token_and_equal_keys():
    # one token: the only key is its own, so o = v
    x, w_qkv, w_o = _qkv_parts(S=1, seed=5)
    _, parts = ao.group_attention(x, w_qkv, w_o, 2, 128, 500000.0, 1.0)
    assert np.max(np.abs(parts["o"][:, :128] - parts["v"])) <= 1e-14
    assert np.max(np.abs(parts["o"][:, 128:] - parts["v"])) <= 1e-14
    # key rows all zero (zero key weights): every visible key scores 0, so o is
    # the running mean of v over positions 0..s
    S = 17
    x, w_qkv, w_o = _qkv_parts(S=S, seed=6)
    w_qkv = w_qkv.copy()
    w_qkv[2 * 128:3 * 128] = 0.0
    _, parts = ao.group_attention(x, w_qkv, w_o, 2, 128, 500000.0, 1.0)
    run_mean = np.cumsum(parts["v"], axis=0) / np.arange(1, S + 1)[:, None]
    assert np.max(np.abs(parts["o"][:, :128] - run_mean)) <= 1e-13


def test_attention_is_causal():
    x, w_qkv, w_o = _qkv_parts(S=30, seed=7)
    a, _ = ao.group_attention(x, w_qkv, w_o, 2, 128, 500000.0, 16.0)
    x2 = x.copy()
    x2[20:] += np.random.default_rng(8).standard_normal(x2[20:].shape)
    b, _ = ao.group_attention(x2, w_qkv, w_o, 2, 128, 500000.0, 16.0)
    assert np.max(np.abs(a[:20] - b[:20])) <= 1e-13
    assert np.max(np.abs(a[20:] - b[20:])) > 1e-3


def test_identical_groups_average_to_one_group():
    inp = synth.make_attention_inputs(dict(synth.ATTN_CONFIGS["attn_tiny_bf16"], S=40))
    c = inp["cfg"]
    x1 = inp["x"][:1]
    g1 = inp["groups"][:1]
    one, d1 = ao.attention_block(x1, g1, c["nq"], c["hd"], c["theta"], c["scale"])
    four, _ = ao.attention_block(np.repeat(x1, 4, axis=0), g1 * 4, c["nq"], c["hd"],
                                 c["theta"], c["scale"])
    assert np.max(np.abs(one - four)) <= 1e-12
    assert np.max(np.abs(one - (x1[0] + d1[0]))) <= 1e-12


def test_attention_inputs_are_seeded_and_bf16():
    a = synth.make_attention_inputs("attn_tiny_bf16")
    b = synth.make_attention_inputs("attn_tiny_bf16")
    assert np.array_equal(a["x"], b["x"])
    assert np.array_equal(a["groups"][1]["w_qkv"], b["groups"][1]["w_qkv"])
    for t in (a["x"], a["groups"][0]["w_qkv"], a["groups"][0]["w_o"]):
        assert np.array_equal(t, synth.round_to_bf16(t))


@pytest.mark.parametrize("hd,nq,theta,scale,S", [
    (128, 2, 500000.0, 16.0, 300),
    (128, 1, 10000.0, 1.0, 129),
    (96, 1, 500000.0, 16.0, 257),
    (96, 3, 10000.0, 16.0, 64),
    (128, 3, 500000.0, 1.0, 97),
    (96, 2, 10000.0, 1.0, 1),
])
def test_rows_form_equals_whole_sequence_form(hd, nq, theta, scale, S):
    """``group_attention_rows`` (the reference of the full-size sampled checks)
    agrees with the pinned ``group_attention`` at every query position: a wrong
    per-row rotary angle, causal bound or head slice there would fail here."""
    rng = np.random.default_rng([hd, nq, S])
    d = 40
    x = rng.standard_normal((S, d))
    w_qkv = rng.standard_normal(((nq + 2) * hd, d)) * 0.15
    w_o = rng.standard_normal((d, nq * hd)) * 0.15
    whole, _ = ao.group_attention(x, w_qkv, w_o, nq, hd, theta, scale)
    rows = np.arange(S)
    part = ao.group_attention_rows(x, w_qkv, w_o, nq, hd, theta, scale, rows)
    assert np.max(np.abs(part - whole)) <= 1e-12 * max(1.0, np.max(np.abs(whole)))
    # an unordered subset (first, last, interior) gives the same rows
    sub = np.unique(np.array([S - 1, 0, S // 2, S // 3]))[::-1]
    part2 = ao.group_attention_rows(x, w_qkv, w_o, nq, hd, theta, scale, sub)
    assert np.max(np.abs(part2 - whole[sub])) <= 1e-12 * max(1.0, np.max(np.abs(whole)))
