"""Pins of the oracle's transformer primitives.

The paper gives no internals of v_theta, so the DiT is this project's
Wan-shaped specification (parity unpinned by the paper).  Every primitive is
pinned here against an independent library routine (torch.nn.functional,
einops) or a mathematical identity, and the assembled network against a
second formulation built from torch library calls (complex-number RoPE,
scaled-dot-product attention, einops patching).
"""
import math

import einops
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import dit
from paper_2607_23159_amd import synth

rng = np.random.default_rng(0)


def t64(a):
    return torch.from_numpy(np.asarray(a, dtype=np.float64))


def test_layer_norm_matches_torch():
    z = rng.standard_normal((7, 40)) * 3 + 1
    ref = F.layer_norm(t64(z), (40,), eps=1e-6).numpy()
    np.testing.assert_allclose(dit.layer_norm(z), ref, rtol=1e-12, atol=1e-12)


def test_rms_norm_matches_torch():
    z = rng.standard_normal((5, 48)) * 2
    g = rng.standard_normal(48)
    ref = F.rms_norm(t64(z), (48,), weight=t64(g), eps=1e-6).numpy()
    np.testing.assert_allclose(dit.rms_norm(z, g), ref, rtol=1e-12, atol=1e-12)


def test_gelu_silu_match_torch():
    x = np.linspace(-6, 6, 1001)
    np.testing.assert_allclose(dit.gelu_tanh(x), F.gelu(t64(x), approximate="tanh").numpy(), rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(dit.silu(x), F.silu(t64(x)).numpy(), rtol=1e-12, atol=1e-14)


def test_linear_matches_torch():
    x = rng.standard_normal((6, 10))
    w = rng.standard_normal((4, 10))
    b = rng.standard_normal(4)
    np.testing.assert_allclose(dit.linear(x, w, b), F.linear(t64(x), t64(w), t64(b)).numpy(), rtol=1e-12)


@pytest.mark.parametrize("lq,lk,heads,dh", [(5, 9, 3, 8), (17, 4, 2, 32), (1, 1, 1, 4)])
def test_attention_matches_sdpa(lq, lk, heads, dh):
    q = rng.standard_normal((lq, heads * dh))
    k = rng.standard_normal((lk, heads * dh))
    v = rng.standard_normal((lk, heads * dh))
    qt = t64(q).reshape(lq, heads, dh).transpose(0, 1)
    kt = t64(k).reshape(lk, heads, dh).transpose(0, 1)
    vt = t64(v).reshape(lk, heads, dh).transpose(0, 1)
    ref = F.scaled_dot_product_attention(qt, kt, vt).transpose(0, 1).reshape(lq, heads * dh).numpy()
    np.testing.assert_allclose(dit.attention(q, k, v, heads), ref, rtol=1e-10, atol=1e-12)


def test_attention_single_key_returns_value():
    q = rng.standard_normal((3, 8))
    k = rng.standard_normal((1, 8))
    v = rng.standard_normal((1, 8))
    np.testing.assert_allclose(dit.attention(q, k, v, 2), np.repeat(v, 3, axis=0), rtol=1e-14)


def test_patchify_matches_einops_and_roundtrips():
    x = rng.standard_normal((3, 2, 6, 8))
    ref = einops.rearrange(x, "c (f pt) (h ph) (w pw) -> (f h w) (c pt ph pw)", pt=1, ph=2, pw=2)
    p = dit.patchify(x, 1, 2, 2)
    np.testing.assert_array_equal(p, ref)
    np.testing.assert_array_equal(dit.unpatchify(p, x.shape, 1, 2, 2), x)


def test_rope_bands():
    assert dit.rope_bands(128) == (22, 21, 21)
    assert dit.rope_bands(32) == (6, 5, 5)


def _rope_complex(x, ang, heads):
    """RoPE as multiplication of complex pairs by exp(i angle)."""
    L, dm = x.shape
    xc = torch.view_as_complex(t64(x).reshape(L, heads, dm // heads // 2, 2).contiguous())
    rot = torch.polar(torch.ones_like(t64(ang)), t64(ang))[:, None, :]
    return torch.view_as_real(xc * rot).reshape(L, dm).numpy()


def test_rope_matches_complex_formulation_and_identities():
    grid = (3, 4, 5)
    dh, heads = 32, 2
    ang = dit.rope_angles(grid, dh)
    L = 60
    x = rng.standard_normal((L, heads * dh))
    y = dit.apply_rope(x, ang, heads)
    np.testing.assert_allclose(y, _rope_complex(x, ang, heads), rtol=1e-12, atol=1e-12)
    # norm preserved per head, identity at token (0,0,0)
    np.testing.assert_allclose(np.linalg.norm(y.reshape(L, heads, dh), axis=-1),
                               np.linalg.norm(x.reshape(L, heads, dh), axis=-1), rtol=1e-12)
    np.testing.assert_array_equal(y[0], x[0])
    # the dot product depends only on position differences: shift both
    # tokens by one step along the width axis
    q, k = rng.standard_normal(dh), rng.standard_normal(dh)
    def tok(f, h, w):
        return (f * grid[1] + h) * grid[2] + w
    def dot(a, b):
        qa = dit.apply_rope(q[None], ang[[a]], 1)[0]
        kb = dit.apply_rope(k[None], ang[[b]], 1)[0]
        return qa @ kb
    assert dot(tok(1, 2, 1), tok(0, 1, 3)) == pytest.approx(dot(tok(2, 3, 2), tok(1, 2, 4)), rel=1e-10)
    # angle values: pair 0 of every axis has frequency 1
    n_f, n_h, n_w = dit.rope_bands(dh)
    assert ang[tok(2, 3, 4), 0] == 2 and ang[tok(2, 3, 4), n_f] == 3 and ang[tok(2, 3, 4), n_f + n_h] == 4
    assert ang[tok(1, 0, 0), 1] == pytest.approx(10000.0 ** (-1.0 / n_f))


def test_rope_angles_match_hand_derived_table():
    """Every band's frequencies, not only pair 0: hand-derived angles
    (powers of ten) at tokens away from the origin on all three axes, for
    head dims 32 and 128 (a wrong band split, denominator or axis order
    moves at least one entry)."""
    import json
    import os
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "rope_angles.json")))
    for e in g["entries"]:
        grid = tuple(e["grid"])
        ang = dit.rope_angles(grid, e["head_dim"])
        f, h, w = e["token"]
        tok = (f * grid[1] + h) * grid[2] + w
        assert ang[tok, e["pair"]] == pytest.approx(e["value"], rel=1e-11, abs=1e-15), e


def test_time_sinusoid_values():
    s = dit.time_sinusoid(0.0, 256)
    np.testing.assert_array_equal(s[:128], np.ones(128))
    np.testing.assert_array_equal(s[128:], np.zeros(128))
    s = dit.time_sinusoid(0.5, 8)
    om = np.array([1.0, 10.0 ** -1, 10.0 ** -2, 10.0 ** -3])
    np.testing.assert_allclose(s, np.concatenate([np.cos(500 * om), np.sin(500 * om)]), rtol=1e-12)


def test_zero_weights_give_head_bias():
    m = synth.MODELS["tiny"]
    W = {k: np.zeros_like(v, dtype=np.float64) for k, v in synth.unflatten(m, synth.make_weights(m)).items()}
    W["head_b"] = rng.standard_normal(m.patch_dim)
    x = rng.standard_normal(m.latent_shape)
    v = dit.velocity(x, 0.5, dit.text_embedding(np.zeros((m.text_len, m.text_dim)), W), W, m)
    expect = dit.unpatchify(np.tile(W["head_b"], (m.tokens, 1)), m.latent_shape, 1, 2, 2)
    np.testing.assert_allclose(v, expect, rtol=1e-14)


# ---------------------------------------------------- assembled network check
def _torch_velocity(x, t, ctx, W, m):
    """Second formulation of the same network from torch library calls."""
    T = {k: t64(v) for k, v in W.items()}
    d, H, dh = m.hidden, m.heads, m.head_dim
    half = m.freq_dim // 2
    om = torch.pow(torch.tensor(10000.0, dtype=torch.float64), -torch.arange(half, dtype=torch.float64) / half)
    s = torch.cat([torch.cos(1000 * t * om), torch.sin(1000 * t * om)])
    e = F.linear(F.silu(F.linear(s, T["time1_w"], T["time1_b"])), T["time2_w"], T["time2_b"])
    m6 = F.linear(F.silu(e), T["mod_w"], T["mod_b"]).reshape(6, d)
    c = F.linear(F.gelu(F.linear(t64(ctx), T["text1_w"], T["text1_b"]), approximate="tanh"),
                 T["text2_w"], T["text2_b"])
    tok = einops.rearrange(t64(x), "c (f pt) (h ph) (w pw) -> (f h w) (c pt ph pw)", pt=1, ph=2, pw=2)
    z = F.linear(tok, T["patch_w"], T["patch_b"])
    # rotary angles built here from positions and per-band frequencies (not
    # from the oracle's table)
    nf_b = dh // 2 - 2 * (dh // 6)
    nhw_b = dh // 6
    freq = lambda n: torch.pow(torch.tensor(10000.0, dtype=torch.float64),
                               -torch.arange(n, dtype=torch.float64) / n)
    gf, gh, gw = m.grid
    pf, ph_, pw_ = torch.meshgrid(torch.arange(gf, dtype=torch.float64), torch.arange(gh, dtype=torch.float64),
                                  torch.arange(gw, dtype=torch.float64), indexing="ij")
    ang = torch.cat([pf.reshape(-1, 1) * freq(nf_b), ph_.reshape(-1, 1) * freq(nhw_b),
                     pw_.reshape(-1, 1) * freq(nhw_b)], dim=1)
    rot = torch.polar(torch.ones_like(ang), ang)[:, None, :]
    L = z.shape[0]

    def rope(u):
        uc = torch.view_as_complex(u.reshape(L, H, dh // 2, 2).contiguous())
        return torch.view_as_real(uc * rot).reshape(L, d)

    def mha(q, k, v):
        sp = lambda u: u.reshape(u.shape[0], H, dh).transpose(0, 1)
        return F.scaled_dot_product_attention(sp(q), sp(k), sp(v)).transpose(0, 1).reshape(q.shape[0], d)

    for j in range(m.n_blocks):
        p = f"blk{j}."
        sh1, sc1, g1, sh2, sc2, g2 = m6 + T[p + "mod"]
        u = F.layer_norm(z, (d,), eps=1e-6) * (1 + sc1) + sh1
        q, k, v = F.linear(u, T[p + "qkv_w"], T[p + "qkv_b"]).split(d, dim=1)
        q = rope(F.rms_norm(q, (d,), T[p + "q_gain"], eps=1e-6))
        k = rope(F.rms_norm(k, (d,), T[p + "k_gain"], eps=1e-6))
        z = z + g1 * F.linear(mha(q, k, v), T[p + "o_w"], T[p + "o_b"])
        u = F.layer_norm(z, (d,), T[p + "ca_ln_g"], T[p + "ca_ln_b"], eps=1e-6)
        q = F.rms_norm(F.linear(u, T[p + "caq_w"], T[p + "caq_b"]), (d,), T[p + "caq_gain"], eps=1e-6)
        k = F.rms_norm(F.linear(c, T[p + "cak_w"], T[p + "cak_b"]), (d,), T[p + "cak_gain"], eps=1e-6)
        v = F.linear(c, T[p + "cav_w"], T[p + "cav_b"])
        z = z + F.linear(mha(q, k, v), T[p + "cao_w"], T[p + "cao_b"])
        u = F.layer_norm(z, (d,), eps=1e-6) * (1 + sc2) + sh2
        z = z + g2 * F.linear(F.gelu(F.linear(u, T[p + "ffn1_w"], T[p + "ffn1_b"]), approximate="tanh"),
                              T[p + "ffn2_w"], T[p + "ffn2_b"])
    sh, sc = e[None] + T["head_mod"]
    y = F.linear(F.layer_norm(z, (d,), eps=1e-6) * (1 + sc) + sh, T["head_w"], T["head_b"])
    return einops.rearrange(y, "(f h w) (c pt ph pw) -> c (f pt) (h ph) (w pw)", f=m.grid[0], h=m.grid[1],
                            w=m.grid[2], pt=1, ph=2, pw=2).numpy()


@pytest.mark.parametrize("init", ["paper", "stress"])
def test_velocity_matches_torch_formulation(init):
    m = synth.MODELS["tiny"]
    W = {k: v.astype(np.float64) for k, v in synth.unflatten(m, synth.make_weights(m, init=init)).items()}
    x = synth.make_noise(m, 1)[0]
    ctx = synth.make_context(m, 1)
    v = dit.velocity(x, 0.37, dit.text_embedding(ctx, W), W, m)
    ref = _torch_velocity(x, 0.37, ctx, W, m)
    np.testing.assert_allclose(v, ref, rtol=1e-9, atol=1e-11)


def test_last_block_rows_match_full_forward():
    m = synth.MODELS["tiny"]
    W = {k: v.astype(np.float64) for k, v in synth.unflatten(m, synth.make_weights(m, init="stress")).items()}
    x = synth.make_noise(m, 1)[0]
    emb = dit.text_embedding(synth.make_context(m, 1), W)
    full = dit.patchify(dit.velocity(x, 0.6, emb, W, m), 1, 2, 2)
    rows = np.array([0, 5, 77, 255])
    part = dit.velocity(x, 0.6, emb, W, m, last_block_rows=rows)
    np.testing.assert_allclose(part, full[rows], rtol=1e-12, atol=1e-14)
