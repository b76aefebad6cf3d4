"""Oracle: the velocity model v_theta(x, t, c) in plain float64 numpy.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path imports this module;
only the tests, the smoke check and the benchmark's CPU-baseline leg do.

The paper treats the DiT as a black box v_theta(x_t, t, c) that predicts
the flow-matching velocity of a latent video conditioned on a prompt
(Sec. Preliminaries, flow-matching video diffusion).  It gives no internals,
so this module writes out the Wan-shaped transformer the workloads use, one
textbook operation at a time, in the order listed below:

  patchify (1x2x2 patches, tokens ordered (f, h, w), patch vector (c, dy, dx))
  -> patch embedding (linear)
  -> per block: LN + adaLN(shift, scale) -> QKV -> RMSNorm(q), RMSNorm(k)
     -> 3D RoPE -> softmax attention -> out-proj, gated residual
     -> affine LN -> cross-attention to the text embedding (RMSNorm q, k)
     -> out-proj, plain residual
     -> LN + adaLN -> FFN with tanh-GELU -> gated residual
  -> head: LN + adaLN(shift, scale) -> linear -> unpatchify.

Time conditioning: a 256-wide sinusoid of 1000*t -> linear, SiLU, linear
(embedding e) -> SiLU, linear (6d modulation m); block j uses m + P_j, the
head uses e + P_head.  Text conditioning: linear, tanh-GELU, linear.

Parity unpinned by the paper: the paper does not define the DiT.  Each
primitive is pinned in the tests against library routines (torch layer
norm, RMSNorm, GELU, SiLU, scaled-dot-product attention, einops) and
identities (RoPE preserves norms, is the identity at position 0 and makes
q.k depend only on the position difference; zero weights give v = head
bias).
"""
from __future__ import annotations

import math
from typing import Dict, Optional, Sequence

import numpy as np

EPS = 1e-6


def as64(a) -> np.ndarray:
    return np.asarray(a, dtype=np.float64)


# ----------------------------------------------------------------- primitives
def linear(x: np.ndarray, w: np.ndarray, b: Optional[np.ndarray]) -> np.ndarray:
    """x W^T + b with W stored [out][in]."""
    y = x @ as64(w).T
    if b is not None:
        y = y + as64(b)
    return y


def layer_norm(z: np.ndarray, eps: float = EPS) -> np.ndarray:
    """Normalise each row to zero mean and unit (biased) variance."""
    mu = z.mean(axis=-1, keepdims=True)
    var = ((z - mu) ** 2).mean(axis=-1, keepdims=True)
    return (z - mu) / np.sqrt(var + eps)


def rms_norm(z: np.ndarray, gain: np.ndarray, eps: float = EPS) -> np.ndarray:
    """Divide each row by its root mean square, then scale by the gain."""
    ms = (z * z).mean(axis=-1, keepdims=True)
    return z / np.sqrt(ms + eps) * as64(gain)


def gelu_tanh(x: np.ndarray) -> np.ndarray:
    """GELU, tanh approximation (Hendrycks & Gimpel)."""
    return 0.5 * x * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (x + 0.044715 * x ** 3)))


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def softmax_rows(s: np.ndarray) -> np.ndarray:
    s = s - s.max(axis=-1, keepdims=True)
    e = np.exp(s)
    return e / e.sum(axis=-1, keepdims=True)


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, heads: int) -> np.ndarray:
    """Multi-head softmax(q k^T / sqrt(dh)) v.

    q [Lq][heads*dh], k and v [Lk][heads*dh]; head h uses columns
    h*dh .. h*dh+dh-1.  Returns [Lq][heads*dh].
    """
    lq, dm = q.shape
    dh = dm // heads
    out = np.empty((lq, dm), dtype=np.float64)
    scale = 1.0 / math.sqrt(dh)
    for h in range(heads):
        sl = slice(h * dh, (h + 1) * dh)
        p = softmax_rows((q[:, sl] @ k[:, sl].T) * scale)
        out[:, sl] = p @ v[:, sl]
    return out


# ------------------------------------------------------------ token geometry
def patchify(x: np.ndarray, pt: int, ph: int, pw: int) -> np.ndarray:
    """[C][F][H][W] -> [L][C*pt*ph*pw]; token (f, h, w) row-major, patch
    vector ordered (c, dt, dy, dx)."""
    c, f, hh, ww = x.shape
    nf, nh, nw = f // pt, hh // ph, ww // pw
    out = np.empty((nf * nh * nw, c * pt * ph * pw), dtype=np.float64)
    tok = 0
    for i in range(nf):
        for j in range(nh):
            for k in range(nw):
                blk = x[:, i * pt:(i + 1) * pt, j * ph:(j + 1) * ph, k * pw:(k + 1) * pw]
                out[tok] = blk.reshape(-1)
                tok += 1
    return out


def unpatchify(y: np.ndarray, shape: Sequence[int], pt: int, ph: int, pw: int) -> np.ndarray:
    """Inverse of :func:`patchify`."""
    c, f, hh, ww = shape
    nf, nh, nw = f // pt, hh // ph, ww // pw
    x = np.empty((c, f, hh, ww), dtype=np.float64)
    tok = 0
    for i in range(nf):
        for j in range(nh):
            for k in range(nw):
                x[:, i * pt:(i + 1) * pt, j * ph:(j + 1) * ph, k * pw:(k + 1) * pw] = \
                    y[tok].reshape(c, pt, ph, pw)
                tok += 1
    return x


def rope_bands(head_dim: int):
    """Rotation pairs per axis: height and width get floor(dh/6) pairs each,
    time gets the rest; pairs are ordered time, height, width."""
    half = head_dim // 2
    n_h = n_w = head_dim // 6
    n_f = half - n_h - n_w
    return n_f, n_h, n_w


def rope_angles(grid: Sequence[int], head_dim: int) -> np.ndarray:
    """Angle of every rotation pair at every token: [L][dh/2].

    Pair p of an axis with n pairs turns at frequency 10000^(-p/n); the angle
    is (token position on that axis) * frequency.
    """
    nf_, nh_, nw_ = grid
    n_f, n_h, n_w = rope_bands(head_dim)
    L = nf_ * nh_ * nw_
    ang = np.empty((L, n_f + n_h + n_w), dtype=np.float64)
    om_f = 10000.0 ** (-np.arange(n_f) / n_f)
    om_h = 10000.0 ** (-np.arange(n_h) / n_h)
    om_w = 10000.0 ** (-np.arange(n_w) / n_w)
    tok = 0
    for i in range(nf_):
        for j in range(nh_):
            for k in range(nw_):
                ang[tok, :n_f] = i * om_f
                ang[tok, n_f:n_f + n_h] = j * om_h
                ang[tok, n_f + n_h:] = k * om_w
                tok += 1
    return ang


def apply_rope(x: np.ndarray, ang: np.ndarray, heads: int) -> np.ndarray:
    """Rotate adjacent pairs (x_2p, x_2p+1) of every head by the pair angle."""
    L, dm = x.shape
    dh = dm // heads
    xr = x.reshape(L, heads, dh // 2, 2)
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    a, b = xr[..., 0], xr[..., 1]
    out = np.empty_like(xr)
    out[..., 0] = a * c - b * s
    out[..., 1] = a * s + b * c
    return out.reshape(L, dm)


# ------------------------------------------------------------- conditioning
def time_sinusoid(t: float, freq_dim: int = 256) -> np.ndarray:
    """[cos(1000 t w_k), sin(1000 t w_k)], w_k = 10000^(-k/half)."""
    half = freq_dim // 2
    om = 10000.0 ** (-np.arange(half, dtype=np.float64) / half)
    arg = 1000.0 * float(t) * om
    return np.concatenate([np.cos(arg), np.sin(arg)])


def time_embedding(t: float, W: Dict[str, np.ndarray], freq_dim: int = 256):
    """Returns (e [d], m [6d])."""
    s = time_sinusoid(t, freq_dim)
    e = linear(silu(linear(s, W["time1_w"], W["time1_b"])), W["time2_w"], W["time2_b"])
    m = linear(silu(e), W["mod_w"], W["mod_b"])
    return e, m


def text_embedding(ctx: np.ndarray, W: Dict[str, np.ndarray]) -> np.ndarray:
    return linear(gelu_tanh(linear(as64(ctx), W["text1_w"], W["text1_b"])),
                  W["text2_w"], W["text2_b"])


# ------------------------------------------------------------------ network
def block_forward(z: np.ndarray, j: int, m6: np.ndarray, ctx_emb: np.ndarray,
                  ang: np.ndarray, W: Dict[str, np.ndarray], heads: int,
                  rows: Optional[np.ndarray] = None,
                  attn_io: Optional[dict] = None) -> np.ndarray:
    """One transformer block.  z [L][d] float64; returns the new residual.

    ``rows`` (optional) restricts the output to those token rows: keys and
    values of the self-attention still come from every token, all other
    operations are row-wise.  The result is then [len(rows)][d].

    ``attn_io`` (optional) serves attention-output broadcasting: its entries
    "self" and "cross" are either None (compute that attention branch) or a
    [L][d] array used in place of the branch's output, where the output is
    taken after the branch's output projection and before the self-attention
    gate.  The outputs actually used are written back to "self_out" and
    "cross_out".
    """
    p = f"blk{j}."
    d = z.shape[1]
    mod = m6.reshape(6, d) + as64(W[p + "mod"])
    sh1, sc1, g1, sh2, sc2, g2 = mod
    reuse_self = attn_io.get("self") if attn_io is not None else None
    reuse_cross = attn_io.get("cross") if attn_io is not None else None
    if attn_io is not None and rows is not None:
        raise ValueError("attention-output broadcasting needs every row")

    # self-attention
    if reuse_self is not None:
        zr, y = z, as64(reuse_self)
    else:
        u = layer_norm(z) * (1.0 + sc1) + sh1
        qkv = linear(u, W[p + "qkv_w"], W[p + "qkv_b"])
        k = apply_rope(rms_norm(qkv[:, d:2 * d], W[p + "k_gain"]), ang, heads)
        v = qkv[:, 2 * d:]
        if rows is None:
            zr, q_in, ang_q = z, qkv[:, :d], ang
        else:
            zr, q_in, ang_q = z[rows], qkv[rows, :d], ang[rows]
        q = apply_rope(rms_norm(q_in, W[p + "q_gain"]), ang_q, heads)
        o = attention(q, k, v, heads)
        y = linear(o, W[p + "o_w"], W[p + "o_b"])
    zr = zr + g1 * y
    if attn_io is not None:
        attn_io["self_out"] = y

    # cross-attention to the text embedding
    if reuse_cross is not None:
        yc = as64(reuse_cross)
    else:
        u = layer_norm(zr) * as64(W[p + "ca_ln_g"]) + as64(W[p + "ca_ln_b"])
        q = rms_norm(linear(u, W[p + "caq_w"], W[p + "caq_b"]), W[p + "caq_gain"])
        kc = rms_norm(linear(ctx_emb, W[p + "cak_w"], W[p + "cak_b"]), W[p + "cak_gain"])
        vc = linear(ctx_emb, W[p + "cav_w"], W[p + "cav_b"])
        yc = linear(attention(q, kc, vc, heads), W[p + "cao_w"], W[p + "cao_b"])
    zr = zr + yc
    if attn_io is not None:
        attn_io["cross_out"] = yc

    # feed-forward
    u = layer_norm(zr) * (1.0 + sc2) + sh2
    h = gelu_tanh(linear(u, W[p + "ffn1_w"], W[p + "ffn1_b"]))
    zr = zr + g2 * linear(h, W[p + "ffn2_w"], W[p + "ffn2_b"])
    return zr


def velocity(x: np.ndarray, t: float, ctx_emb: np.ndarray, W: Dict[str, np.ndarray],
             cfg, last_block_rows: Optional[np.ndarray] = None,
             attn_io: Optional[Sequence[dict]] = None) -> np.ndarray:
    """v_theta(x, t, c) for one latent x [C][F][H][W] (float64 result).

    ``ctx_emb`` is the text embedding (output of :func:`text_embedding`).
    ``last_block_rows`` restricts the last block and the head to the given
    tokens; the result is then the head output [len(rows)][patch_dim] rather
    than a latent (used to check single-block models at full size on a
    sample of tokens).  ``attn_io`` (one dict per block, see
    :func:`block_forward`) reuses and reports attention outputs.
    """
    pt, ph, pw = cfg.patch_t, cfg.patch_h, cfg.patch_w
    e, m = time_embedding(t, W, cfg.freq_dim)
    ang = rope_angles(cfg.grid, cfg.head_dim)
    z = linear(patchify(as64(x), pt, ph, pw), W["patch_w"], W["patch_b"])
    for j in range(cfg.n_blocks):
        rows = last_block_rows if j == cfg.n_blocks - 1 else None
        z = block_forward(z, j, m, ctx_emb, ang, W, cfg.heads, rows,
                          None if attn_io is None else attn_io[j])
    hm = e[None, :] + as64(W["head_mod"])
    sh, sc = hm[0], hm[1]
    y = linear(layer_norm(z) * (1.0 + sc) + sh, W["head_w"], W["head_b"])
    if last_block_rows is not None:
        return y
    return unpatchify(y, cfg.latent_shape, pt, ph, pw)
