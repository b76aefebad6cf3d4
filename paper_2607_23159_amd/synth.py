"""Seeded synthetic inputs and the workload registry.

This module is the only code shared by the GPU path's callers and by the
CPU oracle.  It draws random numbers and lays them out; it holds none of
the method's arithmetic (no transformer, no cache rule, no update, no
score).  Everything is drawn from seeded torch CPU generators so a
(config, seed) pair always produces the same arrays.

Workloads stand in for the paper's video models (Sec. Reproducibility,
table of model-card generation configurations): random-init weights of the
Wan2.1/2.2 transformer shapes, N(0,1) text embeddings shaped like the
umT5 context (512 x 4096), N(0,1) latent noise per candidate seed
(Sec. Preliminaries: the seed fixes x_1 ~ N(0, I)).

Weight layout (the order of the flat weight array handed to
``cs_model_init``): every matrix is stored [out][in] row-major, the way a
linear layer maps an input row x to x W^T + b.  The order is given by
:func:`weight_spec`.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Tuple

import numpy as np
import torch

# Seeds used for every workload (candidate i's noise uses NOISE_SEED0 + i,
# mirroring the paper's per-candidate torch.Generator seeded with the seed).
WEIGHT_SEED = 0
CTX_COND_SEED = 1
CTX_UNCOND_SEED = 2
SCORER_SEED = 3
NOISE_SEED0 = 100

CACHE_OFF, CACHE_ADAPTIVE, CACHE_STATIC, CACHE_PAB = 0, 1, 2, 3
DTYPE_BF16, DTYPE_FP32 = 0, 1


@dataclasses.dataclass(frozen=True)
class ModelCfg:
    n_blocks: int
    hidden: int
    heads: int
    head_dim: int
    ffn: int
    text_dim: int
    text_len: int
    in_ch: int
    lat_f: int
    lat_h: int
    lat_w: int
    freq_dim: int = 256
    patch_t: int = 1
    patch_h: int = 2
    patch_w: int = 2
    dtype: int = DTYPE_BF16

    @property
    def out_ch(self) -> int:
        return self.in_ch

    @property
    def patch_dim(self) -> int:
        return self.in_ch * self.patch_t * self.patch_h * self.patch_w

    @property
    def grid(self) -> Tuple[int, int, int]:
        return (self.lat_f // self.patch_t, self.lat_h // self.patch_h,
                self.lat_w // self.patch_w)

    @property
    def tokens(self) -> int:
        f, h, w = self.grid
        return f * h * w

    @property
    def latent_shape(self) -> Tuple[int, int, int, int]:
        return (self.in_ch, self.lat_f, self.lat_h, self.lat_w)

    @property
    def latent_numel(self) -> int:
        return self.in_ch * self.lat_f * self.lat_h * self.lat_w

    def with_dtype(self, dtype: int) -> "ModelCfg":
        return dataclasses.replace(self, dtype=dtype)


@dataclasses.dataclass(frozen=True)
class RolloutCfg:
    n_cand: int
    n_steps: int
    n_branch: int = 1
    k_warm: int = 5
    k_cool: int = 5
    tau: float = 0.1
    guidance: float = 5.0
    mode: int = CACHE_ADAPTIVE
    static_k: int = 2
    shift: float = 1.0
    # attention-output broadcast ranges (CACHE_PAB): self- and cross-attention
    # outputs are recomputed every pab_self / pab_cross steps
    pab_self: int = 2
    pab_cross: int = 6


# --------------------------------------------------------------------------
# Workload registry.  Shapes follow the public model cards of the models the
# paper runs (Sec. Reproducibility); latent = 16 (or 48) channels at 1/4
# temporal and 1/8 (or 1/16) spatial compression of 81x480x832 (121x704x1280).
# --------------------------------------------------------------------------
_WAN13B = dict(n_blocks=30, hidden=1536, heads=12, head_dim=128, ffn=8960,
               text_dim=4096, text_len=512, in_ch=16, lat_f=21, lat_h=60,
               lat_w=104)

MODELS: Dict[str, ModelCfg] = {
    # 2 blocks, hidden 128, 4x32 heads, 256 tokens: oracle finishes in seconds.
    "tiny": ModelCfg(n_blocks=2, hidden=128, heads=4, head_dim=32, ffn=512,
                     text_dim=128, text_len=32, in_ch=16, lat_f=4, lat_h=16,
                     lat_w=16, dtype=DTYPE_FP32),
    # Ragged geometry: 3x9x11 = 297 tokens (no tile size divides it), 100-wide
    # latent rows, 4 heads x 64.
    "ragged": ModelCfg(n_blocks=2, hidden=256, heads=4, head_dim=64, ffn=512,
                       text_dim=64, text_len=19, in_ch=16, lat_f=3, lat_h=18,
                       lat_w=22, dtype=DTYPE_FP32),
    # Wan widths, 2 blocks, 384 tokens: full-width parity at oracle cost.
    "wan_mid": ModelCfg(n_blocks=2, hidden=1536, heads=12, head_dim=128,
                        ffn=8960, text_dim=4096, text_len=512, in_ch=16,
                        lat_f=3, lat_h=16, lat_w=32),
    # Wan2.2-5B and Wan2.1-14B widths, 2 blocks, 384 tokens: the widest
    # projections (K up to 5120, N up to 15360) and 24 / 40 heads at oracle cost.
    "wan5b_mid": ModelCfg(n_blocks=2, hidden=3072, heads=24, head_dim=128,
                          ffn=14336, text_dim=4096, text_len=512, in_ch=48,
                          lat_f=3, lat_h=16, lat_w=32),
    "wan14b_mid": ModelCfg(n_blocks=2, hidden=5120, heads=40, head_dim=128,
                           ffn=13824, text_dim=4096, text_len=512, in_ch=16,
                           lat_f=3, lat_h=16, lat_w=32),
    # One Wan2.1-1.3B block at the full 32,760-token latent.
    "wan13b_block1": ModelCfg(**dict(_WAN13B, n_blocks=1)),
    "wan13b": ModelCfg(**_WAN13B),
    "wan5b": ModelCfg(n_blocks=30, hidden=3072, heads=24, head_dim=128,
                      ffn=14336, text_dim=4096, text_len=512, in_ch=48,
                      lat_f=31, lat_h=44, lat_w=80),
    "wan14b": ModelCfg(n_blocks=40, hidden=5120, heads=40, head_dim=128,
                       ffn=13824, text_dim=4096, text_len=512, in_ch=16,
                       lat_f=21, lat_h=60, lat_w=104),
}

# Warmup / cooldown: 5 at T=50 (Sec. Method, adaptive skip rule); at T=10 the
# proportional value round(0.1*T) = 1 is used so that anything can skip.
WORKLOADS: Dict[str, Tuple[str, RolloutCfg]] = {
    "tiny": ("tiny", RolloutCfg(n_cand=4, n_steps=10, k_warm=1, k_cool=1,
                                tau=0.1)),
    "ragged": ("ragged", RolloutCfg(n_cand=3, n_steps=8, k_warm=1, k_cool=1,
                                    tau=0.1)),
    "wan_mid": ("wan_mid", RolloutCfg(n_cand=4, n_steps=10, k_warm=1,
                                      k_cool=1, tau=0.1)),
    "wan13b_full": ("wan13b", RolloutCfg(n_cand=1, n_steps=50,
                                         mode=CACHE_OFF, tau=0.0)),
    "wan13b_cached": ("wan13b", RolloutCfg(n_cand=8, n_steps=50, tau=0.1)),
    "wan5b_cached": ("wan5b", RolloutCfg(n_cand=4, n_steps=50, tau=0.1)),
    "wan14b_cached": ("wan14b", RolloutCfg(n_cand=4, n_steps=50, tau=0.1)),
}


def timestep_grid(n_steps: int, shift: float = 1.0) -> np.ndarray:
    """Decreasing grid t_1 = 1 > ... > t_{T+1} = 0 (Sec. Preliminaries).

    Uniform in [0, 1]; an optional time shift t -> s t / (1 + (s-1) t)
    keeps the end points.  Returned as float32 (what the library takes).
    """
    u = 1.0 - np.arange(n_steps + 1, dtype=np.float64) / n_steps
    if shift != 1.0:
        u = shift * u / (1.0 + (shift - 1.0) * u)
    u[0], u[-1] = 1.0, 0.0
    return u.astype(np.float32)


# --------------------------------------------------------------------------
# Weight layout
# --------------------------------------------------------------------------
# init kinds: "n" = N(0, std), "one" = 1, "zero" = 0, "gate" = mod table
# (N(0, std); the stress init adds 1 to its gate rows).
def weight_spec(m: ModelCfg) -> List[Tuple[str, Tuple[int, ...], str]]:
    d, p, F = m.hidden, m.patch_dim, m.ffn
    spec: List[Tuple[str, Tuple[int, ...], str]] = [
        ("patch_w", (d, p), "n"), ("patch_b", (d,), "n"),
        ("text1_w", (d, m.text_dim), "n"), ("text1_b", (d,), "n"),
        ("text2_w", (d, d), "n"), ("text2_b", (d,), "n"),
        ("time1_w", (d, m.freq_dim), "n"), ("time1_b", (d,), "n"),
        ("time2_w", (d, d), "n"), ("time2_b", (d,), "n"),
        ("mod_w", (6 * d, d), "n"), ("mod_b", (6 * d,), "n"),
    ]
    for j in range(m.n_blocks):
        b = f"blk{j}."
        spec += [
            (b + "mod", (6, d), "gate"),
            (b + "qkv_w", (3 * d, d), "n"), (b + "qkv_b", (3 * d,), "n"),
            (b + "q_gain", (d,), "one"), (b + "k_gain", (d,), "one"),
            (b + "o_w", (d, d), "n"), (b + "o_b", (d,), "n"),
            (b + "ca_ln_g", (d,), "one"), (b + "ca_ln_b", (d,), "zero"),
            (b + "caq_w", (d, d), "n"), (b + "caq_b", (d,), "n"),
            (b + "cak_w", (d, d), "n"), (b + "cak_b", (d,), "n"),
            (b + "cav_w", (d, d), "n"), (b + "cav_b", (d,), "n"),
            (b + "caq_gain", (d,), "one"), (b + "cak_gain", (d,), "one"),
            (b + "cao_w", (d, d), "n"), (b + "cao_b", (d,), "n"),
            (b + "ffn1_w", (F, d), "n"), (b + "ffn1_b", (F,), "n"),
            (b + "ffn2_w", (d, F), "n"), (b + "ffn2_b", (d,), "n"),
        ]
    spec += [("head_mod", (2, d), "n"), ("head_w", (p, d), "n"),
             ("head_b", (p,), "n")]
    return spec


def weight_count(m: ModelCfg) -> int:
    return sum(int(np.prod(s)) for _, s, _ in weight_spec(m))


def make_weights(m: ModelCfg, seed: int = WEIGHT_SEED, init: str = "paper",
                 std: Optional[float] = None) -> np.ndarray:
    """Flat float32 weight array in :func:`weight_spec` order.

    ``init="paper"``: every matrix, bias and modulation table N(0, 0.02),
    norm gains 1, layer-norm shift 0 (random init of the workload).
    ``init="stress"``: N(0, 0.05) weights, the gate rows of every block's
    modulation table shifted by +1, and norm gains 1 + N(0, 0.1), so the
    attention and feed-forward branches reach the output with weight
    comparable to the residual stream (used by parity tests).
    """
    if std is None:
        std = 0.02 if init == "paper" else 0.05
    n = weight_count(m)
    g = torch.Generator().manual_seed(seed)
    flat = torch.randn(n, generator=g, dtype=torch.float32)
    flat.mul_(std)
    out = flat.numpy()
    off = 0
    for name, shape, kind in weight_spec(m):
        k = int(np.prod(shape))
        view = out[off:off + k].reshape(shape)
        if kind == "one":
            if init == "stress":
                view *= (0.1 / std)
                view += 1.0
            else:
                view[...] = 1.0
        elif kind == "zero":
            if init != "stress":
                view[...] = 0.0
        elif kind == "gate" and init == "stress":
            view[2] += 1.0
            view[5] += 1.0
        off += k
    return out


def unflatten(m: ModelCfg, flat: np.ndarray) -> Dict[str, np.ndarray]:
    """Named views into a flat weight array (no copy)."""
    out: Dict[str, np.ndarray] = {}
    off = 0
    for name, shape, _ in weight_spec(m):
        k = int(np.prod(shape))
        out[name] = flat[off:off + k].reshape(shape)
        off += k
    assert off == flat.size, (off, flat.size)
    return out


def make_context(m: ModelCfg, seed: int) -> np.ndarray:
    """Text-embedding stand-in: N(0,1) [text_len][text_dim] float32."""
    g = torch.Generator().manual_seed(seed)
    return torch.randn(m.text_len, m.text_dim, generator=g).numpy()


def make_noise(m: ModelCfg, n_cand: int, seed0: int = NOISE_SEED0) -> np.ndarray:
    """x_1 ~ N(0, I) per candidate, [N][C][F][H][W] float32; candidate i is
    drawn from its own generator seeded seed0 + i."""
    out = np.empty((n_cand,) + m.latent_shape, dtype=np.float32)
    for i in range(n_cand):
        g = torch.Generator().manual_seed(seed0 + i)
        out[i] = torch.randn(m.latent_shape, generator=g).numpy()
    return out


def make_scorer(m: ModelCfg, seed: int = SCORER_SEED) -> np.ndarray:
    """Fixed random projection vector w ~ N(0,1) of length D."""
    g = torch.Generator().manual_seed(seed)
    return torch.randn(m.latent_numel, generator=g).numpy()


def make_latent_batch(shape: Tuple[int, ...], seed: int, scale: float = 1.0) -> np.ndarray:
    """Generic N(0, scale^2) float32 array (kernel-level test inputs)."""
    g = torch.Generator().manual_seed(seed)
    return (torch.randn(shape, generator=g) * scale).numpy()


@dataclasses.dataclass
class Workload:
    name: str
    model: ModelCfg
    roll: RolloutCfg
    weights: np.ndarray
    ctx: List[np.ndarray]            # one per branch: [cond, uncond]
    noise: np.ndarray
    scorer: np.ndarray
    timesteps: np.ndarray

    def named_weights(self) -> Dict[str, np.ndarray]:
        return unflatten(self.model, self.weights)


def make_workload(name: str, *, n_branch: int = 1, dtype: Optional[int] = None,
                  init: str = "paper", n_cand: Optional[int] = None,
                  n_steps: Optional[int] = None, tau: Optional[float] = None,
                  mode: Optional[int] = None, model: Optional[str] = None,
                  ctx_seed: int = CTX_COND_SEED, noise_seed0: int = NOISE_SEED0,
                  **roll_overrides) -> Workload:
    """A workload by name.  ``ctx_seed`` draws the conditional text context
    (a stand-in prompt; the unconditional one keeps its own seed) and
    ``noise_seed0`` the first candidate's noise seed."""
    mname, roll = WORKLOADS[name] if name in WORKLOADS else (name, RolloutCfg(1, 10))
    if model is not None:
        mname = model
    m = MODELS[mname]
    if dtype is not None:
        m = m.with_dtype(dtype)
    kw = dict(n_branch=n_branch, **roll_overrides)
    if n_cand is not None:
        kw["n_cand"] = n_cand
    if n_steps is not None:
        kw["n_steps"] = n_steps
    if tau is not None:
        kw["tau"] = tau
    if mode is not None:
        kw["mode"] = mode
    roll = dataclasses.replace(roll, **kw)
    ctx = [make_context(m, ctx_seed)]
    if roll.n_branch == 2:
        ctx.append(make_context(m, CTX_UNCOND_SEED))
    return Workload(name=name, model=m, roll=roll,
                    weights=make_weights(m, init=init), ctx=ctx,
                    noise=make_noise(m, roll.n_cand, noise_seed0), scorer=make_scorer(m),
                    timesteps=timestep_grid(roll.n_steps, roll.shift))
