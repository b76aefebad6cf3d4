"""GPU checks at full size in the launch configurations the bench times
(Wan2.1-1.3B: 8 streams of 32,760 tokens in one transformer call; one
Wan2.2-5B block: 4 streams of 27,280 tokens; one Wan2.1-14B block: 4
streams of 32,760 tokens).

The oracle cannot run whole full-size rollouts, so they are checked on
sampled outputs it computes one by one (one block, sampled tokens) and
through properties that hold at any size: per-stream batch invariance,
tau = 0 reproducing the uncached rollout bit for bit, tau = inf computing
only the forced windows, PAB with range 1 reproducing the uncached rollout,
and a candidate's rollout not depending on which other seeds share its
batch."""
import dataclasses
import math
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

from oracle import dit as odit
from paper_2607_23159_amd import binding as B
from paper_2607_23159_amd import synth
from paper_2607_23159_amd.search import GpuModel, run_rollout
from parity import TOL, rel_l2, row_errors


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()


def _block_sampled(m, n, rows, sampled, single):
    """One block on n full-length latents in one call: sampled tokens of the
    streams in `sampled` against the oracle, the streams in `single` bitwise
    equal to their own single-stream calls."""
    w = synth.make_weights(m, init="stress")
    gm = GpuModel(m, w)
    W = {k: v.astype(np.float64) for k, v in synth.unflatten(m, w).items()}
    x = synth.make_noise(m, n, seed0=900)
    ctx = synth.make_context(m, 1)
    xd = torch.from_numpy(x.reshape(n, -1)).cuda()
    cd = torch.from_numpy(ctx).cuda()
    vn = gm.velocity(xd, 0.6, cd)
    emb = odit.text_embedding(ctx, W)
    for i in sampled:
        vp = odit.patchify(vn[i].cpu().numpy().reshape(x.shape[1:]), m.patch_t, m.patch_h, m.patch_w)
        ref = odit.velocity(x[i], 0.6, emb, W, m, last_block_rows=rows)
        err = rel_l2(vp[rows], ref)
        tok = row_errors(vp[rows], ref)
        say(f"  stream {i} sampled rel_l2={err:.3e} per-token {np.round(tok, 5).tolist()}")
        assert err < TOL[0] / 2
        assert tok.max() < TOL[0] / 2      # every sampled token on its own, same bar
    for i in single:
        one = gm.velocity(xd[i:i + 1].contiguous(), 0.6, cd)
        assert torch.equal(one[0], vn[i])
    gm.close()


def test_block_8_streams_full_length_sampled():
    """One Wan2.1-1.3B block, 8 latents of 32,760 tokens in one call (the
    bench's row count, 262,080 GEMM rows): sampled tokens of two streams
    against the oracle, and every stream bitwise equal to its own
    single-stream call."""
    say("one block, 8 streams x 32760 tokens, bf16")
    _block_sampled(synth.MODELS["wan13b_block1"], 8, np.array([0, 255, 256, 16384, 32511, 32759]),
                   (0, 7), (0, 3, 7))


def test_block_16_streams_full_length_sampled():
    """One Wan2.1-1.3B block, 16 latents of 32,760 tokens in one call, the
    launch shape of a guided (two-branch) rollout of 8 seeds: 524,160 GEMM
    rows, an FFN hidden activation of 4.7e9 elements (offsets past 2^32).
    Sampled tokens of the first and last stream against the oracle; the last
    stream bitwise equal to its single-stream call."""
    say("one block, 16 streams x 32760 tokens, bf16")
    _block_sampled(synth.MODELS["wan13b_block1"], 16, np.array([0, 255, 256, 16384, 32511, 32759]),
                   (0, 15), (15,))


def test_block_wan5b_4_streams_full_length_sampled():
    """One Wan2.2-5B block (d = 3072, 24 heads, FFN 14336), 4 latents of
    27,280 tokens in one call, the 5B workload's launch shape: 71 full
    query tiles of 384 and a 16-query last one per head, 426 full key tiles
    of 64 and a 16-key last one.  Sampled tokens across those boundaries
    against the oracle; streams bitwise equal to single-stream calls."""
    say("one Wan2.2-5B block, 4 streams x 27280 tokens, bf16")
    m = dataclasses.replace(synth.MODELS["wan5b"], n_blocks=1)
    L = (m.lat_f // m.patch_t) * (m.lat_h // m.patch_h) * (m.lat_w // m.patch_w)
    assert L == 27280
    _block_sampled(m, 4, np.array([0, 383, 384, 13640, 27263, 27264, L - 1]), (0, 3), (0, 3))


def test_block_wan14b_4_streams_full_length_sampled():
    """One Wan2.1-14B block (d = 5120, 40 heads, FFN 13824), 4 latents of
    32,760 tokens in one call, the 14B workload's launch shape: every
    residual projection (K = 5120 and 13824) runs on the one-wave-per-SIMD
    GEMM with the deep residual epilogue.  Sampled tokens of one stream
    against the oracle; streams bitwise equal to single-stream calls."""
    say("one Wan2.1-14B block, 4 streams x 32760 tokens, bf16")
    m = dataclasses.replace(synth.MODELS["wan14b"], n_blocks=1)
    _block_sampled(m, 4, np.array([0, 383, 384, 16384, 32639, 32640, 32759]), (3,), (0, 3))


@pytest.fixture(scope="module")
def full_model():
    m = synth.MODELS["wan13b"]
    w = synth.make_weights(m)
    gm = GpuModel(m, w)
    yield m, w, gm
    gm.close()


def _short(m, w, n_cand, seed0=100, n_branch=1, **kw):
    roll = synth.RolloutCfg(n_cand=n_cand, n_steps=4, k_warm=1, k_cool=1, n_branch=n_branch, **kw)
    ctx = [synth.make_context(m, synth.CTX_COND_SEED)]
    if n_branch == 2:
        ctx.append(synth.make_context(m, synth.CTX_UNCOND_SEED))
    return synth.Workload(name="wan13b_short", model=m, roll=roll, weights=w,
                          ctx=ctx,
                          noise=synth.make_noise(m, n_cand, seed0=seed0),
                          scorer=synth.make_scorer(m), timesteps=synth.timestep_grid(4))


def test_full_model_rollout_properties(full_model):
    """Full 30-block model, 2 seeds, 4 steps."""
    m, w, gm = full_model
    wl = _short(m, w, 2)
    say("full model: tau=0 vs off")
    a = run_rollout(gm, wl, tau=0.0)
    b = run_rollout(gm, wl, mode=synth.CACHE_OFF)
    assert a.computed == a.calls
    assert np.array_equal(a.latents, b.latents) and np.array_equal(a.scores, b.scores)
    say("full model: tau=inf forced only")
    c = run_rollout(gm, wl, tau=math.inf)
    assert (c.masks.sum(axis=0) == 2).all()
    say("full model: PAB range 1 vs off")
    p = run_rollout(gm, wl, mode=synth.CACHE_PAB, pab_self=1, pab_cross=1)
    assert np.array_equal(p.latents, b.latents)
    say("full model: seed 101 alone vs in the batch")
    one = _short(m, w, 1, seed0=101)
    assert np.array_equal(one.noise[0], wl.noise[1])
    s = run_rollout(gm, one, tau=0.1)
    t = run_rollout(gm, wl, tau=0.1)
    assert np.array_equal(s.masks[:, 0], t.masks[:, 1])
    assert np.array_equal(s.latents[0], t.latents[1])


def test_full_model_guided_rollout_properties(full_model):
    """Full 30-block model with guidance (B = 2, w = 5), 2 seeds, 4 steps:
    tau = 0 reproduces the uncached guided rollout bit for bit, tau = inf
    computes only the forced windows and both branches decide alike (they
    see the same latent), and a seed's guided rollout is the same alone and
    in a batch."""
    m, w, gm = full_model
    wl = _short(m, w, 2, n_branch=2)
    say("full model, B=2: tau=0 vs off")
    a = run_rollout(gm, wl, tau=0.0)
    b = run_rollout(gm, wl, mode=synth.CACHE_OFF)
    assert a.computed == a.calls == 2 * 2 * 4
    assert np.array_equal(a.latents, b.latents) and np.array_equal(a.scores, b.scores)
    say("full model, B=2: tau=inf forced only")
    c = run_rollout(gm, wl, tau=math.inf)
    assert c.masks.shape == (4, 4) and (c.masks.sum(axis=0) == 2).all()
    assert np.array_equal(c.masks[:, 0::2], c.masks[:, 1::2])
    say("full model, B=2: seed 101 alone vs in the batch")
    one = _short(m, w, 1, seed0=101, n_branch=2)
    s = run_rollout(gm, one, tau=0.1)
    t = run_rollout(gm, wl, tau=0.1)
    assert np.array_equal(s.latents[0], t.latents[1])


def test_full_model_mixed_compute_and_skip_batches(full_model):
    """Full 30-block model, 4 seeds of 32,760 tokens, 4 steps replaying a
    schedule in which the seeds decide differently (steps with 1, 2 and 3 of
    the 4 streams computing, so the compacted transformer batch and the
    skip axpy run side by side in one step): every seed's latent equals its
    own single-seed replay of the same schedule bit for bit."""
    m, w, gm = full_model
    wl = _short(m, w, 4)
    ovr = np.array([[1, 1, 1, 1],
                    [1, 0, 1, 0],
                    [0, 1, 1, 0],
                    [1, 0, 0, 0]], np.uint8)
    say("full model: mixed compute/skip replay, 4 seeds")
    g = run_rollout(gm, wl, override=ovr)
    assert np.array_equal(g.masks, ovr)
    assert g.computed == int(ovr.sum())
    for i in range(4):
        say(f"  seed {100 + i} alone")
        one = _short(m, w, 1, seed0=100 + i)
        s = run_rollout(gm, one, override=ovr[:, i:i + 1])
        assert np.array_equal(s.latents[0], g.latents[i])
