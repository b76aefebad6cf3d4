"""Allocation-free scoring entry point (cs_score_noalloc) against cs_score.

Both compute s_i = <w, x_i> / sqrt(D) with the same kernels and the same
fixed summation order, so the allocation-free call must reproduce the
rollout's cs_score bit for bit on the same latents.  Two calls in a row on
one GPU share the library's static scratch array; the second, with a
smaller input, must not see the first call's leftovers."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

from paper_2607_23159_amd import binding as B
from paper_2607_23159_amd import synth
from paper_2607_23159_amd.search import GpuModel, Inputs


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()


def _rollout_scores_and_latents(name, n_steps_run, n_branch=1):
    """cs_score of a rollout after a few steps, and its latents on the device."""
    wl = synth.make_workload(name, n_branch=n_branch, init="stress", dtype=synth.DTYPE_FP32)
    gm = GpuModel(wl.model, wl.weights)
    inp = Inputs(wl)
    r = wl.roll
    h = B.cs_rollout_init(gm.h, B.RolloutDesc(r, wl.timesteps), inp.x1, inp.ctx[0],
                          inp.ctx[1] if n_branch == 2 else None)
    try:
        for k in range(1, n_steps_run + 1):
            B.cs_denoise_step(h, k)
        s = B.cs_score(h, inp.w, r.n_cand)
        lat = torch.empty_like(inp.x1)
        B.cs_rollout_latents(h, lat)
        torch.cuda.synchronize()
    finally:
        B.cs_rollout_free(h)
    gm.close()
    return s, lat, inp.w, wl.model.latent_numel


def test_noalloc_scores_equal_cs_score_on_two_calls():
    # first call: the ragged geometry (D = 19,008: 3 chunks, the last partial)
    s1, x1, w1, D1 = _rollout_scores_and_latents("ragged", 3, n_branch=2)
    n1 = x1.shape[0]
    out1 = torch.full((n1,), float("nan"), dtype=torch.float64, device="cuda")
    B.cs_score_noalloc(x1, w1, n1, D1, out1)
    torch.cuda.synchronize()
    assert np.array_equal(out1.cpu().numpy(), s1), (out1.cpu().numpy(), s1)
    # second call right after, smaller input: 2 of the tiny workload's
    # latents (D = 16,384: 2 chunks, fewer partials than the first call left)
    s2, x2, w2, D2 = _rollout_scores_and_latents("tiny", 4)
    assert D2 < D1
    out2 = torch.full((2,), float("nan"), dtype=torch.float64, device="cuda")
    B.cs_score_noalloc(x2[:2].contiguous(), w2, 2, D2, out2)
    torch.cuda.synchronize()
    assert np.array_equal(out2.cpu().numpy(), s2[:2]), (out2.cpu().numpy(), s2[:2])


def test_noalloc_rejects_sizes_beyond_its_scratch_and_bad_arguments():
    x = torch.zeros(8, dtype=torch.float32, device="cuda")
    out = torch.zeros(1, dtype=torch.float64, device="cuda")
    lib = B.lib()
    big_n, D = 65535, 8192 * 9           # 65535 * 9 partials > 512 Ki
    assert big_n * 9 > 512 * 1024
    st = lib.cs_score_noalloc(x.data_ptr(), x.data_ptr(), big_n, D, out.data_ptr(), None)
    assert st == B.CS_E_INVAL and "scratch capacity" in B.cs_last_error()
    assert lib.cs_score_noalloc(x.data_ptr(), x.data_ptr(), 1, 6, out.data_ptr(), None) == B.CS_E_INVAL
    assert lib.cs_score_noalloc(None, x.data_ptr(), 1, 8, out.data_ptr(), None) == B.CS_E_INVAL
    assert lib.cs_score_noalloc(x.data_ptr(), x.data_ptr(), 0, 8, out.data_ptr(), None) == B.CS_E_INVAL
    assert lib.cs_score_noalloc(x.data_ptr() + 4, x.data_ptr(), 1, 4, out.data_ptr(), None) == B.CS_E_INVAL
    # a valid call still works after the rejected ones
    B.cs_score_noalloc(x, x, 1, 8, out)
    torch.cuda.synchronize()
    assert out.item() == 0.0
