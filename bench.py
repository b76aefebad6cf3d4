"""Benchmark: cached candidate denoise-steps/s on one MI355X.

One step = one CachedSearch exploration pass (Alg. 1) over one batch of
synthetic inputs: rollout init (cache reset, text keys/values), T Euler
steps of N candidates with the cache decision, transformer on the computed
calls, skip/refresh/CFG/Euler update, then scoring and ranking.  The
full-compute reference rollout of the same seeds (cache off) is tau
independent; with --reference it is run once before the timed region and
the cached ranking is compared with it (Spearman rho, top-1).

Printed: one JSON line with the metric, the roofline of the dominant kernel
(self-attention, timed by HIP events on the rollout stream inside the
library), and the CPU oracle timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0
TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "self_attention_traffic_wan13b_n8_tau0.1.md")
ATTN_SOURCES = [os.path.join(ROOT, "paper_2607_23159_amd", "csrc", f)
                for f in ("attn_kernel.hpp", "k_attn.hip", "common.hpp")]


def attn_source_hash() -> str:
    import hashlib
    h = hashlib.sha256()
    for f in ATTN_SOURCES:
        h.update(open(f, "rb").read())
    return h.hexdigest()[:16]


def measured_traffic(workload: str, n_branch: int):
    """HBM bytes per self-attention launch from the committed counter
    summary, or None when it does not exist, covers another workload, or the
    kernel sources changed since the counters were taken."""
    try:
        txt = open(TRAFFIC_PROFILE).read()
    except OSError:
        return None
    fields = dict(l.split(":", 1) for l in txt.splitlines() if l.startswith("- ") and ":" in l)
    get = lambda k: fields.get("- " + k, "").strip().strip("`")
    if get("kernel_source_sha256") != attn_source_hash():
        return None
    if get("workload") != workload or get("n_branch") != str(n_branch):
        return None
    try:
        return float(get("bytes_per_launch"))
    except ValueError:
        return None


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=1)
    p.add_argument("--warmup", type=int, default=0)
    p.add_argument("--workload", default="wan13b_cached")
    p.add_argument("--tau", type=float, default=None)
    p.add_argument("--n-cand", type=int, default=None)
    p.add_argument("--n-steps", type=int, default=None)
    p.add_argument("--cfg", action="store_true", help="two guidance branches (w = 5.0)")
    p.add_argument("--fp32", action="store_true", help="fp32 transformer arithmetic")
    p.add_argument("--reference", action="store_true", help="also run the full rollouts for rho")
    p.add_argument("--tau-sweep", default="", help="comma-separated extra tau values, one rollout each")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-profile", action="store_true", help="no per-kernel HIP event timing")
    p.add_argument("--mode", choices=["adaptive", "static", "pab"], default="adaptive",
                   help="reuse engine: the drift-indicator cache, the static schedule, or "
                        "attention-output broadcasting")
    p.add_argument("--pab-self", type=int, default=2, help="self-attention broadcast range")
    p.add_argument("--pab-cross", type=int, default=6, help="cross-attention broadcast range")
    p.add_argument("--calibration-copy", type=int, default=0,
                   help="bytes of one plain device-to-device copy made before timing (a "
                        "known-size reference for HBM counter runs)")
    return p.parse_args()


def cpu_baseline(model_cfg, computed_per_cand_step: float, n_branch: int):
    """The float64 oracle on a bounded sample of the workload: one
    transformer block at full token count with R1 and R2 sampled query rows
    (keys/values of all tokens), extrapolated linearly to all rows, times
    the block count, times the transformer calls per candidate-step the GPU
    run measured."""
    import dataclasses

    import numpy as np

    from oracle import dit
    from paper_2607_23159_amd import synth

    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        cores = os.cpu_count() or 1
    m1 = dataclasses.replace(model_cfg, n_blocks=1)
    W = {k: v.astype(np.float64) for k, v in synth.unflatten(m1, synth.make_weights(m1)).items()}
    x = synth.make_noise(m1, 1)[0]
    emb = dit.text_embedding(synth.make_context(m1, 1), W)
    L = m1.tokens
    times = {}
    R1, R2 = 256, 2048
    for nr in (R1, R2):
        rows = np.linspace(0, L - 1, nr).astype(np.int64)
        t0 = time.perf_counter()
        dit.velocity(x, 0.5, emb, W, m1, last_block_rows=rows)
        times[nr] = time.perf_counter() - t0
    per_row = (times[R2] - times[R1]) / (R2 - R1)
    fixed = times[R1] - R1 * per_row
    block_s = fixed + per_row * L
    eval_s = block_s * model_cfg.n_blocks
    cand_step_s = eval_s * computed_per_cand_step
    return {"value": 1.0 / cand_step_s, "unit": "candidate-steps/s", "cores": int(cores),
            "kind": "oracle",
            "sample": (f"float64 oracle, one {model_cfg.hidden}-wide block at {L} tokens with {R1} and {R2} "
                       f"sampled query rows ({times[R1]:.1f} s, {times[R2]:.1f} s), extrapolated to all "
                       f"rows x {model_cfg.n_blocks} blocks = {eval_s:.0f} s per transformer call, "
                       f"x {computed_per_cand_step:.3f} calls per candidate-step (measured on the GPU run, "
                       f"B={n_branch})")}


def progress(msg: str) -> None:
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU: this build has no multi-GPU path "
              "(candidates would shard across GPUs with no per-step traffic); run with --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2607_23159_amd import binding as B
    from paper_2607_23159_amd import synth
    from paper_2607_23159_amd.search import GpuModel, Inputs

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    B.lib()
    dtype = synth.DTYPE_FP32 if args.fp32 else synth.DTYPE_BF16
    nb = 2 if args.cfg else 1
    t_gen = time.perf_counter()
    mode = {"adaptive": synth.CACHE_ADAPTIVE, "static": synth.CACHE_STATIC,
            "pab": synth.CACHE_PAB}[args.mode]
    wl = synth.make_workload(args.workload, n_branch=nb, dtype=dtype, n_cand=args.n_cand,
                             n_steps=args.n_steps, tau=args.tau, mode=mode,
                             pab_self=args.pab_self, pab_cross=args.pab_cross)
    m, r = wl.model, wl.roll
    gen_s = time.perf_counter() - t_gen
    progress(f"inputs generated ({gen_s:.1f} s); uploading weights")
    gm = GpuModel(m, wl.weights)
    inp = Inputs(wl)
    progress("model ready")
    wl.weights = None
    N, T = r.n_cand, r.n_steps
    S = N * nb

    reused = [0, 0]   # self / cross attention reuses, accumulated by rollout()

    def rollout(mode=None, label="cached"):
        desc = B.RolloutDesc(r, wl.timesteps, **({} if mode is None else {"mode": mode}))
        h = B.cs_rollout_init(gm.h, desc, inp.x1, inp.ctx[0], inp.ctx[1] if nb == 2 else None)
        try:
            for k in range(1, T + 1):
                B.cs_denoise_step(h, k)
                if k % 10 == 0:
                    progress(f"{label} rollout: step {k}/{T}")
            scores = B.cs_score(h, inp.w, N)
            st = B.cs_rollout_stats(h)
            reused[0] += int(st.self_reused)
            reused[1] += int(st.cross_reused)
            return scores, int(st.computed), int(st.calls)
        finally:
            B.cs_rollout_free(h)

    if args.calibration_copy > 0:
        src = torch.empty(args.calibration_copy, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        progress(f"calibration copy of {args.calibration_copy} bytes done")

    # prime: load every kernel once (one transformer call), untimed
    v = torch.empty_like(inp.x1[:1])
    B.cs_velocity(gm.h, inp.x1[:1], 1, 1.0, inp.ctx[0], v)
    torch.cuda.synchronize()

    ref_scores = None
    full_s = None
    if args.reference:
        torch.cuda.synchronize()
        t_ref = time.perf_counter()
        ref_scores, _, _ = rollout(mode=synth.CACHE_OFF, label="full reference")
        full_s = time.perf_counter() - t_ref

    for _ in range(args.warmup):
        rollout(label="warmup")
    torch.cuda.synchronize()

    if not args.no_profile:
        B.cs_profile_enable(gm.h, True)
        B.cs_profile_reset(gm.h)
    computed = calls = 0
    rho = top1 = None
    reused[0] = reused[1] = 0
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        scores, c, n = rollout(label="timed")
        computed += c
        calls += n
        if N < 2:
            pass                     # one candidate: nothing to rank (cs_rank needs n >= 2)
        elif ref_scores is not None:
            _, _, rho, top1 = B.cs_rank(scores, ref_scores)
        else:
            B.cs_rank(scores, scores)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = wall * 1e3 / args.steps
    value = N * T * args.steps / wall

    fam = {}
    if not args.no_profile:
        for f, name in enumerate(B.KERNEL_FAMILIES):
            fam[name] = B.cs_profile_read(gm.h, f)
        B.cs_profile_enable(gm.h, False)

    L, d = m.tokens, m.hidden
    evals = computed                                   # stream evaluations in the timed region
    self_evals = computed - reused[0]                  # of which ran self-attention
    cross_evals = computed - reused[1]                 # ... and cross-attention
    roof = None
    if fam:
        sa_ms, sa_n = fam["self_attn"]
        flops = 4.0 * L * L * d * m.n_blocks * self_evals   # QK^T and PV, 2 flop per MAC
        ach = flops / (sa_ms * 1e-3) / 1e12 if sa_ms > 0 else 0.0
        peak = PEAK_FP32_TFLOPS if args.fp32 else PEAK_BF16_TFLOPS
        roof = {"bound": "mfma", "kernel": "k_flash (self-attention)", "achieved": round(ach, 1),
                "peak": peak, "unit": "TFLOP/s", "frac": round(ach / peak, 4),
                "traffic": measured_traffic(args.workload, nb) if not args.fp32 else None,
                "launches": sa_n, "avg_launch_ms": round(sa_ms / max(sa_n, 1), 3),
                "flop_per_launch": flops / max(sa_n, 1)}
        g_ms, g_n = fam["gemm"]
        F = m.ffn
        # QKV + out-projection (4 d^2) on self-attention evaluations, cross q +
        # out-projection (2 d^2) on cross-attention evaluations, FFN (2 d F),
        # patch embedding and head on every evaluation
        gflops = (2.0 * L * m.n_blocks * (4 * d * d * self_evals + 2 * d * d * cross_evals + 2 * d * F * evals)
                  + 4.0 * L * d * m.patch_dim * evals)
        roof["gemm_tflops"] = round(gflops / (g_ms * 1e-3) / 1e12, 1) if g_ms > 0 else None
        roof["family_ms"] = {k: round(vv[0], 2) for k, vv in fam.items()}
        # streaming kernels against the HBM roofline, algorithmic bytes:
        # decision reads x and every branch's x_ref on each step past the
        # forced windows; the fused update reads and writes x, reads v (or
        # Delta when skipped) per stream and, when the cache keeps state,
        # writes Delta, x_ref per computed stream; scoring reads x and w per
        # candidate
        D = int(np.prod(wl.noise.shape[1:]))
        K = args.steps
        adaptive = r.mode == synth.CACHE_ADAPTIVE
        dec_launches = (T - r.k_warm - r.k_cool) * K if adaptive else 0
        stream_bytes = {
            "decide": 4.0 * D * N * (1 + nb) * dec_launches,
            "update": 4.0 * D * (2 * N * T * K + S * T * K
                                 + (2 * computed if r.mode in (synth.CACHE_ADAPTIVE, synth.CACHE_STATIC) else 0)),
            "score": 8.0 * D * N * K,
        }
        # each family's time is the sum of HIP-event brackets around its
        # calls, so it includes every call's dispatch and event overhead:
        # small against the 40 ms attention launches, but of the order of
        # the 20-60 us these kernels take (rates below are lower bounds; a
        # kernel trace gives the kernels alone)
        roof["streaming"] = {"timing": "per-call HIP-event brackets incl. dispatch overhead (lower bound)"}
        for name, nbytes in stream_bytes.items():
            ms, n = fam[name]
            gbs = nbytes / (ms * 1e-3) / 1e9 if ms > 0 and nbytes > 0 else None
            roof["streaming"][name] = {"bytes": nbytes, "ms": round(ms, 3), "calls": n,
                                       "GB/s": None if gbs is None else round(gbs, 1),
                                       "frac": None if gbs is None else round(gbs / PEAK_HBM_GBS, 4)}

    # tau sweep (each value: one timed cached rollout, compared with the
    # reference when it was run)
    sweep = []
    for tv in [float(x) for x in args.tau_sweep.split(",") if x.strip()]:
        r_t = __import__("dataclasses").replace(r, tau=tv)
        desc = B.RolloutDesc(r_t, wl.timesteps)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        h = B.cs_rollout_init(gm.h, desc, inp.x1, inp.ctx[0], inp.ctx[1] if nb == 2 else None)
        try:
            for k in range(1, T + 1):
                B.cs_denoise_step(h, k)
                if k % 10 == 0:
                    progress(f"tau={tv} rollout: step {k}/{T}")
            sc = B.cs_score(h, inp.w, N)
            st = B.cs_rollout_stats(h)
        finally:
            B.cs_rollout_free(h)
        dt_s = time.perf_counter() - t1
        rec = {"tau": tv, "candidate_steps_per_s": round(N * T / dt_s, 4),
               "skip_fraction": round(1 - st.computed / st.calls, 4), "ms_per_rollout": round(dt_s * 1e3, 1)}
        if ref_scores is not None and N >= 2:
            _, _, rho_t, top1_t = B.cs_rank(sc, ref_scores)
            rec.update({"rho_vs_full": rho_t, "top1_vs_full": top1_t,
                        "regret": float(max(ref_scores) - ref_scores[int(np.argmax(sc))])})
        sweep.append(rec)

    # cost model (Sec. Method, cost analysis): per-rollout costs of the
    # cached (C_c) and full (C_f) N-candidate batches, per candidate
    costs = None
    if full_s is not None:
        cc = wall / args.steps / N
        cf = full_s / N
        gamma = cc / cf
        costs = {"C_c_s": round(cc, 3), "C_f_s": round(cf, 3), "gamma": round(gamma, 4),
                 "break_even_N": round(1.0 / (1.0 - gamma), 3) if gamma < 1 else None,
                 "keep_s": round(N * cc, 2), "commit_s": round(N * cc + cf, 2),
                 "best_of_N_full_s": round(N * cf, 2)}

    cpu = None
    if not args.no_cpu_baseline:
        progress("timing the CPU oracle on a sample")
        try:
            cpu = cpu_baseline(m, computed / (N * T * args.steps), nb)
        except Exception as e:  # report, never hide
            cpu = {"value": None, "error": repr(e)}

    out = {
        "metric": "cached candidate denoise-steps/s (N seeds, 1 GPU)",
        "value": round(value, 4),
        "unit": "candidate-steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 1),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if args.fp32 else "bf16",
        "data": "synthetic",
        "config": {"workload": (f"{args.workload}: Wan-shaped DiT {m.n_blocks} blocks d={d} "
                                f"{m.heads}x{m.head_dim} ffn={m.ffn}, {L} tokens, N={N} seeds, "
                                f"T={T}, " + (f"PAB ranges self {r.pab_self} cross {r.pab_cross}"
                                               if mode == synth.CACHE_PAB else
                                               f"tau={r.tau}" if mode == synth.CACHE_ADAPTIVE else
                                               f"static period {r.static_k}")
                                + f", B={nb}, random init"),
                   "n_cand": N, "n_steps": T, "tau": r.tau, "n_branch": nb,
                   "cache_mode": r.mode},
        "skip_fraction": round(1.0 - computed / max(calls, 1), 4),
        "attn_reuse_fraction": ({"self": round(reused[0] / max(calls, 1), 4),
                                 "cross": round(reused[1] / max(calls, 1), 4)}
                                if mode == synth.CACHE_PAB else None),
        "rho_vs_full": rho,
        "top1_vs_full": top1,
        "tau_sweep": sweep or None,
        "costs": costs,
        "roofline": roof,
        "cpu_baseline": cpu,
        "input_gen_s": round(gen_s, 1),
    }
    print(json.dumps(out), flush=True)
    gm.close()


if __name__ == "__main__":
    main()
