"""Host logic of bench.py (no GPU): the one-GPU guard and the lookup of the
measured HBM traffic of the self-attention kernel in its counter summary."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402  (stdlib-only at import time)


@pytest.mark.parametrize("argv,env", [(["--gpus", "2"], {}), (["--gpus", "8"], {}),
                                      ([], {"WORLD_SIZE": "2"})])
def test_more_than_one_gpu_is_refused(argv, env):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py")] + argv,
                       env={**os.environ, **env}, capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""          # no JSON line for a refused run


def _summary(tmp_path, sha, workload="wan13b_cached", n_branch="1", nbytes="7522578237"):
    p = tmp_path / "traffic.md"
    p.write_text("# traffic\n\nsome text: not a field\n\n"
                 f"- workload: `{workload}`\n- n_branch: {n_branch}\n"
                 f"- kernel_source_sha256: {sha}\n- bytes_per_launch: {nbytes}\n")
    return str(p)


def test_measured_traffic_follows_the_kernel_sources(tmp_path, monkeypatch):
    sha = bench.attn_source_hash()
    assert len(sha) == 16 and int(sha, 16) >= 0
    monkeypatch.setattr(bench, "TRAFFIC_PROFILE", _summary(tmp_path, sha))
    assert bench.measured_traffic("wan13b_cached", 1) == 7522578237.0
    # another workload or branch count: the counters do not apply
    assert bench.measured_traffic("wan5b_cached", 1) is None
    assert bench.measured_traffic("wan13b_cached", 2) is None
    # kernel sources changed since the counters were taken
    stale = "0" * 16 if sha != "0" * 16 else "1" * 16
    monkeypatch.setattr(bench, "TRAFFIC_PROFILE", _summary(tmp_path, stale))
    assert bench.measured_traffic("wan13b_cached", 1) is None
    # unreadable value, missing file
    monkeypatch.setattr(bench, "TRAFFIC_PROFILE", _summary(tmp_path, sha, nbytes="n/a"))
    assert bench.measured_traffic("wan13b_cached", 1) is None
    monkeypatch.setattr(bench, "TRAFFIC_PROFILE", str(tmp_path / "absent.md"))
    assert bench.measured_traffic("wan13b_cached", 1) is None


def test_committed_traffic_summary_is_well_formed():
    """The committed summary names the default workload and a positive byte
    count; its hash is either current (the bench reports the traffic) or
    stale (the bench reports null), never unparsable."""
    txt = open(bench.TRAFFIC_PROFILE).read()
    fields = dict(l.split(":", 1) for l in txt.splitlines() if l.startswith("- ") and ":" in l)
    assert fields["- workload"].strip().strip("`") == "wan13b_cached"
    assert fields["- n_branch"].strip() == "1"
    assert float(fields["- bytes_per_launch"]) > 0
    v = bench.measured_traffic("wan13b_cached", 1)
    current = fields["- kernel_source_sha256"].strip().strip("`") == bench.attn_source_hash()
    assert (v is not None) == current


# ---------------------------------------------------------------- step units
def test_timed_rollouts_round_up_to_whole_rollouts():
    assert bench.timed_rollouts(20, 50) == 1      # the driver's --steps 20 at T = 50
    assert bench.timed_rollouts(50, 50) == 1
    assert bench.timed_rollouts(51, 50) == 2
    assert bench.timed_rollouts(100, 50) == 2
    assert bench.timed_rollouts(1, 10) == 1
    assert bench.timed_rollouts(25, 10) == 3
    with pytest.raises(ValueError):
        bench.timed_rollouts(0, 50)


def test_default_arguments_time_one_rollout_with_warmup_steps():
    a = bench.parse([])
    assert (a.steps, a.warmup, a.gpus, a.workload) == (50, 5, 1, "wan13b_cached")
    assert bench.timed_rollouts(a.steps, 50) == 1
    d = bench.parse(["--steps", "20", "--warmup", "5"])
    assert bench.timed_rollouts(d.steps, 50) == 1
    with pytest.raises(SystemExit):
        bench.parse(["--steps", "0"])
    with pytest.raises(SystemExit):
        bench.parse(["--warmup", "-1"])


def test_budget_refuses_a_leg_that_would_overrun():
    now = [100.0]
    b = bench.Budget(480.0, start=100.0, clock=lambda: now[0])
    assert b.fits(480.0) and not b.fits(480.5)
    now[0] = 400.0                        # 300 s used
    assert b.elapsed() == 300.0 and b.left() == 180.0
    assert b.fits(179.0) and not b.fits(181.0)


def test_leg_estimates_scale_with_the_measured_rollout():
    # 40 s rollout of N = 8, T = 50, B = 1 with 160 of 400 calls computed
    e = bench.leg_estimates(40.0, 160, 8, 50, 1)
    assert e["reference"] == pytest.approx(40.0 / 160 * 400 * 1.05)     # 105 s
    assert e["cfg"] == pytest.approx(40.0 * 2.0 * 1.15)
    assert e["sweep_higher"] == pytest.approx(42.0)
    assert e["sweep_lower"] == pytest.approx(54.0)
    # nothing computed beyond the forced steps cannot make the full rollout cheaper than it is
    e0 = bench.leg_estimates(10.0, 0, 4, 10, 2)
    assert e0["reference"] > 0
    # a worst-case driver run fits the default budget: 2 min of start-up,
    # 20 s of inputs, 5 warmup steps, the timed rollout, the CPU leg and
    # every optional leg at the measured 1.3B rates
    total = 120 + 20 + 4 + 40 + 15 + e["reference"] + e["cfg"] + e["sweep_lower"] + e["sweep_higher"]
    assert total < 600


def test_n_compute_histogram_counts_steps_per_batch_size():
    import numpy as np
    masks = [np.array([1, 1, 1, 1], np.uint8)] * 5 + [np.array([1, 0, 1, 0], np.uint8)] * 2 + \
        [np.zeros(4, np.uint8)] * 3
    assert bench.n_compute_histogram(masks) == {"0": 3, "2": 2, "4": 5}
    assert bench.n_compute_histogram([]) == {}


def test_cpu_model_name_is_a_string():
    s = bench.cpu_model_name()
    assert isinstance(s, str) and s


@pytest.mark.parametrize("T,kw,kc", [(50, 5, 5), (10, 1, 1), (12, 0, 0), (8, 2, 3), (1, 0, 0)])
def test_static_computes_matches_the_oracle_schedule(T, kw, kc):
    """The bench's count of computed steps per stream under the static
    schedule equals what the oracle's rollout computes (velocity -x, any
    latent), for every period."""
    import numpy as np
    from oracle import rollout as orl
    x1 = np.ones((1, 2, 1, 2, 2))
    fns = [lambda x, t: -x]
    grid = [1.0 - k / T for k in range(T + 1)]
    for k in range(1, T + 2):
        res = orl.cached_rollout(x1, fns, grid, tau=0.0, k_warm=kw, k_cool=kc, guidance=1.0,
                                 mode=orl.CACHE_STATIC, static_k=k)
        assert bench.static_computes(T, kw, kc, k) == res.n_compute, (T, kw, kc, k)


def test_matched_static_period():
    # T = 50, windows 5/5: period 4 computes 10 + 10 = 20 of 50 (skip 0.6)
    assert bench.static_computes(50, 5, 5, 4) == 20
    assert bench.matched_static_period(50, 5, 5, 0.6) == 4
    assert bench.matched_static_period(50, 5, 5, 0.0) == 1
    # the closest achievable fraction, shorter period on ties
    k = bench.matched_static_period(50, 5, 5, 0.56)
    fr = lambda k: 1 - bench.static_computes(50, 5, 5, k) / 50
    assert all(abs(fr(k) - 0.56) <= abs(fr(j) - 0.56) for j in range(1, 51))


def test_decision_log_records(tmp_path):
    """The decision log has one JSON line per (step, candidate, branch) with
    the indicator (null where the call was forced) and the decision."""
    import json
    import numpy as np
    from paper_2607_23159_amd.search import decision_records, write_decision_log
    masks = np.array([[1, 1, 1, 1], [0, 1, 0, 0], [1, 1, 1, 1]], np.uint8)
    a = np.array([[np.nan] * 4, [0.05, 0.2, 0.07, 0.09], [np.nan] * 4])
    p = tmp_path / "d.jsonl"
    assert write_decision_log(str(p), masks, a, 2) == 12
    recs = [json.loads(l) for l in p.read_text().splitlines()]
    assert recs == decision_records(masks, a, 2)
    assert recs[0] == {"k": 1, "i": 0, "b": 0, "a": None, "decision": "compute"}
    assert recs[5] == {"k": 2, "i": 0, "b": 1, "a": 0.2, "decision": "compute"}
    assert recs[6] == {"k": 2, "i": 1, "b": 0, "a": 0.07, "decision": "skip"}
    assert sum(r["decision"] == "skip" for r in recs) == 3


def test_cpu_leg_runs_the_whole_oracle_rollout_only_for_small_workloads():
    from paper_2607_23159_amd import synth
    tiny = synth.MODELS["tiny"]
    assert bench.eval_flop(tiny) * 4 * 10 <= bench.ORACLE_FULL_ROLLOUT_FLOP
    for name in ("wan_mid", "wan13b", "wan5b"):
        assert bench.eval_flop(synth.MODELS[name]) * 8 * 50 > bench.ORACLE_FULL_ROLLOUT_FLOP
    # the 1.3B shape's per-call count used in the roofline analysis
    assert bench.eval_flop(synth.MODELS["wan13b"]) == pytest.approx(2.83e14, rel=0.02)


def test_cost_model_reproduces_the_papers_worked_example():
    """The cost model (Eqs. costs and breakeven) applied to the per-rollout
    costs the paper measures gives its printed search costs at N = 4 and 8,
    the cost fractions of best-of-N, gamma and the break-even width
    (tests/golden/cost_model_wan13b.json, with its citation)."""
    import json
    import os
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "cost_model_wan13b.json")))
    for row in g["rows"]:
        c = bench.cost_model(g["C_c_s"], g["C_f_s"], row["N"])
        for key, printed in (("best_of_N_full_s", row["best_of_N_s"]), ("keep_s", row["keep_s"]),
                             ("commit_s", row["commit_s"])):
            assert abs(c[key] - printed) <= 0.005 * printed, (row["N"], key, c[key], printed)
        assert abs(c["keep_s"] / c["best_of_N_full_s"] - row["keep_frac"]) <= 0.0015
        assert abs(c["commit_s"] / c["best_of_N_full_s"] - row["commit_frac"]) <= 0.0015
        assert abs(c["gamma"] - g["gamma"]) <= 0.005
        assert abs(c["break_even_N"] - g["break_even_N"]) <= 0.005
    # commit beats best-of-N exactly beyond the break-even width
    c = bench.cost_model(g["C_c_s"], g["C_f_s"], 2)
    assert c["commit_s"] > c["best_of_N_full_s"]
    c = bench.cost_model(g["C_c_s"], g["C_f_s"], 3)
    assert c["commit_s"] < c["best_of_N_full_s"]
    assert bench.cost_model(5.0, 5.0, 4)["break_even_N"] is None
