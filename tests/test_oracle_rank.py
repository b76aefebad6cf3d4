"""Pins of the oracle's ranking and Spearman correlation.

Checked against brute force over rank assignments, scipy's Spearman, the
no-ties closed form 1 - 6 S / (n (n^2 - 1)), and the N = 8 medians the paper
prints (tests/golden/spearman_lattice.json).
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
import scipy.stats

from oracle import rank

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _brute_avg_ranks(s):
    """Average rank by counting: rank = 1 + #smaller + (#equal - 1)/2."""
    out = []
    for v in s:
        less = sum(1 for u in s if u < v)
        eq = sum(1 for u in s if u == v)
        out.append(1 + less + (eq - 1) / 2)
    return out


@pytest.mark.parametrize("n", [2, 3, 4, 5, 6, 7])
def test_spearman_matches_closed_form_all_permutations(n):
    base = list(range(n))
    for perm in itertools.permutations(base):
        s2 = sum((a - b) ** 2 for a, b in zip(base, perm))
        rho = rank.spearman([float(v) for v in base], [float(v) for v in perm])
        assert rho == pytest.approx(1 - 6 * s2 / (n * (n * n - 1)), abs=1e-12)


def test_spearman_with_ties_matches_scipy_and_counting():
    r = np.random.default_rng(4)
    for _ in range(300):
        n = int(r.integers(2, 9))
        a = r.integers(0, 4, n).astype(float)
        b = r.integers(0, 4, n).astype(float)
        assert rank.average_ranks(list(a)) == _brute_avg_ranks(list(a))
        got = rank.spearman(list(a), list(b))
        if len(set(a)) < 2 or len(set(b)) < 2:
            assert math.isnan(got)
        else:
            assert got == pytest.approx(scipy.stats.spearmanr(a, b).statistic, abs=1e-12)


def test_paper_medians_lie_on_the_n8_lattice():
    g = json.load(open(os.path.join(GOLD, "spearman_lattice.json")))
    n = g["n"]
    base = list(range(n))

    def rho_with_sum(s2):
        for perm in itertools.permutations(base):
            if sum((a - b) ** 2 for a, b in zip(base, perm)) == s2:
                return rank.spearman([float(v) for v in base], [float(v) for v in perm])
        raise AssertionError(s2)

    for p in g["points"]:
        assert round(rho_with_sum(p["sum_d2"]), 3) == pytest.approx(p["printed"], abs=1e-9)
    for p in g["midpoints"]:
        mid = (rho_with_sum(p["sum_d2"][0]) + rho_with_sum(p["sum_d2"][1])) / 2
        assert round(mid, 3) == pytest.approx(p["printed"], abs=1e-9)


def test_order_and_top1_and_regret():
    s_full = [0.3, 0.9, 0.1, 0.9]
    s_cached = [0.5, 0.2, 0.8, 0.4]
    oc, of, rho, top1, regret = rank.rank_report(s_cached, s_full)
    assert of == [1, 3, 0, 2]           # tie at 0.9 -> lower index first
    assert oc == [2, 0, 3, 1]
    assert top1 == 0
    assert regret == pytest.approx(0.9 - 0.1)
    assert math.isnan(rank.spearman([1.0], [2.0]))
    assert math.isnan(rank.spearman([1.0, 1.0], [2.0, 3.0]))


# -------------------------------------------- planted mistakes are caught
import inspect


def _planted(fn_name, old, new):
    src = inspect.getsource(getattr(rank, fn_name))
    assert old in src, old
    ns = dict(rank.__dict__)
    exec(compile(src.replace(old, new), "<planted>", "exec"), ns)
    return ns[fn_name]


def _pins_hold():
    try:
        test_spearman_with_ties_matches_scipy_and_counting()
        test_order_and_top1_and_regret()
        for n in (2, 3, 4):
            test_spearman_matches_closed_form_all_permutations(n)
    except AssertionError:
        return False
    return True


@pytest.mark.parametrize("fn_name,old,new", [
    ("average_ranks", "mean_rank = (pos + end) / 2.0 + 1.0", "mean_rank = pos + 1.0"),   # ordinal ties
    ("order_desc", "key=lambda i: (-float(s[i]), i)", "key=lambda i: (float(s[i]), i)"),  # ascending
    ("order_desc", "key=lambda i: (-float(s[i]), i)", "key=lambda i: (-float(s[i]), -i)"),  # tie order
    ("pearson", "return sxy / math.sqrt(sxx * syy)", "return sxy / (sxx * syy)"),          # normaliser
])
def test_planted_rank_mistake_breaks_a_pin(monkeypatch, fn_name, old, new):
    assert _pins_hold()
    monkeypatch.setattr(rank, fn_name, _planted(fn_name, old, new))
    assert not _pins_hold()
