"""Host-side checks of the C ABI: the library loads, exports every symbol
the header declares, validates arguments before touching a device, and its
host ranking agrees with the oracle's (no GPU needed)."""
import math
import os
import re
import subprocess

import numpy as np
import pytest

from oracle import rank as orank
from paper_2607_23159_amd import binding as B
from paper_2607_23159_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "cs.h")


def _declared():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(cs_[a-z_0-9]+)\s*\(", txt)))


def test_library_exports_every_declared_symbol():
    assert os.path.exists(B.LIB_PATH), "library not built"
    out = subprocess.run(["nm", "-D", "--defined-only", B.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r"\sT\s(cs_\w+)", out))
    decl = _declared()
    assert len(decl) >= 18
    missing = [s for s in decl if s not in exported]
    assert not missing, missing
    B.lib()  # loads and binds every signature


@pytest.mark.parametrize("name", ["tiny", "wan_mid", "wan5b_mid", "wan14b_mid", "wan13b", "wan5b", "wan14b"])
def test_weight_count_matches_generator_layout(name):
    m = synth.MODELS[name]
    assert B.cs_model_weight_count(B.model_desc(m)) == synth.weight_count(m)


def test_model_desc_validation():
    m = synth.MODELS["tiny"]
    bad = B.model_desc(m)
    bad.hidden = 100
    with pytest.raises(B.CsError) as e:
        B.cs_model_weight_count(bad)
    assert e.value.status == B.CS_E_INVAL and "heads" in str(e.value)
    bad = B.model_desc(m)
    bad.head_dim, bad.heads = 16, 8
    with pytest.raises(B.CsError) as e:
        B.cs_model_weight_count(bad)
    assert e.value.status == B.CS_E_UNSUPPORTED
    bad = B.model_desc(m)
    bad.lat_w = 15
    with pytest.raises(B.CsError):
        B.cs_model_weight_count(bad)


def test_model_init_rejects_bad_arguments_before_device_work():
    m = synth.MODELS["tiny"]
    d = B.model_desc(m)
    with pytest.raises(B.CsError) as e:
        B.cs_model_init(d, None, synth.weight_count(m))
    assert e.value.status == B.CS_E_INVAL
    with pytest.raises(B.CsError) as e:
        B.cs_model_init(d, 12345, synth.weight_count(m) - 1)
    assert e.value.status == B.CS_E_INVAL and "expected" in str(e.value)


def test_rollout_calls_reject_null_handles():
    lib = B.lib()
    assert lib.cs_denoise_step(None, 1) == B.CS_E_INVAL
    assert lib.cs_cache_decide(None, 1, None, None, None) == B.CS_E_INVAL
    assert lib.cs_score(None, None, None) == B.CS_E_INVAL
    assert lib.cs_rollout_init(None, None, None, None, None, None) == B.CS_E_INVAL
    assert lib.cs_velocity(None, None, 1, 0.5, None, None) == B.CS_E_INVAL
    assert lib.cs_profile_read(None, 0, None, None) == B.CS_E_INVAL
    assert "NULL" in B.cs_last_error()


def test_cs_rank_matches_oracle_and_handles_ties():
    r = np.random.default_rng(9)
    for _ in range(200):
        n = int(r.integers(2, 12))
        sc = r.integers(0, 5, n).astype(float) if r.random() < 0.5 else r.standard_normal(n)
        sf = r.standard_normal(n)
        oc, of, rho, top1 = B.cs_rank(sc, sf)
        ooc, oof, orho, otop1, _ = orank.rank_report(list(sc), list(sf))
        assert oc == ooc and of == oof and top1 == otop1
        if math.isnan(orho):
            assert math.isnan(rho)
        else:
            assert rho == pytest.approx(orho, abs=1e-12)


def test_cs_rank_argument_errors():
    with pytest.raises(B.CsError) as e:
        B.cs_rank([1.0], [2.0])
    assert e.value.status == B.CS_E_INVAL
    with pytest.raises(B.CsError):
        B.cs_rank([1.0, float("nan")], [2.0, 1.0])
    _, _, rho, _ = B.cs_rank([1.0, 1.0, 1.0], [1.0, 2.0, 3.0])
    assert math.isnan(rho)


def test_binding_fails_loudly_without_library(tmp_path):
    import importlib
    import subprocess
    import sys
    code = ("import paper_2607_23159_amd.binding as b; b.LIB_PATH = '/nonexistent/libcachedsearch.so'; "
            "b._lib = None\ntry:\n    b.lib()\nexcept RuntimeError as e:\n    print('raised', e)\n")
    out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, cwd=ROOT)
    assert "raised" in out.stdout and "not built" in out.stdout
