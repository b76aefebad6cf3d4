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


def test_cs_rank_order_only_form():
    """With no full-rollout scores the library still orders the candidates
    (keep mode's argmax, pruned search's top-k): decreasing score, ties to
    the lower index, the same order the oracle's ranking gives; n = 1 is
    allowed there; outputs that need the reference must be NULL."""
    r = np.random.default_rng(11)
    for _ in range(100):
        n = int(r.integers(1, 12))
        s = r.integers(0, 4, n).astype(float) if r.random() < 0.5 else r.standard_normal(n)
        oc, of, rho, top1 = B.cs_rank(s, None)
        assert of is None and rho is None and top1 is None
        assert oc == orank.order_desc(list(s))
    import ctypes as C
    lib = B.lib()
    a = (C.c_double * 3)(1.0, 2.0, 3.0)
    o = (C.c_int32 * 3)()
    rho = C.c_double()
    assert lib.cs_rank(a, None, 3, o, None, C.byref(rho), None) == B.CS_E_INVAL
    assert lib.cs_rank(a, None, 0, o, None, None, None) == B.CS_E_INVAL
    assert lib.cs_rank(None, None, 3, o, None, None, None) == B.CS_E_INVAL


def test_binding_checks_tensor_arguments():
    """Tensors handed to the binding must be contiguous float32 device
    tensors of at least the size the library will touch; the checks run
    before any library call (here on the CPU, so every tensor is refused
    for not being on a device)."""
    import torch
    with pytest.raises(ValueError, match="device tensor"):
        B._ptr(torch.zeros(4), name="x")
    class Fake:
        is_cuda = True
        def __init__(self, dtype, contig=True, n=8):
            self.dtype, self._c, self._n = dtype, contig, n
        def is_contiguous(self):
            return self._c
        def numel(self):
            return self._n
        def data_ptr(self):
            return 4096
    assert B._ptr(Fake(torch.float32), 8) == 4096
    with pytest.raises(ValueError, match="dtype"):
        B._ptr(Fake(torch.float16), 8)
    with pytest.raises(ValueError, match="contiguous"):
        B._ptr(Fake(torch.float32, contig=False), 8)
    with pytest.raises(ValueError, match="elements"):
        B._ptr(Fake(torch.float32, n=7), 8)
    assert B._ptr(None) is None and B._ptr(1234) == 1234
