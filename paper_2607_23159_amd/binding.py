"""Thin ctypes binding of ``libcachedsearch.so`` (the C ABI in include/cs.h).

Functions keep the C names and only marshal arguments: device buffers are
passed as integers or as objects with ``data_ptr()`` (torch tensors), HIP
streams as integers or objects with ``cuda_stream``.  Every non-OK status
raises :class:`CsError` carrying the library's message.  There is no
fallback: if the library is not built, importing anything that calls it
fails loudly.
"""
from __future__ import annotations

import ctypes as C
import math
import os
from typing import Optional, Sequence, Tuple

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libcachedsearch.so")

CS_OK, CS_E_INVAL, CS_E_NOMEM, CS_E_DEVICE, CS_E_STATE, CS_E_UNSUPPORTED = range(6)
CS_BF16, CS_FP32 = 0, 1
CS_CACHE_OFF, CS_CACHE_ADAPTIVE, CS_CACHE_STATIC, CS_CACHE_PAB = 0, 1, 2, 3
(CS_K_SELF_ATTN, CS_K_CROSS_ATTN, CS_K_GEMM, CS_K_NORM, CS_K_DECIDE, CS_K_UPDATE, CS_K_SCORE,
 CS_K_OTHER) = range(8)
KERNEL_FAMILIES = ["self_attn", "cross_attn", "gemm", "norm", "decide", "update", "score", "other"]


class CsError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"cs status {status}: {msg}")
        self.status = status


class cs_model_desc(C.Structure):
    _fields_ = [(n, C.c_int32) for n in (
        "n_blocks", "hidden", "heads", "head_dim", "ffn", "text_dim", "text_len", "freq_dim",
        "in_ch", "lat_f", "lat_h", "lat_w", "patch_t", "patch_h", "patch_w", "dtype")]


class cs_rollout_desc(C.Structure):
    _fields_ = [("n_cand", C.c_int32), ("n_steps", C.c_int32), ("n_branch", C.c_int32),
                ("k_warm", C.c_int32), ("k_cool", C.c_int32), ("static_k", C.c_int32),
                ("mode", C.c_int32), ("tau", C.c_float), ("guidance", C.c_float),
                ("timesteps", C.POINTER(C.c_float)),
                ("pab_self_range", C.c_int32), ("pab_cross_range", C.c_int32)]


class cs_rollout_stats_t(C.Structure):
    _fields_ = [("steps_done", C.c_int32), ("calls", C.c_int64), ("computed", C.c_int64),
                ("self_reused", C.c_int64), ("cross_reused", C.c_int64), ("n_cand", C.c_int32)]


_lib: Optional[C.CDLL] = None


def lib() -> C.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run paper_2607_23159_amd.build.build()")
    L = C.CDLL(LIB_PATH)
    vp, i32, i64, f32, sz = C.c_void_p, C.c_int32, C.c_int64, C.c_float, C.c_size_t
    pf, pd, pu8, pi32 = C.c_void_p, C.POINTER(C.c_double), C.c_void_p, C.POINTER(C.c_int32)
    sig = {
        "cs_model_weight_count": (i32, [C.POINTER(cs_model_desc), C.POINTER(sz)]),
        "cs_model_init": (i32, [C.POINTER(cs_model_desc), pf, sz, vp, C.POINTER(vp)]),
        "cs_model_free": (None, [vp]),
        "cs_velocity": (i32, [vp, pf, i32, f32, pf, pf]),
        "cs_rollout_init": (i32, [vp, C.POINTER(cs_rollout_desc), pf, pf, pf, C.POINTER(vp)]),
        "cs_rollout_free": (None, [vp]),
        "cs_cache_decide": (i32, [vp, i32, pu8, pu8, pd]),
        "cs_denoise_step": (i32, [vp, i32]),
        "cs_score": (i32, [vp, pf, pd]),
        "cs_score_noalloc": (i32, [pf, pf, i32, i64, pf, vp]),
        "cs_rollout_latents": (i32, [vp, pf]),
        "cs_rollout_stats": (i32, [vp, C.POINTER(cs_rollout_stats_t)]),
        "cs_rollout_enable_preview": (i32, [vp, i32]),
        "cs_preview_score": (i32, [vp, pf, pd]),
        "cs_rollout_retain": (i32, [vp, pi32, i32]),
        "cs_rollout_export": (i32, [vp, vp, C.POINTER(sz)]),
        "cs_rollout_import": (i32, [vp, vp, sz]),
        "cs_rank": (i32, [pd, pd, i32, pi32, pi32, pd, pi32]),
        "cs_profile_enable": (i32, [vp, i32]),
        "cs_profile_reset": (i32, [vp]),
        "cs_profile_read": (i32, [vp, i32, pd, C.POINTER(i64)]),
        "cs_last_error": (C.c_char_p, []),
        "cs_debug_set_alloc_cap": (None, [sz]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    _lib = L
    return L


def _check(status: int) -> None:
    if status != CS_OK:
        raise CsError(status, lib().cs_last_error().decode(errors="replace"))


def _ptr(x, numel: Optional[int] = None, dtype: str = "float32", name: str = "buffer") -> Optional[int]:
    """Device address of ``x``: None, a raw integer address (passed through
    unchecked), or a tensor, which must be a contiguous device tensor of the
    given dtype holding at least ``numel`` elements."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if not getattr(x, "is_cuda", False):
        raise ValueError(f"{name}: a device tensor is required (got {getattr(x, 'device', type(x))})")
    if str(x.dtype).rsplit(".", 1)[-1] != dtype:
        raise ValueError(f"{name}: dtype {x.dtype}, {dtype} required")
    if not x.is_contiguous():
        raise ValueError(f"{name}: tensor must be contiguous")
    if numel is not None and x.numel() < numel:
        raise ValueError(f"{name}: {x.numel()} elements, {numel} required")
    return int(x.data_ptr())


# Latent size D of every live model handle and the model of every live
# rollout handle, so that tensor arguments can be checked against the sizes
# the library will read or write.
_model_D = {}
_rollout_model = {}


def _latent_numel(model: int) -> Optional[int]:
    return _model_D.get(model)


def _stream(s) -> Optional[int]:
    if s is None:
        return None
    if isinstance(s, int):
        return s
    return int(s.cuda_stream)


# ------------------------------------------------------------ descriptors
def model_desc(cfg, dtype: Optional[int] = None) -> cs_model_desc:
    """cs_model_desc from any object with the ModelCfg fields."""
    return cs_model_desc(cfg.n_blocks, cfg.hidden, cfg.heads, cfg.head_dim, cfg.ffn, cfg.text_dim,
                         cfg.text_len, cfg.freq_dim, cfg.in_ch, cfg.lat_f, cfg.lat_h, cfg.lat_w,
                         cfg.patch_t, cfg.patch_h, cfg.patch_w,
                         cfg.dtype if dtype is None else dtype)


class RolloutDesc:
    """cs_rollout_desc plus the timestep array it points to."""

    def __init__(self, roll, timesteps: Sequence[float], **override):
        kw = dict(n_cand=roll.n_cand, n_steps=roll.n_steps, n_branch=roll.n_branch,
                  k_warm=roll.k_warm, k_cool=roll.k_cool, static_k=roll.static_k,
                  mode=roll.mode, tau=roll.tau, guidance=roll.guidance,
                  pab_self=getattr(roll, "pab_self", 2), pab_cross=getattr(roll, "pab_cross", 6))
        kw.update(override)
        self.t = np.ascontiguousarray(np.asarray(timesteps, dtype=np.float32))
        self.c = cs_rollout_desc(kw["n_cand"], kw["n_steps"], kw["n_branch"], kw["k_warm"],
                                 kw["k_cool"], kw["static_k"], kw["mode"],
                                 float(kw["tau"]), float(kw["guidance"]),
                                 self.t.ctypes.data_as(C.POINTER(C.c_float)),
                                 int(kw["pab_self"]), int(kw["pab_cross"]))


# ------------------------------------------------------------------- calls
def cs_model_weight_count(desc: cs_model_desc) -> int:
    n = C.c_size_t(0)
    _check(lib().cs_model_weight_count(C.byref(desc), C.byref(n)))
    return n.value


def cs_model_init(desc: cs_model_desc, weights, n_weights: int, stream=None) -> int:
    out = C.c_void_p()
    _check(lib().cs_model_init(C.byref(desc), _ptr(weights, n_weights, name="weights"), n_weights,
                               _stream(stream), C.byref(out)))
    _model_D[out.value] = desc.in_ch * desc.lat_f * desc.lat_h * desc.lat_w
    return out.value


def cs_model_free(model: int) -> None:
    lib().cs_model_free(model)
    _model_D.pop(model, None)


def cs_velocity(model: int, x, n: int, t: float, ctx, v) -> None:
    D = _latent_numel(model)
    nD = None if D is None else n * D
    _check(lib().cs_velocity(model, _ptr(x, nD, name="x"), n, float(t), _ptr(ctx, name="ctx"),
                             _ptr(v, nD, name="v")))


def cs_rollout_init(model: int, desc: RolloutDesc, x1, ctx_cond, ctx_uncond=None) -> int:
    out = C.c_void_p()
    D = _latent_numel(model)
    _check(lib().cs_rollout_init(model, C.byref(desc.c),
                                 _ptr(x1, None if D is None else desc.c.n_cand * D, name="x1"),
                                 _ptr(ctx_cond, name="ctx_cond"), _ptr(ctx_uncond, name="ctx_uncond"),
                                 C.byref(out)))
    _rollout_model[out.value] = model
    return out.value


def cs_rollout_free(r: int) -> None:
    lib().cs_rollout_free(r)
    _rollout_model.pop(r, None)


def _rollout_D(r: int) -> Optional[int]:
    return _latent_numel(_rollout_model.get(r, 0))


def cs_cache_decide(r: int, step: int, n_streams: int, override_mask: Optional[np.ndarray] = None,
                    want: bool = True) -> Tuple[Optional[np.ndarray], Optional[np.ndarray]]:
    """Returns (mask [n_streams] uint8, a [n_streams] float64) when ``want``."""
    ovr = None
    if override_mask is not None:
        ovr = np.ascontiguousarray(np.asarray(override_mask, dtype=np.uint8).reshape(-1))
        assert ovr.size == n_streams
    mask = np.zeros(n_streams, np.uint8) if want else None
    a = np.zeros(n_streams, np.float64) if want else None
    _check(lib().cs_cache_decide(
        r, step, None if ovr is None else ovr.ctypes.data, None if mask is None else mask.ctypes.data,
        None if a is None else a.ctypes.data_as(C.POINTER(C.c_double))))
    return mask, a


def cs_denoise_step(r: int, step: int) -> None:
    _check(lib().cs_denoise_step(r, step))


def _current_n_cand(r: int, n_cand: int) -> None:
    cur = cs_rollout_stats(r).n_cand
    if n_cand != cur:
        raise ValueError(f"n_cand {n_cand} does not match the rollout's current {cur} candidates")


def cs_score(r: int, w, n_cand: int) -> np.ndarray:
    _current_n_cand(r, n_cand)
    out = np.zeros(n_cand, np.float64)
    _check(lib().cs_score(r, _ptr(w, _rollout_D(r), name="w"), out.ctypes.data_as(C.POINTER(C.c_double))))
    return out


def cs_score_noalloc(x, w, n: int, D: int, scores, stream=None) -> None:
    """Enqueue the scores of n latents x [n][D] into the device float64
    tensor ``scores`` [n]; allocates nothing and does not synchronise."""
    _check(lib().cs_score_noalloc(_ptr(x, n * D, name="x"), _ptr(w, D, name="w"), int(n), int(D),
                                  _ptr(scores, n, dtype="float64", name="scores"), _stream(stream)))


def cs_rollout_latents(r: int, dst) -> None:
    D = _rollout_D(r)
    n = cs_rollout_stats(r).n_cand
    _check(lib().cs_rollout_latents(r, _ptr(dst, None if D is None else n * D, name="dst")))


def cs_rollout_enable_preview(r: int, on: bool = True) -> None:
    _check(lib().cs_rollout_enable_preview(r, 1 if on else 0))


def cs_preview_score(r: int, w, n_cand: int) -> np.ndarray:
    _current_n_cand(r, n_cand)
    out = np.zeros(n_cand, np.float64)
    _check(lib().cs_preview_score(r, _ptr(w, _rollout_D(r), name="w"),
                                  out.ctypes.data_as(C.POINTER(C.c_double))))
    return out


def cs_rollout_retain(r: int, keep: Sequence[int]) -> None:
    k = np.ascontiguousarray(np.asarray(keep, dtype=np.int32))
    _check(lib().cs_rollout_retain(r, k.ctypes.data_as(C.POINTER(C.c_int32)), int(k.size)))


def cs_rollout_stats(r: int) -> cs_rollout_stats_t:
    s = cs_rollout_stats_t()
    _check(lib().cs_rollout_stats(r, C.byref(s)))
    return s


def cs_rollout_export(r: int) -> bytes:
    n = C.c_size_t(0)
    _check(lib().cs_rollout_export(r, None, C.byref(n)))
    buf = C.create_string_buffer(n.value)
    _check(lib().cs_rollout_export(r, buf, C.byref(n)))
    return buf.raw[:n.value]


def cs_rollout_import(r: int, data: bytes) -> None:
    buf = C.create_string_buffer(data, len(data))
    _check(lib().cs_rollout_import(r, buf, len(data)))


def cs_rank(s_cached: Sequence[float], s_full: Optional[Sequence[float]]):
    """(order_cached, order_full, rho, top1_agree); with ``s_full`` None only
    the order of ``s_cached`` is computed (the rest is None)."""
    a = np.ascontiguousarray(np.asarray(s_cached, np.float64))
    n = a.size
    oc = np.zeros(n, np.int32)
    pd = C.POINTER(C.c_double)
    pi = C.POINTER(C.c_int32)
    if s_full is None:
        _check(lib().cs_rank(a.ctypes.data_as(pd), None, n, oc.ctypes.data_as(pi), None, None, None))
        return oc.tolist(), None, None, None
    b = np.ascontiguousarray(np.asarray(s_full, np.float64))
    if b.size != n:
        raise ValueError(f"score vectors of different lengths {n} and {b.size}")
    of = np.zeros(n, np.int32)
    rho = C.c_double(0.0)
    top1 = C.c_int32(0)
    _check(lib().cs_rank(a.ctypes.data_as(pd), b.ctypes.data_as(pd), n, oc.ctypes.data_as(pi),
                         of.ctypes.data_as(pi), C.byref(rho), C.byref(top1)))
    return oc.tolist(), of.tolist(), rho.value, top1.value


def cs_profile_enable(model: int, on: bool) -> None:
    _check(lib().cs_profile_enable(model, 1 if on else 0))


def cs_profile_reset(model: int) -> None:
    _check(lib().cs_profile_reset(model))


def cs_profile_read(model: int, family: int) -> Tuple[float, int]:
    ms = C.c_double(0.0)
    n = C.c_int64(0)
    _check(lib().cs_profile_read(model, family, C.byref(ms), C.byref(n)))
    return ms.value, n.value


def cs_last_error() -> str:
    return lib().cs_last_error().decode(errors="replace")
