"""ctypes front end of the fp64 CPU oracle (``oracle.c``).

TEST INFRASTRUCTURE ONLY: the test-suite, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` are the only callers.  The HIP library
never imports this package and this package never imports the HIP library.

Every function takes plain numpy arrays (bf16 tensors are ``uint16`` arrays of
bf16 bit patterns) and returns numpy arrays.
"""
from __future__ import annotations

import ctypes
import math
import os

import numpy as np

from . import build as _build

_LIB = None

_u16p = np.ctypeslib.ndpointer(dtype=np.uint16, flags="C_CONTIGUOUS")
_f32p = np.ctypeslib.ndpointer(dtype=np.float32, flags="C_CONTIGUOUS")
_f64p = np.ctypeslib.ndpointer(dtype=np.float64, flags="C_CONTIGUOUS")
_i32p = np.ctypeslib.ndpointer(dtype=np.int32, flags="C_CONTIGUOUS")
_u8p = np.ctypeslib.ndpointer(dtype=np.uint8, flags="C_CONTIGUOUS")
_c_int, _c_i64, _c_dbl, _c_flt, _c_i32 = (ctypes.c_int, ctypes.c_int64, ctypes.c_double,
                                          ctypes.c_float, ctypes.c_int32)


def lib():
    """Load liboracle.so, compiling it first only if it is not built yet."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        L = ctypes.CDLL(_build.LIB)
        L.orc_threads.restype = _c_int
        L.orc_set_threads.argtypes = [_c_int]
        L.orc_pool.restype = _c_int
        L.orc_pool.argtypes = [_u16p, _c_i64, _c_int, _c_int, _f64p, _f64p]
        L.orc_probe.restype = _c_int
        L.orc_probe.argtypes = [_u16p, _u16p, _c_int, _c_int, _c_int, _c_int, _c_int, _c_int,
                                _c_int, _c_dbl, ctypes.c_void_p, _c_i64, _f64p, _f64p]
        L.orc_budget.restype = _c_int
        L.orc_budget.argtypes = [_f32p, _c_i64, _c_flt, _c_dbl, _c_dbl, _c_i32, _c_i32, _f64p]
        L.orc_select.restype = _c_int
        L.orc_select.argtypes = [_f32p, _f32p, _c_int, _c_int, _c_int, _c_int, _c_int, _c_flt,
                                 _c_dbl, _c_dbl, _c_i32, _c_i32, _c_i32, _u8p, _i32p, _i32p,
                                 _i32p]
        L.orc_select_mode.restype = _c_int
        L.orc_select_mode.argtypes = [_f32p, _f32p, _c_int, _c_int, _c_int, _c_int, _c_int,
                                      _c_int, _c_int, _c_flt, _c_dbl, _c_dbl, _c_i32, _c_i32,
                                      _c_i32, _u8p, _i32p, _i32p, _i32p]
        L.orc_budget_segment.restype = _c_int
        L.orc_budget_segment.argtypes = [_f32p, _c_i64, _c_flt, _c_dbl, _c_dbl, _c_i32, _c_i32,
                                         _f64p]
        L.orc_group_entropy.restype = None
        L.orc_group_entropy.argtypes = [_f32p, _c_i64, _c_int, _f32p]
        L.orc_attention.restype = _c_int
        L.orc_attention.argtypes = [_u16p, _u16p, _u16p, _c_int, _c_int, _c_int, _c_int, _c_int,
                                    _c_int, _c_int, _c_dbl, _c_int, ctypes.c_void_p,
                                    ctypes.c_void_p, _c_i32, _i32p, _c_i64, _f64p]
        _LIB = L
    return _LIB


def threads() -> int:
    """OpenMP threads the oracle runs with."""
    return lib().orc_threads()


def set_threads(n: int) -> None:
    lib().orc_set_threads(int(n))


def _check(rc: int, what: str) -> None:
    if rc != 0:
        raise ValueError(f"oracle {what} failed with status {rc}")


def _u16(a) -> np.ndarray:
    a = np.ascontiguousarray(a)
    if a.dtype != np.uint16:
        raise TypeError("bf16 tensors are passed as uint16 bit patterns")
    return a


def pool(x: np.ndarray, L: int):
    """Algorithm 1 on one head: x [rows, D] bf16 bits -> (max, min) [groups, D] fp64."""
    x = _u16(x)
    rows, D = x.shape
    groups = -(-rows // L)
    mx = np.empty((groups, D), np.float64)
    mn = np.empty((groups, D), np.float64)
    _check(lib().orc_pool(x, rows, D, L, mx, mn), "pool")
    return mx, mn


def probe(q, k, Ls: int, Lb: int, probe_scale: float = 1.0, rows=None):
    """Algorithm 2 + row entropy.

    q [B, Hq, N, D], k [B, Hkv, N, D] as bf16 bits.  ``rows``: optional int
    array [n, 3] of (b, h, s); default all.  Returns (log_scores [n, C_B] with
    NaN where j >= n_vis(s), entropy [n]) in fp64; with rows=None the leading
    dimension is reshaped to [B, Hq, C_S].
    """
    q, k = _u16(q), _u16(k)
    B, Hq, N, D = q.shape
    Hkv = k.shape[1]
    CS, CB = -(-N // Ls), -(-N // Lb)
    if rows is None:
        n, selp = B * Hq * CS, None
    else:
        sel = np.ascontiguousarray(np.asarray(rows, np.int32).reshape(-1, 3))
        n, selp = sel.shape[0], sel.ctypes.data
    Lout = np.full((n, CB), np.nan, np.float64)
    H = np.empty((n,), np.float64)
    _check(lib().orc_probe(q, k, B, Hq, Hkv, N, D, Ls, Lb, float(probe_scale), selp, n, Lout, H),
           "probe")
    if rows is None:
        return Lout.reshape(B, Hq, CS, CB), H.reshape(B, Hq, CS)
    return Lout, H


def budget(e, e_t=1e-5, alpha=0.5, delta_t=0.4, base_budget=2048, mult=3):
    """Algorithm 3 on one head's entropies -> (rigid: bool, B [C_S] tokens fp64)."""
    e = np.ascontiguousarray(np.asarray(e, np.float32))
    B = np.empty((max(1, e.shape[0]),), np.float64)
    rigid = lib().orc_budget(e, e.shape[0], float(e_t), float(alpha), float(delta_t),
                             int(base_budget), int(mult), B)
    return bool(rigid), B[: e.shape[0]]


def budget_segment(e, e_t=1e-5, alpha=0.5, delta_t=0.4, base_budget=2048, mult=3):
    """The per-segment rigid rule on one head's entropies -> (all rigid, B)."""
    e = np.ascontiguousarray(np.asarray(e, np.float32))
    B = np.empty((max(1, e.shape[0]),), np.float64)
    rigid = lib().orc_budget_segment(e, e.shape[0], float(e_t), float(alpha), float(delta_t),
                                     int(base_budget), int(mult), B)
    return bool(rigid), B[: e.shape[0]]


def group_entropy(e_group):
    """[G, C_S] entropies of one GQA group -> [C_S] binary32 group means."""
    e = np.ascontiguousarray(np.asarray(e_group, np.float32))
    out = np.empty((e.shape[1],), np.float32)
    lib().orc_group_entropy(e, e.shape[1], e.shape[0], out)
    return out


# classification modes of select()
CLASSIFY_HEAD, CLASSIFY_GQA_GROUP, CLASSIFY_SEGMENT = 0, 1, 2


def kmax(Ls: int, Lb: int, base_budget: int, mult: int) -> int:
    return (mult * base_budget) // Lb + Ls // Lb


def select(log_scores, entropy, N: int, Ls: int, Lb: int, e_t=1e-5, alpha=0.5, delta_t=0.4,
           base_budget=2048, mult=3, kmax_=None, mode=CLASSIFY_HEAD, n_kv_heads=None):
    """Classification, budgets and top-k selection from binary32 inputs.

    log_scores [B, Hq, C_S, C_B] fp32, entropy [B, Hq, C_S] fp32.  mode: one
    of the CLASSIFY_* constants (n_kv_heads is needed for the GQA-group mode).
    Returns dict(rigid [B,Hq] u8, budget [B,Hq,C_S] i32, idx [B,Hq,C_S,kmax] i32,
    cnt [B,Hq,C_S] i32).
    """
    ls = np.ascontiguousarray(log_scores, dtype=np.float32)
    en = np.ascontiguousarray(entropy, dtype=np.float32)
    B, Hq, CS, CB = ls.shape
    km = kmax(Ls, Lb, base_budget, mult) if kmax_ is None else int(kmax_)
    rigid = np.empty((B, Hq), np.uint8)
    bud = np.empty((B, Hq, CS), np.int32)
    idx = np.empty((B, Hq, CS, km), np.int32)
    cnt = np.empty((B, Hq, CS), np.int32)
    hkv = Hq if n_kv_heads is None else int(n_kv_heads)
    _check(lib().orc_select_mode(ls, en, B, Hq, hkv, int(mode), N, Ls, Lb, float(e_t),
                                 float(alpha), float(delta_t), int(base_budget), int(mult), km,
                                 rigid, bud, idx, cnt), "select")
    return {"rigid": rigid, "budget": bud, "idx": idx, "cnt": cnt}


def attention(q, k, v, rows, scale=None, causal=True, block_idx=None, block_cnt=None,
              Ls: int = 128, Lb: int = 64):
    """Causal GQA attention in fp64 for query rows [n, 3] of (b, h, i).

    With block_idx/block_cnt the key set is the listed blocks of the row's
    segment, restricted to keys <= i.  Returns [n, D] fp64.
    """
    q, k, v = _u16(q), _u16(k), _u16(v)
    B, Hq, N, D = q.shape
    Hkv = k.shape[1]
    sc = 1.0 / math.sqrt(D) if scale is None else float(scale)
    r = np.ascontiguousarray(np.asarray(rows, np.int32).reshape(-1, 3))
    out = np.empty((r.shape[0], D), np.float64)
    if block_idx is not None:
        bi = np.ascontiguousarray(block_idx, dtype=np.int32)
        bc = np.ascontiguousarray(block_cnt, dtype=np.int32)
        km = bi.shape[-1]
        bip, bcp = bi.ctypes.data, bc.ctypes.data
    else:
        bi = bc = None
        km, bip, bcp = 0, None, None
    _check(lib().orc_attention(q, k, v, B, Hq, Hkv, N, D, Ls, Lb, sc, 1 if causal else 0, bip,
                               bcp, km, r, r.shape[0], out), "attention")
    return out
