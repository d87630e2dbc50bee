"""CPU oracle for PruneKV -- TEST INFRASTRUCTURE ONLY.

Plain double-precision C (``oracle.c``) behind a thin ctypes layer.  Only the
test suite, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline leg may
import this package; the GPU library never calls it and shares no code with it.

Every function follows a passage of the paper (VisCache, Sec. 3.2 "PruneKV" and
Appendix B, Algorithm 1); see ``oracle.h`` for the per-function citations.
Parity pins for each function live in ``tests/test_oracle_*.py``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading
from concurrent.futures import ThreadPoolExecutor

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_HDR = os.path.join(_HERE, "oracle.h")
_LIB = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None

P_i32 = ctypes.POINTER(ctypes.c_int32)
P_f64 = ctypes.POINTER(ctypes.c_double)


def build(force: bool = False) -> str:
    """Compile liboracle.so: plain C, no vector intrinsics, no FMA contraction."""
    newest = max(os.path.getmtime(_SRC), os.path.getmtime(_HDR))
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < newest:
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fPIC", "-shared", "-std=c11", "-ffp-contract=off",
                               "-fno-fast-math", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def lib():
    global _lib
    with _lock:
        if _lib is None:
            path = _LIB if os.path.exists(_LIB) else build()
            L = ctypes.CDLL(path)
            vp, i32, f64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_double
            L.orc_budget.argtypes = [i32, i32, f64, i32, f64, i32, i32, P_i32, P_i32, P_i32, P_f64, P_f64]
            L.orc_budget.restype = ctypes.c_int
            L.orc_scores_unit.argtypes = [i32, i32, i32, vp, vp, vp]
            L.orc_scores_unit_prefill.argtypes = [i32, i32, i32, i32, vp, vp, vp, vp, vp]
            L.orc_select.argtypes = [i32, vp, i32, i32, vp, vp]
            L.orc_gather.argtypes = [i32, i32, vp, vp, vp]
            L.orc_fuse.argtypes = [i32, i32, i32, vp, vp, vp, f64, f64, vp]
            L.orc_attend.argtypes = [i32, i32, vp, vp, vp, f64, vp]
            L.orc_quant_rows.argtypes = [i32, i32, vp, vp, vp]
            L.orc_dequant_rows.argtypes = [i32, i32, vp, vp, vp]
            L.orc_prune_unit.argtypes = [i32, i32, i32, vp, vp, vp, i32, i32, f64, f64,
                                         vp, vp, vp, vp, vp]
            _lib = L
    return _lib


def _p(a: np.ndarray):
    assert a.flags.c_contiguous
    return a.ctypes.data


SCHEDULES = {"parabolic": 0, "fixed": 1, "arithmetic": 2, "geometric": 3}


def budget(L: int, n: int, rr: float, h: int = 0, m: float = 0.75, schedule: int = 0, drop_all: bool = False):
    """Returns dict(k=int32[L], n_surv, h, b=float64[L], q) or raises ValueError."""
    k = np.zeros(L, dtype=np.int32)
    b = np.zeros(L, dtype=np.float64)
    ns, ho, q = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_double()
    rc = lib().orc_budget(L, n, rr, h, m, int(schedule), int(drop_all), k.ctypes.data_as(P_i32), ctypes.byref(ns),
                          ctypes.byref(ho), b.ctypes.data_as(P_f64), ctypes.byref(q))
    if rc != 0:
        raise ValueError("invalid budget parameters")
    return dict(k=k, n_surv=int(ns.value), h=int(ho.value), b=b, q=float(q.value))


def scores_unit(K: np.ndarray, Q: np.ndarray) -> np.ndarray:
    """K: uint16 bf16 bits [n, d]; Q: float32 [rows, d].  Returns fp64 S[n]."""
    K = np.ascontiguousarray(K, dtype=np.uint16)
    Q = np.ascontiguousarray(Q, dtype=np.float32).reshape(-1, K.shape[1])
    S = np.zeros(K.shape[0], dtype=np.float64)
    lib().orc_scores_unit(K.shape[0], K.shape[1], Q.shape[0], _p(K), _p(Q), _p(S))
    return S


def scores_unit_prefill(K: np.ndarray, Kt: np.ndarray, Q: np.ndarray, with_text: bool = False):
    """Prefill scoring of one unit.  K: uint16 bf16 bits [n, d] (visual keys);
    Kt: uint16 [T, d] (text keys); Q: float32 [G, n + T, d] (every token's
    query, visual tokens first).  Returns fp64 S[n], or (S, St[T]) with
    with_text."""
    K = np.ascontiguousarray(K, dtype=np.uint16)
    d = K.shape[1]
    Kt = np.ascontiguousarray(Kt, dtype=np.uint16).reshape(-1, d)
    n, T = K.shape[0], Kt.shape[0]
    Q = np.ascontiguousarray(Q, dtype=np.float32).reshape(-1, n + T, d)
    S = np.zeros(max(n, 1), dtype=np.float64)
    St = np.zeros(max(T, 1), dtype=np.float64)
    lib().orc_scores_unit_prefill(n, T, d, Q.shape[0], _p(K), _p(Kt) if T else None, _p(Q), _p(S), _p(St))
    return (S[:n], St[:T]) if with_text else S[:n]


def select(score: np.ndarray, k: int, n_surv: int):
    s = np.ascontiguousarray(score, dtype=np.float32)
    kept = np.zeros(max(k, 1), dtype=np.int32)
    drop = np.zeros(max(n_surv - k, 1), dtype=np.int32)
    lib().orc_select(s.shape[0], _p(s), k, n_surv, _p(kept), _p(drop))
    return kept[:k], drop[:n_surv - k]


def gather(K: np.ndarray, kept: np.ndarray) -> np.ndarray:
    K = np.ascontiguousarray(K, dtype=np.uint16)
    kept = np.ascontiguousarray(kept, dtype=np.int32)
    out = np.zeros((max(len(kept), 1), K.shape[1]), dtype=np.uint16)
    lib().orc_gather(K.shape[1], len(kept), _p(kept), _p(K), _p(out))
    return out[:len(kept)]


def fuse(V: np.ndarray, kept: np.ndarray, drop: np.ndarray, tau: float = 1.0,
         mu: float = 0.7) -> np.ndarray:
    V = np.ascontiguousarray(V, dtype=np.uint16)
    kept = np.ascontiguousarray(kept, dtype=np.int32)
    drop = np.ascontiguousarray(drop, dtype=np.int32)
    out = np.zeros((max(len(kept), 1), V.shape[1]), dtype=np.float64)
    lib().orc_fuse(V.shape[1], len(kept), len(drop), _p(V), _p(kept) if len(kept) else None,
                   _p(drop) if len(drop) else None, tau, mu, _p(out))
    return out[:len(kept)]


def attend(q: np.ndarray, K: np.ndarray, V: np.ndarray, scale: float) -> np.ndarray:
    q = np.ascontiguousarray(q, dtype=np.uint16)
    K = np.ascontiguousarray(K, dtype=np.uint16)
    V = np.ascontiguousarray(V, dtype=np.uint16)
    out = np.zeros(q.shape[-1], dtype=np.float64)
    lib().orc_attend(q.shape[-1], K.shape[0], _p(q), _p(K), _p(V), scale, _p(out))
    return out


def quant_rows(x: np.ndarray):
    """4-bit rows: bf16 bits [n][d] -> (codes uint8 [n][d/2], meta fp32 [n][d/32][2] = (scale, lo))."""
    x = np.ascontiguousarray(x, dtype=np.uint16)
    n, d = x.shape
    codes = np.zeros((max(n, 1), d // 2), dtype=np.uint8)
    meta = np.zeros((max(n, 1), d // 32, 2), dtype=np.float32)
    lib().orc_quant_rows(n, d, _p(x), _p(codes), _p(meta))
    return codes[:n], meta[:n]


def dequant_rows(codes: np.ndarray, meta: np.ndarray) -> np.ndarray:
    """Inverse of quant_rows up to the 4-bit grid: bf16 bits [n][d]."""
    codes = np.ascontiguousarray(codes, dtype=np.uint8)
    meta = np.ascontiguousarray(meta, dtype=np.float32)
    n, d = codes.shape[0], codes.shape[1] * 2
    out = np.zeros((max(n, 1), d), dtype=np.uint16)
    lib().orc_dequant_rows(n, d, _p(codes), _p(meta), _p(out))
    return out[:n]


def prune_unit(K: np.ndarray, V: np.ndarray, Q: np.ndarray, k: int, n_surv: int,
               tau: float = 1.0, mu: float = 0.7):
    """One layer/head-specific unit end to end.  Returns dict(kept, drop, K_out, V_out, S32)."""
    K = np.ascontiguousarray(K, dtype=np.uint16)
    V = np.ascontiguousarray(V, dtype=np.uint16)
    Q = np.ascontiguousarray(Q, dtype=np.float32).reshape(-1, K.shape[1])
    n, d = K.shape
    kept = np.zeros(max(k, 1), dtype=np.int32)
    drop = np.zeros(max(n_surv - k, 1), dtype=np.int32)
    K_out = np.zeros((max(k, 1), d), dtype=np.uint16)
    V_out = np.zeros((max(k, 1), d), dtype=np.float64)
    S32 = np.zeros(max(n, 1), dtype=np.float32)
    lib().orc_prune_unit(n, d, Q.shape[0], _p(K), _p(V), _p(Q), k, n_surv, tau, mu,
                         _p(kept), _p(drop), _p(K_out), _p(V_out), _p(S32))
    return dict(kept=kept[:k], drop=drop[:n_surv - k], K_out=K_out[:k], V_out=V_out[:k],
                S32=S32[:n])


def global_scores(S_units) -> np.ndarray:
    """Shared ranking across layers (the paper's ablation on shared vs
    layer-specific ranking): s_v = sum over every layer and kv head of the
    unit scores, summed in fp64 in (layer, head) order, then rounded to fp32."""
    acc = None
    for S in S_units:
        acc = np.array(S, dtype=np.float64) if acc is None else acc + S
    return acc.astype(np.float32)


def run_units(fn, items, threads: int | None = None):
    """Run independent units on a thread pool (ctypes releases the GIL);
    each unit itself is single-threaded."""
    threads = threads or min(16, os.cpu_count() or 1)
    with ThreadPoolExecutor(max_workers=threads) as ex:
        return list(ex.map(fn, items))
