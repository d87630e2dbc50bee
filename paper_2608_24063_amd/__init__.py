"""Python binding of libviscache (PruneKV on MI355X / gfx950).

Thin ctypes layer over the C ABI declared in ``include/viscache.h``: the same
entry-point names, argument marshalling only.  Every step of the computation
runs in the library's HIP kernels; PyTorch only supplies device memory and the
current stream.  If the shared library has not been built, loading fails
loudly -- there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libviscache.so")

VC_OK, VC_ERR_ARG, VC_ERR_SHAPE, VC_ERR_BUDGET, VC_ERR_WORKSPACE, VC_ERR_UNSUPPORTED, VC_ERR_HIP = range(7)
VC_RANK_LAYER_HEAD, VC_RANK_GLOBAL = 0, 1
VC_SCHED_PARABOLIC, VC_SCHED_FIXED, VC_SCHED_ARITHMETIC, VC_SCHED_GEOMETRIC = 0, 1, 2, 3
VC_SCORE_WINDOW, VC_SCORE_PREFILL = 0, 1

P = ctypes.POINTER
c_i32, c_i64, c_f32, c_f64, c_vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_double, ctypes.c_void_p


class vc_params(ctypes.Structure):
    _fields_ = [("retention", c_f64), ("h", c_i32), ("m", c_f64), ("tau", c_f32), ("mu", c_f32),
                ("rank_mode", c_i32), ("v_out_fp32", c_i32), ("schedule", c_i32), ("drop_all", c_i32),
                ("score_queries", c_i32)]


class vc_shape(ctypes.Structure):
    _fields_ = [("B", c_i32), ("L", c_i32), ("Hq", c_i32), ("Hkv", c_i32), ("d", c_i32),
                ("W", c_i32), ("n_vis", P(c_i32))]


class vc_prune_io(ctypes.Structure):
    _fields_ = [("k_in", P(c_vp)), ("v_in", P(c_vp)), ("q_win", P(c_vp)), ("k_out", P(c_vp)),
                ("v_out", P(c_vp)), ("idx_out", P(c_vp)), ("drop_out", P(c_vp)), ("k_text", P(c_vp))]


class vc_decode_shape(ctypes.Structure):
    _fields_ = [("B", c_i32), ("L", c_i32), ("Hq", c_i32), ("Hkv", c_i32), ("d", c_i32)]


class vc_cache(ctypes.Structure):
    _fields_ = [("k_pool", c_vp), ("v_pool", c_vp), ("row_off", c_vp), ("cap", c_vp), ("len", c_vp)]


class vc_qcache(ctypes.Structure):
    _fields_ = [("k_codes", c_vp), ("k_meta", c_vp), ("v_codes", c_vp), ("v_meta", c_vp),
                ("qrow_off", c_vp), ("nq", c_vp)]


class VisCacheError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {strerror(status)} (status {status})")
        self.status = status


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded library.  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: run __graft_entry__.build() first")
        L = ctypes.CDLL(LIB_PATH)
        L.viscache_default_params.argtypes = [P(vc_params), c_f64]
        L.viscache_default_params.restype = None
        L.viscache_budget.argtypes = [P(vc_shape), P(vc_params), P(c_i32), P(c_i32), P(c_i32)]
        L.viscache_out_rows.argtypes = [P(vc_shape), P(vc_params), P(c_i64)]
        L.viscache_prune_workspace_bytes.argtypes = [P(vc_shape), P(vc_params)]
        L.viscache_prune_workspace_bytes.restype = ctypes.c_size_t
        L.viscache_prune_score_offsets.argtypes = [P(vc_shape), P(vc_params), P(ctypes.c_size_t),
                                                   P(ctypes.c_size_t)]
        L.viscache_prune.argtypes = [P(vc_shape), P(vc_params), P(vc_prune_io), c_vp, ctypes.c_size_t, c_vp]
        L.viscache_prune_staged.argtypes = [P(vc_shape), P(vc_params), P(vc_prune_io), c_vp, ctypes.c_size_t,
                                            c_vp, P(c_vp)]
        L.viscache_decode_workspace_bytes.argtypes = [P(vc_decode_shape), c_i64]
        L.viscache_decode_workspace_bytes.restype = ctypes.c_size_t
        L.viscache_append_kv.argtypes = [P(vc_decode_shape), P(vc_cache), c_vp, c_vp, c_vp]
        L.viscache_decode_attn.argtypes = [P(vc_decode_shape), P(vc_cache), c_vp, c_vp, c_f32, c_i64,
                                           c_vp, ctypes.c_size_t, c_vp]
        L.viscache_decode_step_workspace_bytes.argtypes = [P(vc_decode_shape), c_i64]
        L.viscache_decode_step_workspace_bytes.restype = ctypes.c_size_t
        L.viscache_decode_step.argtypes = [P(vc_decode_shape), P(vc_cache), c_vp, c_vp, c_vp, c_vp, c_f32,
                                           c_i64, c_vp, ctypes.c_size_t, c_vp]
        L.viscache_decode_step_q4.argtypes = [P(vc_decode_shape), P(vc_cache), P(vc_qcache), c_vp, c_vp, c_vp,
                                              c_vp, c_f32, c_i64, c_vp, ctypes.c_size_t, c_vp]
        L.viscache_decode_step_noalloc.argtypes = [P(vc_decode_shape), P(vc_cache), c_vp, c_vp, c_vp, c_vp, c_f32,
                                                   c_i64, c_vp]
        L.viscache_decode_plan_bytes.argtypes = [P(vc_decode_shape), c_i64]
        L.viscache_decode_plan_bytes.restype = ctypes.c_size_t
        L.viscache_decode_plan.argtypes = [P(vc_decode_shape), P(c_i32), P(c_i64), P(c_i32), c_i64, c_vp,
                                           ctypes.c_size_t]
        L.viscache_decode_step_planned.argtypes = [P(vc_decode_shape), P(vc_cache), P(vc_qcache), c_vp,
                                                   ctypes.c_size_t, c_vp, c_vp, c_vp, c_vp, c_f32, c_i64, c_vp,
                                                   ctypes.c_size_t, c_vp]
        L.viscache_quantize_rows.argtypes = [c_i32, c_i64, c_vp, c_vp, c_vp, c_vp]
        L.viscache_strerror.argtypes = [c_i32]
        L.viscache_strerror.restype = ctypes.c_char_p
        for name in ("viscache_budget", "viscache_out_rows", "viscache_prune", "viscache_prune_score_offsets",
                     "viscache_prune_staged",
                     "viscache_append_kv", "viscache_decode_attn", "viscache_decode_step",
                     "viscache_decode_step_q4", "viscache_decode_step_noalloc", "viscache_decode_plan",
                     "viscache_decode_step_planned", "viscache_quantize_rows"):
            getattr(L, name).restype = c_i32
        _lib = L
    return _lib


def strerror(status: int) -> str:
    return lib().viscache_strerror(status).decode()


def _check(status: int, what: str) -> None:
    if status != VC_OK:
        raise VisCacheError(status, what)


# ---- parameter / shape construction -----------------------------------------

def make_params(retention: float, h: int = 0, m: float = 0.75, tau: float = 1.0, mu: float = 0.7,
                rank_mode: int = VC_RANK_LAYER_HEAD, v_out_fp32: bool = False,
                schedule: int = VC_SCHED_PARABOLIC, drop_all: bool = False,
                score_queries: int = VC_SCORE_WINDOW) -> vc_params:
    p = vc_params()
    lib().viscache_default_params(ctypes.byref(p), retention)
    p.h, p.m, p.tau, p.mu, p.rank_mode, p.v_out_fp32 = h, m, tau, mu, rank_mode, int(v_out_fp32)
    p.schedule, p.drop_all, p.score_queries = int(schedule), int(drop_all), int(score_queries)
    return p


def make_shape(B: int, L: int, Hq: int, Hkv: int, d: int, W: int, n_vis) -> vc_shape:
    arr = (c_i32 * B)(*[int(x) for x in n_vis])
    s = vc_shape(B, L, Hq, Hkv, d, W, ctypes.cast(arr, P(c_i32)))
    s._keep = arr  # keep the host array alive with the struct
    return s


# ---- the C entry points, same names ------------------------------------------

def viscache_budget(shape: vc_shape, params: vc_params):
    """Returns (k[B*L], n_surv[B*L], h) as Python lists."""
    n = shape.B * shape.L
    k, ns, h = (c_i32 * n)(), (c_i32 * n)(), c_i32()
    _check(lib().viscache_budget(ctypes.byref(shape), ctypes.byref(params), k, ns, ctypes.byref(h)),
           "viscache_budget")
    return list(k), list(ns), h.value


def viscache_out_rows(shape: vc_shape, params: vc_params):
    rows = (c_i64 * (shape.L * (shape.B + 1)))()
    _check(lib().viscache_out_rows(ctypes.byref(shape), ctypes.byref(params), rows), "viscache_out_rows")
    return list(rows)


def viscache_prune_workspace_bytes(shape: vc_shape, params: vc_params) -> int:
    return int(lib().viscache_prune_workspace_bytes(ctypes.byref(shape), ctypes.byref(params)))


def viscache_prune_score_offsets(shape: vc_shape, params: vc_params):
    """(scores_off, shared_off or None): byte offsets of the scores in the workspace."""
    a, b = ctypes.c_size_t(), ctypes.c_size_t()
    _check(lib().viscache_prune_score_offsets(ctypes.byref(shape), ctypes.byref(params), ctypes.byref(a),
                                              ctypes.byref(b)), "viscache_prune_score_offsets")
    return a.value, (None if b.value == ctypes.c_size_t(-1).value else b.value)


def _ptrs(seq):
    arr = (c_vp * len(seq))(*[int(x) if x else None for x in seq])
    return arr


VC_PRUNE_EVENTS = 7


def _io(k_in, v_in, q_win, k_out, v_out, idx_out, drop_out, k_text):
    arrs = [_ptrs(x) for x in (k_in, v_in, q_win, k_out, v_out, idx_out)]
    opt = [_ptrs(x) if x is not None else None for x in (drop_out, k_text)]
    io = vc_prune_io(*[ctypes.cast(a, P(c_vp)) for a in arrs],
                     *[ctypes.cast(a, P(c_vp)) if a is not None else None for a in opt])
    io._keep = (arrs, opt)
    return io


def make_prune_io(k_in, v_in, q_win, k_out, v_out, idx_out, drop_out=None, k_text=None) -> vc_prune_io:
    """A vc_prune_io over sequences of L device addresses (ints, 0 for none),
    keeping its pointer arrays alive; reusable while the buffers stay put."""
    return _io(k_in, v_in, q_win, k_out, v_out, idx_out, drop_out, k_text)


def prune_with_io(shape: vc_shape, params: vc_params, io: vc_prune_io, workspace: int, workspace_bytes: int,
                  stream: int, events=None) -> None:
    """viscache_prune (or viscache_prune_staged with `events`, VC_PRUNE_EVENTS
    raw hipEvent_t handles) on a prebuilt vc_prune_io."""
    if events is None:
        _check(lib().viscache_prune(ctypes.byref(shape), ctypes.byref(params), ctypes.byref(io), workspace,
                                    workspace_bytes, stream), "viscache_prune")
    else:
        ev = (c_vp * VC_PRUNE_EVENTS)(*[int(e) for e in events])
        _check(lib().viscache_prune_staged(ctypes.byref(shape), ctypes.byref(params), ctypes.byref(io), workspace,
                                           workspace_bytes, stream, ev), "viscache_prune_staged")


def viscache_prune(shape: vc_shape, params: vc_params, k_in, v_in, q_win, k_out, v_out, idx_out,
                   workspace: int, workspace_bytes: int, stream: int, drop_out=None, k_text=None) -> None:
    """k_in ... idx_out, drop_out, k_text: sequences of L device addresses (ints, 0 for none)."""
    io = _io(k_in, v_in, q_win, k_out, v_out, idx_out, drop_out, k_text)
    _check(lib().viscache_prune(ctypes.byref(shape), ctypes.byref(params), ctypes.byref(io),
                                workspace, workspace_bytes, stream), "viscache_prune")


def viscache_prune_staged(shape: vc_shape, params: vc_params, k_in, v_in, q_win, k_out, v_out, idx_out,
                          workspace: int, workspace_bytes: int, stream: int, events, drop_out=None,
                          k_text=None) -> None:
    """As viscache_prune; `events` = VC_PRUNE_EVENTS raw hipEvent_t handles (ints)."""
    io = _io(k_in, v_in, q_win, k_out, v_out, idx_out, drop_out, k_text)
    ev = (c_vp * VC_PRUNE_EVENTS)(*[int(e) for e in events])
    _check(lib().viscache_prune_staged(ctypes.byref(shape), ctypes.byref(params), ctypes.byref(io),
                                       workspace, workspace_bytes, stream, ev), "viscache_prune_staged")


def viscache_decode_workspace_bytes(shape: vc_decode_shape, max_rows: int) -> int:
    return int(lib().viscache_decode_workspace_bytes(ctypes.byref(shape), max_rows))


def viscache_append_kv(shape: vc_decode_shape, cache: vc_cache, k_new: int, v_new: int, stream: int) -> None:
    _check(lib().viscache_append_kv(ctypes.byref(shape), ctypes.byref(cache), k_new, v_new, stream),
           "viscache_append_kv")


def viscache_decode_attn(shape: vc_decode_shape, cache: vc_cache, q: int, out: int, scale: float,
                         max_rows: int, workspace: int, workspace_bytes: int, stream: int) -> None:
    _check(lib().viscache_decode_attn(ctypes.byref(shape), ctypes.byref(cache), q, out, scale, max_rows,
                                      workspace, workspace_bytes, stream), "viscache_decode_attn")


def viscache_decode_step_workspace_bytes(shape: vc_decode_shape, max_rows: int) -> int:
    return int(lib().viscache_decode_step_workspace_bytes(ctypes.byref(shape), max_rows))


def viscache_decode_step(shape: vc_decode_shape, cache: vc_cache, k_new: int, v_new: int, q: int, out: int,
                         scale: float, max_rows: int, workspace: int, workspace_bytes: int,
                         stream: int) -> None:
    _check(lib().viscache_decode_step(ctypes.byref(shape), ctypes.byref(cache), k_new, v_new, q, out, scale,
                                      max_rows, workspace, workspace_bytes, stream), "viscache_decode_step")


def viscache_decode_step_q4(shape: vc_decode_shape, cache: vc_cache, qcache: vc_qcache, k_new: int,
                            v_new: int, q: int, out: int, scale: float, max_rows: int, workspace: int,
                            workspace_bytes: int, stream: int) -> None:
    _check(lib().viscache_decode_step_q4(ctypes.byref(shape), ctypes.byref(cache), ctypes.byref(qcache), k_new,
                                         v_new, q, out, scale, max_rows, workspace, workspace_bytes, stream),
           "viscache_decode_step_q4")


VC_DECODE_NOALLOC_BYTES = 16 << 20
VC_DECODE_NOALLOC_UNITS = 65536


def viscache_decode_step_noalloc(shape: vc_decode_shape, cache: vc_cache, k_new: int, v_new: int, q: int, out: int,
                                 scale: float, max_rows: int, stream: int) -> None:
    """viscache_decode_step with the library's own per-device scratch (no
    workspace argument; allocates nothing)."""
    _check(lib().viscache_decode_step_noalloc(ctypes.byref(shape), ctypes.byref(cache), k_new, v_new, q, out, scale,
                                              max_rows, stream), "viscache_decode_step_noalloc")


def viscache_decode_plan_bytes(shape: vc_decode_shape, max_rows: int) -> int:
    return int(lib().viscache_decode_plan_bytes(ctypes.byref(shape), max_rows))


def viscache_decode_plan(shape: vc_decode_shape, cap, row_off, max_rows: int, len_hint=None) -> bytes:
    """The piece table of caches with capacities `cap`, first pool rows
    `row_off` and (optionally) current lengths `len_hint` (host sequences),
    built on the host; returns its bytes."""
    n = len(cap)
    cap_a = (c_i32 * n)(*[int(x) for x in cap])
    off_a = (c_i64 * n)(*[int(x) for x in row_off])
    hint_a = (c_i32 * n)(*[int(x) for x in len_hint]) if len_hint is not None else None
    nbytes = viscache_decode_plan_bytes(shape, max_rows)
    buf = (ctypes.c_int32 * max(nbytes // 4, 1))()
    _check(lib().viscache_decode_plan(ctypes.byref(shape), cap_a, off_a, hint_a, max_rows, ctypes.addressof(buf),
                                      nbytes), "viscache_decode_plan")
    return bytes(buf)[:nbytes]


def viscache_decode_step_planned(shape: vc_decode_shape, cache: vc_cache, qcache, plan: int, plan_bytes: int,
                                 k_new: int, v_new: int, q: int, out: int, scale: float, max_rows: int,
                                 workspace: int, workspace_bytes: int, stream: int) -> None:
    """viscache_decode_step (qcache None) or viscache_decode_step_q4 over a
    device copy of a piece table."""
    qc = ctypes.byref(qcache) if qcache is not None else None
    _check(lib().viscache_decode_step_planned(ctypes.byref(shape), ctypes.byref(cache), qc, plan, plan_bytes, k_new,
                                              v_new, q, out, scale, max_rows, workspace, workspace_bytes, stream),
           "viscache_decode_step_planned")


def viscache_quantize_rows(d: int, rows: int, src: int, codes: int, meta: int, stream: int) -> None:
    _check(lib().viscache_quantize_rows(d, rows, src, codes, meta, stream), "viscache_quantize_rows")


def viscache_strerror(status: int) -> str:
    return strerror(status)


EXPORTED = ("viscache_default_params", "viscache_budget", "viscache_out_rows",
            "viscache_prune_workspace_bytes", "viscache_prune_score_offsets", "viscache_prune",
            "viscache_prune_staged", "viscache_decode_workspace_bytes",
            "viscache_append_kv", "viscache_decode_attn", "viscache_decode_step_workspace_bytes",
            "viscache_decode_step", "viscache_decode_step_q4", "viscache_decode_step_noalloc",
            "viscache_decode_plan_bytes", "viscache_decode_plan", "viscache_decode_step_planned",
            "viscache_quantize_rows", "viscache_strerror")
