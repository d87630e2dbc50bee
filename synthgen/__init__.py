"""Seeded synthetic workloads for PruneKV.

This module is shared by the CPU oracle's tests and by the GPU path's tests and
benchmark.  It only generates data (counter-based random numbers and the
frame-centroid / outlier / relevant-frame model described in ``synthgen.c``); it
holds none of the compression method's arithmetic.

The five workload shapes mirror the paper's setting (long videos encoded as
frames of visual tokens in a grouped-query-attention decoder); the paper's own
datasets are replaced by these seeded tensors.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "synthgen.c")
_LIB = os.path.join(_HERE, "libsynthgen.so")
_lock = threading.Lock()
_lib = None


def build(force: bool = False) -> str:
    """Compile libsynthgen.so with gcc (plain C, pthreads)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fPIC", "-shared", "-std=c11", "-ffp-contract=off",
                               _SRC, "-o", tmp, "-lm", "-lpthread"])
        os.replace(tmp, _LIB)
    return _LIB


class _Cfg(ctypes.Structure):
    _fields_ = [("seed", ctypes.c_uint64), ("B", ctypes.c_int32), ("L", ctypes.c_int32),
                ("Hq", ctypes.c_int32), ("Hkv", ctypes.c_int32), ("d", ctypes.c_int32),
                ("W", ctypes.c_int32), ("tokens_per_frame", ctypes.c_int32),
                ("frames", ctypes.c_int32), ("frame_jitter", ctypes.c_int32),
                ("n_relevant", ctypes.c_int32), ("outlier_frac", ctypes.c_double)]


def lib():
    global _lib
    with _lock:
        if _lib is None:
            path = _LIB if os.path.exists(_LIB) else build()
            L = ctypes.CDLL(path)
            P = ctypes.POINTER
            L.sg_n_vis.argtypes = [P(_Cfg), P(ctypes.c_int32)]
            L.sg_outlier_flags.argtypes = [P(_Cfg), ctypes.c_int32, ctypes.c_int32, P(ctypes.c_uint8)]
            L.sg_relevant_frames.argtypes = [P(_Cfg), ctypes.c_int32, P(ctypes.c_int32)]
            L.sg_frames_of.argtypes = [P(_Cfg), ctypes.c_int32]
            L.sg_frames_of.restype = ctypes.c_int32
            L.sg_kv_layer.argtypes = [P(_Cfg), ctypes.c_int, ctypes.c_int32, ctypes.c_void_p, ctypes.c_int]
            L.sg_q_layer.argtypes = [P(_Cfg), ctypes.c_int32, ctypes.c_void_p]
            L.sg_qall_layer.argtypes = [P(_Cfg), ctypes.c_int32, ctypes.c_void_p]
            L.sg_ktext_layer.argtypes = [P(_Cfg), ctypes.c_int32, ctypes.c_void_p]
            L.sg_normal_bf16.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int64, ctypes.c_void_p]
            L.sg_uniform.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int64, ctypes.c_void_p]
            _lib = L
    return _lib


@dataclasses.dataclass(frozen=True)
class Workload:
    """One seeded workload: model shape, video shape, compression target."""
    name: str
    seed: int
    B: int
    L: int
    Hq: int
    Hkv: int
    d: int
    W: int
    tokens_per_frame: int
    frames: int
    retention: float
    frame_jitter: int = 0
    n_relevant: int = 2
    outlier_frac: float = 0.01
    decode_steps: int = 128

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv

    def _c(self) -> _Cfg:
        return _Cfg(self.seed, self.B, self.L, self.Hq, self.Hkv, self.d, self.W,
                    self.tokens_per_frame, self.frames, self.frame_jitter, self.n_relevant,
                    self.outlier_frac)

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)

    # ---- metadata ---------------------------------------------------------
    def n_vis(self) -> np.ndarray:
        out = np.zeros(self.B, dtype=np.int32)
        c = self._c()
        lib().sg_n_vis(ctypes.byref(c), out.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)))
        return out

    def outlier_flags(self, b: int) -> np.ndarray:
        n = int(self.n_vis()[b])
        out = np.zeros(max(n, 1), dtype=np.uint8)
        c = self._c()
        lib().sg_outlier_flags(ctypes.byref(c), b, n, out.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8)))
        return out[:n]

    def relevant_frames(self, b: int) -> np.ndarray:
        c = self._c()
        F = lib().sg_frames_of(ctypes.byref(c), b)
        out = np.zeros(max(1, min(self.n_relevant, F)), dtype=np.int32)
        lib().sg_relevant_frames(ctypes.byref(c), b, out.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)))
        return out[:min(self.n_relevant, F)]

    def seq_offsets(self) -> np.ndarray:
        n = self.n_vis().astype(np.int64)
        return np.concatenate([[0], np.cumsum(n)])

    def kv_rows(self) -> int:
        return int(self.n_vis().astype(np.int64).sum()) * self.Hkv

    # ---- tensors ----------------------------------------------------------
    def kv_layer(self, role: str, layer: int, out: np.ndarray | None = None,
                 threads: int | None = None) -> np.ndarray:
        """bf16 bits (uint16) [sum_b Hkv*n_b, d]; role 'K' or 'V'."""
        rows = self.kv_rows()
        if out is None:
            out = np.empty((rows, self.d), dtype=np.uint16)
        assert out.dtype == np.uint16 and out.shape == (rows, self.d) and out.flags.c_contiguous
        c = self._c()
        nt = threads or min(16, os.cpu_count() or 1)
        lib().sg_kv_layer(ctypes.byref(c), 0 if role == "K" else 1, layer, out.ctypes.data, nt)
        return out

    def q_layer(self, layer: int) -> np.ndarray:
        """fp32 [B, Hq, W, d] window queries (values exactly representable in bf16)."""
        out = np.empty((self.B, self.Hq, self.W, self.d), dtype=np.float32)
        c = self._c()
        lib().sg_q_layer(ctypes.byref(c), layer, out.ctypes.data)
        return out

    def qall_rows(self) -> int:
        """Rows of the all-token queries: sum_b Hq * (n_b + W)."""
        return int((self.n_vis().astype(np.int64) + self.W).sum()) * self.Hq

    def qall_layer(self, layer: int) -> np.ndarray:
        """fp32 [sum_b Hq*(n_b+W), d]: the query of every prefill token (visual
        tokens first, then the W text tokens), packed over sequences: row
        (b, h, i) at qoff_b*Hq + h*(n_b + W) + i, qoff_b = sum_{b'<b} (n_b' + W)."""
        out = np.empty((self.qall_rows(), self.d), dtype=np.float32)
        c = self._c()
        lib().sg_qall_layer(ctypes.byref(c), layer, out.ctypes.data)
        return out

    def ktext_layer(self, layer: int) -> np.ndarray:
        """bf16 bits [B, Hkv, W, d]: keys of the W text tokens."""
        out = np.empty((self.B, self.Hkv, self.W, self.d), dtype=np.uint16)
        c = self._c()
        lib().sg_ktext_layer(ctypes.byref(c), layer, out.ctypes.data)
        return out


def normal_bf16(seed: int, stream: int, shape) -> np.ndarray:
    """N(0,1) values rounded to bf16, as uint16 bits."""
    out = np.empty(shape, dtype=np.uint16)
    lib().sg_normal_bf16(seed, stream, out.size, out.ctypes.data)
    return out


def uniform(seed: int, stream: int, count: int) -> np.ndarray:
    out = np.empty(count, dtype=np.float64)
    lib().sg_uniform(seed, stream, count, out.ctypes.data)
    return out


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to float32 (exact)."""
    return (bits.astype(np.uint32) << 16).view(np.float32)


# The five workloads.  Shapes follow 3B/7B/72B-class video LLM decoders with
# grouped-query attention; visual tokens come as frames of tokens.
TINY = Workload("tiny", 0x5EED0001, B=1, L=4, Hq=8, Hkv=2, d=64, W=32,
                tokens_per_frame=64, frames=8, retention=0.25)
VLLM7B = Workload("vllm7b", 0x5EED0002, B=1, L=28, Hq=28, Hkv=4, d=128, W=64,
                  tokens_per_frame=196, frames=16, retention=0.28)
LONGVIDEO = Workload("longvideo", 0x5EED0003, B=1, L=28, Hq=28, Hkv=4, d=128, W=64,
                     tokens_per_frame=196, frames=64, retention=0.19, n_relevant=4)
VLLM72B = Workload("vllm72b", 0x5EED0004, B=1, L=80, Hq=64, Hkv=8, d=128, W=128,
                   tokens_per_frame=256, frames=32, retention=0.22, outlier_frac=0.02)
BATCHED = Workload("batched", 0x5EED0005, B=8, L=28, Hq=28, Hkv=4, d=128, W=64,
                   tokens_per_frame=144, frames=128, retention=0.19, frame_jitter=32,
                   decode_steps=256)

WORKLOADS = {w.name: w for w in (TINY, VLLM7B, LONGVIDEO, VLLM72B, BATCHED)}
