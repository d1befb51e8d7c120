"""Seeded synthetic inputs shared by the GPU path's tests/bench and the oracle.

The generator itself (SplitMix64 counters, Box-Muller normals, Student-t(3),
exact-count outlier tokens, one bf16 rounding) is defined once in
``synth_core.h``; ``libtpsynth_host.so`` evaluates it on the CPU and
``libtpsynth_dev.so`` on the GPU, bit-identically.  Nothing here computes any
part of the eviction method.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))

TAG_Q, TAG_K, TAG_V, TAG_KG, TAG_VG = 1, 2, 3, 5, 6  # TAG_KG / TAG_VG: keys / values of the guide tokens
DIST_NORMAL, DIST_STUDENT_T3 = 0, 1


class SynSpec(ctypes.Structure):
    _fields_ = [
        ("seed", ctypes.c_uint64),
        ("tag", ctypes.c_int32),
        ("dist", ctypes.c_int32),
        ("out_frac", ctypes.c_double),
        ("out_scale", ctypes.c_double),
    ]


@dataclass(frozen=True)
class Stream:
    """One generated tensor: seed, tag (Q/K/V), distribution and outlier rows."""

    seed: int
    tag: int
    dist: int = DIST_NORMAL
    out_frac: float = 0.0
    out_scale: float = 1.0

    def spec(self) -> SynSpec:
        return SynSpec(self.seed, self.tag, self.dist, self.out_frac, self.out_scale)


_host = None
_dev = None


def _load_host():
    global _host
    if _host is None:
        path = os.path.join(_HERE, "libtpsynth_host.so")
        if not os.path.exists(path):
            raise ImportError(f"{path} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(path)
        i64, u64 = ctypes.c_int64, ctypes.c_uint64
        lib.syn_host_rows.argtypes = [ctypes.c_void_p, ctypes.POINTER(SynSpec), i64, i64, i64, i64, i64, i64, i64]
        lib.syn_host_rows.restype = None
        lib.syn_host_fill.argtypes = [ctypes.c_void_p, ctypes.POINTER(SynSpec), i64, i64, i64, i64, i64, i64, i64]
        lib.syn_host_fill.restype = None
        lib.syn_probe_log.argtypes = [ctypes.c_double]
        lib.syn_probe_log.restype = ctypes.c_double
        lib.syn_probe_cos_turns.argtypes = [ctypes.c_double]
        lib.syn_probe_cos_turns.restype = ctypes.c_double
        lib.syn_probe_normal.argtypes = [u64, u64]
        lib.syn_probe_normal.restype = ctypes.c_double
        lib.syn_probe_to_bf16.argtypes = [ctypes.c_double]
        lib.syn_probe_to_bf16.restype = ctypes.c_uint16
        lib.syn_probe_perm.argtypes = [u64, u64, u64]
        lib.syn_probe_perm.restype = u64
        lib.syn_probe_at.argtypes = [u64, u64]
        lib.syn_probe_at.restype = u64
        _host = lib
    return _host


def _load_dev():
    global _dev
    if _dev is None:
        path = os.path.join(_HERE, "libtpsynth_dev.so")
        if not os.path.exists(path):
            raise ImportError(f"{path} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(path)
        i64 = ctypes.c_int64
        lib.syn_dev_fill.argtypes = [ctypes.c_void_p, ctypes.POINTER(SynSpec), i64, i64, i64, i64, i64, i64, i64,
                                     ctypes.c_void_p]
        lib.syn_dev_fill.restype = ctypes.c_int
        _dev = lib
    return _dev


def host_lib():
    return _load_host()


def rows(stream: Stream, seq: int, layer: int, head: int, n_seq: int, d: int, t0: int = 0, n: int | None = None):
    """bf16 bits [n, d] of tokens t0..t0+n-1 of the (seq, layer, head) row set (uint16)."""
    if n is None:
        n = n_seq - t0
    out = np.empty((n, d), dtype=np.uint16)
    sp = stream.spec()
    _load_host().syn_host_rows(out.ctypes.data, ctypes.byref(sp), seq, layer, head, n_seq, t0, n, d)
    return out


def host_tensor(stream: Stream, L: int, H: int, lens, d: int):
    """bf16 bits of a [L][H][sum(lens)][d] tensor holding the sequences back to back (uint16)."""
    lens = [int(x) for x in lens]
    ntot = sum(lens)
    out = np.empty((L, H, ntot, d), dtype=np.uint16)
    sp = stream.spec()
    off = 0
    lib = _load_host()
    for b, n in enumerate(lens):
        lib.syn_host_fill(out.ctypes.data, ctypes.byref(sp), b, L, H, ntot, off, n, d)
        off += n
    return out


def device_fill(ptr: int, stream: Stream, L: int, H: int, lens, d: int, hip_stream: int = 0):
    """Fill the device [L][H][sum(lens)][d] bf16 tensor at ``ptr`` with the same values as
    ``host_tensor`` would produce."""
    lens = [int(x) for x in lens]
    ntot = sum(lens)
    sp = stream.spec()
    off = 0
    lib = _load_dev()
    for b, n in enumerate(lens):
        rc = lib.syn_dev_fill(ctypes.c_void_p(ptr), ctypes.byref(sp), b, L, H, ntot, off, n, d,
                              ctypes.c_void_p(hip_stream))
        if rc != 0:
            raise RuntimeError(f"syn_dev_fill failed with hipError {rc}")
        off += n


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float64."""
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
