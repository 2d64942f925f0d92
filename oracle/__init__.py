"""Oracle for exact softmax attention -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product library
(``paper_2609_29219_amd``) never imports it, and this package imports nothing
from the product.

The arithmetic lives in ``oracle_attn.c`` (plain fp64 C, OpenMP over output
rows).  This module only builds that file with gcc and marshals numpy arrays
into it.  Inputs are bf16 bit patterns as ``numpy.uint16`` arrays (or CPU
bfloat16 tensors), contiguous ``[B][H][S][d]``; outputs are fp64.

What each function follows in the paper:
  * ``attn`` / ``attn_probs`` / ``attn_rows`` -- the Flash Attention workload of
    the Evaluation section (matrix multiplication, softmax, value
    aggregation), written as the textbook definition.
  * ``attn_gqa`` -- the same definition with grouped-query heads and the
    row log-sum-exp (variants beyond the paper's evaluation).
  * ``decode_split`` -- the Flash Decode decomposition in the HEG paragraph of
    the latency-modelling section (local softmax per chunk, gather partials,
    global softmax, final output).
  * ``gemm`` -- the GEMM workload of the Evaluation section, C = A B, as its
    plain definition.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle_attn.c")
_LIB_PATH = os.path.join(_HERE, "liboracle_attn.so")
_default = None


def build(force: bool = False, src: str = _SRC, out: str = _LIB_PATH) -> str:
    """Compile an oracle source with gcc (-O2 -fopenmp, no fast-math)."""
    if force or not os.path.exists(out) or os.path.getmtime(out) < os.path.getmtime(src):
        tmp = out + ".tmp"
        cmd = ["gcc", "-O2", "-fno-fast-math", "-ffp-contract=off", "-fopenmp",
               "-fPIC", "-shared", "-std=c11", src, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, out)
    return out


def _bits(a) -> np.ndarray:
    """Accept a numpy uint16 array or a CPU bfloat16 tensor; return uint16."""
    if not isinstance(a, np.ndarray):
        import torch
        a = a.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)
    if a.dtype != np.uint16:
        raise TypeError("oracle inputs are bf16 bit patterns (uint16)")
    return np.ascontiguousarray(a)


def _p(a, t):
    return a.ctypes.data_as(ctypes.POINTER(t))


def _check(rc: int, what: str):
    if rc != 0:
        raise ValueError(f"oracle {what} rejected its arguments (code {rc})")


def _sizes(q, k, v, nq, nkv):
    if q.size != nq or k.size != nkv or v.size != nkv:
        raise ValueError("oracle input sizes do not match the given dimensions")


class Oracle:
    """ctypes handle on one compiled copy of oracle_attn.c."""

    def __init__(self, lib_path: str):
        lib = ctypes.CDLL(lib_path)
        u16p = ctypes.POINTER(ctypes.c_uint16)
        f64p = ctypes.POINTER(ctypes.c_double)
        i64p = ctypes.POINTER(ctypes.c_int64)
        ci, cf = ctypes.c_int, ctypes.c_float
        lib.oracle_attn.argtypes = [u16p, u16p, u16p, f64p, ci, ci, ci, ci, ci, cf, ci]
        lib.oracle_attn_probs.argtypes = [u16p, u16p, u16p, f64p, f64p, ci, ci, ci, ci, ci,
                                          cf, ci]
        lib.oracle_attn_rows.argtypes = [u16p, u16p, u16p, f64p, i64p, ctypes.c_int64,
                                         ci, ci, ci, ci, ci, cf, ci]
        lib.oracle_decode_split.argtypes = [u16p, u16p, u16p, f64p, ci, ci, ci, ci, cf, ci,
                                            f64p, f64p, f64p]
        lib.oracle_attn_gqa.argtypes = [u16p, u16p, u16p, f64p, f64p, ci, ci, ci, ci, ci, ci,
                                        cf, ci]
        lib.oracle_gemm.argtypes = [u16p, u16p, f64p, f64p, ci, ci, ci, ci, i64p, ctypes.c_int64]
        lib.oracle_num_threads.argtypes = []
        for fn in (lib.oracle_attn, lib.oracle_attn_probs, lib.oracle_attn_rows,
                   lib.oracle_decode_split, lib.oracle_num_threads, lib.oracle_attn_gqa,
                   lib.oracle_gemm):
            fn.restype = ctypes.c_int
        self.lib = lib
        self.path = lib_path

    def num_threads(self) -> int:
        return self.lib.oracle_num_threads()

    def attn(self, q, k, v, B, H, Sq, Skv, d, scale, causal) -> np.ndarray:
        """O = softmax(scale * Q K^T [causal]) V in fp64, shape [B,H,Sq,d]."""
        q, k, v = _bits(q), _bits(k), _bits(v)
        _sizes(q, k, v, B * H * Sq * d, B * H * Skv * d)
        o = np.empty((B, H, Sq, d), dtype=np.float64)
        rc = self.lib.oracle_attn(_p(q, ctypes.c_uint16), _p(k, ctypes.c_uint16),
                                  _p(v, ctypes.c_uint16), _p(o, ctypes.c_double),
                                  B, H, Sq, Skv, d, float(scale), int(bool(causal)))
        _check(rc, "attn")
        return o

    def attn_gqa(self, q, k, v, B, Hq, Hkv, Sq, Skv, d, scale, causal):
        """(O, lse): grouped-query heads (query head h reads key/value head
        h // (Hq // Hkv)) and the natural-log log-sum-exp of every row's
        scores; shapes [B,Hq,Sq,d] and [B,Hq,Sq]."""
        q, k, v = _bits(q), _bits(k), _bits(v)
        _sizes(q, k, v, B * Hq * Sq * d, B * Hkv * Skv * d)
        o = np.empty((B, Hq, Sq, d), dtype=np.float64)
        lse = np.empty((B, Hq, Sq), dtype=np.float64)
        rc = self.lib.oracle_attn_gqa(_p(q, ctypes.c_uint16), _p(k, ctypes.c_uint16),
                                      _p(v, ctypes.c_uint16), _p(o, ctypes.c_double),
                                      _p(lse, ctypes.c_double), B, Hq, Hkv, Sq, Skv, d,
                                      float(scale), int(bool(causal)))
        _check(rc, "attn_gqa")
        return o, lse

    def attn_probs(self, q, k, v, B, H, Sq, Skv, d, scale, causal):
        """(O, P) with P = the softmax weights, shape [B,H,Sq,Skv]."""
        q, k, v = _bits(q), _bits(k), _bits(v)
        _sizes(q, k, v, B * H * Sq * d, B * H * Skv * d)
        o = np.empty((B, H, Sq, d), dtype=np.float64)
        p = np.empty((B, H, Sq, Skv), dtype=np.float64)
        rc = self.lib.oracle_attn_probs(_p(q, ctypes.c_uint16), _p(k, ctypes.c_uint16),
                                        _p(v, ctypes.c_uint16), _p(o, ctypes.c_double),
                                        _p(p, ctypes.c_double), B, H, Sq, Skv, d,
                                        float(scale), int(bool(causal)))
        _check(rc, "attn_probs")
        return o, p

    def attn_rows(self, q, k, v, rows, B, H, Sq, Skv, d, scale, causal) -> np.ndarray:
        """Output rows for flat row indices ``rows`` into [B*H*Sq]; [n, d]."""
        q, k, v = _bits(q), _bits(k), _bits(v)
        _sizes(q, k, v, B * H * Sq * d, B * H * Skv * d)
        rows = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
        o = np.empty((rows.size, d), dtype=np.float64)
        rc = self.lib.oracle_attn_rows(_p(q, ctypes.c_uint16), _p(k, ctypes.c_uint16),
                                       _p(v, ctypes.c_uint16), _p(o, ctypes.c_double),
                                       _p(rows, ctypes.c_int64), rows.size, B, H, Sq, Skv,
                                       d, float(scale), int(bool(causal)))
        _check(rc, "attn_rows")
        return o

    def decode_split(self, q, k, v, B, H, Skv, d, scale, n_splits, return_partials=False):
        """Flash-Decode by split partials and a global-softmax combine; [B,H,d].

        With ``return_partials`` also returns (m, l, u): per-split running max,
        sum of exponentials and unnormalised value sums (NaN past the
        effective split count).
        """
        q, k, v = _bits(q), _bits(k), _bits(v)
        _sizes(q, k, v, B * H * d, B * H * Skv * d)
        o = np.empty((B, H, d), dtype=np.float64)
        n = int(n_splits)
        null = ctypes.POINTER(ctypes.c_double)()
        pm = pl = pu = None
        if return_partials:
            pm = np.full((B, H, max(n, 1)), np.nan)
            pl = np.full((B, H, max(n, 1)), np.nan)
            pu = np.full((B, H, max(n, 1), d), np.nan)
        rc = self.lib.oracle_decode_split(
            _p(q, ctypes.c_uint16), _p(k, ctypes.c_uint16), _p(v, ctypes.c_uint16),
            _p(o, ctypes.c_double), B, H, Skv, d, float(scale), n,
            _p(pm, ctypes.c_double) if pm is not None else null,
            _p(pl, ctypes.c_double) if pl is not None else null,
            _p(pu, ctypes.c_double) if pu is not None else null)
        _check(rc, "decode_split")
        if return_partials:
            return o, (pm, pl, pu)
        return o


    def gemm(self, a, b, M, N, K, b_nk=False, rows=None, with_abs=False):
        """C = A B in fp64 ([M,N], or [len(rows),N] for a row subset); a is
        [M,K], b is [K,N] or, with b_nk, [N,K].  With with_abs also returns
        sum_k |a_mk b_kn| (the scale of any summation order's rounding)."""
        a, b = _bits(a), _bits(b)
        if a.size != M * K or b.size != K * N:
            raise ValueError("oracle input sizes do not match the given dimensions")
        null64 = ctypes.POINTER(ctypes.c_int64)()
        nullf = ctypes.POINTER(ctypes.c_double)()
        if rows is not None:
            rows = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
        n_out = M if rows is None else rows.size
        c = np.empty((n_out, N), dtype=np.float64)
        absc = np.empty((n_out, N), dtype=np.float64) if with_abs else None
        rc = self.lib.oracle_gemm(_p(a, ctypes.c_uint16), _p(b, ctypes.c_uint16),
                                  _p(c, ctypes.c_double),
                                  _p(absc, ctypes.c_double) if with_abs else nullf, M, N, K,
                                  int(bool(b_nk)),
                                  _p(rows, ctypes.c_int64) if rows is not None else null64,
                                  0 if rows is None else rows.size)
        _check(rc, "gemm")
        return (c, absc) if with_abs else c


def default() -> Oracle:
    """The oracle built from oracle_attn.c (compiled on first use)."""
    global _default
    if _default is None:
        _default = Oracle(build())
    return _default


def num_threads() -> int:
    return default().num_threads()


def attn(*a, **kw):
    return default().attn(*a, **kw)


def attn_probs(*a, **kw):
    return default().attn_probs(*a, **kw)


def attn_gqa(*a, **kw):
    return default().attn_gqa(*a, **kw)


def attn_rows(*a, **kw):
    return default().attn_rows(*a, **kw)


def decode_split(*a, **kw):
    return default().decode_split(*a, **kw)


def gemm(*a, **kw):
    return default().gemm(*a, **kw)
