"""ctypes front end of the float64 C oracle (dla_oracle.c).

TEST INFRASTRUCTURE: only tests/, the smoke check and the benchmark's CPU
baseline leg may import this module.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "dla_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None


def build_oracle(force: bool = False, extra_flags: Optional[list] = None,
                 out: Optional[str] = None) -> str:
    """Compile dla_oracle.c with gcc (OpenMP).  extra_flags/out let the tests
    build deliberately broken variants of the oracle."""
    out = out or _LIB
    if force or not os.path.exists(out) or os.path.getmtime(out) < os.path.getmtime(_SRC):
        cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-shared", "-fPIC", _SRC, "-o", out + ".tmp",
               "-lm"] + list(extra_flags or [])
        subprocess.run(cmd, check=True)
        os.replace(out + ".tmp", out)
    return out


def _load(path: Optional[str] = None):
    global _lib
    if path is None and _lib is not None:
        return _lib
    lib = ctypes.CDLL(path or build_oracle())
    P = ctypes.c_void_p
    lib.dla_oracle_forward.restype = ctypes.c_int
    lib.dla_oracle_forward.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int32,
                                       ctypes.c_int32, ctypes.c_int32, P, P, P, P, P, P,
                                       ctypes.c_double, ctypes.c_double, ctypes.c_double, P, P,
                                       ctypes.c_int32, P, P, P, P, P, P, P, P, P, P, P, P, P]
    lib.dla_oracle_threads.restype = ctypes.c_int
    if path is None:
        _lib = lib
    return lib


def oracle_threads() -> int:
    return int(_load().dla_oracle_threads())


@dataclasses.dataclass
class OracleCache:
    """Chronological state cache: true (decayed) states at the last token."""
    m: np.ndarray      # [n_heads] int32
    n: np.ndarray      # [n_heads, C] int64
    ibar: np.ndarray   # [n_heads, C] float64
    S: np.ndarray      # [n_heads, C, dk, dv] float64

    @staticmethod
    def empty(n_heads: int, C: int, dk: int, dv: int) -> "OracleCache":
        return OracleCache(np.zeros(n_heads, np.int32), np.zeros((n_heads, C), np.int64),
                           np.zeros((n_heads, C)), np.zeros((n_heads, C, dk, dv)))

    def copy(self) -> "OracleCache":
        return OracleCache(self.m.copy(), self.n.copy(), self.ibar.copy(), self.S.copy())


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def oracle_forward(k, v, g, C: int, tau: float, *, q=None, lam=None, beta=None, eps: float = 1e-6,
                   eps_rms: float = 1e-6, b_override=None, m_override=None, full: bool = True,
                   want_out: bool = True, want_mag: bool = False, want_u: bool = False,
                   cache: Optional[OracleCache] = None, lib_path: Optional[str] = None):
    """Run the oracle on float64 inputs shaped [n_heads, T, d] (g: [n_heads, T],
    lam: [n_heads, T, C]; beta: [n_heads, T] step sizes of the delta rule, or
    None for the gated form).  Returns a dict with out, b, merge, score, m,
    margin_b, margin_m, mag (with want_mag: the sum over states of |lambda|
    ||S_j||_F ||q||, which bounds the sizes of the readout's terms; with out),
    u (with want_u: [n_heads, T, d_v], the vector of each token's write k_t
    u_t^T) and the final cache.  The cache argument is
    updated in place when given."""
    k = np.ascontiguousarray(k, np.float64)
    v = np.ascontiguousarray(v, np.float64)
    g = np.ascontiguousarray(g, np.float64)
    nh, T, dk = k.shape
    dv = v.shape[2]
    if q is not None:
        q = np.ascontiguousarray(q, np.float64)
    if lam is not None:
        lam = np.ascontiguousarray(lam, np.float64)
        assert lam.shape == (nh, T, C)
    if beta is not None:
        beta = np.ascontiguousarray(beta, np.float64)
        assert beta.shape == (nh, T)
    if cache is None:
        cache = OracleCache.empty(nh, C, dk, dv)
    want_out = want_out and full and q is not None
    res = {
        "out": np.zeros((nh, T, dv)) if want_out else None,
        "b": np.zeros((nh, T), np.int8),
        "merge": np.zeros((nh, T), np.int32),
        "score": np.zeros((nh, T)),
        "m": np.zeros((nh, T), np.int32),
        "margin_b": np.zeros((nh, T)),
        "margin_m": np.zeros((nh, T)),
        "mag": np.zeros((nh, T)) if (want_out and want_mag) else None,
        "u": np.zeros((nh, T, dv)) if want_u else None,
    }
    bo = None if b_override is None else np.ascontiguousarray(b_override, np.int8)
    mo = None if m_override is None else np.ascontiguousarray(m_override, np.int32)
    lib = _load(lib_path)
    rc = lib.dla_oracle_forward(nh, T, C, dk, dv, _p(q), _p(k), _p(v), _p(g), _p(beta), _p(lam),
                                tau, eps,
                                eps_rms, _p(bo), _p(mo), 1 if full else 0, _p(res["out"]),
                                _p(res["b"]), _p(res["merge"]), _p(res["score"]), _p(res["m"]),
                                _p(res["margin_b"]), _p(res["margin_m"]), _p(res["mag"]),
                                _p(res["u"]), _p(cache.m),
                                _p(cache.n), _p(cache.ibar), _p(cache.S))
    if rc != 0:
        raise ValueError(f"oracle error {rc}")
    res["cache"] = cache
    return res
