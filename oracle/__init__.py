"""CPU float64 oracle for tree-WY verification of the gated delta rule.

TEST INFRASTRUCTURE ONLY: imported by the test suite, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.  It shares no code
with the HIP library.  The arithmetic lives in ``oracle.c`` (plain C, float64);
this module only compiles it with gcc and marshals numpy arrays.

Functions (inputs are upcast to float64; a unit is one (sequence, head) pair):
  verify(S0, q, k, v, alpha, beta, parent, states=False) -> (o, vt[, states])
  commit(S0, k, v, alpha, beta, parent, path, path_len) -> state of the accepted node
  chain(S, k, v, alpha, beta) -> state after running eq. 1 over the tokens
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(_HERE, "oracle.c")
LIB_PATH = os.path.join(_HERE, "liboracle.so")


def build(src: str = SOURCE, out: str = LIB_PATH) -> str:
    """Compile the oracle with gcc (OpenMP across independent units)."""
    tmp = out + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-Wall", "-Wextra",
           "-o", tmp, src]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


class OracleError(ValueError):
    pass


_ERRORS = {-1: "parent index outside [-1, t-1]", -2: "not a root-to-node path",
           -3: "bad sizes or out of memory"}


def _f64(x) -> np.ndarray:
    return np.ascontiguousarray(x, dtype=np.float64)


def _i32(x) -> np.ndarray:
    return np.ascontiguousarray(x, dtype=np.int32)


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


class Oracle:
    """Bound to one compiled oracle library.

    `lib` may instead be any object with the library's four functions and the
    same arguments (sizes as ints, arrays as ctypes pointers): the test suite
    passes one that forwards each call to a sanitizer build of oracle.c."""

    def __init__(self, lib_path: str = LIB_PATH, lib=None):
        if lib is None:
            lib = ctypes.CDLL(lib_path)
            P, I = ctypes.c_void_p, ctypes.c_int
            lib.oracle_threads.restype = I
            lib.oracle_gdn_tree.argtypes = [I, I, I, I] + [P] * 10
            lib.oracle_gdn_tree.restype = I
            lib.oracle_gdn_chain.argtypes = [I, I, I, I] + [P] * 5
            lib.oracle_gdn_chain.restype = I
            lib.oracle_commit.argtypes = [I, I, I, I, I] + [P] * 9
            lib.oracle_commit.restype = I
        self._lib = lib
        self.path = lib_path

    @staticmethod
    def _check(rc: int) -> None:
        if rc != 0:
            raise OracleError(_ERRORS.get(rc, "oracle error %d" % rc))

    def threads(self) -> int:
        return int(self._lib.oracle_threads())

    def verify(self, S0, q, k, v, alpha, beta, parent, states: bool = False):
        """S0 [U,dv,dk]; q,k [U,N,dk]; v [U,N,dv]; alpha,beta [U,N]; parent [U,N]."""
        S0, q, k, v, alpha, beta = map(_f64, (S0, q, k, v, alpha, beta))
        parent = _i32(parent)
        U, N, dk = q.shape
        dv = v.shape[2]
        if not (S0.shape == (U, dv, dk) and k.shape == q.shape and v.shape == (U, N, dv)
                and alpha.shape == (U, N) and beta.shape == (U, N) and parent.shape == (U, N)):
            raise OracleError("inconsistent shapes")
        o = np.empty((U, N, dv))
        vt = np.empty((U, N, dv))
        st = np.empty((U, N, dv, dk)) if states else None
        self._check(self._lib.oracle_gdn_tree(U, N, dk, dv, _ptr(S0), _ptr(q), _ptr(k), _ptr(v),
                                              _ptr(alpha), _ptr(beta), _ptr(parent), _ptr(o),
                                              _ptr(vt), _ptr(st)))
        return (o, vt, st) if states else (o, vt)

    def chain(self, S, k, v, alpha, beta):
        """Run eq. 1 over T tokens per unit.  S [U,dv,dk]; k [U,T,dk]; v [U,T,dv]."""
        S = _f64(S).copy()
        k, v, alpha, beta = map(_f64, (k, v, alpha, beta))
        U, T, dk = k.shape
        dv = v.shape[2]
        if S.shape != (U, dv, dk):
            raise OracleError("inconsistent shapes")
        self._check(self._lib.oracle_gdn_chain(U, T, dk, dv, _ptr(S), _ptr(k), _ptr(v),
                                               _ptr(alpha), _ptr(beta)))
        return S

    def commit(self, S0, k, v, alpha, beta, parent, path, path_len):
        """State of the accepted node (S0 for an empty path).  path [U,L_max], path_len [U]."""
        S0, k, v, alpha, beta = map(_f64, (S0, k, v, alpha, beta))
        parent, path, path_len = _i32(parent), _i32(path), _i32(path_len)
        U, N, dk = k.shape
        dv = v.shape[2]
        L_max = path.shape[1]
        out = np.empty((U, dv, dk))
        self._check(self._lib.oracle_commit(U, N, dk, dv, L_max, _ptr(S0), _ptr(k), _ptr(v),
                                            _ptr(alpha), _ptr(beta), _ptr(parent), _ptr(path),
                                            _ptr(path_len), _ptr(out)))
        return out


_default: Optional[Oracle] = None


def default() -> Oracle:
    """The oracle built from oracle.c next to this file (compiled on first use if absent)."""
    global _default
    if _default is None:
        if not os.path.exists(LIB_PATH):
            build()
        _default = Oracle(LIB_PATH)
    return _default


def threads() -> int:
    return default().threads()


def verify(*a, **kw):
    return default().verify(*a, **kw)


def chain(*a, **kw):
    return default().chain(*a, **kw)


def commit(*a, **kw):
    return default().commit(*a, **kw)
