"""Python binding of libtreewy.so (ctypes).  Argument marshalling only.

Every computation runs in the HIP kernels behind the C ABI declared in
include/treewy.h; this module checks tensor shapes, dtypes and devices,
allocates outputs with PyTorch when the caller gives none, and passes raw
device pointers and the current HIP stream.  There is no CPU fallback: if the
library has not been built, importing this module raises.

Function names match the C ABI:
  treewy_verify(S0, q, k, v, alpha, beta, parent) -> (o, U)
  treewy_commit(S0, U, k, alpha, path, path_len, parent=None) -> S_new
  treewy_commit_verify(S_old, U_prev, k_prev, alpha_prev, path, path_len,
                       q, k, v, alpha, beta, parent, parent_prev=None) -> (S_new, o, U)
  treewy_snapshot_verify(S0, q, k, v, alpha, beta, parent) -> (o, snapshots)
  treewy_snapshot_commit(S0, snapshots, accepted) -> S_new
  treewy_path_from_node(parent, accepted, L_max) -> (path, path_len)
  treewy_accept_greedy(parent, draft_token, target_token, root_token, L_max) -> (path, path_len, bonus)
  treewy_chain_prefill(S0, q, k, v, alpha, beta) -> (S_T, o)
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libtreewy.so")

if not os.path.exists(LIB_PATH):
    raise ImportError("libtreewy.so is not built; run `python -m paper_2608_20961_amd.build` first")

lib = ctypes.CDLL(LIB_PATH)

TREEWY_OK, TREEWY_ERR_INVALID_ARG, TREEWY_ERR_UNSUPPORTED, TREEWY_ERR_HIP = 0, 1, 2, 3
TREEWY_F32, TREEWY_BF16 = 0, 1
FLAG_BAD_PARENT, FLAG_BAD_PATH = 1, 2

_P, _I = ctypes.c_void_p, ctypes.c_int
lib.treewy_verify.argtypes = [_P] * 7 + [_I] * 7 + [_P] * 4
lib.treewy_verify.restype = _I
lib.treewy_commit.argtypes = [_P] * 6 + [_I, _P] + [_I] * 7 + [_P] * 3
lib.treewy_commit.restype = _I
lib.treewy_commit_verify.argtypes = [_P] * 6 + [_I, _P, _I] + [_P] * 6 + [_I] * 7 + [_P] * 5
lib.treewy_commit_verify.restype = _I
lib.treewy_snapshot_verify.argtypes = [_P] * 7 + [_I] * 6 + [_P] * 4
lib.treewy_snapshot_verify.restype = _I
lib.treewy_snapshot_commit.argtypes = [_P] * 3 + [_I] * 5 + [_P] * 3
lib.treewy_snapshot_commit.restype = _I
lib.treewy_path_from_node.argtypes = [_P, _P, _I, _I, _I, _P, _P, _P, _P]
lib.treewy_path_from_node.restype = _I
lib.treewy_accept_greedy.argtypes = [_P] * 4 + [_I] * 3 + [_P] * 5
lib.treewy_accept_greedy.restype = _I
lib.treewy_chain_prefill.argtypes = [_P] * 6 + [_I] * 7 + [_P] * 4
lib.treewy_chain_prefill.restype = _I
lib.treewy_status_string.argtypes = [_I]
lib.treewy_status_string.restype = ctypes.c_char_p

EXPORTED = ("treewy_verify", "treewy_commit", "treewy_commit_verify", "treewy_snapshot_verify",
            "treewy_snapshot_commit", "treewy_path_from_node", "treewy_accept_greedy", "treewy_chain_prefill",
            "treewy_status_string")


class TreewyError(RuntimeError):
    def __init__(self, status: int, call: str):
        super().__init__("%s: %s (status %d)" % (call, lib.treewy_status_string(status).decode(), status))
        self.status = status


def _check(status: int, call: str) -> None:
    if status != TREEWY_OK:
        raise TreewyError(status, call)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _need(t: torch.Tensor, name: str, dtype, shape) -> None:
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch.Tensor" % name)
    if t.device.type != "cuda":
        raise ValueError("%s must be on a GPU" % name)
    if t.device.index is not None and t.device.index != torch.cuda.current_device():
        raise ValueError("%s is on %s but the current device is cuda:%d (kernels launch on the current device)"
                         % (name, t.device, torch.cuda.current_device()))
    if t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if tuple(t.shape) != tuple(shape):
        raise ValueError("%s must have shape %s, got %s" % (name, tuple(shape), tuple(t.shape)))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)


def _state_dtype(S: torch.Tensor) -> int:
    """float32 state, or bfloat16 state (with bfloat16 inputs; the library checks)."""
    if S.dtype == torch.float32:
        return TREEWY_F32
    if S.dtype == torch.bfloat16:
        return TREEWY_BF16
    raise TypeError("the state must be float32 or bfloat16, got %s" % S.dtype)


def _in_dtype(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return TREEWY_BF16
    if t.dtype == torch.float32:
        return TREEWY_F32
    raise TypeError("q/k/v must be bfloat16 or float32, got %s" % t.dtype)


def treewy_verify(S0, q, k, v, alpha, beta, parent, o=None, U=None, err=None, stream=None
                  ) -> Tuple[torch.Tensor, torch.Tensor]:
    B, H, N, dk = q.shape
    dv = v.shape[-1]
    dt = q.dtype
    _need(S0, "S0", S0.dtype, (B, H, dv, dk))
    _need(q, "q", dt, (B, H, N, dk)); _need(k, "k", dt, (B, H, N, dk)); _need(v, "v", dt, (B, H, N, dv))
    _need(alpha, "alpha", torch.float32, (B, H, N)); _need(beta, "beta", torch.float32, (B, H, N))
    _need(parent, "parent", torch.int32, (B, N))
    if o is None:
        o = torch.empty((B, H, N, dv), dtype=dt, device=q.device)
    if U is None:
        U = torch.empty((B, H, N, dv), dtype=torch.float32, device=q.device)
    _need(o, "o", dt, (B, H, N, dv)); _need(U, "U", torch.float32, (B, H, N, dv))
    if err is not None:
        _need(err, "err", torch.int32, (B,))
    _check(lib.treewy_verify(_ptr(S0), _ptr(q), _ptr(k), _ptr(v), _ptr(alpha), _ptr(beta), _ptr(parent),
                             N, B, H, dk, dv, _in_dtype(q), _state_dtype(S0), _ptr(o), _ptr(U), _ptr(err),
                             _stream(stream)),
           "treewy_verify")
    return o, U


def treewy_commit(S0, U, k, alpha, path, path_len, parent=None, S_new=None, err=None, stream=None
                  ) -> torch.Tensor:
    B, H, N, dk = k.shape
    dv = U.shape[-1]
    L_max = path.shape[1]
    _need(S0, "S0", S0.dtype, (B, H, dv, dk)); _need(U, "U", torch.float32, (B, H, N, dv))
    _need(k, "k", k.dtype, (B, H, N, dk)); _need(alpha, "alpha", torch.float32, (B, H, N))
    _need(path, "path", torch.int32, (B, L_max)); _need(path_len, "path_len", torch.int32, (B,))
    if parent is not None:
        _need(parent, "parent", torch.int32, (B, N))
    if S_new is None:
        S_new = torch.empty_like(S0)
    _need(S_new, "S_new", S0.dtype, (B, H, dv, dk))
    if err is not None:
        _need(err, "err", torch.int32, (B,))
    _check(lib.treewy_commit(_ptr(S0), _ptr(U), _ptr(k), _ptr(alpha), _ptr(path), _ptr(path_len), L_max,
                             _ptr(parent), N, B, H, dk, dv, _in_dtype(k), _state_dtype(S0), _ptr(S_new),
                             _ptr(err), _stream(stream)), "treewy_commit")
    return S_new


def treewy_commit_verify(S_old, U_prev, k_prev, alpha_prev, path, path_len, q, k, v, alpha, beta, parent,
                         parent_prev=None, S_new=None, o=None, U=None, err=None, stream=None
                         ) -> Tuple[torch.Tensor, torch.Tensor, torch.Tensor]:
    B, H, N, dk = q.shape
    dv = v.shape[-1]
    N_prev = k_prev.shape[2]
    L_max = path.shape[1]
    dt = q.dtype
    _need(S_old, "S_old", S_old.dtype, (B, H, dv, dk))
    _need(U_prev, "U_prev", torch.float32, (B, H, N_prev, dv)); _need(k_prev, "k_prev", dt, (B, H, N_prev, dk))
    _need(alpha_prev, "alpha_prev", torch.float32, (B, H, N_prev))
    _need(path, "path", torch.int32, (B, L_max)); _need(path_len, "path_len", torch.int32, (B,))
    if parent_prev is not None:
        _need(parent_prev, "parent_prev", torch.int32, (B, N_prev))
    _need(q, "q", dt, (B, H, N, dk)); _need(k, "k", dt, (B, H, N, dk)); _need(v, "v", dt, (B, H, N, dv))
    _need(alpha, "alpha", torch.float32, (B, H, N)); _need(beta, "beta", torch.float32, (B, H, N))
    _need(parent, "parent", torch.int32, (B, N))
    if S_new is None:
        S_new = torch.empty_like(S_old)
    if o is None:
        o = torch.empty((B, H, N, dv), dtype=dt, device=q.device)
    if U is None:
        U = torch.empty((B, H, N, dv), dtype=torch.float32, device=q.device)
    _need(S_new, "S_new", S_old.dtype, (B, H, dv, dk))
    _need(o, "o", dt, (B, H, N, dv)); _need(U, "U", torch.float32, (B, H, N, dv))
    if err is not None:
        _need(err, "err", torch.int32, (B,))
    _check(lib.treewy_commit_verify(_ptr(S_old), _ptr(U_prev), _ptr(k_prev), _ptr(alpha_prev), _ptr(path),
                                    _ptr(path_len), L_max, _ptr(parent_prev), N_prev, _ptr(q), _ptr(k), _ptr(v),
                                    _ptr(alpha), _ptr(beta), _ptr(parent), N, B, H, dk, dv, _in_dtype(q),
                                    _state_dtype(S_old), _ptr(S_new), _ptr(o), _ptr(U), _ptr(err),
                                    _stream(stream)),
           "treewy_commit_verify")
    return S_new, o, U


def treewy_snapshot_verify(S0, q, k, v, alpha, beta, parent, o=None, snapshots=None, err=None,
                           stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    B, H, N, dk = q.shape
    dv = v.shape[-1]
    dt = q.dtype
    _need(S0, "S0", torch.float32, (B, H, dv, dk))
    _need(q, "q", dt, (B, H, N, dk)); _need(k, "k", dt, (B, H, N, dk)); _need(v, "v", dt, (B, H, N, dv))
    _need(alpha, "alpha", torch.float32, (B, H, N)); _need(beta, "beta", torch.float32, (B, H, N))
    _need(parent, "parent", torch.int32, (B, N))
    if o is None:
        o = torch.empty((B, H, N, dv), dtype=dt, device=q.device)
    if snapshots is None:
        snapshots = torch.empty((B, H, N, dv, dk), dtype=torch.float32, device=q.device)
    _need(o, "o", dt, (B, H, N, dv)); _need(snapshots, "snapshots", torch.float32, (B, H, N, dv, dk))
    if err is not None:
        _need(err, "err", torch.int32, (B,))
    _check(lib.treewy_snapshot_verify(_ptr(S0), _ptr(q), _ptr(k), _ptr(v), _ptr(alpha), _ptr(beta),
                                      _ptr(parent), N, B, H, dk, dv, _in_dtype(q), _ptr(o),
                                      _ptr(snapshots), _ptr(err), _stream(stream)),
           "treewy_snapshot_verify")
    return o, snapshots


def treewy_snapshot_commit(S0, snapshots, accepted, S_new=None, err=None, stream=None) -> torch.Tensor:
    B, H, N, dv, dk = snapshots.shape
    _need(S0, "S0", torch.float32, (B, H, dv, dk))
    _need(snapshots, "snapshots", torch.float32, (B, H, N, dv, dk))
    _need(accepted, "accepted", torch.int32, (B,))
    if S_new is None:
        S_new = torch.empty_like(S0)
    _need(S_new, "S_new", torch.float32, (B, H, dv, dk))
    if err is not None:
        _need(err, "err", torch.int32, (B,))
    _check(lib.treewy_snapshot_commit(_ptr(S0), _ptr(snapshots), _ptr(accepted), N, B, H, dk, dv,
                                      _ptr(S_new), _ptr(err), _stream(stream)), "treewy_snapshot_commit")
    return S_new


def treewy_path_from_node(parent, accepted, L_max, path=None, path_len=None, err=None, stream=None
                          ) -> Tuple[torch.Tensor, torch.Tensor]:
    B, N = parent.shape
    _need(parent, "parent", torch.int32, (B, N)); _need(accepted, "accepted", torch.int32, (B,))
    if path is None:
        path = torch.empty((B, L_max), dtype=torch.int32, device=parent.device)
    if path_len is None:
        path_len = torch.empty((B,), dtype=torch.int32, device=parent.device)
    _need(path, "path", torch.int32, (B, L_max)); _need(path_len, "path_len", torch.int32, (B,))
    if err is not None:
        _need(err, "err", torch.int32, (B,))
    _check(lib.treewy_path_from_node(_ptr(parent), _ptr(accepted), N, B, L_max, _ptr(path), _ptr(path_len),
                                     _ptr(err), _stream(stream)), "treewy_path_from_node")
    return path, path_len


def treewy_accept_greedy(parent, draft_token, target_token, root_token, L_max: int, path=None, path_len=None,
                         bonus=None, err=None, stream=None) -> Tuple[torch.Tensor, torch.Tensor, torch.Tensor]:
    B, N = parent.shape
    _need(parent, "parent", torch.int32, (B, N))
    _need(draft_token, "draft_token", torch.int32, (B, N))
    _need(target_token, "target_token", torch.int32, (B, N))
    _need(root_token, "root_token", torch.int32, (B,))
    dev = parent.device
    if path is None:
        path = torch.empty((B, L_max), dtype=torch.int32, device=dev)
    if path_len is None:
        path_len = torch.empty((B,), dtype=torch.int32, device=dev)
    if bonus is None:
        bonus = torch.empty((B,), dtype=torch.int32, device=dev)
    _need(path, "path", torch.int32, (B, L_max)); _need(path_len, "path_len", torch.int32, (B,))
    _need(bonus, "bonus", torch.int32, (B,))
    if err is not None:
        _need(err, "err", torch.int32, (B,))
    _check(lib.treewy_accept_greedy(_ptr(parent), _ptr(draft_token), _ptr(target_token), _ptr(root_token), N, B,
                                    L_max, _ptr(path), _ptr(path_len), _ptr(bonus), _ptr(err), _stream(stream)),
           "treewy_accept_greedy")
    return path, path_len, bonus


def treewy_chain_prefill(S0, q, k, v, alpha, beta, S_T=None, o=None, err=None, stream=None
                         ) -> Tuple[torch.Tensor, torch.Tensor]:
    """Gated delta rule over a chain of T tokens per unit (chunks of 32 tokens,
    64 with fp32 tokens; one launch): returns the final state and every
    token's output."""
    B, H, T, dk = q.shape
    dv = v.shape[-1]
    dt = q.dtype
    _need(S0, "S0", S0.dtype, (B, H, dv, dk))
    _need(q, "q", dt, (B, H, T, dk)); _need(k, "k", dt, (B, H, T, dk)); _need(v, "v", dt, (B, H, T, dv))
    _need(alpha, "alpha", torch.float32, (B, H, T)); _need(beta, "beta", torch.float32, (B, H, T))
    if S_T is None:
        S_T = torch.empty_like(S0)
    if o is None:
        o = torch.empty((B, H, T, dv), dtype=dt, device=q.device)
    _need(S_T, "S_T", S0.dtype, (B, H, dv, dk)); _need(o, "o", dt, (B, H, T, dv))
    if err is not None:
        _need(err, "err", torch.int32, (B,))
    _check(lib.treewy_chain_prefill(_ptr(S0), _ptr(q), _ptr(k), _ptr(v), _ptr(alpha), _ptr(beta), T, B, H, dk, dv,
                                    _in_dtype(q), _state_dtype(S0), _ptr(S_T), _ptr(o), _ptr(err), _stream(stream)),
           "treewy_chain_prefill")
    return S_T, o
