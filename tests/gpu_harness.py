"""Shared plumbing for the GPU parity tests: seeded inputs -> oracle on the
CPU and the HIP library on the GPU -> per-unit comparison.

S0 is the gated delta rule run from zero over each unit's warm-up tokens; here
the oracle computes it (float64, rounded once to float32), so no input of the
oracle ever comes from the GPU.  At full sizes only a sample of units is
checked; the other units reuse a sampled unit's S0 so the launch still covers
the full [B, H] grid.
"""
from __future__ import annotations

import numpy as np
import torch

import oracle
from paper_2608_20961_amd import workload as wl

DEV = torch.device("cuda:0")
TOL = {"f32": 1e-4, "bf16": 2e-2}


def say(msg: str) -> None:
    print(msg, flush=True)


def rel_err(x: np.ndarray, ref: np.ndarray) -> float:
    """Normwise max relative error of one (sequence, head) slice."""
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if ref.size == 0:
        return 0.0
    return float(np.max(np.abs(x - ref)) / max(float(np.max(np.abs(ref))), 1e-30))


def warm_state(w: wl.Workload, units: np.ndarray, seed: int, cfg_key: int) -> np.ndarray:
    """S0 of the given units, float32 [len(units), d_v, d_k]."""
    out = np.empty((len(units), w.d_v, w.d_k), dtype=np.float32)
    for i, u in enumerate(units):
        tok = wl.warmup_tokens(w, seed=seed, units=slice(int(u), int(u) + 1), cfg_key=cfg_key)
        S = oracle.chain(np.zeros((1, w.d_v, w.d_k)), tok["k"], tok["v"], tok["alpha"], tok["beta"])
        out[i] = S[0].astype(np.float32)
    return out


class Case:
    """One input set on host and device, with oracle references for `check_units`."""

    def __init__(self, w: wl.Workload, seed: int = 0, cfg_key: int = 99, check_units=None,
                 inputs=None, S0=None):
        self.w, self.seed = w, seed
        self.x = inputs if inputs is not None else wl.make_inputs(w, seed=seed, cfg_key=cfg_key)
        U = w.units
        self.check = np.arange(U) if check_units is None else np.asarray(check_units)
        if S0 is None:
            S0_chk = warm_state(w, self.check, seed, cfg_key)
            S0 = S0_chk[np.searchsorted(self.check, np.arange(U)) % len(self.check)]
            S0[self.check] = S0_chk
        self.S0 = np.ascontiguousarray(S0, dtype=np.float32).reshape(U, w.d_v, w.d_k)

    # ---- oracle on the checked units ----------------------------------------
    def unit_view(self, name):
        w = self.w
        a = self.x[name]
        return a.reshape(w.units, *a.shape[2:])[self.check]

    def oracle(self, states=False):
        w, c = self.w, self.check
        par_u = np.repeat(self.x["parent"], w.H, axis=0)[c]
        args = (self.S0[c], self.unit_view("q"), self.unit_view("k"), self.unit_view("v"),
                self.unit_view("alpha"), self.unit_view("beta"), par_u)
        res = oracle.verify(*args, states=states)
        S_acc = oracle.commit(self.S0[c], self.unit_view("k"), self.unit_view("v"), self.unit_view("alpha"),
                              self.unit_view("beta"), par_u, np.repeat(self.x["path"], w.H, axis=0)[c],
                              np.repeat(self.x["path_len"], w.H, axis=0)[c])
        return res + (S_acc,)

    # ---- device tensors -------------------------------------------------------
    def device(self):
        w = self.w
        dt = torch.bfloat16 if w.in_dtype == "bf16" else torch.float32

        def inp(a):
            return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV).to(dt)

        def f32(a):
            return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV)

        def i32(a):
            return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(DEV)

        return dict(S0=f32(self.S0.reshape(w.B, w.H, w.d_v, w.d_k)), q=inp(self.x["q"]), k=inp(self.x["k"]),
                    v=inp(self.x["v"]), alpha=f32(self.x["alpha"]), beta=f32(self.x["beta"]),
                    parent=i32(self.x["parent"]), path=i32(self.x["path"]), path_len=i32(self.x["path_len"]))


def units_of(t: torch.Tensor, w: wl.Workload, check) -> np.ndarray:
    a = t.float().cpu().numpy()
    return a.reshape(w.units, *a.shape[2:])[check]


def assert_close(name: str, got: np.ndarray, ref: np.ndarray, tol: float) -> float:
    worst = 0.0
    for i in range(len(ref)):
        e = rel_err(got[i], ref[i])
        worst = max(worst, e)
        assert e <= tol, "%s: unit %d max rel err %.3e > %.1e" % (name, i, e, tol)
    return worst
