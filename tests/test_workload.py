"""Input generator and accounting (CPU only)."""
import json
import os

import numpy as np
import pytest
import torch

from paper_2608_20961_amd import accounting as acc
from paper_2608_20961_amd import workload as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _check_tree(par, N, max_depth, caps):
    assert par.shape == (N,) and wl.is_topological(par)
    depth = wl.tree_depths(par)
    assert depth.max() == max_depth
    kids = np.bincount(par[par >= 0], minlength=N)
    assert (par == -1).sum() <= caps[0]
    for t in range(N):
        assert kids[t] <= caps[min(depth[t], len(caps) - 1)]
    # DFS pre-order: every subtree occupies a contiguous index range
    for t in range(N):
        sub = [s for s in range(N) if t in wl.ancestors_and_self(par, s)]
        assert sub == list(range(t, t + len(sub)))


@pytest.mark.parametrize("cfg", [2, 3, 4])
def test_random_trees_respect_recipe(cfg):
    w = wl.WORKLOADS[cfg]
    rng = np.random.default_rng(cfg)
    for _ in range(20):
        _check_tree(wl.random_tree(rng, w.N, w.max_depth, w.caps), w.N, w.max_depth, w.caps)


def test_width_trees_match_paper_tables():
    g = _golden("tree_shapes.json")
    for shape, N in g["table2_shape_to_N"]:
        par = wl.width_tree(shape)
        assert len(par) == N and wl.is_topological(par)
        assert wl.tree_depths(par).max() == len(shape)
    for shape, N, blocks in g["table4_shape_N_blocks"]:
        assert acc.snapshot_blocks(len(wl.width_tree(shape))) == blocks
        assert acc.treewy_blocks(N) == 1
    assert list(wl.width_tree([1, 1, 1])) == list(wl.chain_tree(3))


def test_memory_model_matches_paper():
    g = _golden("memory_model.json")
    for name, m in acc.MODELS.items():
        kv = acc.kv_bytes_per_token(m["n_softmax"], m["n_kv_heads"], m["d_head"])
        assert kv == g["kv_per_token_KiB"][name] * acc.KiB
        assert abs(kv * 32768 / acc.GiB - g["kv_per_seq_32k_GiB"][name]) < 0.005
        st = acc.gdn_state_bytes_per_seq(m["n_gdn"], m["n_v_heads"], m["d_v"], m["d_k"])
        assert st == g["gdn_state_per_seq_MiB"][name] * acc.MiB
        assert acc.snapshot_blocks(3) * st == g["snapshot_k3_per_seq_MiB"][name] * acc.MiB
        assert acc.pseudo_value_ratio(m["d_k"]) == g["pseudo_value_smaller_by"]
    assert acc.snapshot_blocks(3) == g["snapshot_k3_times_committed"]


@pytest.mark.parametrize("cfg", [0, 1, 2])
def test_inputs_reproducible_and_shaped(cfg):
    w = wl.WORKLOADS[cfg]
    small = wl.scaled(w, B=min(w.B, 4), H=min(w.H, 3))
    a = wl.make_inputs(small, seed=3, cfg_key=cfg)
    b = wl.make_inputs(small, seed=3, cfg_key=cfg)
    c = wl.make_inputs(small, seed=4, cfg_key=cfg)
    for key in a:
        assert np.array_equal(a[key], b[key])
    assert not np.array_equal(a["q"], c["q"])
    B, H, N, d = small.B, small.H, small.N, small.d_k
    assert a["q"].shape == (B, H, N, d) and a["v"].shape == (B, H, N, d)
    assert a["alpha"].shape == (B, H, N) and a["parent"].shape == (B, N)
    lo, hi = w.alpha_range
    assert a["alpha"].min() >= lo and a["alpha"].max() <= hi
    assert a["beta"].min() >= 0.05 and a["beta"].max() <= 0.95
    norms = np.linalg.norm(a["k"].astype(np.float64), axis=-1)
    assert np.allclose(norms, 1.0, atol=1e-2 if w.in_dtype == "bf16" else 1e-6)
    if w.in_dtype == "bf16":
        assert np.array_equal(wl.round_to_bf16(a["q"]), a["q"])


@pytest.mark.parametrize("cfg", [0, 1, 2, 3, 4])
def test_paths_are_root_to_node(cfg):
    w = wl.WORKLOADS[cfg]
    small = wl.scaled(w, B=min(w.B, 40), H=1)
    x = wl.make_inputs(small, seed=1, cfg_key=cfg)
    for b in range(small.B):
        L = x["path_len"][b]
        path = list(x["path"][b, :L])
        assert np.all(x["path"][b, L:] == -1)
        if L:
            assert path == wl.ancestors_and_self(x["parent"][b], path[-1])
        if w.accept == "prefix3":
            assert path == [0, 1, 2]
        if w.accept == "depth_1_to_8":
            assert 1 <= L <= 8


def test_bf16_rounding_matches_torch():
    x = np.random.default_rng(0).standard_normal(100000).astype(np.float32) * 3
    x[:4] = [1.00390625, 1.01171875, -2.0078125, 0.0]     # exact ties
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(wl.round_to_bf16(x), ref)


def test_warmup_tokens_slice_reproducible():
    w = wl.scaled(wl.WORKLOADS[1], B=2, H=3)
    full = wl.warmup_tokens(w, seed=0, cfg_key=1)
    part = wl.warmup_tokens(w, seed=0, units=slice(2, 5), cfg_key=1)
    assert full["k"].shape == (6, 256, 128)
    assert np.array_equal(full["k"][2:5], part["k"]) and np.array_equal(full["beta"][2:5], part["beta"])


def test_bytes_model_c3():
    w = wl.WORKLOADS[3]
    # S0 537 MB, q/k/v 403 MB, o 134 MB, U 268 MB, alpha/beta 4 MB for 8192 units
    assert abs(acc.verify_bytes(w) / 1e9 - 1.346) < 0.001
    s = acc.speculative_state_bytes(w)
    assert s["treewy_U"] == 256 * acc.MiB and s["snapshot_states"] == 32 * acc.GiB
