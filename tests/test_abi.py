"""The C-ABI library loads, exports what include/treewy.h declares, and its
host-side checks return the documented status codes (no kernel runs here)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "treewy.h")


@pytest.fixture(scope="module")
def tw():
    from paper_2608_20961_amd import treewy
    return treewy


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(treewy_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    assert names == sorted(["treewy_verify", "treewy_commit", "treewy_commit_verify", "treewy_snapshot_verify",
                            "treewy_snapshot_commit", "treewy_path_from_node", "treewy_accept_greedy",
                            "treewy_chain_prefill", "treewy_status_string"])


def test_library_exports_every_declared_symbol(tw):
    for name in declared_functions():
        assert hasattr(tw.lib, name), name
    assert set(tw.EXPORTED) == set(declared_functions())


def test_status_strings(tw):
    for s in range(4):
        assert tw.lib.treewy_status_string(s)
    assert tw.lib.treewy_status_string(99) == b"unknown status"


A = ctypes.c_void_p(16)   # aligned stand-in pointers: never dereferenced by the host checks
M = ctypes.c_void_p(18)   # misaligned


def _verify(tw, fn="treewy_verify", S0=A, q=A, N=8, B=2, H=2, dk=128, dv=128, dt=1, o=A, U=A, st=0):
    if fn == "treewy_verify":
        return tw.lib.treewy_verify(S0, q, A, A, A, A, A, N, B, H, dk, dv, dt, st, o, U, None, None)
    return getattr(tw.lib, fn)(S0, q, A, A, A, A, A, N, B, H, dk, dv, dt, o, U, None, None)


@pytest.mark.parametrize("fn", ["treewy_verify", "treewy_snapshot_verify"])
def test_verify_host_checks(tw, fn):
    assert _verify(tw, fn, dk=64) == tw.TREEWY_ERR_UNSUPPORTED
    assert _verify(tw, fn, dv=96) == tw.TREEWY_ERR_UNSUPPORTED
    # verify walks trees of up to 256 nodes in chunks; the snapshot baseline stops at 64
    assert _verify(tw, fn, N=257 if fn == "treewy_verify" else 65) == tw.TREEWY_ERR_UNSUPPORTED
    assert _verify(tw, fn, N=-1) == tw.TREEWY_ERR_INVALID_ARG
    assert _verify(tw, fn, B=-3) == tw.TREEWY_ERR_INVALID_ARG
    assert _verify(tw, fn, dt=7) == tw.TREEWY_ERR_INVALID_ARG
    assert _verify(tw, fn, S0=None) == tw.TREEWY_ERR_INVALID_ARG
    assert _verify(tw, fn, U=None) == tw.TREEWY_ERR_INVALID_ARG
    assert _verify(tw, fn, S0=M) == tw.TREEWY_ERR_INVALID_ARG
    if fn == "treewy_verify":
        assert _verify(tw, fn, st=2) == tw.TREEWY_ERR_INVALID_ARG
        assert _verify(tw, fn, dt=0, st=1) == tw.TREEWY_ERR_UNSUPPORTED
    # nothing to do: returns before touching any pointer or the GPU
    assert _verify(tw, fn, N=0, S0=None) == tw.TREEWY_OK
    assert _verify(tw, fn, B=0, S0=None) == tw.TREEWY_OK
    assert _verify(tw, fn, H=0, S0=None) == tw.TREEWY_OK


def test_commit_host_checks(tw):
    f = tw.lib.treewy_commit

    def call(S0=A, path=A, plen=A, L_max=8, N=8, B=2, H=2, dk=128, dt=1, S_new=A, st=0):
        return f(S0, A, A, A, path, plen, L_max, None, N, B, H, dk, 128, dt, st, S_new, None, None)

    assert call(dk=64) == tw.TREEWY_ERR_UNSUPPORTED
    assert call(L_max=257) == tw.TREEWY_ERR_UNSUPPORTED
    assert call(N=257) == tw.TREEWY_ERR_UNSUPPORTED
    assert call(L_max=-1) == tw.TREEWY_ERR_INVALID_ARG
    assert call(plen=None) == tw.TREEWY_ERR_INVALID_ARG
    assert call(path=None) == tw.TREEWY_ERR_INVALID_ARG
    assert call(S_new=M) == tw.TREEWY_ERR_INVALID_ARG
    assert call(dt=2) == tw.TREEWY_ERR_INVALID_ARG
    assert call(st=5) == tw.TREEWY_ERR_INVALID_ARG
    assert call(B=0, S0=None) == tw.TREEWY_OK


def test_commit_verify_host_checks(tw):
    f = tw.lib.treewy_commit_verify

    def call(S_old=A, U_prev=A, k_prev=A, path=A, plen=A, L_max=8, N_prev=8, q=A, N=8, B=2, H=2, dk=128,
             dt=1, S_new=A, o=A, U=A, st=0):
        return f(S_old, U_prev, k_prev, A, path, plen, L_max, None, N_prev, q, A, A, A, A, A, N, B, H, dk, 128,
                 dt, st, S_new, o, U, None, None)

    assert call(dk=64) == tw.TREEWY_ERR_UNSUPPORTED
    assert call(N=65) == tw.TREEWY_ERR_UNSUPPORTED
    assert call(N_prev=65) == tw.TREEWY_ERR_UNSUPPORTED
    assert call(L_max=65) == tw.TREEWY_ERR_UNSUPPORTED
    assert call(N_prev=-1) == tw.TREEWY_ERR_INVALID_ARG
    assert call(L_max=-1) == tw.TREEWY_ERR_INVALID_ARG
    assert call(dt=3) == tw.TREEWY_ERR_INVALID_ARG
    assert call(st=3) == tw.TREEWY_ERR_INVALID_ARG
    assert call(dt=0, st=1) == tw.TREEWY_ERR_UNSUPPORTED     # a bf16 state needs bf16 inputs
    assert call(S_old=None) == tw.TREEWY_ERR_INVALID_ARG
    assert call(plen=None) == tw.TREEWY_ERR_INVALID_ARG
    assert call(path=None) == tw.TREEWY_ERR_INVALID_ARG
    assert call(U_prev=None) == tw.TREEWY_ERR_INVALID_ARG
    assert call(q=None) == tw.TREEWY_ERR_INVALID_ARG
    assert call(o=None) == tw.TREEWY_ERR_INVALID_ARG
    assert call(S_new=M) == tw.TREEWY_ERR_INVALID_ARG
    assert call(k_prev=M) == tw.TREEWY_ERR_INVALID_ARG
    # U over U_prev is allowed only when both rounds have the same N
    assert call(U_prev=A, U=A, N_prev=4) == tw.TREEWY_ERR_INVALID_ARG
    assert call(B=0, S_old=None) == tw.TREEWY_OK
    assert call(H=0, S_old=None) == tw.TREEWY_OK


def test_snapshot_commit_and_path_host_checks(tw):
    assert tw.lib.treewy_snapshot_commit(A, A, None, 8, 2, 2, 128, 128, A, None, None) == tw.TREEWY_ERR_INVALID_ARG
    assert tw.lib.treewy_snapshot_commit(A, A, A, 8, 2, 2, 128, 64, A, None, None) == tw.TREEWY_ERR_UNSUPPORTED
    assert tw.lib.treewy_path_from_node(A, A, 257, 2, 8, A, A, None, None) == tw.TREEWY_ERR_UNSUPPORTED
    assert tw.lib.treewy_path_from_node(A, A, 8, 2, 257, A, A, None, None) == tw.TREEWY_ERR_UNSUPPORTED
    assert tw.lib.treewy_path_from_node(A, None, 8, 2, 8, A, A, None, None) == tw.TREEWY_ERR_INVALID_ARG
    assert tw.lib.treewy_path_from_node(None, None, 8, 0, 8, None, None, None, None) == tw.TREEWY_OK


def test_accept_greedy_host_checks(tw):
    f = tw.lib.treewy_accept_greedy

    def call(parent=A, draft=A, target=A, root=A, N=8, B=2, L_max=8, path=A, plen=A):
        return f(parent, draft, target, root, N, B, L_max, path, plen, None, None, None)

    assert call(N=257) == tw.TREEWY_ERR_UNSUPPORTED
    assert call(L_max=257) == tw.TREEWY_ERR_UNSUPPORTED
    assert call(N=-1) == tw.TREEWY_ERR_INVALID_ARG
    assert call(B=-1) == tw.TREEWY_ERR_INVALID_ARG
    assert call(root=None) == tw.TREEWY_ERR_INVALID_ARG
    assert call(draft=None) == tw.TREEWY_ERR_INVALID_ARG
    assert call(plen=None) == tw.TREEWY_ERR_INVALID_ARG
    assert call(path=None) == tw.TREEWY_ERR_INVALID_ARG
    assert call(B=0, root=None, plen=None) == tw.TREEWY_OK


def test_chain_prefill_host_checks(tw):
    f = tw.lib.treewy_chain_prefill

    def call(S0=A, q=A, T=100, B=2, H=2, dk=128, dt=1, st=0, S_T=A, o=A):
        return f(S0, q, A, A, A, A, T, B, H, dk, 128, dt, st, S_T, o, None, None)

    assert call(T=-1) == tw.TREEWY_ERR_INVALID_ARG
    assert call(dk=64) == tw.TREEWY_ERR_UNSUPPORTED
    assert call(dt=0, st=1) == tw.TREEWY_ERR_UNSUPPORTED
    assert call(st=4) == tw.TREEWY_ERR_INVALID_ARG
    assert call(S0=None) == tw.TREEWY_ERR_INVALID_ARG
    assert call(o=None) == tw.TREEWY_ERR_INVALID_ARG
    assert call(q=M) == tw.TREEWY_ERR_INVALID_ARG
    assert call(T=1 << 29, B=4) == tw.TREEWY_ERR_UNSUPPORTED
    assert call(B=0, S0=None) == tw.TREEWY_OK
    assert call(T=0, S_T=A, S0=A) == tw.TREEWY_OK           # in place, nothing to copy


def test_binding_raises_with_status(tw):
    with pytest.raises(tw.TreewyError) as e:
        tw._check(tw.TREEWY_ERR_UNSUPPORTED, "treewy_verify")
    assert e.value.status == tw.TREEWY_ERR_UNSUPPORTED and "unsupported" in str(e.value)


def test_binding_refuses_without_library(tmp_path):
    """The binding has no fallback: a copy of it next to no libtreewy.so
    raises ImportError on import."""
    import shutil
    import subprocess
    import sys
    src = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_2608_20961_amd",
                       "treewy.py")
    pkg = tmp_path / "nolib"
    pkg.mkdir()
    (pkg / "__init__.py").write_text("")
    shutil.copy(src, pkg / "treewy.py")
    r = subprocess.run([sys.executable, "-c", "import nolib.treewy"], cwd=str(tmp_path), capture_output=True,
                       text=True, timeout=300)
    assert r.returncode != 0
    assert "ImportError" in r.stderr and "not built" in r.stderr
