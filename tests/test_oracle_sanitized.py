"""Every oracle pin again, against oracle.c built with AddressSanitizer and
UndefinedBehaviorSanitizer (CPU only).

The sanitizer build is a standalone executable (tests/oracle_sanitized.c
linked with oracle/oracle.c), so its runtimes load first without touching the
Python process.  `_Forward` stands in for the ctypes library inside
oracle.Oracle: each call copies the input arrays into a request, the
executable runs the same C function on heap buffers of exactly those sizes,
and the outputs are copied back.  A sanitizer report ends the executable, so
the pin that caused it fails, and the final check reads the report.
"""
import ctypes
import os
import shutil
import struct
import subprocess
import tempfile

import pytest

import oracle
from tests import pins

HERE = os.path.dirname(os.path.abspath(__file__))
SAN_FLAGS = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer",
             "-g", "-O1", "-fopenmp", "-std=c11", "-Wall", "-Wextra"]


class _Forward:
    """The oracle library's four functions, forwarded to the sanitizer build."""

    def __init__(self, exe):
        env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:exitcode=23",
                   UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1:exitcode=24")
        self.err = tempfile.TemporaryFile()
        self.proc = subprocess.Popen([exe], stdin=subprocess.PIPE, stdout=subprocess.PIPE, stderr=self.err, env=env)

    def _send(self, op, sizes, arrays):
        msg = struct.pack("=%di" % (1 + len(sizes)), op, *sizes)
        msg += b"".join(ctypes.string_at(p.value, n) for p, n in arrays)
        self.proc.stdin.write(msg)
        self.proc.stdin.flush()
        (status,) = struct.unpack("=i", self._read(4))
        return status

    def _read(self, n):
        data = self.proc.stdout.read(n)
        if len(data) != n:
            raise RuntimeError("the sanitizer build stopped (report below in the final check)")
        return data

    def _recv(self, outputs):
        for p, n in outputs:
            if p is not None:
                ctypes.memmove(p.value, self._read(n), n)

    def oracle_threads(self):
        self._send(1, [], [])
        return struct.unpack("=i", self._read(4))[0]

    def oracle_gdn_tree(self, U, N, dk, dv, S0, q, k, v, alpha, beta, parent, o, vt, states):
        un = U * N
        rc = self._send(2, [U, N, dk, dv, int(states is not None)],
                        [(S0, 8 * U * dv * dk), (q, 8 * un * dk), (k, 8 * un * dk), (v, 8 * un * dv),
                         (alpha, 8 * un), (beta, 8 * un), (parent, 4 * un)])
        if rc == 0:
            self._recv([(o, 8 * un * dv), (vt, 8 * un * dv), (states, 8 * un * dv * dk)])
        return rc

    def oracle_gdn_chain(self, U, T, dk, dv, S, k, v, alpha, beta):
        ut = U * T
        rc = self._send(3, [U, T, dk, dv], [(S, 8 * U * dv * dk), (k, 8 * ut * dk), (v, 8 * ut * dv),
                                            (alpha, 8 * ut), (beta, 8 * ut)])
        if rc == 0:
            self._recv([(S, 8 * U * dv * dk)])
        return rc

    def oracle_commit(self, U, N, dk, dv, L_max, S0, k, v, alpha, beta, parent, path, path_len, out):
        un = U * N
        rc = self._send(4, [U, N, dk, dv, L_max],
                        [(S0, 8 * U * dv * dk), (k, 8 * un * dk), (v, 8 * un * dv), (alpha, 8 * un),
                         (beta, 8 * un), (parent, 4 * un), (path, 4 * U * L_max), (path_len, 4 * U)])
        if rc == 0:
            self._recv([(out, 8 * U * dv * dk)])
        return rc

    def close(self):
        if self.proc.poll() is None:
            try:
                self.proc.stdin.write(struct.pack("=i", 0))
                self.proc.stdin.flush()
            except BrokenPipeError:
                pass
        rc = self.proc.wait(timeout=60)
        self.err.seek(0)
        return rc, self.err.read().decode(errors="replace")


@pytest.fixture(scope="module")
def sanitized():
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    d = tempfile.mkdtemp(prefix="oracle_san_")
    exe = os.path.join(d, "oracle_sanitized")
    subprocess.run(["gcc", *SAN_FLAGS, "-o", exe, os.path.join(HERE, "oracle_sanitized.c"), oracle.SOURCE],
                   check=True)
    fwd = _Forward(exe)
    yield oracle.Oracle(lib_path=exe, lib=fwd), fwd
    fwd.close()
    shutil.rmtree(d, ignore_errors=True)


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda p: p.__name__)
def test_pin_under_sanitizers(sanitized, pin):
    orc, _ = sanitized
    pin(orc)


def test_sanitizers_report_nothing(sanitized):
    """Runs after the pins (same module): the executable exits cleanly, with
    no AddressSanitizer, LeakSanitizer or UBSan report."""
    orc, fwd = sanitized
    assert orc.threads() >= 1
    rc, report = fwd.close()
    assert rc == 0 and "Sanitizer" not in report and "runtime error" not in report, report[-4000:]


def test_sanitizer_build_catches_planted_overflow():
    """A copy of oracle.c reading one key element past the end of the last
    key must stop the sanitizer build with a heap-buffer-overflow report (so
    the clean run above means something)."""
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    src = open(oracle.SOURCE).read()
    old = "for (int c = 0; c < dk; ++c) Pk += Pr[c] * k[c];"
    assert src.count(old) == 1, "mutation site vanished"
    d = tempfile.mkdtemp(prefix="oracle_san_bad_")
    try:
        bad_src = os.path.join(d, "oracle_bad.c")
        with open(bad_src, "w") as f:
            f.write(src.replace(old, "for (int c = 0; c <= dk; ++c) Pk += Pr[c < dk ? c : 0] * k[c];"))
        exe = os.path.join(d, "oracle_bad")
        subprocess.run(["gcc", *SAN_FLAGS, "-o", exe, os.path.join(HERE, "oracle_sanitized.c"), bad_src], check=True)
        fwd = _Forward(exe)
        with pytest.raises(RuntimeError):
            pins.pin_chain_literal(oracle.Oracle(lib_path=exe, lib=fwd))
        rc, report = fwd.close()
        assert rc != 0 and "heap-buffer-overflow" in report, report[-2000:]
    finally:
        shutil.rmtree(d, ignore_errors=True)
