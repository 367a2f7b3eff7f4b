"""Benchmark: tree-WY verify + commit of one GDN layer on one MI355X.

A step is one pass of the hot path over one batch: treewy_verify (every draft
node's output and the pseudo-values, one solve per (sequence, head)) followed
by treewy_commit (the accepted node's state, out of place so the inputs stay
fixed).  The headline workload is the 397B-shaped wide tree: B = 128
sequences, H = 64 value heads, d_k = d_v = 128, N = 64 draft nodes (max depth
8), bf16 q/k/v and fp32 state.  Inputs are resident in HBM before the timed
region.

Prints ONE JSON line.  Besides the headline (verified draft nodes per second
for the layer) it carries the per-kernel HBM rooflines, a block per other
workload (the 4-node fp32 chain, the 35B-shaped chain and tree, and the
32-node stress tree with the full-state-snapshot comparison: bytes moved and
speculative memory of both methods), the fused call, the bf16 state, the chain
prefill, 128-node trees, and the float64 oracle timed on the host's cores as
a CPU baseline.  Every other GPU section runs first and the headline's timed
steps after them, so that they run at the clocks the GPU holds under
sustained load; the oracle runs last.

  python bench.py [--steps K] [--warmup W] [--workload 0..4] [--gpus 1]
                  [--configs 0,1,2,4 | --no-configs] [--no-snapshot]
                  [--no-cpu-baseline] [--copy-calibration]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0          # MI355X HBM3E, vendor figure
METRIC = "verified draft nodes/sec per GDN layer + commit GB/s (% HBM peak), 1 GPU"


def log(msg):
    print("[bench] " + msg, file=sys.stderr, flush=True)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    # (the first few dozen launches of a section run while the GPU's clocks
    # settle under the sustained HBM load; 30 untimed steps cover that)
    p.add_argument("--warmup", type=int, default=30)
    p.add_argument("--workload", type=int, default=3)
    p.add_argument("--seed", type=int, default=0)
    p.add_argument("--no-snapshot", action="store_true")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--prefill-tokens", type=int, default=1024,
                   help="tokens per sequence for the chain-prefill measurement (0 skips it)")
    p.add_argument("--no-big-tree", action="store_true", help="skip the 128-node tree (chunked verify)")
    p.add_argument("--cpu-seconds", type=float, default=12.0, help="target oracle time for the CPU baseline")
    p.add_argument("--configs", default="0,1,2,4",
                   help="other workloads measured first, each in a block of its own (comma-separated ids)")
    p.add_argument("--no-configs", action="store_true", help="skip the other workloads' blocks")
    p.add_argument("--config-cpu-seconds", type=float, default=2.0,
                   help="target oracle time for each other workload's CPU baseline")
    p.add_argument("--copy-calibration", action="store_true",
                   help="only run a plain 1 GiB device copy (for scaling HBM counters)")
    return p.parse_args()


def _code_only(text: str) -> str:
    """C/HIP source with comments removed and whitespace collapsed, so that a
    comment edit does not count as a kernel change."""
    out, i, n = [], 0, len(text)
    while i < n:
        c = text[i]
        if c in "\"'":                            # string or char literal, copied whole
            j = i + 1
            while j < n and text[j] != c:
                j += 2 if text[j] == "\\" else 1
            out.append(text[i:j + 1])
            i = j + 1
        elif text.startswith("//", i):
            j = text.find("\n", i)
            i = n if j < 0 else j
        elif text.startswith("/*", i):
            j = text.find("*/", i + 2)
            i = n if j < 0 else j + 2
        else:
            out.append(c)
            i += 1
    return " ".join("".join(out).split())


def kernel_source_hash() -> str:
    """Hash of the code (comments excluded) of every source under csrc/."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2608_20961_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        with open(os.path.join(csrc, name), encoding="utf-8") as f:
            h.update(name.encode() + _code_only(f.read()).encode())
    return h.hexdigest()[:16]


def load_traffic(kernel: str, workload: str, src_hash: str):
    """HBM bytes per launch from committed rocprofv3 counter summaries, if they
    were taken on the current kernel sources (else None)."""
    path = os.path.join(ROOT, "profiles", "traffic_%s_%s.txt" % (kernel, workload))
    if not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            key, val = line.split(":", 1)
            vals[key.strip()] = val.strip()
    if vals.get("source_hash") != src_hash:
        return None
    try:
        return float(vals["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def copy_calibration(torch):
    n = 1 << 28                                    # 2^28 floats = 1 GiB
    src = torch.ones(n, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes_each_way": 4 * n, "launches": 5}), flush=True)


def device_inputs(torch, tw, wl, w, seed, x):
    """The seeded host inputs `x` on the device; S0 made on the device by the
    library's chain prefill over the workload's warm-up tokens in float32
    (the float32 kernels, so a profile's statistics for the timed bf16
    kernels cover only the timed launches)."""
    dev = torch.device("cuda:0")
    dt = torch.bfloat16 if w.in_dtype == "bf16" else torch.float32

    def put(a, dtype):
        return torch.from_numpy(np.ascontiguousarray(a)).to(dev).to(dtype)

    d = dict(q=put(x["q"], dt), k=put(x["k"], dt), v=put(x["v"], dt), alpha=put(x["alpha"], torch.float32),
             beta=put(x["beta"], torch.float32), parent=put(x["parent"], torch.int32),
             path=put(x["path"], torch.int32), path_len=put(x["path_len"], torch.int32))
    S = torch.zeros((w.B, w.H, w.d_v, w.d_k), dtype=torch.float32, device=dev)
    k, v, a, b = wl.warmup_chunk_torch(w, seed, 0, w.warm_tokens, dev, torch.float32)
    tw.treewy_chain_prefill(S, k, k, v, a, b, S_T=S)
    torch.cuda.synchronize()
    del k, v, a, b
    d["S0"] = S
    return x, d


class TimingEvent:
    """A HIP event used only for timing, created with hipEventDisableSystemFence.

    By default recording an event ends with a system-scope fence, which
    writes back and invalidates the L2 caches: between two timed launches it
    adds its own cost to the interval and leaves the next launch cold caches
    that no serving loop would give it.  HIP offers this flag for events that
    only measure time; the elapsed times are read after a device-wide
    synchronize.  The events come from the HIP runtime torch has loaded, so
    they record on torch's streams."""
    DISABLE_SYSTEM_FENCE = 0x20000000
    _hip = None

    @classmethod
    def runtime(cls):
        if cls._hip is None:
            import ctypes
            path = "libamdhip64.so"
            for line in open("/proc/self/maps"):
                if "libamdhip64" in line:
                    path = line.split()[-1]
                    break
            cls._hip = ctypes.CDLL(path)
        return cls._hip

    def __init__(self):
        import ctypes
        self._c = ctypes
        self.ev = ctypes.c_void_p()
        rc = self.runtime().hipEventCreateWithFlags(ctypes.byref(self.ev), ctypes.c_uint(self.DISABLE_SYSTEM_FENCE))
        if rc != 0:
            raise RuntimeError("hipEventCreateWithFlags failed (%d)" % rc)

    def record(self, stream):
        rc = self.runtime().hipEventRecord(self.ev, self._c.c_void_p(stream.cuda_stream))
        if rc != 0:
            raise RuntimeError("hipEventRecord failed (%d)" % rc)

    def elapsed_time(self, end):
        ms = self._c.c_float()
        rc = self.runtime().hipEventElapsedTime(self._c.byref(ms), self.ev, end.ev)
        if rc != 0:
            raise RuntimeError("hipEventElapsedTime failed (%d)" % rc)
        return ms.value

    def __del__(self):
        if self._hip is not None and self.ev:
            self._hip.hipEventDestroy(self.ev)


SETTLE_MS = 40.0
# Every timed section in launch order: its tag, its warm-up and timed steps
# (so that a kernel trace of this command can be split into sections).
LAUNCH_LOG = []


def time_steps(torch, launches, steps, warmup, flush=None, stats=None, settle_ms=0.0, tag=None, per_step=None):
    """Run `launches` (a list of callables, one step) W + K times; return the
    average step time and the average time of each launch (HIP timing
    events on the stream the kernels run on).  With `flush`, it runs between
    steps (outside every launch's events) and the step time is the sum of the
    launch times.  With `stats` (a list), the p10 / p50 / p90 of each
    launch's times are appended to it.  With `settle_ms`, warm-up steps go on
    past W until that much wall time has passed: the GPU's clocks take tens
    of milliseconds of sustained work to reach their level under load (a
    fused launch timed after 5 warm-up launches ran 388 us against 335 us
    once settled), and the headline aside every section is timed settled.
    `tag` names the section in LAUNCH_LOG; `per_step` lists how many kernels
    each callable launches when that is not one."""
    t0 = time.perf_counter()
    n = 0
    while n < warmup or (time.perf_counter() - t0) * 1e3 < settle_ms:
        if flush is not None and n >= warmup:
            flush()
        for f in launches:
            f()
        n += 1
        if settle_ms > 0 and n % 8 == 0:
            torch.cuda.synchronize()                # (wall time then follows the GPU)
    torch.cuda.synchronize()
    LAUNCH_LOG.append({"tag": tag, "warmup_steps": n, "timed_steps": steps,
                       "kernels_per_step": per_step if per_step is not None else [1] * len(launches)})
    stream = torch.cuda.current_stream()
    ev = [[TimingEvent() for _ in range(len(launches) + 1)] for _ in range(steps)]
    t0 = TimingEvent()
    t1 = TimingEvent()
    torch.cuda.synchronize()
    t0.record(stream)
    for i in range(steps):
        if flush is not None:
            flush()
        ev[i][0].record(stream)
        for j, f in enumerate(launches):
            f()
            ev[i][j + 1].record(stream)
    t1.record(stream)
    torch.cuda.synchronize()
    times = [[ev[i][j].elapsed_time(ev[i][j + 1]) for i in range(steps)] for j in range(len(launches))]
    per = [float(np.mean(t)) for t in times]
    total = sum(per) if flush is not None else t0.elapsed_time(t1) / steps
    if stats is not None:
        stats.extend([round(float(x), 5) for x in np.percentile(t, (10, 50, 90))] for t in times)
    return total, per


def roofline(bytes_per_launch, ms, traffic):
    gbps = bytes_per_launch / (ms * 1e-3) / 1e9
    return {"bound": "hbm", "achieved": round(gbps, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
            "frac": round(gbps / PEAK_HBM_GBPS, 4), "traffic": traffic,
            "algorithmic_bytes": int(bytes_per_launch), "avg_launch_ms": round(ms, 5)}


def _cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, wl, x, seed, target_s, max_units=None):
    """The float64 oracle (verify + commit) on a bounded sample of units.

    S0 of each sampled unit is the oracle's own warm-up over the unit's
    warm-up tokens (untimed); the timed part is verify + commit.  The sample
    grows from a 64-unit probe to about `target_s` seconds of oracle time, and
    at most `max_units` units."""
    import oracle
    orc = oracle.default()
    H, N = w.H, w.N

    def warm(units):
        S0 = np.empty((len(units), w.d_v, w.d_k))
        for lo in range(0, len(units), 256):
            part = units[lo:lo + 256]
            toks = [wl.warmup_tokens(w, seed=seed, units=slice(int(u), int(u) + 1)) for u in part]
            cat = {n: np.concatenate([t[n] for t in toks]) for n in ("k", "v", "alpha", "beta")}
            S0[lo:lo + len(part)] = orc.chain(np.zeros((len(part), w.d_v, w.d_k)), cat["k"], cat["v"],
                                              cat["alpha"], cat["beta"])
        return S0.astype(np.float32)

    def run(units, S0):
        b = units // H
        sel = lambda a: a.reshape(w.units, *a.shape[2:])[units].astype(np.float64)
        q, k, v, al, be = (sel(x[n]) for n in ("q", "k", "v", "alpha", "beta"))
        par = x["parent"][b]
        t0 = time.perf_counter()
        orc.verify(S0, q, k, v, al, be, par)
        orc.commit(S0, k, v, al, be, par, x["path"][b], x["path_len"][b])
        return time.perf_counter() - t0

    probe = np.arange(min(64, w.units))
    dt = run(probe, warm(probe))
    count = int(min(w.units, max(len(probe), len(probe) * target_s / max(dt, 1e-6))))
    if max_units is not None:
        count = max(len(probe), min(count, max_units))
    units = wl.sample_units(w, count, seed=1)
    dt = run(units, warm(units))
    nodes_per_s = (len(units) / H) * N / dt       # a sequence's N nodes cost H units of work
    return {"value": round(nodes_per_s, 1), "unit": "nodes/s", "cores": orc.threads(), "kind": "oracle",
            "cpu_model": _cpu_model(), "host_cpus": os.cpu_count(),
            "sample": "%d of %d (sequence, head) units of the same workload; float64 verify + commit "
                      "took %.2f s; nodes/s = units/H * N / time" % (len(units), w.units, dt)}


def make_flush(torch, acc, w, path_len):
    """A workload whose step fits in the 256 MiB last-level cache would be
    served from it step after step: then 512 MiB are read between steps
    (outside the timed launches).  A read leaves the caches holding clean
    lines; a write (zero-fill) would leave dirty ones, whose write-back the
    next timed launch would pay for (at the 16-node workload that cost verify
    60%).  None for workloads that do not fit."""
    if acc.verify_bytes(w) + acc.commit_bytes(w, path_len) >= (1 << 30):
        return None
    scratch = torch.ones(1 << 27, device="cuda")

    def flush():
        scratch.max()
    return flush


def snapshot_comparison(torch, tw, acc, w, x, d, o, ms_treewy_step, steps):
    """Full-state snapshotting (approach (i) of Section "The memory problem")
    on the same inputs: its verify writes every node's state, its commit
    copies the accepted one.  Reports time, bytes moved and speculative
    memory for both methods.  The snapshot buffer is allocated here and freed
    before returning."""
    S_new = torch.empty_like(d["S0"])
    snaps = torch.empty((w.B, w.H, w.N, w.d_v, w.d_k), dtype=torch.float32, device="cuda")
    acc_node = torch.tensor([int(x["path"][b, x["path_len"][b] - 1]) if x["path_len"][b] else -1
                             for b in range(w.B)], dtype=torch.int32, device="cuda")
    o2 = torch.empty_like(o)

    def sverify():
        tw.treewy_snapshot_verify(d["S0"], d["q"], d["k"], d["v"], d["alpha"], d["beta"], d["parent"],
                                  o=o2, snapshots=snaps)

    def scommit():
        tw.treewy_snapshot_commit(d["S0"], snaps, acc_node, S_new=S_new)

    ms_s, (ms_sv, ms_sc) = time_steps(torch, [sverify, scommit], steps, 1, tag=w.name + ".snapshot")
    sb = acc.snapshot_verify_bytes(w)
    reload = acc.snapshot_reload_bytes(w, x["parent"])
    spec = acc.speculative_state_bytes(w)
    tw_bytes = acc.verify_bytes(w) + acc.commit_bytes(w, x["path_len"])
    snap_bytes = sb + acc.snapshot_commit_bytes(w)
    out = {
        "workload": w.describe(), "ms_per_step": round(ms_s, 4), "steps": steps,
        "nodes_per_s": round(w.B * w.N / (ms_s * 1e-3), 1),
        "verify": dict(roofline(sb, ms_sv, None), parent_reload_bytes=int(reload),
                       frac_with_reloads=round((sb + reload) / (ms_sv * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4)),
        "commit": roofline(acc.snapshot_commit_bytes(w), ms_sc, None),
        "bytes_moved_per_step": {"treewy": int(tw_bytes), "snapshot": int(snap_bytes),
                                 "snapshot_with_reloads": int(snap_bytes + reload),
                                 "ratio": round(snap_bytes / tw_bytes, 2)},
        "speculative_state_bytes": {"treewy_U": spec["treewy_U"], "treewy_U_k_alpha": spec["treewy_U_k_alpha"],
                                    "snapshot_states": spec["snapshot_states"],
                                    "committed_state": spec["committed_state"],
                                    "ratio_U": round(spec["snapshot_states"] / spec["treewy_U"], 1)},
        "treewy_speedup": round(ms_s / ms_treewy_step, 2),
    }
    del snaps, S_new, o2
    return out


def launch_context(torch, tw, acc, w, d, flush, steps):
    """For a workload small enough to be flushed between launches, what the
    single flushed launch is measured against: a plain device copy that moves
    the verify's algorithmic bytes (half read, half written) under the same
    flush and events, and the verify run back to back over R distinct input
    sets, as consecutive layers would be, with R x the bytes >= 1 GiB so that
    no set is still in the last-level cache when its turn comes (per-launch
    time = the interval / R)."""
    vb = acc.verify_bytes(w)
    half = torch.empty(vb // 8, dtype=torch.float32, device="cuda").fill_(1.0)
    dst = torch.empty_like(half)
    _, (ms_copy,) = time_steps(torch, [lambda: dst.copy_(half)], steps, 3, flush, settle_ms=SETTLE_MS,
                               tag=w.name + ".copy")
    del half, dst
    R = int(min(32, max(2, -(-(1 << 30) // vb))))
    sets = []
    for _ in range(R):
        c = {n: d[n].clone() for n in ("S0", "q", "k", "v", "alpha", "beta", "parent")}
        c["U"] = torch.empty((w.B, w.H, w.N, w.d_v), dtype=torch.float32, device="cuda")
        c["o"] = torch.empty((w.B, w.H, w.N, w.d_v), dtype=d["q"].dtype, device="cuda")
        sets.append(c)

    def layers():
        for c in sets:
            tw.treewy_verify(c["S0"], c["q"], c["k"], c["v"], c["alpha"], c["beta"], c["parent"], o=c["o"], U=c["U"])
    # Captured in one HIP graph (as a serving loop would run a decode step),
    # so that the host's per-call cost does not pace the launches.
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        layers()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    LAUNCH_LOG.append({"tag": w.name + ".graph_warm", "warmup_steps": 1, "timed_steps": 0, "kernels_per_step": [R]})
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        layers()
    _, (ms_r,) = time_steps(torch, [graph.replay], max(3, steps // 4), 1, settle_ms=SETTLE_MS,
                            tag=w.name + ".graph", per_step=[R])
    del graph, sets
    torch.cuda.empty_cache()
    return {"copy_same_bytes": dict(roofline(vb, ms_copy, None), what="torch copy_ of verify_bytes / 2 each way, "
                                                                      "flushed and timed like the verify"),
            "verify_back_to_back": dict(roofline(vb, ms_r / R, None), input_sets=R,
                                        what="R launches over R distinct input sets captured in one HIP graph; "
                                             "one replay's interval / R")}


def measure_workload(torch, tw, wl, acc, w, x, d, args, src_hash, snapshot):
    """One workload's block on the GPU: verify + commit steps (the headline's
    step on this workload), the fused call and optionally the snapshot
    comparison, on the host inputs `x` already resident on the device as `d`.
    Returns the block (the oracle's CPU baseline runs after all GPU work)."""
    U = torch.empty((w.B, w.H, w.N, w.d_v), dtype=torch.float32, device="cuda")
    o = torch.empty((w.B, w.H, w.N, w.d_v), dtype=d["q"].dtype, device="cuda")
    S_new = torch.empty_like(d["S0"])
    S0_commit = d["S0"].clone()

    def verify():
        tw.treewy_verify(d["S0"], d["q"], d["k"], d["v"], d["alpha"], d["beta"], d["parent"], o=o, U=U)

    def commit():
        tw.treewy_commit(S0_commit, U, d["k"], d["alpha"], d["path"], d["path_len"], parent=d["parent"],
                         S_new=S_new)

    flush = make_flush(torch, acc, w, x["path_len"])
    dist = []
    ms_step, (ms_v, ms_c) = time_steps(torch, [verify, commit], args.steps, args.warmup, flush, dist,
                                       settle_ms=SETTLE_MS, tag=w.name + ".verify_commit")
    S_f, o_f, U_f = torch.empty_like(d["S0"]), torch.empty_like(o), torch.empty_like(U)

    def fused():
        tw.treewy_commit_verify(S0_commit, U, d["k"], d["alpha"], d["path"], d["path_len"], d["q"], d["k"], d["v"],
                                d["alpha"], d["beta"], d["parent"], parent_prev=d["parent"], S_new=S_f, o=o_f,
                                U=U_f)

    _, (ms_f,) = time_steps(torch, [fused], args.steps, args.warmup, flush, settle_ms=SETTLE_MS,
                            tag=w.name + ".fused")
    nodes = w.B * w.N
    block = {
        "workload": w.describe(), "units": w.units, "ms_per_step": round(ms_step, 5),
        "nodes_per_s": round(nodes / (ms_step * 1e-3), 1), "cache_flushed_between_steps": flush is not None,
        "verify": dict(roofline(acc.verify_bytes(w), ms_v, load_traffic("verify", w.name, src_hash)),
                       launch_ms_p10_p50_p90=dist[0], nodes_per_s=round(nodes / (ms_v * 1e-3), 1)),
        "commit": dict(roofline(acc.commit_bytes(w, x["path_len"]), ms_c, load_traffic("commit", w.name, src_hash)),
                       launch_ms_p10_p50_p90=dist[1]),
        "fused_commit_verify": dict(roofline(acc.commit_verify_bytes(w, x["path_len"]), ms_f,
                                             load_traffic("commit_verify", w.name, src_hash)),
                                    speedup_vs_separate_calls=round(ms_step / ms_f, 3)),
    }
    log("%s: verify %.4f, commit %.4f, fused %.4f ms" % (w.name, ms_v, ms_c, ms_f))
    del S_f, o_f, U_f
    if flush is not None:
        ctx = launch_context(torch, tw, acc, w, d, flush, args.steps)
        ctx["verify_over_copy_time"] = round(ms_v / ctx["copy_same_bytes"]["avg_launch_ms"], 3)
        block["verify"]["launch_context"] = ctx
        log("%s: copy of the same bytes %.4f ms; verify back to back %.4f ms" % (
            w.name, ctx["copy_same_bytes"]["avg_launch_ms"], ctx["verify_back_to_back"]["avg_launch_ms"]))
    if snapshot:
        block["snapshot_comparison"] = snapshot_comparison(torch, tw, acc, w, x, d, o, ms_step,
                                                           max(3, args.steps // 10))
        log("%s: snapshot baseline %.4f ms/step" % (w.name, block["snapshot_comparison"]["ms_per_step"]))
    del d, U, o, S_new, S0_commit
    torch.cuda.empty_cache()
    return block


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py runs on exactly one GPU: the verify/commit path has no cross-GPU step, "
              "and it measures one GPU's share (got --gpus %d)" % args.gpus, file=sys.stderr)
        sys.exit(2)
    import torch
    if args.copy_calibration:
        copy_calibration(torch)
        return
    from paper_2608_20961_amd import accounting as acc
    from paper_2608_20961_amd import treewy as tw
    from paper_2608_20961_amd import workload as wl

    src_hash = kernel_source_hash()
    # Order.  Every workload's inputs are drawn on the host and made resident
    # on the device (with its S0) first.  Then the GPU sections run back to
    # back: the other workloads, each in a block of its own (the 32-node
    # stress tree with the snapshot comparison it exists for), the headline
    # workload's other calls, and last the headline's own W warmup and K
    # timed steps.  The oracle's CPU baselines run after all GPU work.  The
    # GPU's compute clock falls within milliseconds of idling (host work,
    # host-to-device copies) and takes about 10 ms of sustained work to come
    # back, and verify and the fused call (not commit) ran about 10% slower
    # in the launches after such an idle spell; this order times every
    # section at the clocks the GPU holds under sustained load, as in a
    # serving loop.
    w = wl.WORKLOADS[args.workload]
    ids = [] if args.no_configs else [int(c) for c in args.configs.split(",") if c.strip() != ""]
    ids = [i for i in ids if i != args.workload]
    hosts = {i: wl.make_inputs(wl.WORKLOADS[i], seed=args.seed) for i in ids + [args.workload]}
    big = not args.no_big_tree and w.in_dtype == "bf16" and w.B == wl.BIG_TREE.B and w.H == wl.BIG_TREE.H
    xb = wl.make_inputs(wl.BIG_TREE, seed=args.seed) if big else None
    tok = wl.acceptance_tokens(hosts[args.workload]["parent"], seed=args.seed, vocab=4, plant=True)
    log("host inputs drawn")
    devs = {i: device_inputs(torch, tw, wl, wl.WORKLOADS[i], args.seed, hosts[i])[1] for i in ids + [args.workload]}
    Tp = args.prefill_tokens if w.in_dtype == "bf16" else 0
    if Tp > 0:
        kp, vp, ap, bp = wl.warmup_chunk_torch(w, args.seed, 1, Tp, "cuda", torch.bfloat16)
        qp = wl.warmup_chunk_torch(w, args.seed, 2, Tp, "cuda", torch.bfloat16)[0]
    if big:
        wb = wl.BIG_TREE
        put = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a)).to("cuda").to(dt)
        bq, bk, bv = (put(xb[n], torch.bfloat16) for n in ("q", "k", "v"))
        ba, bb = put(xb["alpha"], torch.float32), put(xb["beta"], torch.float32)
        bpar, bpath, bplen = (put(xb[n], torch.int32) for n in ("parent", "path", "path_len"))
    t_d, t_t, t_r = (torch.from_numpy(tok[n]).to("cuda") for n in ("draft", "target", "root"))
    torch.cuda.synchronize()
    log("inputs resident, S0 warmed on the device")
    others, cpu_jobs = {}, []
    for i in ids:
        wo = wl.WORKLOADS[i]
        log("workload " + wo.describe())
        block = measure_workload(torch, tw, wl, acc, wo, hosts[i], devs.pop(i), args, src_hash,
                                 snapshot=not args.no_snapshot and wo.name == "stress-tree32")
        others[wo.name] = block
        cpu_jobs.append((block, wo, hosts[i]))

    log("workload " + w.describe() + " (headline)")
    x, d = hosts[args.workload], devs.pop(args.workload)
    U = torch.empty((w.B, w.H, w.N, w.d_v), dtype=torch.float32, device="cuda")
    o = torch.empty((w.B, w.H, w.N, w.d_v), dtype=d["q"].dtype, device="cuda")
    S_new = torch.empty_like(d["S0"])
    # Commit reads its own copy of S0 (same values, other addresses).  In a
    # serving step the other layers run between a layer's verify and its
    # commit, so the state verify just read is no longer in the 256 MiB
    # last-level cache; reading one buffer twice back to back would credit
    # commit with cache hits it does not get.
    S0_commit = d["S0"].clone()

    def verify():
        tw.treewy_verify(d["S0"], d["q"], d["k"], d["v"], d["alpha"], d["beta"], d["parent"], o=o, U=U)

    def commit():
        tw.treewy_commit(S0_commit, U, d["k"], d["alpha"], d["path"], d["path_len"], parent=d["parent"],
                         S_new=S_new)

    flush = make_flush(torch, acc, w, x["path_len"])
    verify()                                       # U for the fused call's previous round
    torch.cuda.synchronize()
    LAUNCH_LOG.append({"tag": "head.verify_for_U", "warmup_steps": 1, "timed_steps": 0, "kernels_per_step": [1]})
    nodes = w.B * w.N
    result = {}
    # Fused: the previous round's commit inside this round's verify
    # (treewy_commit_verify).  The previous round is this round's own draft
    # and paths, so one launch moves commit + verify bytes minus one read of
    # the state.
    S_fused = torch.empty_like(d["S0"])
    o_f, U_f = torch.empty_like(o), torch.empty_like(U)

    def fused():
        tw.treewy_commit_verify(S0_commit, U, d["k"], d["alpha"], d["path"], d["path_len"], d["q"], d["k"], d["v"],
                                d["alpha"], d["beta"], d["parent"], parent_prev=d["parent"], S_new=S_fused, o=o_f,
                                U=U_f)

    _, (ms_fused,) = time_steps(torch, [fused], args.steps, args.warmup, flush, settle_ms=SETTLE_MS,
                                tag="head.fused")
    log("fused commit+verify: %.4f ms/launch" % ms_fused)
    fb = acc.commit_verify_bytes(w, x["path_len"])
    result["fused_commit_verify"] = dict(
        roofline(fb, ms_fused, load_traffic("commit_verify", w.name, src_hash)),
        kernel="treewy_commit_verify", nodes_per_s=round(nodes / (ms_fused * 1e-3), 1))
    del S_fused, o_f, U_f
    # bf16 state storage: the same step with S0 / S_new in bfloat16 (inputs
    # rounded once from the float32 state).
    ms_step_b = None
    if w.in_dtype == "bf16":
        S0_b = d["S0"].to(torch.bfloat16)
        S0_bc = S0_b.clone()
        S_new_b = torch.empty_like(S0_b)
        o_b, U_b = torch.empty_like(o), torch.empty_like(U)

        def verify_b():
            tw.treewy_verify(S0_b, d["q"], d["k"], d["v"], d["alpha"], d["beta"], d["parent"], o=o_b, U=U_b)

        def commit_b():
            tw.treewy_commit(S0_bc, U_b, d["k"], d["alpha"], d["path"], d["path_len"], parent=d["parent"],
                             S_new=S_new_b)

        def fused_b():
            tw.treewy_commit_verify(S0_bc, U_b, d["k"], d["alpha"], d["path"], d["path_len"], d["q"], d["k"],
                                    d["v"], d["alpha"], d["beta"], d["parent"], parent_prev=d["parent"],
                                    S_new=S_new_b, o=o_f2, U=U_f2)

        o_f2, U_f2 = torch.empty_like(o), torch.empty_like(U)
        ms_step_b, (ms_vb, ms_cb) = time_steps(torch, [verify_b, commit_b], args.steps, args.warmup, flush,
                                               settle_ms=SETTLE_MS, tag="head.bf16_verify_commit")
        _, (ms_fb,) = time_steps(torch, [fused_b], args.steps, args.warmup, flush, settle_ms=SETTLE_MS,
                                 tag="head.bf16_fused")
        log("bf16 state: verify %.4f, commit %.4f, fused %.4f ms" % (ms_vb, ms_cb, ms_fb))
        result["bf16_state"] = {
            "ms_per_step": round(ms_step_b, 5), "nodes_per_s": round(nodes / (ms_step_b * 1e-3), 1),
            "verify": roofline(acc.verify_bytes(w, 2), ms_vb, load_traffic("verify_bf16state", w.name, src_hash)),
            "commit": roofline(acc.commit_bytes(w, x["path_len"], 2), ms_cb,
                               load_traffic("commit_bf16state", w.name, src_hash)),
            "fused_commit_verify": roofline(acc.commit_verify_bytes(w, x["path_len"], 2), ms_fb,
                                            load_traffic("commit_verify_bf16state", w.name, src_hash)),
        }
        del S0_b, S0_bc, S_new_b, o_b, U_b, o_f2, U_f2
    # Chain prefill (bf16 tokens, float32 state) at the workload's B x H.
    if Tp > 0:
        S_p = torch.empty_like(d["S0"])
        o_p = torch.empty_like(vp)

        def prefill():
            tw.treewy_chain_prefill(d["S0"], qp, kp, vp, ap, bp, S_T=S_p, o=o_p)

        _, (ms_pf,) = time_steps(torch, [prefill], max(3, args.steps // 10), 1, settle_ms=SETTLE_MS,
                                 tag="head.prefill")
        pb = acc.prefill_bytes(w, Tp)
        result["chain_prefill"] = dict(roofline(pb, ms_pf, load_traffic("chain_prefill", w.name, src_hash)), tokens=Tp,
                                       tokens_per_s=round(w.B * Tp / (ms_pf * 1e-3), 1))
        log("chain prefill of %d tokens: %.4f ms" % (Tp, ms_pf))
        del kp, vp, ap, bp, qp, S_p, o_p
    # Trees past one 64-node chunk: 128-node trees at the same layer shape
    # (verify walks two chunks per unit; commit follows paths up to 16 long).
    if big:
        o_b = torch.empty((wb.B, wb.H, wb.N, wb.d_v), dtype=torch.bfloat16, device="cuda")
        U_b = torch.empty((wb.B, wb.H, wb.N, wb.d_v), dtype=torch.float32, device="cuda")
        S_nb = torch.empty_like(d["S0"])

        def verify_big():
            tw.treewy_verify(d["S0"], bq, bk, bv, ba, bb, bpar, o=o_b, U=U_b)

        def commit_big():
            tw.treewy_commit(S0_commit, U_b, bk, ba, bpath, bplen, parent=bpar, S_new=S_nb)

        ms_bstep, (ms_bv, ms_bc) = time_steps(torch, [verify_big, commit_big], max(5, args.steps // 2),
                                              max(2, args.warmup // 2), settle_ms=SETTLE_MS, tag="head.tree128")
        nb = wb.B * wb.N
        result["tree128"] = {
            "workload": wb.describe(),
            "ms_per_step": round(ms_bstep, 5),
            "nodes_per_s": round(nb / (ms_bstep * 1e-3), 1),
            "verify": dict(roofline(acc.verify_bytes(wb), ms_bv, load_traffic("verify", wb.name, src_hash)),
                           nodes_per_s=round(nb / (ms_bv * 1e-3), 1)),
            "commit": roofline(acc.commit_bytes(wb, xb["path_len"]), ms_bc,
                               load_traffic("commit", wb.name, src_hash)),
        }
        log("128-node trees: verify %.4f ms, commit %.4f ms" % (ms_bv, ms_bc))
        del bq, bk, bv, ba, bb, bpar, bpath, bplen, o_b, U_b, S_nb
    # Greedy acceptance on the device (tokens: vocabulary of 4, the target
    # agreeing with the drafter along one planted chain per sequence).
    acc_path = torch.empty((w.B, w.max_depth), dtype=torch.int32, device="cuda")
    acc_len = torch.empty((w.B,), dtype=torch.int32, device="cuda")
    acc_bonus = torch.empty((w.B,), dtype=torch.int32, device="cuda")

    def accept():
        tw.treewy_accept_greedy(d["parent"], t_d, t_t, t_r, w.max_depth, path=acc_path, path_len=acc_len,
                                bonus=acc_bonus)

    _, (ms_acc,) = time_steps(torch, [accept], args.steps, args.warmup, settle_ms=SETTLE_MS, tag="head.accept")
    result["accept_greedy"] = {"avg_launch_ms": round(ms_acc, 5), "sequences": w.B, "nodes": w.N,
                               "mean_accepted": round(float(acc_len.float().mean()), 3)}
    # What a plain device-to-device copy reaches on this GPU (read + write
    # bytes): the practical ceiling next to the 8 TB/s vendor peak.
    src = torch.ones(1 << 28, device="cuda")
    dst = torch.empty_like(src)
    _, (ms_copy,) = time_steps(torch, [lambda: dst.copy_(src)], 10, 3, settle_ms=SETTLE_MS, tag="head.copy")
    result["hbm_copy_achievable"] = {"GB_per_s": round(2 * 4 * (1 << 28) / (ms_copy * 1e-3) / 1e9, 1),
                                     "bytes_each_way": 4 * (1 << 28), "avg_launch_ms": round(ms_copy, 5)}
    del src, dst
    spec = acc.speculative_state_bytes(w)
    result["speculative_state_bytes"] = {"treewy_U": spec["treewy_U"], "treewy_U_k_alpha": spec["treewy_U_k_alpha"],
                                         "snapshot_states": spec["snapshot_states"]}
    if not args.no_snapshot:
        result["snapshot_baseline"] = snapshot_comparison(torch, tw, acc, w, x, d, o, 1.0, max(3, args.steps // 10))
        log("snapshot baseline: %.4f ms/step" % result["snapshot_baseline"]["ms_per_step"])

    # ---- the headline: W warmup steps, then exactly K timed steps ------------
    dist = []
    ms_step, (ms_verify, ms_commit) = time_steps(torch, [verify, commit], args.steps, args.warmup, flush, dist,
                                                 tag="head.verify_commit")
    log("timed %d steps: %.4f ms/step (verify %.4f, commit %.4f)" % (args.steps, ms_step, ms_verify, ms_commit))
    vb = acc.verify_bytes(w)
    cb = acc.commit_bytes(w, x["path_len"])
    rf_verify = roofline(vb, ms_verify, load_traffic("verify", w.name, src_hash))
    rf_commit = roofline(cb, ms_commit, load_traffic("commit", w.name, src_hash))
    dominant = rf_verify if ms_verify >= ms_commit else rf_commit
    head = {
        "metric": METRIC,
        "value": round(nodes / (ms_step * 1e-3), 1),
        "unit": "nodes/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": w.in_dtype, "data": "synthetic",
        "config": {"workload": w.describe(), "B": w.B, "H": w.H, "N": w.N, "d_k": w.d_k, "d_v": w.d_v,
                   "step": "treewy_verify + treewy_commit (out of place)", "accumulate": "f32",
                   "state": "f32", "parallelism": "none (1 GPU)",
                   "cache_flushed_between_steps": flush is not None,
                   "timed_after": "the other workloads' blocks and this workload's other sections"},
        "roofline": dict(dominant, kernel="treewy_verify" if dominant is rf_verify else "treewy_commit"),
        "verify": dict(rf_verify, launch_ms_p10_p50_p90=dist[0], nodes_per_s=round(nodes / (ms_verify * 1e-3), 1),
                       head_nodes_per_s=round(w.units * w.N / (ms_verify * 1e-3), 1),
                       useful_tflops=round(acc.verify_flops(w) / (ms_verify * 1e-3) / 1e12, 2)),
        "commit": dict(rf_commit, launch_ms_p10_p50_p90=dist[1], pct_hbm_peak=round(100 * rf_commit["frac"], 2)),
        "kernel_source_hash": src_hash,
    }
    result = dict(head, **result)
    result["fused_commit_verify"]["speedup_vs_separate_calls"] = round(ms_step / ms_fused, 3)
    if ms_step_b is not None:
        result["bf16_state"]["speedup_vs_f32_state"] = round(ms_step / ms_step_b, 3)
    if "snapshot_baseline" in result:
        sb = result["snapshot_baseline"]
        sb["treewy_speedup"] = round(sb["ms_per_step"] / ms_step, 2)
    if others:
        result["configs"] = others

    # ---- CPU baselines (after all GPU work) ---------------------------------
    if not args.no_cpu_baseline:
        for block, wo, xo in cpu_jobs:
            log("cpu baseline (oracle), %s ..." % wo.name)
            block["cpu_baseline"] = cpu_baseline(wo, wl, xo, args.seed, args.config_cpu_seconds, max_units=2048)
        log("cpu baseline (oracle) ...")
        result["cpu_baseline"] = cpu_baseline(w, wl, x, args.seed, args.cpu_seconds)
    result["launch_log"] = LAUNCH_LOG
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
