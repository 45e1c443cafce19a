"""Benchmark: one CURE verify-and-repair step on one MI355X.

A step is one pass of the whole hot path over one batch of synthetic input
already resident in HBM, in two calls:
  1. cure_tree_attn one tree-masked verification attention layer (Sec. 3.5),
  2. cure_margins_accept  the margin pass over every tree node's logits row,
                    with the UFP gate over the draft-chain rows (Sec. 3.3,
                    Eq. 2, Algorithm 1) and the acceptance walk on the rows'
                    top-1 indices as the target argmax (Eq. 1, Eq. 4) -- the
                    same outputs as cure_margins followed by cure_accept.
The separate cure_margins and cure_accept calls are timed too (`kernels`).
The repair-tree builder (cure_repair_tree: ranked alternatives at the UFPs,
Eq. 3 branch budget, parent/token assembly) is timed beside the step, on the
draft-chain rows and UFPs the step's margin pass produced; it is reported
under `repair_tree` and is not part of `value`. So is the commit of the
accepted paths (cure_commit, Sec. 3.5), run on the step's own acceptance
results over a 32-layer cache of the workload's row shape (Llama-3-8B has 32
layers), reported under `commit`.

Timing: each input copy's step is captured once as a HIP graph; W warm-up
replays, then exactly K replays (K steps) bracketed by synchronize() on both
sides, timed by the host clock (ms_per_step) and by HIP events on the launch
stream. Inputs rotate over enough copies (>= 512 MB in total) that each step
reads from HBM rather than the 256 MB last-level cache. A second timed region
launches the calls eagerly with HIP events around each one (behind a spin
kernel, so host launch cost stays off the GPU timeline) to give the per-call
durations used for the roofline.

The printed JSON line's `value` is the step's algorithmic bytes over its time
(GB/s). `roofline` reports the longest call against the HBM peak; its
`traffic` is the calibrated FETCH_SIZE + WRITE_SIZE bytes per call stored in
profiles/traffic_<workload>.json, or null when that file is missing or the
call's kernel sources have changed since the counters were taken.
`read_ceiling` is the rate of a plain streaming read of a 1 GiB buffer
(cure_read_ceiling), the practical ceiling for the roofline fractions.
`cpu_baseline` times the CPU oracle on a bounded sample of the same workload
on this host.
"""

import argparse
import ctypes
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "tree-verify step latency (µs) + KV GB/s vs HBM peak, Llama-3-8B attn shape"
HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0     # dense bf16 matrix-core peak
DEFAULT_WORKLOAD = "llama3_8b_ctx2k_b1"
ROTATE_BYTES = 512 << 20
CSRC = os.path.join(ROOT, "paper_2608_00531_amd", "csrc")
# Kernel sources behind each call: a stored traffic figure is used only while
# these files are unchanged since the counters were taken.
CALL_SOURCES = {"margins": ["margins.hip", "common.hpp", "accept_walk.hpp"],
                "margins_accept": ["margins.hip", "common.hpp", "accept_walk.hpp"],
                "attn": ["tree_attn.hip", "common.hpp"],
                "accept": ["accept.hip", "common.hpp", "accept_walk.hpp"],
                "repair": ["repair.hip", "common.hpp"], "commit": ["commit.hip", "common.hpp"]}
# Layers of the cache the commit runs over (a Llama-3-8B-class target).
COMMIT_LAYERS = 32
# Eq. 3 parameters of the repair-tree builder: the paper's b_min, b_max, and a
# margin scale equal to the UFP threshold tau.
B_MIN, B_MAX = 1, 5


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--workload", default=DEFAULT_WORKLOAD)
    p.add_argument("--cpu-seconds", type=float, default=10.0,
                   help="approximate CPU time spent on the oracle baseline (0 = skip)")
    p.add_argument("--no-rotate", action="store_true",
                   help="reuse one input copy (cache-warm numbers; never the headline)")
    p.add_argument("--sweep", action="store_true",
                   help="acceptance-compute trade-off over the repair budgets 0-64 at "
                        "batch 8, context 8192: one line per budget, then the rate model")
    p.add_argument("--layers", type=int, default=32,
                   help="target layers in the sweep's verification cost model")
    p.add_argument("--accept-trees", type=int, default=2048,
                   help="seeded trees per budget for the sweep's mean accepted length")
    p.add_argument("--no-targets", action="store_true",
                   help="skip the bandwidth-bar workloads (ragged batch, long context, "
                        "32- and 64-node repair budgets) measured beside the headline step")
    p.add_argument("--summary", default=None,
                   help="with --sweep: also write the sweep as a markdown summary to this path")
    return p.parse_args()


class Step:
    """Pre-bound C-ABI calls for one input copy (argument marshalling done once)."""

    def __init__(self, pc, torch, w, copy, stream, commit_cache):
        L = pc.lib()
        self.L = L
        self.stream = stream
        dev = torch.device("cuda")
        i32 = dict(dtype=torch.int32, device=dev)
        f32 = dict(dtype=torch.float32, device=dev)
        B, R, V = w.batch, w.n_max, w.vocab
        self.keep = [copy]
        self.m = {k: torch.empty(B, R, **(f32 if k in ("top1_val", "top2_val", "lse", "margin") else i32))
                  for k in ("top1_val", "top1_idx", "top2_val", "top2_idx", "lse", "margin")}
        self.ufp_pos = torch.empty(B, w.chain_len, **i32)
        self.ufp_cnt = torch.empty(B, **i32)
        self.o = torch.empty(B, R, w.hq, w.d, dtype=torch.bfloat16, device=dev)
        self.lse = torch.empty(B, R, w.hq, **f32)
        self.status = torch.empty(B, **i32)
        self.acc = {k: torch.empty(B, **i32) for k in ("acc_len", "best", "bonus", "resync")}
        self.path = torch.empty(B, R, **i32)
        K, budget, depth = w.chain_len, w.repair_budget, w.branch_depth
        self.rep_nmax = K + budget
        self.rep = {"parent": torch.empty(B, self.rep_nmax, **i32),
                    "token": torch.empty(B, self.rep_nmax, **i32),
                    "n_nodes": torch.empty(B, **i32), "branch_cnt": torch.empty(B, K, **i32)}
        self.host_ctx = np.ascontiguousarray(w.ctx_len, np.int32)
        self.host_nn = np.ascontiguousarray(w.n_nodes, np.int32)
        hc = self.host_ctx.ctypes.data_as(ctypes.c_void_p)
        hn = self.host_nn.ctypes.data_as(ctypes.c_void_p)
        mws = L.cure_margins_workspace_size(B, R, V)
        self.mws = torch.zeros(max(mws, 256), dtype=torch.uint8, device=dev)
        aws = L.cure_tree_attn_workspace_size(B, w.hq, w.hkv, w.d, R, hc, hn, 0)
        self.aws = torch.zeros(max(aws, 256), dtype=torch.uint8, device=dev)
        rws = L.cure_repair_tree_workspace_size(B, K, V, budget, depth)
        self.rws = torch.zeros(max(rws, 256), dtype=torch.uint8, device=dev)
        P = lambda t: ctypes.c_void_p(t.data_ptr())
        s = ctypes.c_void_p(stream)
        self.margins_args = (
            P(copy["logits"]), pc.CURE_BF16 if w.dtype == "bf16" else pc.CURE_F32, B, R, V, V,
            P(self.m["top1_val"]), P(self.m["top1_idx"]), P(self.m["top2_val"]),
            P(self.m["top2_idx"]), P(self.m["lse"]), P(self.m["margin"]), w.chain_len,
            ctypes.c_float(w.tau), w.repair_budget, w.branch_depth, P(self.ufp_pos),
            P(self.ufp_cnt), P(self.mws), self.mws.numel(), s)
        self.attn_args = (
            P(copy["q"]), P(copy["k"]), P(copy["v"]), P(self.o), P(self.lse),
            pc.CURE_BF16 if w.dtype == "bf16" else pc.CURE_F32, pc.CURE_BF16, B, w.hq, w.hkv,
            w.d, ctypes.c_float(w.scale), P(copy["kv_off"]), P(copy["ctx_len"]),
            P(copy["n_nodes"]), P(copy["parent"]), R, hc, hn, 0, 0, P(self.status),
            P(self.aws), self.aws.numel(), s)
        self.accept_args = (
            P(copy["parent"]), P(copy["token"]), P(self.m["top1_idx"]), P(copy["root_tgt"]),
            P(copy["n_nodes"]), w.chain_len, B, R, P(self.acc["acc_len"]), P(self.path),
            P(self.acc["best"]), P(self.acc["bonus"]), P(self.acc["resync"]), s)
        # The margin pass with the acceptance walk as its epilogue: the step's
        # margins and accept in the margin pass's two launches.
        self.margins_accept_args = self.margins_args[:18] + (
            P(copy["parent"]), P(copy["token"]), P(copy["root_tgt"]), P(copy["n_nodes"]),
            P(self.acc["acc_len"]), P(self.path), P(self.acc["best"]), P(self.acc["bonus"]),
            P(self.acc["resync"])) + self.margins_args[18:]
        self.repair_args = (
            P(copy["logits"]), pc.CURE_BF16 if w.dtype == "bf16" else pc.CURE_F32, B, R, V, V,
            P(self.m["margin"]), P(self.ufp_pos), P(self.ufp_cnt), P(copy["chain_tok"]), K,
            budget, depth, ctypes.c_float(w.tau), B_MIN, B_MAX, P(copy["suffix"]),
            self.rep_nmax, P(self.rep["parent"]), P(self.rep["token"]),
            P(self.rep["n_nodes"]), P(self.rep["branch_cnt"]), P(self.rws), self.rws.numel(), s)
        if commit_cache is None:                 # the call is not timed here
            return
        ck, cv = commit_cache
        self.com = {k: torch.empty(B, **i32) for k in
                    ("new_ctx_len", "emit_cnt", "replay_start", "status")}
        self.com["emit"] = torch.empty(B, R + 1, **i32)
        self.commit_args = (
            P(ck), P(cv), pc.CURE_BF16 if w.dtype == "bf16" else pc.CURE_F32, ck.shape[0],
            ck.stride(0), w.hkv, w.d, B, P(copy["kv_off"]), P(copy["ctx_len"]),
            P(copy["n_nodes"]), P(self.path), P(self.acc["acc_len"]), P(copy["token"]),
            P(self.acc["bonus"]), w.chain_len, R, P(self.com["new_ctx_len"]),
            P(self.com["emit"]), P(self.com["emit_cnt"]), P(self.com["replay_start"]),
            P(self.com["status"]), s)

    def margins(self):
        st = self.L.cure_margins(*self.margins_args)
        if st:
            raise RuntimeError("cure_margins status %d" % st)

    def attn(self):
        st = self.L.cure_tree_attn(*self.attn_args)
        if st:
            raise RuntimeError("cure_tree_attn status %d" % st)

    def accept(self):
        st = self.L.cure_accept(*self.accept_args)
        if st:
            raise RuntimeError("cure_accept status %d" % st)

    def margins_accept(self):
        st = self.L.cure_margins_accept(*self.margins_accept_args)
        if st:
            raise RuntimeError("cure_margins_accept status %d" % st)

    def repair(self):
        st = self.L.cure_repair_tree(*self.repair_args)
        if st:
            raise RuntimeError("cure_repair_tree status %d" % st)

    def commit(self):
        st = self.L.cure_commit(*self.commit_args)
        if st:
            raise RuntimeError("cure_commit status %d" % st)

    def run(self):
        """One step, in the method's order: the tree-masked verification
        attention with its merge, then the margin pass over the nodes' logits
        with its UFP gate and the acceptance walk on their argmaxes."""
        self.attn()
        self.margins_accept()


def upload_copy(torch, w):
    def dev(a, bf16=False):
        a = np.ascontiguousarray(a)
        if bf16:
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
        return torch.from_numpy(a).cuda()
    bf = w.dtype == "bf16"
    # Suffix tokens the drafter would propose after each substitution: seeded
    # uniform tokens [batch][chain_len][b_max][branch_depth - 1].
    rng = np.random.default_rng(np.random.SeedSequence([w.seed, 99]))
    suffix = rng.integers(0, w.vocab, size=(w.batch, w.chain_len, B_MAX,
                                           max(w.branch_depth - 1, 1))).astype(np.int32)
    return {
        "logits": dev(w.logits, bf), "q": dev(w.q, bf), "k": dev(w.k, bf), "v": dev(w.v, bf),
        "kv_off": dev(w.kv_off), "ctx_len": dev(w.ctx_len), "n_nodes": dev(w.n_nodes),
        "parent": dev(w.parent), "token": dev(w.token), "root_tgt": dev(w.root_tgt),
        "chain_tok": dev(w.token[:, :w.chain_len]), "suffix": dev(suffix),
    }


def replicate(torch, base):
    """A fresh device copy of the large inputs (so each lives at its own address)."""
    c = dict(base)
    for k in ("logits", "q", "k", "v"):
        c[k] = base[k].clone()
    return c


def spin(torch, us):
    """Queue a spin kernel of about `us` microseconds on the current stream."""
    torch.cuda._sleep(int(us * 2400))          # cycles at ~2.4 GHz


def capture(torch, steps, stream):
    """One HIP graph per input copy, each holding one whole step."""
    graphs = []
    for st in steps:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            st.run()
        graphs.append(g)
    return graphs


def timed_steps(torch, graphs, k, warmup):
    """Exactly k graph replays (one step each), bracketed by synchronize()."""
    n = len(graphs)
    for i in range(warmup):
        graphs[i % n].replay()
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    start.record()
    for i in range(k):
        graphs[i % n].replay()
    end.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    return wall * 1e3 / k, start.elapsed_time(end) / k


class _Dim3(ctypes.Structure):
    _fields_ = [("x", ctypes.c_uint32), ("y", ctypes.c_uint32), ("z", ctypes.c_uint32)]


class _KernelNodeParams(ctypes.Structure):
    _fields_ = [("blockDim", _Dim3), ("extra", ctypes.c_void_p), ("func", ctypes.c_void_p),
                ("gridDim", _Dim3), ("kernelParams", ctypes.c_void_p),
                ("sharedMemBytes", ctypes.c_uint)]


def _hip():
    """The HIP runtime this process already uses (the copy torch loaded)."""
    with open("/proc/self/maps") as f:
        paths = sorted({l.split()[-1] for l in f if "libamdhip64" in l.split()[-1]})
    h = ctypes.CDLL(paths[0])
    vp = ctypes.c_void_p
    h.hipGraphGetNodes.argtypes = [vp, ctypes.POINTER(vp), ctypes.POINTER(ctypes.c_size_t)]
    h.hipGraphNodeGetType.argtypes = [vp, ctypes.POINTER(ctypes.c_int)]
    h.hipGraphKernelNodeGetParams.argtypes = [vp, ctypes.POINTER(_KernelNodeParams)]
    h.hipExtLaunchKernel.argtypes = [vp, _Dim3, _Dim3, vp, ctypes.c_size_t, vp, vp, vp,
                                     ctypes.c_int]
    h.hipEventCreate.argtypes = [ctypes.POINTER(vp)]
    h.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), vp, vp]
    h.hipKernelNameRefByPtr.argtypes = [vp, vp]
    h.hipKernelNameRefByPtr.restype = ctypes.c_char_p
    return h


def _check_hip(err, what):
    if err != 0:
        raise RuntimeError("%s failed with hipError %d" % (what, err))


class KernelReplay:
    """The kernels one library call launches, read back from a HIP graph of
    the call (function, grid, block, arguments), so that each can be launched
    on its own between a start and a stop HIP event (hipExtLaunchKernel): the
    per-kernel durations behind the roofline, measured on the launch stream.
    The captured graph is kept alive: it owns the argument copies."""

    def __init__(self, torch, call, stream):
        self.h = _hip()
        self.stream = stream
        self.graph = torch.cuda.CUDAGraph(keep_graph=True)
        with torch.cuda.graph(self.graph, stream=torch.cuda.ExternalStream(stream)):
            call()
        raw = ctypes.c_void_p(self.graph.raw_cuda_graph())
        n = ctypes.c_size_t(0)
        _check_hip(self.h.hipGraphGetNodes(raw, None, ctypes.byref(n)), "hipGraphGetNodes")
        nodes = (ctypes.c_void_p * n.value)()
        _check_hip(self.h.hipGraphGetNodes(raw, nodes, ctypes.byref(n)), "hipGraphGetNodes")
        self.kernels = []
        for i in range(n.value):
            t = ctypes.c_int(-1)
            _check_hip(self.h.hipGraphNodeGetType(nodes[i], ctypes.byref(t)), "hipGraphNodeGetType")
            if t.value != 0:                        # hipGraphNodeTypeKernel
                continue
            prm = _KernelNodeParams()
            _check_hip(self.h.hipGraphKernelNodeGetParams(nodes[i], ctypes.byref(prm)),
                       "hipGraphKernelNodeGetParams")
            name = self.h.hipKernelNameRefByPtr(prm.func, ctypes.c_void_p(stream))
            self.kernels.append((name.decode() if name else "kernel%d" % i, prm))

    def names(self):
        return [k[0] for k in self.kernels]

    def launch(self, idx, ev0, ev1):
        _, prm = self.kernels[idx]
        _check_hip(self.h.hipExtLaunchKernel(prm.func, prm.gridDim, prm.blockDim,
                                             prm.kernelParams, prm.sharedMemBytes,
                                             ctypes.c_void_p(self.stream), ev0, ev1, 0),
                   "hipExtLaunchKernel")


def _short_kernel_name(name):
    """A kernel's symbol as its readable name without namespace and arguments:
    '_ZN4cure12_GLOBAL__N_113tree_attn_m16ILi128ELi8EEEvNS0_4ArgsE' ->
    'tree_attn_m16<128, 8>' (demangled with c++filt when it is there)."""
    import subprocess
    try:
        out = subprocess.run(["c++filt", name], capture_output=True, text=True,
                             timeout=10).stdout.strip()
    except (OSError, subprocess.SubprocessError):
        return name
    if not out or out == name:
        return name
    for pre in ("cure::(anonymous namespace)::", "cure::", "void "):
        out = out.replace(pre, "")
    return out.split("(")[0].strip()


def _stats(samples):
    a = np.asarray(samples, np.float64)
    return {"mean": round(float(a.mean()), 2), "p10": round(float(np.percentile(a, 10)), 2),
            "p50": round(float(np.percentile(a, 50)), 2),
            "p90": round(float(np.percentile(a, 90)), 2), "n": int(a.size)}


def kernel_times(torch, steps, call, k):
    """Event-timed duration samples (µs) of every kernel that `call` launches,
    each launched on its own K times, rotating over the input copies. Returns
    {kernel name: samples}, in launch order."""
    reps = [KernelReplay(torch, getattr(st, call), st.stream) for st in steps]
    h = reps[0].h
    names = reps[0].names()
    out = {}
    for ki, name in enumerate(names):
        evs = []
        for _ in range(k):
            pair = (ctypes.c_void_p(), ctypes.c_void_p())
            _check_hip(h.hipEventCreate(ctypes.byref(pair[0])), "hipEventCreate")
            _check_hip(h.hipEventCreate(ctypes.byref(pair[1])), "hipEventCreate")
            evs.append(pair)
        torch.cuda.synchronize()
        spin(torch, 5000)
        for i in range(k):
            reps[i % len(reps)].launch(ki, evs[i][0], evs[i][1])
        torch.cuda.synchronize()
        samples = []
        for e0, e1 in evs:
            ms = ctypes.c_float(0)
            _check_hip(h.hipEventElapsedTime(ctypes.byref(ms), e0, e1), "hipEventElapsedTime")
            samples.append(ms.value * 1e3)
            h.hipEventDestroy(e0)
            h.hipEventDestroy(e1)
        out[_short_kernel_name(name)] = samples
    del reps
    return out


CALLS = ("margins", "attn", "accept", "margins_accept", "repair", "commit")


def per_call_samples(torch, steps, k, calls=CALLS, warmup=0):
    """GPU duration samples (µs) of each call, from HIP events around every
    eager launch on the launch stream, k rounds rotating over the input copies.
    A spin kernel queued first keeps the host's launch cost off the GPU
    timeline."""
    n = len(steps)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(len(calls) + 1)] for _ in range(k)]
    for i in range(warmup):
        for name in calls:
            getattr(steps[i % n], name)()
    torch.cuda.synchronize()
    spin(torch, 25000)
    for i in range(k):
        s = steps[i % n]
        ev[i][0].record()
        for j, name in enumerate(calls):
            getattr(s, name)()
            ev[i][j + 1].record()
    torch.cuda.synchronize()
    return {name: [ev[i][j].elapsed_time(ev[i][j + 1]) * 1e3 for i in range(k)]
            for j, name in enumerate(calls)}


def stored_traffic(call, workload):
    """HBM bytes per call from the committed rocprofv3 FETCH_SIZE/WRITE_SIZE summary
    (calibrated against a plain copy), or None when there is none for this workload
    or the call's kernel sources changed since it was taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "traffic_%s.json" % workload)
    if not os.path.exists(path):
        return None
    with open(path) as f:
        entry = json.load(f).get("calls", {}).get(call)
    if not entry:
        return None
    h = hashlib.sha256()
    for name in CALL_SOURCES[call]:
        with open(os.path.join(CSRC, name), "rb") as f:
            h.update(f.read())
    return int(entry["bytes_per_call"]) if h.hexdigest() == entry["sources_sha256"] else None


def attention_flops(w):
    """Algorithmic flops of one cure_tree_attn call: 2 * D for each of Q K^T and P V
    over every visible (query head, key) pair. Node n of sequence b sees the ctx_len[b]
    context rows and the depth(n) + 1 nodes of its root path, with depths taken from the
    workload's parent array; masked pairs are not counted."""
    total = 0
    for b in range(w.batch):
        depth = []
        for n in range(int(w.n_nodes[b])):
            p = int(w.parent[b][n])
            depth.append(0 if p < 0 else depth[p] + 1)
        visible = sum(int(w.ctx_len[b]) + dn + 1 for dn in depth)
        total += 4 * w.hq * w.d * visible
    return total


def repair_bytes(w, step):
    """Algorithmic bytes of one cure_repair_tree call, from what it produced: the
    logits rows of the UFPs that received branches (the rows that must be
    ranked), the UFP list, count and margins, the draft block, the suffix tokens
    of the granted branches, and the parent/token arrays, node count and
    per-UFP branch counts written."""
    bc = step.rep["branch_cnt"].cpu().numpy()
    nn = step.rep["n_nodes"].cpu().numpy()
    eb = w.elem_bytes()
    ranked = int((bc > 0).sum())
    branches = int(bc.sum())
    K = w.chain_len
    total = (ranked * w.vocab * eb + w.batch * (3 * K * 4 + 4)
             + branches * (w.branch_depth - 1) * 4
             + int(nn.sum()) * 8 + w.batch * (4 + K * 4))
    info = {"rows_ranked": ranked, "branches": branches, "nodes": int(nn.sum()),
            "bytes": total}
    return total, info


def read_ceiling(torch, pc, reps=20, nbytes=1 << 30):
    """The practical HBM read rate on this GPU: cure_read_ceiling (a plain
    non-temporal streaming read, one workgroup per 256 KB) over a 1 GiB buffer,
    four times the last-level cache, median of `reps` event-timed reads."""
    buf = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
    pc.cure_read_ceiling(buf)
    torch.cuda.synchronize()
    ev[0].record()
    for i in range(reps):
        pc.cure_read_ceiling(buf)
        ev[i + 1].record()
    torch.cuda.synchronize()
    us = sorted(ev[i].elapsed_time(ev[i + 1]) * 1e3 for i in range(reps))[reps // 2]
    gbs = nbytes / (us * 1e-6) / 1e9
    del buf
    return {"GB/s": round(gbs, 1), "frac_hbm": round(gbs / HBM_PEAK_GBS, 4), "bytes": nbytes,
            "kernel": "cure_read_ceiling (read_ceiling_kernel)"}


def commit_bytes(w, step, layers):
    """Algorithmic bytes of one cure_commit call, from the acceptance results it
    committed: each moved cache row (path[j] != j) read once and written once,
    in K and V of every layer, plus the per-sequence sizes, the path and token
    entries read and the emitted tokens and counters written."""
    acc = step.acc["acc_len"].cpu().numpy()
    path = step.path.cpu().numpy()
    row = w.hkv * w.d * w.elem_bytes()
    moved = 0
    for b in range(w.batch):
        a = max(int(acc[b]), 0)
        moved += a - sum(1 for j in range(a) if int(path[b][j]) == j)
    tokens = int(np.maximum(acc, 0).sum())
    total = (moved * row * 2 * 2 * layers + w.batch * 8 * 4 + tokens * 8
             + (tokens + w.batch) * 4 + w.batch * 16)
    return total, {"layers": layers, "rows_moved": moved, "bytes": total}


def _oracle_steps(w, budget_s):
    """Whole oracle steps of workload w for about budget_s seconds: (steps, s/step)."""
    import oracle
    t0 = time.perf_counter()
    reps = 0
    while True:
        for b in range(w.batch):
            m = oracle.margins(w.logits[b], w.dtype)
            oracle.ufp_select(m["margin_f32"][: w.chain_len], w.tau, w.repair_budget,
                              w.branch_depth)
            oracle.accept(w.parent[b], w.token[b], m["top1_idx"], int(w.root_tgt[b]),
                          int(w.n_nodes[b]), w.chain_len)
        oracle.tree_attention(w.q, w.k, w.v, w.dtype, w.kv_off, w.ctx_len, w.n_nodes,
                              w.parent, w.hq, w.hkv, w.scale)
        reps += 1
        if time.perf_counter() - t0 >= budget_s:
            break
    return reps, (time.perf_counter() - t0) / reps


def cpu_baseline(w, algo_bytes, budget_s):
    """The CPU oracle on this host over the same workload: about budget_s seconds
    with the BLAS thread pool at its default size (the threads the oracle's
    matrix-vector products use; its sorts and walks run on one thread), then
    about budget_s / 2 seconds with one thread in all."""
    import threadpoolctl
    host_cores = len(os.sched_getaffinity(0))
    info = threadpoolctl.threadpool_info()
    threads = max([i.get("num_threads", 1) for i in info if i.get("user_api") == "blas"] or [1])
    reps, dt = _oracle_steps(w, budget_s)
    with threadpoolctl.threadpool_limits(limits=1):
        reps1, dt1 = _oracle_steps(w, budget_s / 2)
    return {"value": round(algo_bytes / dt / 1e9, 4), "unit": "GB/s", "cores": int(threads),
            "host_cores": host_cores, "kind": "oracle", "ms_per_step": round(dt * 1e3, 1),
            "single_thread": {"value": round(algo_bytes / dt1 / 1e9, 4), "unit": "GB/s",
                              "cores": 1, "ms_per_step": round(dt1 * 1e3, 1), "steps": reps1},
            "sample": "%d full oracle step(s) of workload %s (margins+UFP and accept per "
                      "sequence, float64 tree attention for every node and head) with %d "
                      "BLAS threads (sorts and walks on one thread), then %d step(s) on one "
                      "thread; host has %d cores available" % (reps, w.name, threads, reps1,
                                                               host_cores)}


def measure(w, args, torch, pc):
    """Times one workload's step (and the calls beside it); returns the JSON line."""
    from synth import algorithmic_bytes
    ab = algorithmic_bytes(w)
    step_bytes = ab["attention"] + ab["margins"] + ab["accept"]
    base = upload_copy(torch, w)
    per_copy = sum(base[k].numel() * base[k].element_size() for k in ("logits", "q", "k", "v"))
    ncopy = 1 if args.no_rotate else max(3, math.ceil(ROTATE_BYTES / per_copy))
    copies = [base] + [replicate(torch, base) for _ in range(ncopy - 1)]
    # The commit's cache: COMMIT_LAYERS layers of the workload's K and V rows.
    # Its contents do not change the work, so it is left uninitialised.
    cdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    commit_cache = tuple(torch.empty(COMMIT_LAYERS, w.kv_rows, w.hkv, w.d, dtype=cdt,
                                     device="cuda") for _ in range(2))
    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        steps = [Step(pc, torch, w, c, stream.cuda_stream, commit_cache) for c in copies]
        for st in steps:                       # eager reference results, one per copy
            st.run()
            st.repair()
            st.commit()
        torch.cuda.synchronize()
        ref = [(st.m["top1_idx"].clone(), st.acc["acc_len"].clone(), st.o.clone())
               for st in steps]
        graphs = capture(torch, steps, stream)
        ms, ev_ms = timed_steps(torch, graphs, args.steps, args.warmup)
        # Every graph's last replay must reproduce the eager results.
        for st, (t1, al, o) in zip(steps, ref):
            assert torch.equal(st.m["top1_idx"], t1) and torch.equal(st.acc["acc_len"], al)
            assert torch.equal(st.o, o)
        k_calls = min(args.steps, 100)
        call_samples = per_call_samples(torch, steps, k_calls)
        kern = {c: kernel_times(torch, steps, c, k_calls) for c in ("margins_accept", "attn")}
    calls = {c: float(np.mean(v)) for c, v in call_samples.items()}
    status = steps[0].status.cpu().tolist()
    assert status == [0] * w.batch, status
    acc_len = steps[0].acc["acc_len"].float().cpu()
    rep_bytes, rep_info = repair_bytes(w, steps[0])
    com_bytes, com_info = commit_bytes(w, steps[0], COMMIT_LAYERS)
    assert steps[0].com["status"].cpu().tolist() == [0] * w.batch

    call_bytes = {"margins": ab["margins"], "attn": ab["attention"], "accept": ab["accept"],
                  "margins_accept": ab["margins"] + ab["accept"],
                  "repair": rep_bytes, "commit": com_bytes}
    kernels = {}
    for name, us in calls.items():
        gbs = call_bytes[name] / (us * 1e-6) / 1e9
        kernels[name] = dict(us=round(us, 2), **{k: v for k, v in _stats(call_samples[name]).items()
                                                 if k != "mean"},
                             **{"GB/s": round(gbs, 1), "frac_hbm": round(gbs / HBM_PEAK_GBS, 4)})
    # Kernel level: every kernel of the step's calls launched on its own between
    # HIP events. The dominant kernel is the longest; its call's algorithmic
    # bytes are all attributed to it (the others move only partials or results).
    kernel_level = {}
    for c, ks in kern.items():
        for kname, samples in ks.items():
            kernel_level[kname] = dict(call=c, **_stats(samples))
    dom_k = max(kernel_level, key=lambda n: kernel_level[n]["mean"])
    dom = kernel_level[dom_k]["call"]
    dom_us = kernel_level[dom_k]["mean"]
    dom_gbs = call_bytes[dom] / (dom_us * 1e-6) / 1e9
    call_gbs = call_bytes[dom] / (calls[dom] * 1e-6) / 1e9
    value = step_bytes / (ms * 1e-3) / 1e9
    attn_flops = attention_flops(w)
    attn_k = max((n for n in kernel_level if kernel_level[n]["call"] == "attn"),
                 key=lambda n: kernel_level[n]["mean"])
    attn_tf = attn_flops / (kernel_level[attn_k]["mean"] * 1e-6) / 1e12
    attn_tf_call = attn_flops / (calls["attn"] * 1e-6) / 1e12
    line = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": w.name, "batch": w.batch, "ctx_len": int(w.ctx_len.max()),
                   "tree_nodes": int(w.n_nodes.max()), "hq": w.hq, "hkv": w.hkv, "d": w.d,
                   "vocab": w.vocab, "chain_len": w.chain_len, "repair_budget": w.repair_budget,
                   "parallelism": "single-gpu", "input_copies": ncopy},
        "step_latency_us": round(ms * 1e3, 2),
        "kv_gbps": round(ab["attention_kv"] / (calls["attn"] * 1e-6) / 1e9, 1),
        "event_ms_per_step": round(ev_ms, 5),
        "kernels": kernels,
        # Mean accepted draft length of the step's sequences (tokens emitted = +1).
        "acc_len_mean": round(float(acc_len.mean()), 3),
        "kernel_level": kernel_level,
        "roofline": {"bound": "hbm", "kernel": dom_k, "call": dom,
                     "achieved": round(dom_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(dom_gbs / HBM_PEAK_GBS, 4),
                     "kernel_us": dom_us, "bytes": call_bytes[dom],
                     "call_us": round(calls[dom], 2),
                     "call_frac": round(call_gbs / HBM_PEAK_GBS, 4),
                     "traffic": stored_traffic(dom, w.name)},
        # The attention kernel against its other bound, the bf16 matrix cores (it
        # reaches the ridge only for the widest trees).
        "attn_mfma": {"bound": "mfma", "kernel": attn_k,
                      "achieved": round(attn_tf, 1), "peak": MFMA_BF16_PEAK_TFLOPS,
                      "unit": "TFLOP/s", "frac": round(attn_tf / MFMA_BF16_PEAK_TFLOPS, 4),
                      "call_frac": round(attn_tf_call / MFMA_BF16_PEAK_TFLOPS, 4),
                      "flops": attn_flops},
        "repair_tree": dict(rep_info, us=round(calls["repair"], 2),
                            roofline={"bound": "hbm", "kernel": "cure_repair_tree (topk_chunk "
                                      "+ repair_assemble)",
                                      "achieved": kernels["repair"]["GB/s"],
                                      "peak": HBM_PEAK_GBS, "unit": "GB/s",
                                      "frac": kernels["repair"]["frac_hbm"],
                                      "traffic": stored_traffic("repair", w.name)}),
        "commit": dict(com_info, us=round(calls["commit"], 2),
                       roofline={"bound": "hbm", "kernel": "cure_commit (commit_kernel)",
                                 "achieved": kernels["commit"]["GB/s"],
                                 "peak": HBM_PEAK_GBS, "unit": "GB/s",
                                 "frac": kernels["commit"]["frac_hbm"],
                                 "traffic": stored_traffic("commit", w.name)}),
    }
    line["read_ceiling"] = read_ceiling(torch, pc)
    if args.cpu_seconds > 0:
        line["cpu_baseline"] = cpu_baseline(w, step_bytes, args.cpu_seconds)
    return line

# The bandwidth bars: the verification attention at 70 % and the margin pass at
# 80 % of the HBM peak, on the workloads where each is judged.
TARGETS = (
    ("llama3_8b_ragged_b16", (("margins", 0.80), ("attn", 0.70))),
    ("llama3_8b_ctx32k_b4", (("attn", 0.70),)),
    ("llama3_8b_ctx8k_b8_budget32", (("attn", 0.70),)),
    ("llama3_8b_ctx8k_b8_budget64", (("attn", 0.70),)),
)


def measure_targets(args, torch, pc):
    """For each bar: the call's duration (HIP events around each eager call)
    and the duration of each of its kernels launched on its own (HIP events on
    the launch stream), with mean, p10, median and p90 over 200 launches after
    20 warm-up calls, rotating over >= 512 MB of input copies; the fraction of
    the HBM peak at call and at kernel level (algorithmic bytes over the mean,
    and over the median); the stored per-call HBM traffic."""
    from synth import algorithmic_bytes, preset
    k = 200
    out = {}
    for wname, checks in TARGETS:
        w = preset(wname)
        ab = algorithmic_bytes(w)
        base = upload_copy(torch, w)
        per_copy = sum(base[c].numel() * base[c].element_size() for c in ("logits", "q", "k", "v"))
        ncopy = max(3, math.ceil(ROTATE_BYTES / per_copy))
        copies = [base] + [replicate(torch, base) for _ in range(ncopy - 1)]
        stream = torch.cuda.Stream()
        names = tuple(c for c, _ in checks)
        with torch.cuda.stream(stream):
            steps = [Step(pc, torch, w, c, stream.cuda_stream, None) for c in copies]
            for st in steps:
                st.run()
            torch.cuda.synchronize()
            assert steps[0].status.cpu().tolist() == [0] * w.batch
            samples = per_call_samples(torch, steps, k, calls=names, warmup=20)
            kern = {c: kernel_times(torch, steps, c, k) for c in names}
        flops = attention_flops(w)
        for c, bar in checks:
            nbytes = ab["margins"] if c == "margins" else ab["attention"]
            cs = _stats(samples[c])
            ks = {n: _stats(v) for n, v in kern[c].items()}
            dom = max(ks, key=lambda n: ks[n]["mean"])
            frac = lambda us: round(nbytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)
            traffic = stored_traffic(c, wname)
            entry = {"workload": wname, "call": c, "bar": bar, "bytes": nbytes,
                     "call_us": cs, "kernels": ks, "dominant_kernel": dom,
                     "frac": {"call": frac(cs["mean"]), "kernel": frac(ks[dom]["mean"]),
                              "call_p50": frac(cs["p50"]), "kernel_p50": frac(ks[dom]["p50"])},
                     "bar_call_us": round(nbytes / (bar * HBM_PEAK_GBS * 1e9) * 1e6, 2),
                     "traffic": traffic,
                     "traffic_ratio": round(traffic / nbytes, 4) if traffic else None}
            if c == "attn":
                tf = lambda us: round(flops / (us * 1e-6) / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4)
                entry["flops"] = flops
                entry["mfma_frac"] = {"call": tf(cs["mean"]), "kernel": tf(ks[dom]["mean"])}
            out["%s@%s" % (c, wname)] = entry
            print("[targets] %s %s: call %.2f us (p50 %.2f), %s %.2f us, frac call %.3f "
                  "kernel %.3f (bar %.2f)" % (wname, c, cs["mean"], cs["p50"], dom,
                                              ks[dom]["mean"], entry["frac"]["call"],
                                              entry["frac"]["kernel"], bar),
                  file=sys.stderr, flush=True)
        del steps, copies, base, w
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
    return out


SWEEP_BUDGETS = (0, 8, 16, 32, 64)
# Parameters of a Llama-3-8B-class target for the sweep's cost model: its
# weights are streamed once per verification pass.
TARGET_PARAMS = 8.03e9
TARGET_BYTES_PER_PARAM = 2


def mean_accepted(pc, torch, budget, n_trees, seed):
    """Mean accepted length E[a] (and E[a] + 1 tokens per step) over n_trees
    seeded trees of the sweep's shape (chain 16, depth-4 branches at seeded
    positions), against the synthetic target that agrees with each node with
    probability 0.8 i.i.d., computed by cure_accept on the GPU."""
    from synth import make_workload
    w = make_workload("accept_sample", dtype="f32", batch=n_trees, hq=1, hkv=1, d=4, vocab=64,
                      ctx_lens=[1] * n_trees, chain_len=16, n_ufp=budget // 4, branch_depth=4,
                      seed=700 + seed, p_agree=0.8)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()
    out = pc.cure_accept(t(w.parent), t(w.token), t(w.tgt_planted), t(w.root_tgt), t(w.n_nodes),
                         w.chain_len)
    acc = out["acc_len"].float().cpu().numpy()
    assert acc.min() >= 0
    return float(acc.mean()), float(acc.std() / math.sqrt(len(acc))), float(out["resync"].float().mean())


def tpot_model(c_d_us, c_v_us, mean_accepted):
    """Sec. 3.1's cost model per sequence: one decoding step costs the draft
    overhead C_d plus the verification cost C_v and emits the E[a] accepted
    draft tokens plus the bonus token, so the time per output token is
    (C_d + C_v) / (E[a] + 1) (microseconds)."""
    return (c_d_us + c_v_us) / (mean_accepted + 1.0)


def rate_model(mean_accepted, batch, c_d_us, c_v_us):
    """Sec. 3.1's generation rate, (E[a] + 1) / (C_d + C_v) per sequence, for a
    batch of sequences verified together: output tokens per second."""
    return batch / (tpot_model(c_d_us, c_v_us, mean_accepted) * 1e-6)


def speedup(tpot_ref, tpot):
    """Speedup as Table 1 reports it (Sec. 4.1's metric): the ratio of the
    reference's time per output token to the method's."""
    return tpot_ref / tpot


def accept_gain(accepted_ref, accepted):
    """Relative gain in accepted tokens per step over a reference (Sec. 4.2
    quotes the gain over the single-path parallel draft this way)."""
    return accepted / accepted_ref - 1.0


def verify_cost(layers, attn_us, margins_us, accept_us, weights_us):
    """C_v(N) of the sweep: every target layer's verification attention over the
    tree, the margin pass over the node logits, the acceptance walk, and one
    streaming read of the target's weights."""
    return layers * attn_us + margins_us + accept_us + weights_us


def rate_table(rows, t_weights_us, layers, batch, ratios=(0.25, 0.5, 1.0, 2.0)):
    """The sweep's rate model over measured rows.

    rows: dicts with budget, tree_nodes, mean_accepted and the measured attn_us,
    margins_us, accept_us of that budget's step. For each draft cost C_d =
    ratio x t_weights it adds the modelled tokens/s of every row and picks the
    budget with the highest rate (its gain over budget 0 is the speedup of its
    time per output token over budget 0's). Returns (table, best)."""
    table = []
    for row in rows:
        cv = verify_cost(layers, row["attn_us"], row["margins_us"], row["accept_us"], t_weights_us)
        table.append({"budget": row["budget"], "tree_nodes": row["tree_nodes"],
                      "mean_accepted": row["mean_accepted"], "attn_us": row["attn_us"],
                      "c_v_us": round(cv, 1), "_cv": cv})
    best = {}
    for ratio in ratios:
        cd = ratio * t_weights_us
        scored = []
        for row in table:
            rate = rate_model(row["mean_accepted"], batch, cd, row["_cv"])
            row["tokens_per_s_cd%.2g" % ratio] = round(rate, 1)
            scored.append((rate, -row["budget"], row))
        top = max(scored, key=lambda s: (s[0], s[1]))[2]
        base = table[0]
        gain = speedup(tpot_model(cd, base["_cv"], base["mean_accepted"]),
                       tpot_model(cd, top["_cv"], top["mean_accepted"]))
        best["cd_%.2g_x_weights" % ratio] = {
            "budget": top["budget"],
            "tokens_per_s": round(rate_model(top["mean_accepted"], batch, cd, top["_cv"]), 1),
            "gain_vs_budget0": round(gain, 4)}
    for row in table:
        del row["_cv"]
    return table, best


def write_sweep_summary(args, rows, summary):
    """The sweep as a short markdown summary: per budget the tree size, the
    measured call times, E[a] with its standard error, and the modelled rate per
    draft cost, then the best budget per draft cost."""
    cmd = "python3 bench.py --sweep --steps %d --warmup %d --cpu-seconds %g --accept-trees %d " \
          "--layers %d --summary %s" % (args.steps, args.warmup, args.cpu_seconds,
                                        args.accept_trees, args.layers, args.summary)
    out = ["# Acceptance-compute sweep: batch 8, context 8192, chain 16, depth-4 branches", "",
           "Command (from the repository root):", "", "    " + cmd, "",
           "Measured on this GPU: the per-call times (HIP events, mean of the eager "
           "calls) and E[a] (cure_accept over %d seeded trees per budget against the "
           "synthetic target that agrees with each node with probability 0.8). Modelled: "
           "C_v = %d x attention + margins + accept + one read of the target's weights "
           "(%.1f µs at the margin pass's %.1f GB/s), and C_d in multiples of that "
           "read. Rate = (E[a] + 1) x %d / (C_d + C_v)."
           % (args.accept_trees, summary["layers"], summary["t_weights_us"],
              summary["weights_gbps"], summary["batch"]), ""]
    ratios = [k for k in summary["rows"][0] if k.startswith("tokens_per_s_cd")]
    head = ["budget", "nodes", "attention µs", "attention frac of 8 TB/s", "margins µs",
            "accept µs", "step µs", "E[a] ± se", "C_v µs"] + \
           ["tok/s, C_d = %s x weights" % k[len("tokens_per_s_cd"):] for k in ratios]
    out.append("| " + " | ".join(head) + " |")
    out.append("|" + "---|" * len(head))
    for r, t in zip(rows, summary["rows"]):
        cells = [r["budget"], r["tree_nodes"], r["attn_us"], r["attn_frac_hbm"], r["margins_us"],
                 r["accept_us"], r["step_us"], "%.3f ± %.3f" % (r["mean_accepted"],
                                                             r["mean_accepted_se"]),
                 t["c_v_us"]] + [t[k] for k in ratios]
        out.append("| " + " | ".join(str(c) for c in cells) + " |")
    out += ["", "Best budget per draft cost:", ""]
    for k, v in summary["best_budget"].items():
        out.append("* C_d = %s x weights: budget %d, %.1f tok/s, %.4f x budget 0's rate"
                   % (k[len("cd_"):-len("_x_weights")], v["budget"], v["tokens_per_s"],
                      v["gain_vs_budget0"]))
    os.makedirs(os.path.dirname(os.path.abspath(args.summary)), exist_ok=True)
    with open(args.summary, "w") as f:
        f.write("\n".join(out) + "\n")


def sweep(args, torch, pc):
    """Acceptance-compute trade-off (Sec. 3.1's rate model): for each repair
    budget, the measured verify step and the mean accepted length, then the
    modelled generation rate (E[a] + 1) / (C_d + C_v(N)) with

      C_v(N) = layers x t_attn(N) + t_margins(N) + t_accept + t_weights,

    t_attn, t_margins, t_accept measured here for the budget's tree (N nodes
    per sequence), t_weights = the target's weight bytes at the measured margin
    pass bandwidth (one streaming read of the weights per verification pass),
    and a synthetic draft cost C_d given as multiples of t_weights (the paper's
    drafter is a target-sized block-parallel model: one forward, C_d ~ t_weights).
    The budget that maximises the rate is reported per C_d; with --summary the
    per-budget figures and that choice are also written as a markdown table."""
    from synth import preset
    rows = []
    batch = None
    for budget in SWEEP_BUDGETS:
        w = preset("llama3_8b_ctx8k_b8_budget%d" % budget)
        batch = w.batch
        line = measure(w, args, torch, pc)
        ea, ea_se, resync = mean_accepted(pc, torch, budget, args.accept_trees, budget)
        line["sweep"] = {"budget": budget, "tree_nodes": int(w.n_nodes.max()),
                         "mean_accepted": round(ea, 4), "mean_accepted_se": round(ea_se, 4),
                         "resync_rate": round(resync, 4), "accept_trees": args.accept_trees}
        print(json.dumps(line), flush=True)
        k = line["kernels"]
        rows.append({"budget": budget, "tree_nodes": int(w.n_nodes.max()),
                     "mean_accepted": round(ea, 4), "mean_accepted_se": round(ea_se, 4),
                     "attn_us": k["attn"]["us"], "margins_us": k["margins"]["us"],
                     "accept_us": k["accept"]["us"], "step_us": line["step_latency_us"],
                     "margins_gbps": k["margins"]["GB/s"],
                     "attn_frac_hbm": k["attn"]["frac_hbm"]})
        del w
    # Weight streaming at the bandwidth the margin pass reached on this GPU.
    bw = max(r["margins_gbps"] for r in rows) * 1e9
    t_weights = TARGET_PARAMS * TARGET_BYTES_PER_PARAM / bw * 1e6
    table, best = rate_table(rows, t_weights, args.layers, batch)
    summary = {
        "model": "rate = (E[a] + 1) * batch / (C_d + C_v(N)); C_v = layers * attn + margins + "
                 "accept + weight streaming; C_d synthetic, in multiples of the weight stream",
        "layers": args.layers, "batch": batch, "t_weights_us": round(t_weights, 1),
        "weights_gbps": round(bw / 1e9, 1), "rows": table, "best_budget": best}
    print(json.dumps({"sweep_summary": summary}), flush=True)
    if args.summary:
        write_sweep_summary(args, rows, summary)


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(--gpus %d requested)" % args.gpus, file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2608_00531_amd as pc
    from synth import preset

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.sweep:
        sweep(args, torch, pc)
        return
    line = measure(preset(args.workload), args, torch, pc)
    if not args.no_targets:
        line["targets"] = measure_targets(args, torch, pc)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
