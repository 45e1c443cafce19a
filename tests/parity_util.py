"""Shared helpers for the GPU parity tests: upload a synthetic workload, run the
HIP path through the C ABI, run the oracle on the same bytes, compare.

Tolerances (fixed for this path): indices, UFP lists, accepted lengths and
paths bit-exact; margins and log-sum-exp within 1e-3 absolute; attention output
within 1e-5 (fp32 inputs) or 2e-2 (bf16 inputs) max-abs of the float64 oracle
on the same input bytes, attention log-sum-exp within 1e-4 / 4e-3.
"""

import sys
import time

import numpy as np
import torch

import oracle
import paper_2608_00531_amd as pc

MARGIN_TOL = 1e-3
ATTN_TOL = {"f32": 1e-5, "bf16": 2e-2}
# Attention log-sum-exp (no bound is fixed for it, so it is derived from the
# arithmetic). bf16: the matrix-core kernels sum the probabilities as rounded
# to bf16 for the P V product (so the output's normalisation matches its
# numerator); each term then carries a relative error of at most 2^-8, the
# unit roundoff of bf16's 8-bit significand, so the sum's relative error is at
# most 2^-8 and the log-sum-exp is off by at most ln(1 + 2^-8) = 3.9e-3, which
# a node that sees only a few keys (one of them dominant) reaches. fp32: the
# vector-ALU kernel sums ~10^3 fp32 terms, relative error ~ L * 2^-24.
LSE_TOL = {"f32": 1e-4, "bf16": 4e-3}


def say(*msg):
    print("[parity]", *msg, flush=True)
    sys.stdout.flush()


def to_dev(a, dtype):
    """numpy -> cuda tensor. dtype 'bf16' means a is raw uint16 bf16 bits."""
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def upload(w):
    d = {
        "logits": to_dev(w.logits, w.dtype),
        "q": to_dev(w.q, w.dtype), "k": to_dev(w.k, w.dtype), "v": to_dev(w.v, w.dtype),
        "kv_off": torch.from_numpy(w.kv_off).cuda(),
        "ctx_len": torch.from_numpy(w.ctx_len).cuda(),
        "n_nodes": torch.from_numpy(w.n_nodes).cuda(),
        "parent": torch.from_numpy(w.parent).cuda(),
        "token": torch.from_numpy(w.token).cuda(),
        "root_tgt": torch.from_numpy(w.root_tgt).cuda(),
    }
    return d


def gpu_margins(w, dev, gate=True):
    return pc.cure_margins(dev["logits"], chain_len=w.chain_len if gate else 0, tau=w.tau,
                           repair_budget=w.repair_budget, branch_depth=w.branch_depth,
                           gate=gate)


def check_margins(w, got, rows=None, sample_batches=None):
    """Compare GPU margins (dict of tensors [batch, rows]) with the oracle."""
    bs = range(w.batch) if sample_batches is None else sample_batches
    for b in bs:
        ref = oracle.margins(w.logits[b], w.dtype)
        g = {k: v[b].cpu().numpy() for k, v in got.items() if v.dim() == 2 and k != "ufp_pos"}
        assert np.array_equal(g["top1_idx"], ref["top1_idx"]), ("top1_idx", b)
        assert np.array_equal(g["top2_idx"], ref["top2_idx"]), ("top2_idx", b)
        assert np.array_equal(g["top1_val"], ref["top1_val"]), ("top1_val", b)
        assert np.array_equal(g["top2_val"], ref["top2_val"]), ("top2_val", b)
        assert np.array_equal(g["margin"], ref["margin_f32"], equal_nan=True), ("margin", b)
        fin = np.isfinite(ref["lse"])
        assert np.array_equal(np.isfinite(g["lse"]), fin)
        assert np.max(np.abs(g["lse"][fin] - ref["lse"][fin]), initial=0) <= MARGIN_TOL, ("lse", b)
        if "ufp_pos" in got:
            want = oracle.ufp_select(ref["margin_f32"][: w.chain_len], w.tau, w.repair_budget,
                                     w.branch_depth)
            pos = got["ufp_pos"][b].cpu().numpy()
            cnt = int(got["ufp_cnt"][b])
            assert cnt == len(want), ("ufp_cnt", b, cnt, want)
            assert list(pos[:cnt]) == want, ("ufp_pos", b)
            assert np.all(pos[cnt:] == -1)


def gpu_attn(w, dev, out_dtype=None, kv_split=0, flags=0):
    return pc.cure_tree_attn(dev["q"], dev["k"], dev["v"], dev["kv_off"], dev["ctx_len"],
                             dev["n_nodes"], dev["parent"], w.ctx_len, w.n_nodes, w.scale,
                             out_dtype=out_dtype, kv_split=kv_split, flags=flags)


def oracle_attn(w, sample=None):
    return oracle.tree_attention(w.q, w.k, w.v, w.dtype, w.kv_off, w.ctx_len, w.n_nodes,
                                 w.parent, w.hq, w.hkv, w.scale, sample=sample)


def check_attn(w, o, lse, ref_o, ref_lse, sample=None):
    o = o.float().cpu().numpy()
    lse = lse.cpu().numpy()
    pairs = sample if sample is not None else [
        (b, n) for b in range(w.batch) for n in range(int(w.n_nodes[b]))]
    worst_o = worst_l = 0.0
    for b, n in pairs:
        worst_o = max(worst_o, float(np.max(np.abs(o[b, n] - ref_o[b, n]))))
        worst_l = max(worst_l, float(np.max(np.abs(lse[b, n] - ref_lse[b, n]))))
    say("attention max-abs O %.3g  LSE %.3g over %d nodes" % (worst_o, worst_l, len(pairs)))
    assert worst_o <= ATTN_TOL[w.dtype], worst_o
    assert worst_l <= LSE_TOL[w.dtype], worst_l


def check_accept(w, got, tgt):
    for b in range(w.batch):
        ref = oracle.accept(w.parent[b], w.token[b], tgt[b], int(w.root_tgt[b]),
                            int(w.n_nodes[b]), w.chain_len)
        assert int(got["acc_len"][b]) == ref["acc_len"], b
        assert int(got["best"][b]) == ref["best"], b
        assert int(got["bonus"][b]) == ref["bonus"], b
        assert int(got["resync"][b]) == ref["resync"], b
        path = got["path"][b].cpu().numpy()
        assert list(path[: ref["acc_len"]]) == ref["path"], b
        assert np.all(path[ref["acc_len"]:] == -1), b


class Timer:
    def __init__(self, what):
        self.what = what

    def __enter__(self):
        self.t = time.time()
        return self

    def __exit__(self, *a):
        say("%s: %.2fs" % (self.what, time.time() - self.t))
