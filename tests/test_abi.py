"""C-ABI checks that need no GPU: the library loads, exports every entry point
declared in include/cure.h, and rejects bad arguments before touching a device.

Calls here pass fake device pointers, so every call is built to stop at a
host-side argument check: none may reach a kernel launch (these tests must be
safe on a GPU machine too).
"""

import ctypes
import os
import re

import numpy as np
import pytest

import paper_2608_00531_amd as pc
from paper_2608_00531_amd import build as pbuild

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                      "include", "cure.h")


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(pbuild.LIB_PATH):
        pbuild.build_library()
    return pc.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(cure_[a-z_0-9]+)\s*\(", text)))


def test_header_declares_the_three_entry_points():
    names = declared_functions()
    for fn in ("cure_margins", "cure_tree_attn", "cure_accept"):
        assert fn in names


def test_every_declared_symbol_is_exported(L):
    for name in declared_functions():
        assert hasattr(L, name), name


def test_status_strings_and_version(L):
    assert L.cure_status_string(0) == b"CURE_OK"
    assert L.cure_status_string(3) == b"CURE_ERR_BAD_TREE"
    assert L.cure_status_string(99) == b"CURE_ERR_UNKNOWN"
    assert L.cure_version() >= 100


def _margins(L, **kw):
    # vocab 100000 over 4 rows always plans several chunks per row, so a
    # missing workspace is reported before any launch.
    args = dict(logits=1, dtype=1, batch=1, rows=4, vocab=100000, ld=100000,
                top1_val=1, top1_idx=1, top2_val=1, top2_idx=1, lse=1, margin=1,
                chain_len=2, tau=1.0, repair_budget=4, branch_depth=2, ufp_pos=1, ufp_cnt=1,
                workspace=None, ws_bytes=0, stream=None)
    args.update(kw)
    return L.cure_margins(*args.values())


def test_margins_argument_errors(L):
    assert _margins(L, dtype=7) == pc.CURE_ERR_INVALID_ARG
    assert _margins(L, vocab=1, ld=1) == pc.CURE_ERR_INVALID_ARG
    assert _margins(L, ld=50000) == pc.CURE_ERR_INVALID_ARG
    assert _margins(L, logits=None) == pc.CURE_ERR_INVALID_ARG
    assert _margins(L, margin=None) == pc.CURE_ERR_INVALID_ARG
    assert _margins(L, chain_len=5) == pc.CURE_ERR_INVALID_ARG        # > rows
    assert _margins(L, branch_depth=0) == pc.CURE_ERR_INVALID_ARG
    assert _margins(L, ufp_cnt=None) == pc.CURE_ERR_INVALID_ARG      # half a gate
    assert _margins(L, rows=2000, chain_len=1500) == pc.CURE_ERR_UNSUPPORTED
    assert _margins(L) == pc.CURE_ERR_WORKSPACE                        # no workspace
    assert _margins(L, batch=0) == pc.CURE_OK                          # empty: nothing to do
    assert _margins(L, batch=-1) == pc.CURE_ERR_INVALID_ARG


def test_margins_accept_argument_errors(L):
    # cure_margins' host checks, then the acceptance walk's, before any device
    # is touched (vocab 100000 over 4 rows splits the rows, so a missing
    # workspace is reported rather than a launch).
    def call(**kw):
        args = dict(logits=1, dtype=1, batch=1, rows=4, vocab=100000, ld=100000,
                    top1_val=1, top1_idx=1, top2_val=1, top2_idx=1, lse=1, margin=1,
                    chain_len=2, tau=1.0, repair_budget=4, branch_depth=2, ufp_pos=1,
                    ufp_cnt=1, parent=1, token=1, root_tgt=1, n_nodes=1, acc_len=1, path=1,
                    best=1, bonus=1, resync=1, workspace=None, ws_bytes=0, stream=None)
        args.update(kw)
        return L.cure_margins_accept(*args.values())
    assert call(dtype=7) == pc.CURE_ERR_INVALID_ARG
    assert call(logits=None) == pc.CURE_ERR_INVALID_ARG
    assert call(ufp_cnt=None) == pc.CURE_ERR_INVALID_ARG              # half a gate
    assert call(chain_len=5) == pc.CURE_ERR_INVALID_ARG               # > rows with the gate
    assert call(ufp_pos=None, ufp_cnt=None, chain_len=-1) == pc.CURE_ERR_INVALID_ARG
    for k in ("parent", "token", "root_tgt", "n_nodes", "acc_len", "path", "best", "bonus",
              "resync"):
        assert call(**{k: None}) == pc.CURE_ERR_INVALID_ARG, k
    assert call(rows=257) == pc.CURE_ERR_UNSUPPORTED                    # not a tree's nodes
    assert call() == pc.CURE_ERR_WORKSPACE                              # no workspace
    assert call(batch=0) == pc.CURE_OK
    assert call(batch=-1) == pc.CURE_ERR_INVALID_ARG


def test_margins_noalloc_argument_errors(L):
    # The same host checks as cure_margins, before any device is touched.
    def call(**kw):
        args = dict(logits=1, dtype=1, batch=1, rows=4, vocab=100000, ld=100000,
                    top1_val=1, top1_idx=1, top2_val=1, top2_idx=1, lse=1, margin=1,
                    chain_len=2, tau=1.0, repair_budget=4, branch_depth=2, ufp_pos=1,
                    ufp_cnt=1, stream=None)
        args.update(kw)
        return L.cure_margins_noalloc(*args.values())
    assert call(dtype=7) == pc.CURE_ERR_INVALID_ARG
    assert call(vocab=1, ld=1) == pc.CURE_ERR_INVALID_ARG
    assert call(logits=None) == pc.CURE_ERR_INVALID_ARG
    assert call(ufp_cnt=None) == pc.CURE_ERR_INVALID_ARG
    assert call(chain_len=5) == pc.CURE_ERR_INVALID_ARG
    assert call(rows=2000, chain_len=1500) == pc.CURE_ERR_UNSUPPORTED
    assert call(batch=0) == pc.CURE_OK
    assert call(batch=-1) == pc.CURE_ERR_INVALID_ARG
    assert L.cure_margins_noalloc_scratch_bytes() == 256 * 1024


def test_margins_workspace_size_grows_with_rows(L):
    a = L.cure_margins_workspace_size(1, 32, 128256)
    b = L.cure_margins_workspace_size(16, 48, 128256)
    assert a > 0 and b > a and b % 256 == 0


def _attn(L, **kw):
    ctx = np.array([10], np.int32)
    nn = np.array([3], np.int32)
    args = dict(q=1, k=1, v=1, o=1, lse=None, dtype=1, out_dtype=1, batch=1, hq=4, hkv=2,
                d=64, scale=0.125, kv_off=1, ctx_len=1, n_nodes=1, parent=1, n_max=3,
                host_ctx_len=ctx.ctypes.data_as(ctypes.c_void_p),
                host_n_nodes=nn.ctypes.data_as(ctypes.c_void_p), kv_split=0, flags=0,
                tree_status=None, workspace=None, ws_bytes=0, stream=None)
    args.update(kw)
    return L.cure_tree_attn(*args.values())


def test_tree_attn_argument_errors(L):
    assert _attn(L, d=96) == pc.CURE_ERR_UNSUPPORTED
    assert _attn(L, n_max=300) == pc.CURE_ERR_UNSUPPORTED
    assert _attn(L, hq=5) == pc.CURE_ERR_INVALID_ARG
    assert _attn(L, dtype=3) == pc.CURE_ERR_INVALID_ARG
    assert _attn(L, q=None) == pc.CURE_ERR_INVALID_ARG
    assert _attn(L, parent=None) == pc.CURE_ERR_INVALID_ARG
    assert _attn(L, host_ctx_len=None) == pc.CURE_ERR_INVALID_ARG
    bad_n = np.array([4], np.int32)                                    # more nodes than n_max
    assert _attn(L, host_n_nodes=bad_n.ctypes.data_as(ctypes.c_void_p)) == pc.CURE_ERR_INVALID_ARG
    assert _attn(L, batch=0) == pc.CURE_OK


def test_tree_attn_alignment_errors(L):
    # The matrix-core path (bf16, d 64) moves q, k, v and o as vectors: o must
    # be 8-byte (bf16) or 16-byte (fp32) aligned; split partials need a
    # 16-byte aligned workspace on every path.
    ok = dict(q=4096, k=4096, v=4096)
    assert _attn(L, o=4100, **ok) == pc.CURE_ERR_INVALID_ARG                   # bf16 out, 4 mod 8
    assert _attn(L, o=4104, out_dtype=pc.CURE_F32, **ok) == pc.CURE_ERR_INVALID_ARG
    assert _attn(L, q=4104, k=4096, v=4096, o=4096) == pc.CURE_ERR_INVALID_ARG  # MFMA operands
    # 1000 context rows in 2 splits need partials, so the workspace is checked.
    ctx = np.array([1000], np.int32)
    assert _attn(L, o=4096, kv_split=2, workspace=4104, ws_bytes=1 << 24,
                 host_ctx_len=ctx.ctypes.data_as(ctypes.c_void_p), **ok) == pc.CURE_ERR_INVALID_ARG


def test_tree_attn_workspace_size_tracks_splits(L):
    ctx = np.array([32768] * 4, np.int32)
    nn = np.array([32] * 4, np.int32)
    cp, np_ = ctx.ctypes.data_as(ctypes.c_void_p), nn.ctypes.data_as(ctypes.c_void_p)
    one = L.cure_tree_attn_workspace_size(4, 32, 8, 128, 32, cp, np_, 1)
    eight = L.cure_tree_attn_workspace_size(4, 32, 8, 128, 32, cp, np_, 8)
    assert one == 0                                      # a single split needs no partials
    assert eight >= 4 * 32 * 32 * 8 * 129 * 4


def test_accept_argument_errors(L):
    args = [1, 1, 1, 1, 1, 4, 2, 8, 1, 1, 1, 1, 1, None]
    bad = list(args)
    bad[7] = 300                                                       # n_max > 256
    assert L.cure_accept(*bad) == pc.CURE_ERR_UNSUPPORTED
    bad = list(args)
    bad[0] = None
    assert L.cure_accept(*bad) == pc.CURE_ERR_INVALID_ARG
    bad = list(args)
    bad[6] = 0
    assert L.cure_accept(*bad) == pc.CURE_OK                           # empty batch


def test_binding_fails_loudly_without_gpu_tensors():
    import torch
    with pytest.raises(pc.CureError):
        pc.cure_margins(torch.zeros(2, 16))


def _repair(L, **kw):
    # 16 chain rows, vocab 32000, budget 16 in depth-4 branches: 4 UFP slots, so
    # a missing workspace is reported before any launch.
    args = dict(logits=1, dtype=1, batch=1, rows=16, vocab=32000, ld=32000, margin=1,
                ufp_pos=1, ufp_cnt=1, chain_tok=1, chain_len=16, budget=16, depth=4,
                scale=1.0, b_min=1, b_max=5, suffix=None, n_max=32, parent=1, token=1,
                n_nodes=1, branch_cnt=None, workspace=None, ws_bytes=0, stream=None)
    args.update(kw)
    return L.cure_repair_tree(*args.values())


def test_repair_argument_errors(L):
    E, U = pc.CURE_ERR_INVALID_ARG, pc.CURE_ERR_UNSUPPORTED
    assert _repair(L, dtype=3) == E
    assert _repair(L, batch=-1) == E
    assert _repair(L, batch=0) == pc.CURE_OK
    assert _repair(L, chain_len=0) == E
    assert _repair(L, rows=8) == E                         # rows < chain_len
    assert _repair(L, depth=0) == E
    assert _repair(L, budget=-1) == E
    assert _repair(L, b_min=-1) == E
    assert _repair(L, b_min=3, b_max=2) == E
    assert _repair(L, b_min=0, b_max=0) == E
    assert _repair(L, vocab=5, ld=5) == E                  # fewer than b_max + 1 entries
    assert _repair(L, ld=100) == E
    for bad in (0.0, -1.0, float("nan"), float("inf")):
        assert _repair(L, scale=bad) == E
    assert _repair(L, n_max=31) == E                       # a full tree would not fit
    for name in ("logits", "margin", "ufp_pos", "ufp_cnt", "chain_tok", "parent", "token",
                 "n_nodes"):
        assert _repair(L, **{name: None}) == E, name
    assert _repair(L, b_max=8) == U
    assert _repair(L, rows=1025, chain_len=1025, n_max=2000) == U
    assert _repair(L, vocab=524289, ld=524289) == U
    assert _repair(L) == pc.CURE_ERR_WORKSPACE


def test_repair_workspace_size(L):
    f = L.cure_repair_tree_workspace_size
    assert f(1, 16, 32000, 3, 4) == 0                      # budget below one branch
    assert f(0, 16, 32000, 16, 4) == 0
    one = f(1, 16, 32000, 16, 4)
    assert one > 0 and one % 256 == 0
    assert f(4, 16, 32000, 16, 4) >= 4 * one - 512
    assert f(1, 16, 128256, 16, 4) > one                   # more chunks per row
    assert f(1, 16, 32000, 64, 4) > one                    # more UFP slots


def _commit(L, **kw):
    args = dict(k=1, v=1, dtype=1, n_layers=2, layer_stride=4096, hkv=8, d=128, batch=2,
                kv_off=1, ctx_len=2, n_nodes=1, path=1, acc_len=1, token=1, bonus=1,
                chain_len=16, n_max=32, new_ctx_len=3, emit=1, emit_cnt=1, replay_start=1,
                status=1, stream=None)
    args.update(kw)
    return L.cure_commit(*args.values())


def test_commit_argument_errors(L):
    E, U = pc.CURE_ERR_INVALID_ARG, pc.CURE_ERR_UNSUPPORTED
    assert _commit(L, dtype=3) == E
    assert _commit(L, batch=-1) == E
    assert _commit(L, n_layers=-1) == E
    assert _commit(L, hkv=0) == E
    assert _commit(L, d=0) == E
    assert _commit(L, chain_len=-1) == E
    assert _commit(L, layer_stride=0) == E                 # several layers need a stride
    assert _commit(L, new_ctx_len=2) == E                  # aliases ctx_len
    for name in ("kv_off", "ctx_len", "n_nodes", "path", "acc_len", "token", "bonus",
                 "new_ctx_len", "emit", "emit_cnt", "replay_start", "status", "k", "v"):
        assert _commit(L, **{name: None}) == E, name
    assert _commit(L, n_max=257) == U
    assert _commit(L, hkv=1, d=3, dtype=0) == U            # 12-byte rows
    assert _commit(L, hkv=1, d=4, dtype=1) == U            # 8-byte rows
    assert _commit(L, batch=70000) == U
    assert _commit(L, batch=0) == pc.CURE_OK               # empty: nothing to do


def test_read_ceiling_argument_errors(L):
    assert L.cure_read_ceiling_chunks(0) == 0
    assert L.cure_read_ceiling_chunks(1) == 1
    assert L.cure_read_ceiling_chunks(256 << 10) == 1
    assert L.cure_read_ceiling_chunks((256 << 10) + 16) == 2
    assert L.cure_read_ceiling(None, 0, None, None) == pc.CURE_OK      # nothing to read
    assert L.cure_read_ceiling(None, 64, 1, None) == pc.CURE_ERR_INVALID_ARG
    assert L.cure_read_ceiling(1, 64, None, None) == pc.CURE_ERR_INVALID_ARG
    assert L.cure_read_ceiling(1, 60, 1, None) == pc.CURE_ERR_INVALID_ARG  # not 16-byte multiple


def _attn_ws(L, ctx, nn, hq=32, hkv=8, d=128, n_max=32, kv_split=0):
    c = np.ascontiguousarray(ctx, np.int32)
    n = np.ascontiguousarray(nn, np.int32)
    return L.cure_tree_attn_workspace_size(len(c), hq, hkv, d, n_max,
                                           c.ctypes.data_as(ctypes.c_void_p),
                                           n.ctypes.data_as(ctypes.c_void_p), kv_split)


def _partials_bytes(batch, hq, n_max, splits, d):
    rows = batch * hq * n_max * splits                  # fp32 rows, then their LSEs,
    up = lambda x: (x + 255) // 256 * 256               # each array 256-byte aligned
    return up(rows * d * 4) + up(rows * 4)


def test_automatic_split_plan_hand_worked(L):
    # The split plan of the 256-CU GPU, worked by hand: the shortest split (a
    # multiple of the 64-token tile, at least 256 tokens) whose workgroups
    # (splits x kv-heads x row blocks, one per CU) are all resident at once.
    # One sequence, 2048 + 32 tokens: 8 kv-heads fit 32 splits, so 256-token
    # splits, ceil(2080 / 256) = 9 of them.
    assert _attn_ws(L, [2048], [32]) == _partials_bytes(1, 32, 32, 9, 128)
    # Four sequences of 32768 + 32 tokens: 32 workgroups per split index, so 8
    # splits per sequence, ceil(32800 / 8) = 4100 -> 4160 tokens.
    assert _attn_ws(L, [32768] * 4, [32] * 4) == _partials_bytes(4, 32, 32, 8, 128)
    # Forced splits: ceil(2080 / 3) = 694 -> 704-token splits, 3 of them.
    assert _attn_ws(L, [2048], [32], kv_split=3) == _partials_bytes(1, 32, 32, 3, 128)
    # A sequence that fits one split needs no partials at all.
    assert _attn_ws(L, [100, 200], [8, 8], kv_split=1) == 0
    # No sequence with tree nodes: nothing to plan.
    assert _attn_ws(L, [500, 700], [0, 0]) == 0
