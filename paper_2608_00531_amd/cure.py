"""Python binding for libcure (ctypes). Argument marshalling only.

Each function has the name of the C entry point it calls and runs on the
current torch stream of the tensors' device. PyTorch provides the device memory
(outputs and workspaces are allocated as torch tensors) and the stream; every
step of the computation runs in libcure's HIP kernels. If the library is not
built, the first call raises -- there is no fallback implementation.
"""

import ctypes
import os
import threading

import numpy as np
import torch


CURE_OK = 0
CURE_ERR_INVALID_ARG = 1
CURE_ERR_UNSUPPORTED = 2
CURE_ERR_BAD_TREE = 3
CURE_ERR_HIP = 4
CURE_ERR_WORKSPACE = 5
CURE_F32 = 0
CURE_BF16 = 1
CURE_ATTN_FORCE_VALU = 1
CURE_MAX_TREE_NODES = 256

_lock = threading.Lock()
_lib = None
_workspaces = {}

_vp, _i32, _i64, _f32, _sz, _u32 = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64,
                                    ctypes.c_float, ctypes.c_size_t, ctypes.c_uint32)

_SIGNATURES = {
    "cure_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "cure_version": (ctypes.c_int, []),
    "cure_margins_workspace_size": (_sz, [_i32, _i32, _i32]),
    "cure_margins": (ctypes.c_int, [_vp, _i32, _i32, _i32, _i32, _i64,
                                    _vp, _vp, _vp, _vp, _vp, _vp,
                                    _i32, _f32, _i32, _i32, _vp, _vp, _vp, _sz, _vp]),
    "cure_margins_accept": (ctypes.c_int, [_vp, _i32, _i32, _i32, _i32, _i64,
                                           _vp, _vp, _vp, _vp, _vp, _vp,
                                           _i32, _f32, _i32, _i32, _vp, _vp,
                                           _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                           _vp, _sz, _vp]),
    "cure_margins_noalloc_scratch_bytes": (_sz, []),
    "cure_margins_noalloc": (ctypes.c_int, [_vp, _i32, _i32, _i32, _i32, _i64,
                                            _vp, _vp, _vp, _vp, _vp, _vp,
                                            _i32, _f32, _i32, _i32, _vp, _vp, _vp]),
    "cure_tree_attn_workspace_size": (_sz, [_i32, _i32, _i32, _i32, _i32, _vp, _vp, _i32]),
    "cure_tree_attn": (ctypes.c_int, [_vp, _vp, _vp, _vp, _vp, _i32, _i32, _i32, _i32, _i32,
                                      _i32, _f32, _vp, _vp, _vp, _vp, _i32, _vp, _vp, _i32,
                                      _u32, _vp, _vp, _sz, _vp]),
    "cure_accept": (ctypes.c_int, [_vp, _vp, _vp, _vp, _vp, _i32, _i32, _i32,
                                   _vp, _vp, _vp, _vp, _vp, _vp]),
    "cure_repair_tree_workspace_size": (_sz, [_i32, _i32, _i32, _i32, _i32]),
    "cure_repair_tree": (ctypes.c_int, [_vp, _i32, _i32, _i32, _i32, _i64, _vp, _vp, _vp, _vp,
                                        _i32, _i32, _i32, _f32, _i32, _i32, _vp, _i32,
                                        _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
    "cure_read_ceiling_chunks": (_sz, [_sz]),
    "cure_read_ceiling": (ctypes.c_int, [_vp, _sz, _vp, _vp]),
    "cure_commit": (ctypes.c_int, [_vp, _vp, _i32, _i32, _i64, _i32, _i32, _i32,
                                   _vp, _vp, _vp, _vp, _vp, _vp, _vp, _i32, _i32,
                                   _vp, _vp, _vp, _vp, _vp, _vp]),
}


class CureError(RuntimeError):
    pass


def library_path():
    return os.path.join(os.path.dirname(os.path.abspath(__file__)), "_lib", "libcure.so")


def lib():
    """The loaded libcure (ctypes.CDLL). Raises if the library has not been built."""
    global _lib
    with _lock:
        if _lib is None:
            path = library_path()
            if not os.path.exists(path):
                raise CureError("libcure is not built (%s missing); run "
                                "`python -m paper_2608_00531_amd.build`" % path)
            l = ctypes.CDLL(path)
            for name, (res, args) in _SIGNATURES.items():
                fn = getattr(l, name)
                fn.restype = res
                fn.argtypes = args
            _lib = l
        return _lib


def _check(status, what):
    if status != CURE_OK:
        name = lib().cure_status_string(status).decode()
        raise CureError("%s failed: %s" % (what, name))


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _dtype_code(t):
    if t.dtype == torch.float32:
        return CURE_F32
    if t.dtype == torch.bfloat16:
        return CURE_BF16
    raise CureError("unsupported dtype %s (float32 or bfloat16)" % t.dtype)


def _stream(device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _workspace(kind, device, nbytes):
    """Zero-filled device workspace, reused per (kind, device, stream)."""
    if nbytes == 0:
        return None, 0
    key = (kind, device.index, torch.cuda.current_stream(device).cuda_stream)
    ws = _workspaces.get(key)
    if ws is None or ws.numel() < nbytes:
        ws = torch.zeros(max(nbytes, 256), dtype=torch.uint8, device=device)
        _workspaces[key] = ws
    return ws, ws.numel()


def _require_cuda(*ts):
    for t in ts:
        if t is not None and not t.is_cuda:
            raise CureError("tensor arguments must live on the GPU")


def cure_margins(logits, chain_len=0, tau=float("inf"), repair_budget=0, branch_depth=1,
                 gate=True):
    """Margin pass over logits [batch, rows, vocab] (or [rows, vocab]).

    Returns a dict of tensors shaped [batch, rows]: top1_val, top1_idx, top2_val,
    top2_idx, lse, margin; with gate=True also ufp_pos [batch, chain_len] and
    ufp_cnt [batch].
    """
    _require_cuda(logits)
    x = logits if logits.dim() == 3 else logits.unsqueeze(0)
    if x.stride(2) != 1 or x.stride(0) != x.shape[1] * x.stride(1):
        x = x.contiguous()
    batch, rows, vocab = x.shape
    dev = x.device
    f = dict(dtype=torch.float32, device=dev)
    i = dict(dtype=torch.int32, device=dev)
    out = {
        "top1_val": torch.empty(batch, rows, **f), "top1_idx": torch.empty(batch, rows, **i),
        "top2_val": torch.empty(batch, rows, **f), "top2_idx": torch.empty(batch, rows, **i),
        "lse": torch.empty(batch, rows, **f), "margin": torch.empty(batch, rows, **f),
    }
    ufp_pos = ufp_cnt = None
    if gate:
        ufp_pos = torch.empty(batch, chain_len, **i)
        ufp_cnt = torch.empty(batch, **i)
        out["ufp_pos"], out["ufp_cnt"] = ufp_pos, ufp_cnt
    L = lib()
    ws, wsb = _workspace("margins", dev, L.cure_margins_workspace_size(batch, rows, vocab))
    st = L.cure_margins(_ptr(x), _dtype_code(x), batch, rows, vocab, x.stride(1),
                        _ptr(out["top1_val"]), _ptr(out["top1_idx"]), _ptr(out["top2_val"]),
                        _ptr(out["top2_idx"]), _ptr(out["lse"]), _ptr(out["margin"]),
                        chain_len, tau, repair_budget, branch_depth, _ptr(ufp_pos),
                        _ptr(ufp_cnt), _ptr(ws), wsb, _stream(dev))
    _check(st, "cure_margins")
    return out


def cure_margins_accept(logits, parent, token, root_tgt, n_nodes, chain_len, tau=float("inf"),
                        repair_budget=0, branch_depth=1, gate=True):
    """Margin pass over a tree's node logits [batch, n_max, vocab] followed by
    the acceptance walk on their argmaxes, in one call. parent/token int32
    [batch, n_max], root_tgt/n_nodes int32 [batch] (GPU tensors). Returns
    cure_margins' dict plus cure_accept's (acc_len, path, best, bonus, resync)."""
    _require_cuda(logits, parent, token, root_tgt, n_nodes)
    x = logits if logits.dim() == 3 else logits.unsqueeze(0)
    if x.stride(2) != 1 or x.stride(0) != x.shape[1] * x.stride(1):
        x = x.contiguous()
    batch, rows, vocab = x.shape
    dev = x.device
    f = dict(dtype=torch.float32, device=dev)
    i = dict(dtype=torch.int32, device=dev)
    out = {
        "top1_val": torch.empty(batch, rows, **f), "top1_idx": torch.empty(batch, rows, **i),
        "top2_val": torch.empty(batch, rows, **f), "top2_idx": torch.empty(batch, rows, **i),
        "lse": torch.empty(batch, rows, **f), "margin": torch.empty(batch, rows, **f),
        "acc_len": torch.empty(batch, **i), "path": torch.empty(batch, rows, **i),
        "best": torch.empty(batch, **i), "bonus": torch.empty(batch, **i),
        "resync": torch.empty(batch, **i),
    }
    ufp_pos = ufp_cnt = None
    if gate:
        ufp_pos = torch.empty(batch, chain_len, **i)
        ufp_cnt = torch.empty(batch, **i)
        out["ufp_pos"], out["ufp_cnt"] = ufp_pos, ufp_cnt
    tree = [t.contiguous() for t in (parent, token, root_tgt, n_nodes)]
    L = lib()
    ws, wsb = _workspace("margins", dev, L.cure_margins_workspace_size(batch, rows, vocab))
    st = L.cure_margins_accept(_ptr(x), _dtype_code(x), batch, rows, vocab, x.stride(1),
                               _ptr(out["top1_val"]), _ptr(out["top1_idx"]),
                               _ptr(out["top2_val"]), _ptr(out["top2_idx"]), _ptr(out["lse"]),
                               _ptr(out["margin"]), chain_len, tau, repair_budget, branch_depth,
                               _ptr(ufp_pos), _ptr(ufp_cnt), *[_ptr(t) for t in tree],
                               _ptr(out["acc_len"]), _ptr(out["path"]), _ptr(out["best"]),
                               _ptr(out["bonus"]), _ptr(out["resync"]), _ptr(ws), wsb,
                               _stream(dev))
    _check(st, "cure_margins_accept")
    return out


def cure_margins_noalloc(logits, chain_len=0, tau=float("inf"), repair_budget=0,
                         branch_depth=1, gate=True):
    """As cure_margins, through the allocation-free entry point: no workspace
    is passed; the library's fixed scratch array serves the call."""
    _require_cuda(logits)
    x = logits if logits.dim() == 3 else logits.unsqueeze(0)
    if x.stride(2) != 1 or x.stride(0) != x.shape[1] * x.stride(1):
        x = x.contiguous()
    batch, rows, vocab = x.shape
    dev = x.device
    f = dict(dtype=torch.float32, device=dev)
    i = dict(dtype=torch.int32, device=dev)
    out = {
        "top1_val": torch.empty(batch, rows, **f), "top1_idx": torch.empty(batch, rows, **i),
        "top2_val": torch.empty(batch, rows, **f), "top2_idx": torch.empty(batch, rows, **i),
        "lse": torch.empty(batch, rows, **f), "margin": torch.empty(batch, rows, **f),
    }
    ufp_pos = ufp_cnt = None
    if gate:
        ufp_pos = torch.empty(batch, chain_len, **i)
        ufp_cnt = torch.empty(batch, **i)
        out["ufp_pos"], out["ufp_cnt"] = ufp_pos, ufp_cnt
    st = lib().cure_margins_noalloc(_ptr(x), _dtype_code(x), batch, rows, vocab, x.stride(1),
                                    _ptr(out["top1_val"]), _ptr(out["top1_idx"]),
                                    _ptr(out["top2_val"]), _ptr(out["top2_idx"]),
                                    _ptr(out["lse"]), _ptr(out["margin"]), chain_len, tau,
                                    repair_budget, branch_depth, _ptr(ufp_pos), _ptr(ufp_cnt),
                                    _stream(dev))
    _check(st, "cure_margins_noalloc")
    return out


def _host_i32(a):
    a = np.ascontiguousarray(np.asarray(a, dtype=np.int32))
    return a, a.ctypes.data_as(ctypes.c_void_p)


def cure_tree_attn_workspace_size(batch, hq, hkv, d, n_max, host_ctx_len, host_n_nodes,
                                  kv_split=0):
    c, cp = _host_i32(host_ctx_len)
    n, np_ = _host_i32(host_n_nodes)
    return lib().cure_tree_attn_workspace_size(batch, hq, hkv, d, n_max, cp, np_, kv_split)


def cure_tree_attn(q, k, v, kv_off, ctx_len, n_nodes, parent, host_ctx_len, host_n_nodes,
                   scale, out_dtype=None, kv_split=0, flags=0, with_lse=True):
    """Tree-masked verification attention.

    q [batch, n_max, hq, d]; k, v [rows, hkv, d]; kv_off int64 [batch]; ctx_len,
    n_nodes int32 [batch]; parent int32 [batch, n_max] (all on the GPU);
    host_ctx_len / host_n_nodes: host copies (numpy or lists).
    Returns (o [batch, n_max, hq, d], lse [batch, n_max, hq] or None, tree_status [batch]).
    """
    _require_cuda(q, k, v, kv_off, ctx_len, n_nodes, parent)
    for t in (q, k, v, kv_off, ctx_len, n_nodes, parent):
        if not t.is_contiguous():
            raise CureError("tree attention arguments must be contiguous")
    if kv_off.dtype != torch.int64 or ctx_len.dtype != torch.int32 or \
            n_nodes.dtype != torch.int32 or parent.dtype != torch.int32:
        raise CureError("kv_off must be int64; ctx_len, n_nodes and parent int32")
    batch, n_max, hq, d = q.shape
    hkv = k.shape[1]
    dev = q.device
    out_dtype = q.dtype if out_dtype is None else out_dtype
    o = torch.empty(batch, n_max, hq, d, dtype=out_dtype, device=dev)
    lse = torch.empty(batch, n_max, hq, dtype=torch.float32, device=dev) if with_lse else None
    status = torch.empty(batch, dtype=torch.int32, device=dev)
    hc, hcp = _host_i32(host_ctx_len)
    hn, hnp = _host_i32(host_n_nodes)
    L = lib()
    ws, wsb = _workspace("attn", dev, L.cure_tree_attn_workspace_size(
        batch, hq, hkv, d, n_max, hcp, hnp, kv_split))
    st = L.cure_tree_attn(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), _dtype_code(q),
                          _dtype_code(o), batch, hq, hkv, d, scale, _ptr(kv_off),
                          _ptr(ctx_len), _ptr(n_nodes), _ptr(parent), n_max, hcp, hnp,
                          kv_split, flags, _ptr(status), _ptr(ws), wsb, _stream(dev))
    _check(st, "cure_tree_attn")
    return o, lse, status


def cure_accept(parent, token, tgt, root_tgt, n_nodes, chain_len):
    """Acceptance walk. All arguments int32 GPU tensors: parent/token/tgt
    [batch, n_max], root_tgt/n_nodes [batch]. Returns a dict of tensors."""
    _require_cuda(parent, token, tgt, root_tgt, n_nodes)
    batch, n_max = parent.shape
    dev = parent.device
    i = dict(dtype=torch.int32, device=dev)
    out = {"acc_len": torch.empty(batch, **i), "path": torch.empty(batch, n_max, **i),
           "best": torch.empty(batch, **i), "bonus": torch.empty(batch, **i),
           "resync": torch.empty(batch, **i)}
    args = [t.contiguous() for t in (parent, token, tgt, root_tgt, n_nodes)]
    st = lib().cure_accept(*[_ptr(t) for t in args], chain_len, batch, n_max,
                           _ptr(out["acc_len"]), _ptr(out["path"]), _ptr(out["best"]),
                           _ptr(out["bonus"]), _ptr(out["resync"]), _stream(dev))
    _check(st, "cure_accept")
    return out


def cure_repair_tree(logits, margin, ufp_pos, ufp_cnt, chain_tok, repair_budget, branch_depth,
                     margin_scale, b_min=1, b_max=5, suffix=None, n_max=None):
    """Repair tree per sequence.

    logits [batch, rows, vocab] (or [rows, vocab]) -- the draft block's rows;
    margin [batch, rows] float32, ufp_pos [batch, chain_len], ufp_cnt [batch] as
    cure_margins returned them; chain_tok int32 [batch, chain_len]; suffix int32
    [batch, chain_len, b_max, branch_depth - 1] or None.
    Returns a dict: parent, token [batch, n_max] (valid below n_nodes), n_nodes
    [batch], branch_cnt [batch, chain_len].
    """
    _require_cuda(logits, margin, ufp_pos, ufp_cnt, chain_tok, suffix)
    x = logits if logits.dim() == 3 else logits.unsqueeze(0)
    if x.stride(2) != 1 or x.stride(0) != x.shape[1] * x.stride(1):
        x = x.contiguous()
    batch, rows, vocab = x.shape
    chain_len = chain_tok.shape[-1]
    if margin.dtype != torch.float32 or any(
            t is not None and t.dtype != torch.int32 for t in (ufp_pos, ufp_cnt, chain_tok, suffix)):
        raise CureError("margin must be float32; ufp_pos, ufp_cnt, chain_tok and suffix int32")
    shapes = [(margin, (batch, rows)), (ufp_pos, (batch, chain_len)), (ufp_cnt, (batch,)),
              (chain_tok, (batch, chain_len))]
    if suffix is not None and branch_depth > 1:
        shapes.append((suffix, (batch, chain_len, b_max, branch_depth - 1)))
    for t, shape in shapes:
        if tuple(t.shape) != shape:
            raise CureError("expected shape %s, got %s" % (shape, tuple(t.shape)))
    args = [t.contiguous() for t in (margin, ufp_pos, ufp_cnt, chain_tok)]
    suffix = None if suffix is None or branch_depth == 1 else suffix.contiguous()
    n_max = chain_len + repair_budget if n_max is None else n_max
    dev = x.device
    i = dict(dtype=torch.int32, device=dev)
    out = {"parent": torch.empty(batch, n_max, **i), "token": torch.empty(batch, n_max, **i),
           "n_nodes": torch.empty(batch, **i), "branch_cnt": torch.empty(batch, chain_len, **i)}
    L = lib()
    ws, wsb = _workspace("repair", dev, L.cure_repair_tree_workspace_size(
        batch, chain_len, vocab, repair_budget, branch_depth))
    st = L.cure_repair_tree(_ptr(x), _dtype_code(x), batch, rows, vocab, x.stride(1),
                            *[_ptr(t) for t in args], chain_len, repair_budget, branch_depth,
                            margin_scale, b_min, b_max, _ptr(suffix), n_max,
                            _ptr(out["parent"]), _ptr(out["token"]), _ptr(out["n_nodes"]),
                            _ptr(out["branch_cnt"]), _ptr(ws), wsb, _stream(dev))
    _check(st, "cure_repair_tree")
    return out


def cure_commit(k, v, kv_off, ctx_len, n_nodes, path, acc_len, token, bonus, chain_len,
                layer_stride=None):
    """Commit each sequence's winning path, in place.

    k, v: one layer's cache [rows, hkv, d], or n_layers caches [n_layers, rows,
    hkv, d] (contiguous per layer; layer_stride in elements defaults to the
    distance between layers). kv_off int64 [batch]; ctx_len, n_nodes, acc_len,
    bonus int32 [batch]; path, token int32 [batch, n_max] (all on the GPU; path,
    acc_len and bonus as cure_accept returned them).
    Returns a dict: new_ctx_len [batch], emit [batch, n_max + 1], emit_cnt,
    replay_start and status [batch].
    """
    _require_cuda(k, v, kv_off, ctx_len, n_nodes, path, acc_len, token, bonus)
    if k.shape != v.shape or k.dtype != v.dtype or k.dim() not in (3, 4):
        raise CureError("k and v must have the same shape [n_layers,] rows, hkv, d")
    if kv_off.dtype != torch.int64 or any(t.dtype != torch.int32 for t in
                                          (ctx_len, n_nodes, path, acc_len, token, bonus)):
        raise CureError("kv_off must be int64; the other index arrays int32")
    n_layers = 1 if k.dim() == 3 else k.shape[0]
    hkv, d = k.shape[-2], k.shape[-1]
    for t in (k, v):
        if tuple(t.stride()[-3:]) != (hkv * d, d, 1):
            raise CureError("each layer of k and v must be contiguous")
    if layer_stride is None:
        layer_stride = 0 if k.dim() == 3 else k.stride(0)
    if k.dim() == 4 and (k.stride(0) != layer_stride or v.stride(0) != layer_stride):
        raise CureError("layer_stride does not match the tensors' layer stride")
    batch, n_max = path.shape
    dev = k.device
    i = dict(dtype=torch.int32, device=dev)
    out = {"new_ctx_len": torch.empty(batch, **i), "emit": torch.empty(batch, n_max + 1, **i),
           "emit_cnt": torch.empty(batch, **i), "replay_start": torch.empty(batch, **i),
           "status": torch.empty(batch, **i)}
    args = [t.contiguous() for t in (kv_off, ctx_len, n_nodes, path, acc_len, token, bonus)]
    st = lib().cure_commit(_ptr(k), _ptr(v), _dtype_code(k), n_layers, layer_stride, hkv, d,
                           batch, *[_ptr(t) for t in args], chain_len, n_max,
                           _ptr(out["new_ctx_len"]), _ptr(out["emit"]), _ptr(out["emit_cnt"]),
                           _ptr(out["replay_start"]), _ptr(out["status"]), _stream(dev))
    _check(st, "cure_commit")
    return out


def cure_read_ceiling(buf):
    """Streams a contiguous GPU tensor (size a multiple of 16 bytes) once; returns
    the per-256-KB-chunk XOR of its 32-bit words (int32 tensor)."""
    _require_cuda(buf)
    if not buf.is_contiguous():
        raise CureError("the buffer must be contiguous")
    nbytes = buf.numel() * buf.element_size()
    L = lib()
    out = torch.empty(max(int(L.cure_read_ceiling_chunks(nbytes)), 1), dtype=torch.int32,
                      device=buf.device)
    _check(L.cure_read_ceiling(_ptr(buf), nbytes, _ptr(out), _stream(buf.device)),
           "cure_read_ceiling")
    return out
