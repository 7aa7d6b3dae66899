"""Python binding of libd2sd (the C ABI in include/d2sd.h).

Argument marshalling only: every step runs in the library's HIP kernels.
torch supplies device memory and the stream (``torch.cuda.current_stream()``
unless one is given). Function names are the C names without the ``d2sd_``
prefix. Importing this module fails loudly when libd2sd.so has not been built.
"""

from __future__ import annotations

import ctypes
import os
import re

import numpy as np
# torch ships its own HIP runtime (same soname as the system one). Loading it
# first makes libd2sd bind to that single runtime; a second runtime in the
# process cannot open the device, and torch's streams and device pointers are
# only valid inside the runtime that created them.
import torch  # noqa: F401  (must precede the CDLL load below)

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libd2sd.so")
HEADER = os.path.join(os.path.dirname(_PKG), "include", "d2sd.h")

OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_WORKSPACE_TOO_SMALL, ERR_HIP = 0, 1, 2, 3, 4
F32, BF16 = 0, 1
STAGE_CASCADE, STAGE_PREFIX, STAGE_TREE = 0, 1, 2
MAX_B, HEAD_DIM, PAGE_SIZE = 64, 128, 16


class D2SDError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        self.status = status
        super().__init__(f"{where}: {detail or 'error'} (status {status})")


if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2606_04446_amd.build` "
                      "(the verify path has no fallback)")

_lib = ctypes.CDLL(LIB_PATH)
_c_int, _c_ptr, _c_size = ctypes.c_int, ctypes.c_void_p, ctypes.c_size_t
_c_int_p = ctypes.POINTER(ctypes.c_int)


class AttnArgs(ctypes.Structure):
    """Mirror of d2sd_attn_args (field order and types must match the header)."""

    _fields_ = [
        ("batch", _c_int), ("num_qo_heads", _c_int), ("num_kv_heads", _c_int), ("head_dim", _c_int),
        ("page_size", _c_int), ("dtype", _c_int), ("stage", _c_int), ("sm_scale", ctypes.c_float),
        ("total_nodes", _c_int), ("max_nodes", _c_int), ("max_ctx_len", _c_int), ("num_pages", _c_int),
        ("max_pages", _c_int), ("mask_words", _c_int), ("kv_split", _c_int), ("row_group", _c_int),
        ("packed", _c_int),
        ("q", _c_ptr), ("k_cache", _c_ptr), ("v_cache", _c_ptr), ("page_table", _c_ptr),
        ("ctx_len", _c_ptr), ("k_tree", _c_ptr), ("v_tree", _c_ptr), ("node_indptr", _c_ptr),
        ("anc_mask", _c_ptr), ("out", _c_ptr), ("lse", _c_ptr), ("node_indptr_host", _c_ptr),
    ]

    def keep(self, *objs):
        """Keep host arrays whose addresses the struct holds alive as long as it."""
        self._keep = getattr(self, "_keep", ()) + objs


def _sig(name, restype, *argtypes):
    f = getattr(_lib, name)
    f.restype = restype
    f.argtypes = list(argtypes)
    return f


_status_string = _sig("d2sd_status_string", ctypes.c_char_p, _c_int)
_last_error = _sig("d2sd_last_error", ctypes.c_char_p)
_version = _sig("d2sd_version", _c_int)
_mask_words = _sig("d2sd_mask_words", _c_int, _c_int)
_tree_plan = _sig("d2sd_tree_plan", _c_int, _c_int, _c_int, _c_ptr, _c_ptr, _c_int, _c_ptr, _c_int_p)
_tree_build = _sig("d2sd_tree_build", _c_int, _c_int, _c_int, _c_int, _c_ptr, _c_ptr, _c_ptr, _c_int,
                   _c_int, _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_ptr)
_from_parents = _sig("d2sd_tree_from_parents", _c_int, _c_int, _c_ptr, _c_int, _c_int, _c_int, _c_ptr, _c_ptr,
                     _c_ptr, _c_ptr, _c_ptr)
_select = _sig("d2sd_select_reanchor", _c_int, _c_int, _c_int, _c_int, _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_ptr)
_indptr = _sig("d2sd_tree_indptr", _c_int, _c_int, _c_int, _c_int, _c_ptr, _c_ptr, _c_ptr, _c_ptr)
_commit = _sig("d2sd_commit_accepted_kv", _c_int, _c_int, _c_int, _c_int, _c_int, _c_int, _c_int, _c_int, _c_int,
               _c_int, _c_ptr, _c_int, _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_ptr)
_ws_size = _sig("d2sd_cascade_workspace_size", _c_int, ctypes.POINTER(AttnArgs), ctypes.POINTER(_c_size))
_kv_split = _sig("d2sd_cascade_kv_split", _c_int, ctypes.POINTER(AttnArgs), _c_int_p)
_row_group = _sig("d2sd_cascade_row_group", _c_int, ctypes.POINTER(AttnArgs), _c_int_p, _c_int_p)
_cascade = _sig("d2sd_cascade_verify_attention", _c_int, ctypes.POINTER(AttnArgs), _c_ptr, _c_size, _c_ptr)
_noncascade = _sig("d2sd_noncascade_verify_attention", _c_int, ctypes.POINTER(AttnArgs), _c_ptr)
_cascade_noalloc = _sig("d2sd_cascade_verify_attention_noalloc", _c_int, ctypes.POINTER(AttnArgs), _c_ptr)
_merge = _sig("d2sd_merge_state", _c_int, _c_int, _c_int, _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_ptr,
              _c_ptr)
_accept = _sig("d2sd_accept_path", _c_int, _c_int, _c_int, _c_ptr, _c_int, _c_ptr, _c_ptr, _c_ptr, _c_ptr,
               _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_ptr)
_sample = _sig("d2sd_sample_targets", _c_int, _c_int, _c_ptr, _c_int, _c_int, _c_ptr, _c_ptr, _c_int, _c_int, _c_ptr,
                ctypes.c_float, _c_ptr, _c_ptr, _c_ptr, _c_ptr)
_timing_enable = _sig("d2sd_kernel_timing_enable", _c_int, _c_int)
_timing_collect = _sig("d2sd_kernel_timing_collect", _c_int, _c_int_p, ctypes.POINTER(ctypes.c_double))
_timing_each = _sig("d2sd_kernel_timing_collect_each", _c_int, _c_int, ctypes.POINTER(ctypes.c_float), _c_int_p)
_timing_parts = _sig("d2sd_kernel_timing_collect_parts", _c_int, _c_int, ctypes.POINTER(ctypes.c_float),
                     ctypes.POINTER(ctypes.c_float), _c_int_p)


def _check(status: int, where: str):
    if status != OK:
        raise D2SDError(status, where, _last_error().decode())


def header_functions() -> list:
    """Names of the functions include/d2sd.h declares."""
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(d2sd_[a-z_0-9]+)\s*\(", text)))


def status_string(status: int) -> str:
    return _status_string(status).decode()


def last_error() -> str:
    return _last_error().decode()


def version() -> int:
    return _version()


def mask_words(B: int) -> int:
    return _mask_words(B)


# ---------------------------------------------------------------- helpers --

def _stream(stream):
    import torch
    if stream is None:
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return ctypes.c_void_p(stream)
    return ctypes.c_void_p(stream.cuda_stream)


def _dev(t, name, dtype=None):
    """Device pointer of a contiguous CUDA tensor (None passes NULL)."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    return t.data_ptr()


def _host_i32(a):
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


# ------------------------------------------------------------------- tree --

def tree_plan(B: int, K, p):
    """Host planner: returns (node_indptr int32 [batch+1], mask_words)."""
    K = _host_i32(K)
    p = _host_i32(p)
    if p.ndim == 1:
        p = p.reshape(len(K), -1)
    batch, kmax = len(K), (p.shape[1] if p.size else 0)
    indptr = np.zeros(batch + 1, np.int32)
    w = ctypes.c_int(0)
    _check(_tree_plan(batch, B, K.ctypes.data, p.ctypes.data if p.size else None, kmax, indptr.ctypes.data,
                      ctypes.byref(w)), "d2sd_tree_plan")
    return indptr, w.value


def tree_build(B: int, K, p, node_indptr, total_nodes: int, mask_words_: int, out: dict | None = None,
               stream=None) -> dict:
    """Device tree build. K [batch], p [batch, Kmax], node_indptr [batch+1] are
    int32 device tensors. Returns dict(parent, depth, path_id, anc_mask, path_leaf)."""
    import torch
    batch = K.numel()
    kmax = p.shape[1] if p.dim() == 2 else 0
    dev = K.device
    o = out or {}
    parent = (o["parent"] if "parent" in o else torch.empty(total_nodes, dtype=torch.int32, device=dev))
    depth = (o["depth"] if "depth" in o else torch.empty(total_nodes, dtype=torch.int32, device=dev))
    path_id = (o["path_id"] if "path_id" in o else torch.empty(total_nodes, dtype=torch.int32, device=dev))
    anc_mask = (o["anc_mask"] if "anc_mask" in o else torch.empty((total_nodes, mask_words_), dtype=torch.int32, device=dev))
    path_leaf = (o["path_leaf"] if "path_leaf" in o else torch.empty((batch, kmax + 1), dtype=torch.int32, device=dev))
    i32 = torch.int32
    _check(_tree_build(batch, B, kmax, _dev(K, "K", i32), _dev(p, "p", i32) if kmax else None,
                       _dev(node_indptr, "node_indptr", i32), total_nodes, mask_words_,
                       _dev(parent, "parent", i32), _dev(depth, "depth", i32), _dev(path_id, "path_id", i32),
                       _dev(anc_mask, "anc_mask", i32), _dev(path_leaf, "path_leaf", i32), _stream(stream)),
           "d2sd_tree_build")
    return dict(parent=parent, depth=depth, path_id=path_id, anc_mask=anc_mask, path_leaf=path_leaf)


def tree_from_parents(node_indptr, total_nodes: int, max_nodes: int, parent, mask_words_: int | None = None,
                      out: dict | None = None, stream=None) -> dict:
    """Device tree arrays from a parent array (int32 [ΣN], local indices).
    Returns dict(parent, depth, path_id, anc_mask) shaped as tree_build's outputs."""
    import torch
    batch = node_indptr.numel() - 1
    W = mask_words_ if mask_words_ is not None else (max_nodes + 31) // 32
    dev = parent.device
    o = out or {}
    depth = o["depth"] if "depth" in o else torch.empty(total_nodes, dtype=torch.int32, device=dev)
    path_id = o["path_id"] if "path_id" in o else torch.empty(total_nodes, dtype=torch.int32, device=dev)
    anc_mask = o["anc_mask"] if "anc_mask" in o else torch.empty((total_nodes, W), dtype=torch.int32, device=dev)
    i32 = torch.int32
    _check(_from_parents(batch, _dev(node_indptr, "node_indptr", i32), total_nodes, max_nodes, W,
                         _dev(parent, "parent", i32), _dev(depth, "depth", i32), _dev(path_id, "path_id", i32),
                         _dev(anc_mask, "anc_mask", i32), _stream(stream)), "d2sd_tree_from_parents")
    return dict(parent=parent, depth=depth, path_id=path_id, anc_mask=anc_mask)


def select_reanchor(B: int, conf, K, Kmax: int, p_out=None, r_out=None, want_r: bool = False, stream=None):
    """Device re-anchor selection (Eq. 4-5). conf: float32 [batch, B-1] device
    tensor (conf[b, k-1] = c_k), K: int32 [batch]. Returns (p int32 [batch,
    Kmax], r float64 [batch, B-1] or None)."""
    import torch
    batch = K.numel()
    dev = K.device
    if conf.shape != (batch, B - 1):
        raise ValueError(f"conf must have shape ({batch}, {B - 1}), got {tuple(conf.shape)}")
    p = p_out if p_out is not None else torch.empty((batch, Kmax), dtype=torch.int32, device=dev)
    r = r_out if r_out is not None else (torch.empty((batch, B - 1), dtype=torch.float64, device=dev)
                                         if want_r else None)
    _check(_select(batch, B, Kmax, _dev(conf, "conf", torch.float32), _dev(K, "K", torch.int32),
                   _dev(p, "p_out", torch.int32), _dev(r, "r_out", torch.float64), _stream(stream)),
           "d2sd_select_reanchor")
    return p, r


def tree_indptr(B: int, K, p, out=None, stream=None):
    """Device node offsets (int32 [batch+1]) of the trees of K [batch] and p [batch, Kmax]."""
    import torch
    batch = K.numel()
    kmax = p.shape[1] if p.dim() == 2 else 0
    ip = out if out is not None else torch.empty(batch + 1, dtype=torch.int32, device=K.device)
    i32 = torch.int32
    _check(_indptr(batch, B, kmax, _dev(K, "K", i32), _dev(p, "p", i32) if kmax else None,
                   _dev(ip, "node_indptr", i32), _stream(stream)), "d2sd_tree_indptr")
    return ip


def commit_accepted_kv(B: int, node_indptr, total_nodes: int, path_nodes, accept_len, k_tree, v_tree,
                       page_table, ctx_len, k_cache, v_cache, max_ctx_len: int, stream=None):
    """Append every request's accepted path K/V to its pages (in place on
    k_cache / v_cache) and advance ctx_len (in place). Shapes as in the header."""
    import torch
    code = {torch.float32: F32, torch.bfloat16: BF16}.get(k_cache.dtype)
    if code is None or k_tree.dtype != k_cache.dtype:
        raise ValueError("k/v cache and tree must share dtype float32 or bfloat16")
    i32 = torch.int32
    batch = ctx_len.numel()
    _check(_commit(batch, B, k_cache.shape[1], k_cache.shape[3], k_cache.shape[2], code, k_cache.shape[0],
                   page_table.shape[1], max_ctx_len, _dev(node_indptr, "node_indptr", i32), total_nodes,
                   _dev(path_nodes, "path_nodes", i32), _dev(accept_len, "accept_len", i32),
                   _dev(k_tree, "k_tree"), _dev(v_tree, "v_tree"), _dev(page_table, "page_table", i32),
                   _dev(ctx_len, "ctx_len", i32), _dev(k_cache, "k_cache"), _dev(v_cache, "v_cache"),
                   _stream(stream)), "d2sd_commit_accepted_kv")


# -------------------------------------------------------------- attention --

def attn_args(q, k_cache, v_cache, page_table, ctx_len, k_tree, v_tree, node_indptr, anc_mask, out, lse, *,
              total_nodes: int, max_nodes: int, max_ctx_len: int, stage: int = STAGE_CASCADE,
              sm_scale: float = 0.0, kv_split: int = 0, node_indptr_host=None, row_group: int = 0,
              packed: int = 0) -> AttnArgs:
    """Fill a d2sd_attn_args from tensors (shapes as documented in the header).
    node_indptr_host: optional host copy of node_indptr (the automatic split
    then counts the work items exactly)."""
    import torch
    dt = q.dtype
    code = {torch.float32: F32, torch.bfloat16: BF16}.get(dt)
    if code is None:
        raise ValueError(f"q dtype {dt} unsupported (float32 or bfloat16)")
    i32 = torch.int32
    a = AttnArgs()
    a.batch = ctx_len.numel()
    a.num_qo_heads = q.shape[1]
    a.num_kv_heads = k_cache.shape[1]
    a.head_dim = q.shape[2]
    a.page_size = k_cache.shape[2]
    a.dtype = code
    a.stage = stage
    a.sm_scale = sm_scale
    a.total_nodes = total_nodes
    a.max_nodes = max_nodes
    a.max_ctx_len = max_ctx_len
    a.num_pages = k_cache.shape[0]
    a.max_pages = page_table.shape[1]
    a.mask_words = anc_mask.shape[1] if anc_mask is not None else 0
    a.kv_split = kv_split
    a.row_group = row_group
    a.packed = packed
    a.q = _dev(q, "q", dt)
    a.k_cache = _dev(k_cache, "k_cache", dt)
    a.v_cache = _dev(v_cache, "v_cache", dt)
    a.page_table = _dev(page_table, "page_table", i32)
    a.ctx_len = _dev(ctx_len, "ctx_len", i32)
    a.k_tree = _dev(k_tree, "k_tree", dt)
    a.v_tree = _dev(v_tree, "v_tree", dt)
    a.node_indptr = _dev(node_indptr, "node_indptr", i32)
    a.anc_mask = _dev(anc_mask, "anc_mask", i32)
    a.out = _dev(out, "out", dt)
    a.lse = _dev(lse, "lse", torch.float32)
    if node_indptr_host is not None:
        ip = _host_i32(node_indptr_host)
        if ip.shape != (a.batch + 1,):
            raise ValueError(f"node_indptr_host must have {a.batch + 1} entries, got {ip.shape}")
        a.node_indptr_host = ip.ctypes.data
        a.keep(ip)
    return a


def cascade_workspace_size(args: AttnArgs) -> int:
    n = ctypes.c_size_t(0)
    _check(_ws_size(ctypes.byref(args), ctypes.byref(n)), "d2sd_cascade_workspace_size")
    return n.value


def cascade_row_group(args: AttnArgs) -> int:
    """Query rows per workgroup (128 or 384) of the call's plan."""
    return cascade_shape(args)[0]


def cascade_shape(args: AttnArgs) -> tuple:
    """(rows per workgroup, packed) of the call's plan."""
    n = ctypes.c_int(0)
    pk = ctypes.c_int(0)
    _check(_row_group(ctypes.byref(args), ctypes.byref(n), ctypes.byref(pk)), "d2sd_cascade_row_group")
    return n.value, bool(pk.value)


def cascade_kv_split(args: AttnArgs) -> int:
    n = ctypes.c_int(0)
    _check(_kv_split(ctypes.byref(args), ctypes.byref(n)), "d2sd_cascade_kv_split")
    return n.value


def cascade_verify_attention(q, k_cache, v_cache, page_table, ctx_len, k_tree, v_tree, node_indptr, anc_mask,
                             *, total_nodes: int, max_nodes: int, max_ctx_len: int, stage: int = STAGE_CASCADE,
                             sm_scale: float = 0.0, kv_split: int = 0, out=None, lse=None, workspace=None,
                             want_lse: bool = True, node_indptr_host=None, row_group: int = 0, packed: int = 0,
                             stream=None):
    """Verify attention; returns (out, lse). The workspace is allocated when not given."""
    import torch
    if out is None:
        out = torch.empty_like(q)
    if lse is None and want_lse:
        lse = torch.empty(q.shape[:2], dtype=torch.float32, device=q.device)
    a = attn_args(q, k_cache, v_cache, page_table, ctx_len, k_tree, v_tree, node_indptr, anc_mask, out, lse,
                  total_nodes=total_nodes, max_nodes=max_nodes, max_ctx_len=max_ctx_len, stage=stage,
                  sm_scale=sm_scale, kv_split=kv_split, node_indptr_host=node_indptr_host, row_group=row_group,
                  packed=packed)
    need = cascade_workspace_size(a)
    if workspace is None and need > 0:
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
    ws_ptr = _dev(workspace, "workspace") if workspace is not None else None
    ws_len = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(_cascade(ctypes.byref(a), ws_ptr, ws_len, _stream(stream)), "d2sd_cascade_verify_attention")
    return out, lse


def cascade_verify_attention_noalloc(q, k_cache, v_cache, page_table, ctx_len, k_tree, v_tree, node_indptr,
                                     anc_mask, *, total_nodes: int, max_nodes: int, max_ctx_len: int,
                                     stage: int = STAGE_CASCADE, sm_scale: float = 0.0, kv_split: int = 0, out,
                                     lse=None, node_indptr_host=None, row_group: int = 0, packed: int = 0,
                                     stream=None):
    """Verify attention through the allocation-free entry point: the caller
    passes the outputs, the split partial states use the library's static
    device scratch. Returns (out, lse)."""
    a = attn_args(q, k_cache, v_cache, page_table, ctx_len, k_tree, v_tree, node_indptr, anc_mask, out, lse,
                  total_nodes=total_nodes, max_nodes=max_nodes, max_ctx_len=max_ctx_len, stage=stage,
                  sm_scale=sm_scale, kv_split=kv_split, node_indptr_host=node_indptr_host, row_group=row_group,
                  packed=packed)
    _check(_cascade_noalloc(ctypes.byref(a), _stream(stream)), "d2sd_cascade_verify_attention_noalloc")
    return out, lse


def noncascade_verify_attention(q, k_cache, v_cache, page_table, ctx_len, k_tree, v_tree, node_indptr,
                                anc_mask, *, total_nodes: int, max_nodes: int, max_ctx_len: int,
                                sm_scale: float = 0.0, out=None, lse=None, want_lse: bool = True, stream=None):
    """Comparison baseline: same attention, context re-read per tree node."""
    import torch
    if out is None:
        out = torch.empty_like(q)
    if lse is None and want_lse:
        lse = torch.empty(q.shape[:2], dtype=torch.float32, device=q.device)
    a = attn_args(q, k_cache, v_cache, page_table, ctx_len, k_tree, v_tree, node_indptr, anc_mask, out, lse,
                  total_nodes=total_nodes, max_nodes=max_nodes, max_ctx_len=max_ctx_len)
    _check(_noncascade(ctypes.byref(a), _stream(stream)), "d2sd_noncascade_verify_attention")
    return out, lse


def merge_state(o_a, lse_a, o_b, lse_b, o_out=None, lse_out=None, stream=None):
    """LSE merge of two fp32 states o [rows, D], lse [rows]."""
    import torch
    rows, D = o_a.shape
    f32 = torch.float32
    o_out = torch.empty_like(o_a) if o_out is None else o_out
    lse_out = torch.empty_like(lse_a) if lse_out is None else lse_out
    _check(_merge(rows, D, _dev(o_a, "o_a", f32), _dev(lse_a, "lse_a", f32), _dev(o_b, "o_b", f32),
                  _dev(lse_b, "lse_b", f32), _dev(o_out, "o_out", f32), _dev(lse_out, "lse_out", f32),
                  _stream(stream)), "d2sd_merge_state")
    return o_out, lse_out


# ----------------------------------------------------------------- accept --

def accept_path(B: int, node_indptr, total_nodes: int, parent, depth, path_id, draft_tokens, target_argmax,
                out: dict | None = None, stream=None) -> dict:
    """Greedy longest accepted path; returns dict of device int32 tensors."""
    import torch
    batch = node_indptr.numel() - 1
    dev = node_indptr.device
    o = out or {}
    i32 = torch.int32
    res = dict(
        accept_len=(o["accept_len"] if "accept_len" in o else torch.empty(batch, dtype=i32, device=dev)),
        best_path=(o["best_path"] if "best_path" in o else torch.empty(batch, dtype=i32, device=dev)),
        accept_node=(o["accept_node"] if "accept_node" in o else torch.empty(batch, dtype=i32, device=dev)),
        path_nodes=(o["path_nodes"] if "path_nodes" in o else torch.empty((batch, B), dtype=i32, device=dev)),
        out_tokens=(o["out_tokens"] if "out_tokens" in o else torch.empty((batch, B), dtype=i32, device=dev)),
    )
    _check(_accept(batch, B, _dev(node_indptr, "node_indptr", i32), total_nodes, _dev(parent, "parent", i32),
                   _dev(depth, "depth", i32), _dev(path_id, "path_id", i32),
                   _dev(draft_tokens, "draft_tokens", i32), _dev(target_argmax, "target_argmax", i32),
                   _dev(res["accept_len"], "accept_len", i32), _dev(res["best_path"], "best_path", i32),
                   _dev(res["accept_node"], "accept_node", i32), _dev(res["path_nodes"], "path_nodes", i32),
                   _dev(res["out_tokens"], "out_tokens", i32), _stream(stream)), "d2sd_accept_path")
    return res


# -------------------------------------------------- sampling verification --

def sample_targets(node_indptr, total_nodes: int, max_nodes: int, parent, draft_tokens, logits,
                   temperature: float, uniform=None, want_rep: bool = False, out=None, rep_out=None, stream=None):
    """Target token at every tree node from its logits row (float32 or
    bfloat16 [ΣN, vocab]): a draw by inversion with `uniform` (float32 [ΣN])
    at temperature > 0, the argmax at 0; nodes with one context share the draw
    of their representative. Returns (tokens int32 [ΣN], reps int32 [ΣN] or None)."""
    import torch
    code = {torch.float32: F32, torch.bfloat16: BF16}.get(logits.dtype)
    if code is None:
        raise ValueError(f"logits dtype {logits.dtype} unsupported (float32 or bfloat16)")
    if logits.dim() != 2 or logits.shape[0] < total_nodes:
        raise ValueError(f"logits must be [>= {total_nodes}, vocab], got {tuple(logits.shape)}")
    batch = node_indptr.numel() - 1
    dev = node_indptr.device
    i32 = torch.int32
    tokens = out if out is not None else torch.empty(max(total_nodes, 1), dtype=i32, device=dev)
    reps = rep_out if rep_out is not None else (torch.empty(max(total_nodes, 1), dtype=i32, device=dev)
                                                if want_rep else None)
    _check(_sample(batch, _dev(node_indptr, "node_indptr", i32), total_nodes, max_nodes, _dev(parent, "parent", i32),
                   _dev(draft_tokens, "draft_tokens", i32), logits.shape[1], code, _dev(logits, "logits"),
                   float(temperature), _dev(uniform, "uniform", torch.float32), _dev(reps, "context_rep", i32),
                   _dev(tokens, "target_tokens", i32), _stream(stream)), "d2sd_sample_targets")
    return tokens[:total_nodes], (reps[:total_nodes] if reps is not None else None)


# ---------------------------------------------------------------- timing --

def kernel_timing_enable(on: bool = True):
    _check(_timing_enable(1 if on else 0), "d2sd_kernel_timing_enable")


def kernel_timing_collect():
    """(calls, total_ms) of the attention operations (main kernel + split merge) since the last collect."""
    n = ctypes.c_int(0)
    ms = ctypes.c_double(0.0)
    _check(_timing_collect(ctypes.byref(n), ctypes.byref(ms)), "d2sd_kernel_timing_collect")
    return n.value, ms.value


def kernel_timing_collect_each(capacity: int = 4096):
    """Durations (ms, call order) of the attention operations (main kernel + split merge) since the last collect."""
    buf = (ctypes.c_float * capacity)()
    n = ctypes.c_int(0)
    _check(_timing_each(capacity, buf, ctypes.byref(n)), "d2sd_kernel_timing_collect_each")
    return [float(buf[i]) for i in range(min(n.value, capacity))]


def kernel_timing_collect_parts(capacity: int = 4096):
    """(kernel_ms, merge_ms) lists, call order: the main kernel and the split merge of each call."""
    kb = (ctypes.c_float * capacity)()
    mb = (ctypes.c_float * capacity)()
    n = ctypes.c_int(0)
    _check(_timing_parts(capacity, kb, mb, ctypes.byref(n)), "d2sd_kernel_timing_collect_parts")
    m = min(n.value, capacity)
    return [float(kb[i]) for i in range(m)], [float(mb[i]) for i in range(m)]
