"""MI355X (gfx950) batched tree verification for SLO-customised speculative decoding.

Python binding of the C ABI in ``include/adaserve.h``.  The functions here
only marshal arguments (torch tensors -> device pointers, host mirrors ->
host pointers) and raise on a non-OK status; every step of the computation
runs in the library's HIP kernels.  The library must have been built
(``python -m paper_2501_12162_amd.build``); importing the binding does not
require it, but the first call fails loudly when it is missing.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

from .build import LIB_PATH

ADASERVE_OK = 0
ADASERVE_ERR_INVALID_ARGUMENT = 1
ADASERVE_ERR_UNSUPPORTED = 2
ADASERVE_ERR_WORKSPACE = 3
ADASERVE_ERR_DEVICE = 4
ADASERVE_F32 = 0
ADASERVE_BF16 = 1
MAX_TREE_NODES = 128
TREE_ATTN_SCRATCH_BYTES = 32 << 20

_STATUS_NAMES = {1: "INVALID_ARGUMENT", 2: "UNSUPPORTED", 3: "WORKSPACE", 4: "DEVICE"}

# Every function the header declares, with its ctypes signature.
_P, _I32, _I64, _F32, _SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_size_t
SIGNATURES = {
    "adaserve_tree_attn_workspace_bytes": (_SZ, [_I32, _P, _P, _I32, _I32, _I32, _I32, _I32]),
    "adaserve_tree_attn_verify": (_I32, [_I32, _P, _P, _P, _P, _P, _P, _P, _P, _I32, _P, _I32, _P, _P,
                                         _I32, _I32, _I32, _I32, _F32, _I32, _P, _P, _SZ, _P]),
    "adaserve_tree_attn_verify_noalloc": (_I32, [_I32, _P, _P, _P, _P, _P, _P, _P, _P, _I32, _P, _I32, _P,
                                                 _P, _I32, _I32, _I32, _I32, _F32, _I32, _P, _P]),
    "adaserve_tree_verify_step": (_I32, [_I32, _P, _P, _P, _P, _P, _P, _P, _P, _I32, _P, _I32, _P, _P,
                                         _I32, _I32, _I32, _I32, _F32, _I32, _P, _I64, _I32, _P, _I32,
                                         _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "adaserve_node_argmax": (_I32, [_P, _I64, _I32, _I32, _I32, _P, _P]),
    "adaserve_tree_accept": (_I32, [_I32, _I32, _P, _P, _P, _P, _I32, _P, _P, _P, _P]),
    "adaserve_commit_accepted_kv": (_I32, [_I32, _P, _P, _P, _I32, _P, _P, _P, _P, _I32, _P, _I32, _P,
                                           _I32, _I32, _I32, _I32, _P, _P]),
    "adaserve_select_trees": (_I32, [_I32, _I32, _P, _P, _P, _P, _I32, _I32, _I32, _P, _P, _P, _P]),
    "adaserve_beam_step_workspace_bytes": (_SZ, [_I32, _I32, _I32, _I32, _I32]),
    "adaserve_beam_step": (_I32, [_I32, _I32, _P, _I64, _I32, _I32, _P, _I32, _P, _P, _P, _P, _SZ, _P]),
    "adaserve_tree_accept_sampled_workspace_bytes": (_SZ, [_I32]),
    "adaserve_tree_accept_sampled": (_I32, [_I32, _I32, _P, _P, _P, _P, _P, _I64, _I32, _I32, _P, _P, _I32,
                                            _P, _P, _P, _P, _SZ, _P]),
    "adaserve_last_error": (ctypes.c_char_p, []),
}

_lib = None


class AdaserveError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__("%s (%d): %s" % (_STATUS_NAMES.get(status, "?"), status, message))
        self.status = status


def load_library(path: Optional[str] = None) -> ctypes.CDLL:
    """Load ``libadaserve.so``; raises when it has not been built."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or library_path()
    if not os.path.exists(p):
        raise ImportError("libadaserve.so is not built (%s); run `python -m paper_2501_12162_amd.build`" % p)
    lib = ctypes.CDLL(p)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    if path is None:
        _lib = lib
    return lib


def library_path() -> str:
    """The in-tree build, or the build named by ADASERVE_LIBRARY (the CPU
    sanitizer run points it at an instrumented build of the same sources)."""
    return os.environ.get("ADASERVE_LIBRARY") or LIB_PATH


def _check(status: int) -> None:
    if status != ADASERVE_OK:
        msg = load_library().adaserve_last_error()
        raise AdaserveError(status, msg.decode() if msg else "")


def _dptr(t) -> Optional[int]:
    """Device pointer of a torch tensor (None -> NULL)."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("expected a device tensor")
    if not t.is_contiguous():
        raise ValueError("expected a contiguous tensor")
    return t.data_ptr()


def _host_i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a), dtype=np.int32)


def _stream(stream) -> Optional[int]:
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.bfloat16:
        return ADASERVE_BF16
    if t.dtype == torch.float32:
        return ADASERVE_F32
    raise ValueError("tensors must be bfloat16 or float32")


def adaserve_tree_attn_workspace_bytes(node_indptr_host, prefix_len_host, num_q_heads: int,
                                       num_kv_heads: int, head_dim: int, page_size: int,
                                       dtype: int) -> int:
    ip, pl = _host_i32(node_indptr_host), _host_i32(prefix_len_host)
    n = load_library().adaserve_tree_attn_workspace_bytes(
        int(pl.size), ip.ctypes.data, pl.ctypes.data, int(num_q_heads), int(num_kv_heads),
        int(head_dim), int(page_size), int(dtype))
    if n == ctypes.c_size_t(-1).value:
        _check(ADASERVE_ERR_INVALID_ARGUMENT)
    return int(n)


def adaserve_tree_attn_verify(*, node_indptr, node_indptr_host, parent, q, k_tree, v_tree,
                              k_pages, v_pages, block_table, prefix_len, prefix_len_host,
                              sm_scale: float, out, workspace=None, stream=None) -> None:
    """Tree attention; shapes: q/out [T, Hq, D], k_tree/v_tree [T, Hkv, D],
    k_pages/v_pages [P, Hkv, page_size, D], block_table [B, stride]."""
    ip, pl = _host_i32(node_indptr_host), _host_i32(prefix_len_host)
    T, Hq, D = q.shape
    Hkv = k_tree.shape[1]
    P, ps = k_pages.shape[0], k_pages.shape[2]
    bt_stride = block_table.shape[1] if block_table.dim() == 2 else 0
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = load_library().adaserve_tree_attn_verify(
        int(pl.size), _dptr(node_indptr), ip.ctypes.data, _dptr(parent), _dptr(q), _dptr(k_tree),
        _dptr(v_tree), _dptr(k_pages), _dptr(v_pages), int(P), _dptr(block_table), int(bt_stride),
        _dptr(prefix_len), pl.ctypes.data, int(Hq), int(Hkv), int(D), int(ps), float(sm_scale),
        _dtype_code(q), _dptr(out), _dptr(workspace), int(ws_bytes), _stream(stream))
    _check(st)


def adaserve_tree_attn_verify_noalloc(*, node_indptr, node_indptr_host, parent, q, k_tree, v_tree,
                                      k_pages, v_pages, block_table, prefix_len, prefix_len_host,
                                      sm_scale: float, out, stream=None) -> None:
    """Tree attention with the split-KV partials in the library's static
    scratch (no workspace argument, nothing allocated); arguments as
    ``adaserve_tree_attn_verify``."""
    ip, pl = _host_i32(node_indptr_host), _host_i32(prefix_len_host)
    T, Hq, D = q.shape
    Hkv = k_tree.shape[1]
    P, ps = k_pages.shape[0], k_pages.shape[2]
    bt_stride = block_table.shape[1] if block_table.dim() == 2 else 0
    st = load_library().adaserve_tree_attn_verify_noalloc(
        int(pl.size), _dptr(node_indptr), ip.ctypes.data, _dptr(parent), _dptr(q), _dptr(k_tree),
        _dptr(v_tree), _dptr(k_pages), _dptr(v_pages), int(P), _dptr(block_table), int(bt_stride),
        _dptr(prefix_len), pl.ctypes.data, int(Hq), int(Hkv), int(D), int(ps), float(sm_scale),
        _dtype_code(q), _dptr(out), _stream(stream))
    _check(st)


def adaserve_tree_verify_step(*, node_indptr, node_indptr_host, parent, q, k_tree, v_tree, k_pages, v_pages,
                              block_table, prefix_len, prefix_len_host, sm_scale: float, logits, vocab: int,
                              draft_tokens, max_accept: int, out, target_argmax, accept_len, accept_tokens,
                              accept_nodes, workspace=None, stream=None) -> None:
    """Attention, argmax and acceptance of one verification pass in one call;
    arguments as ``adaserve_tree_attn_verify``, ``adaserve_node_argmax`` and
    ``adaserve_tree_accept`` (logits [T, row_stride])."""
    ip, pl = _host_i32(node_indptr_host), _host_i32(prefix_len_host)
    T, Hq, D = q.shape
    Hkv = k_tree.shape[1]
    P, ps = k_pages.shape[0], k_pages.shape[2]
    bt_stride = block_table.shape[1] if block_table.dim() == 2 else 0
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = load_library().adaserve_tree_verify_step(
        int(pl.size), _dptr(node_indptr), ip.ctypes.data, _dptr(parent), _dptr(q), _dptr(k_tree),
        _dptr(v_tree), _dptr(k_pages), _dptr(v_pages), int(P), _dptr(block_table), int(bt_stride),
        _dptr(prefix_len), pl.ctypes.data, int(Hq), int(Hkv), int(D), int(ps), float(sm_scale),
        _dtype_code(q), _dptr(logits), int(logits.shape[1]), int(vocab), _dptr(draft_tokens), int(max_accept),
        _dptr(out), _dptr(target_argmax), _dptr(accept_len), _dptr(accept_tokens), _dptr(accept_nodes),
        _dptr(workspace), int(ws_bytes), _stream(stream))
    _check(st)


def adaserve_node_argmax(logits, vocab: int, argmax_out, stream=None) -> None:
    """Row argmax of ``logits`` [rows, row_stride] over columns ``0..vocab-1``."""
    rows, stride = logits.shape
    st = load_library().adaserve_node_argmax(_dptr(logits), int(stride), int(rows), int(vocab),
                                             _dtype_code(logits), _dptr(argmax_out), _stream(stream))
    _check(st)


def adaserve_tree_accept(*, node_indptr, parent, draft_tokens, target_argmax, max_accept: int,
                         accept_len, accept_tokens, accept_nodes, stream=None) -> None:
    """Longest accepted path per request (outputs [B], [B, max_accept], [B, max_accept])."""
    B = node_indptr.shape[0] - 1
    st = load_library().adaserve_tree_accept(
        int(B), int(parent.shape[0]), _dptr(node_indptr), _dptr(parent), _dptr(draft_tokens),
        _dptr(target_argmax), int(max_accept), _dptr(accept_len), _dptr(accept_tokens),
        _dptr(accept_nodes), _stream(stream))
    _check(st)


def adaserve_commit_accepted_kv(*, node_indptr, accept_len, accept_nodes, k_tree, v_tree, k_pages,
                                v_pages, block_table, prefix_len, new_prefix_len, stream=None) -> None:
    """Write the accepted paths' K/V rows into the paged cache at L_r .. L_r + len - 1.
    accept_nodes [B, max_accept]; k_tree/v_tree [T, Hkv, D]; k_pages/v_pages [P, Hkv, ps, D]."""
    B = node_indptr.shape[0] - 1
    _, Hkv, D = k_tree.shape
    P, ps = k_pages.shape[0], k_pages.shape[2]
    bt_stride = block_table.shape[1] if block_table.dim() == 2 else 0
    st = load_library().adaserve_commit_accepted_kv(
        int(B), _dptr(node_indptr), _dptr(accept_len), _dptr(accept_nodes), int(accept_nodes.shape[1]),
        _dptr(k_tree), _dptr(v_tree), _dptr(k_pages), _dptr(v_pages), int(P), _dptr(block_table),
        int(bt_stride), _dptr(prefix_len), int(Hkv), int(D), int(ps), _dtype_code(k_tree),
        _dptr(new_prefix_len), _stream(stream))
    _check(st)


def adaserve_select_trees(*, cand_indptr, cand_parent, cand_prob, need, budget: int, n_max: int,
                          tree_size, tree_parent, tree_cand, stream=None) -> None:
    """Draft trees from candidate trees (tree_parent / tree_cand [B, max_nodes], max_nodes >= 128)."""
    B = cand_indptr.shape[0] - 1
    st = load_library().adaserve_select_trees(
        int(B), int(cand_prob.shape[0]), _dptr(cand_indptr), _dptr(cand_parent), _dptr(cand_prob),
        _dptr(need), int(budget), int(n_max), int(tree_parent.shape[1]), _dptr(tree_size),
        _dptr(tree_parent), _dptr(tree_cand), _stream(stream))
    _check(st)



def adaserve_beam_step_workspace_bytes(num_requests: int, beam_in: int, vocab: int, beam_out: int,
                                       dtype: int) -> int:
    n = load_library().adaserve_beam_step_workspace_bytes(int(num_requests), int(beam_in), int(vocab),
                                                          int(beam_out), int(dtype))
    if n == ctypes.c_size_t(-1).value:
        _check(ADASERVE_ERR_INVALID_ARGUMENT)
    return int(n)


def adaserve_beam_step(*, logits, vocab: int, beam_logprob, out_parent, out_token, out_logprob,
                       workspace, stream=None) -> None:
    """One beam-search step.  logits [num_requests * beam_in, row_stride];
    beam_logprob [num_requests, beam_in] float32; outputs [num_requests, beam_out]."""
    B, w_in = beam_logprob.shape
    rows, stride = logits.shape
    if rows != B * w_in:
        raise ValueError("logits has %d rows, beam_logprob asks for %d" % (rows, B * w_in))
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = load_library().adaserve_beam_step(
        int(B), int(w_in), _dptr(logits), int(stride), int(vocab), _dtype_code(logits), _dptr(beam_logprob),
        int(out_parent.shape[1]), _dptr(out_parent), _dptr(out_token), _dptr(out_logprob), _dptr(workspace),
        int(ws_bytes), _stream(stream))
    _check(st)


def adaserve_tree_accept_sampled_workspace_bytes(total_nodes: int) -> int:
    n = load_library().adaserve_tree_accept_sampled_workspace_bytes(int(total_nodes))
    if n == ctypes.c_size_t(-1).value:
        _check(ADASERVE_ERR_INVALID_ARGUMENT)
    return int(n)


def adaserve_tree_accept_sampled(*, node_indptr, parent, draft_tokens, target_logits, draft_logits, vocab: int,
                                 u_accept, u_bonus, max_accept: int, accept_len, accept_tokens, accept_nodes,
                                 workspace, stream=None) -> None:
    """Sampled-decoding tree verification; logits [T, row_stride] (temperature applied),
    u_accept / u_bonus [T] float32; workspace of adaserve_tree_accept_sampled_workspace_bytes(T)
    bytes; outputs as adaserve_tree_accept."""
    B = node_indptr.shape[0] - 1
    T, stride = target_logits.shape
    if draft_logits.shape != target_logits.shape or draft_logits.dtype != target_logits.dtype:
        raise ValueError("draft_logits must match target_logits in shape and dtype")
    st = load_library().adaserve_tree_accept_sampled(
        int(B), int(parent.shape[0]), _dptr(node_indptr), _dptr(parent), _dptr(draft_tokens),
        _dptr(target_logits), _dptr(draft_logits), int(stride), int(vocab), _dtype_code(target_logits),
        _dptr(u_accept), _dptr(u_bonus), int(max_accept), _dptr(accept_len), _dptr(accept_tokens),
        _dptr(accept_nodes), _dptr(workspace), int(0 if workspace is None else workspace.numel() * workspace.element_size()),
        _stream(stream))
    _check(st)
