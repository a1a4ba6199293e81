"""Device-resident verify batch: uploads host arrays once and runs the three
C-ABI steps (attention, argmax, accept) on them.

Marshalling only: tensors are allocated with torch and every computation
is a call into ``libadaserve.so``.
"""
from __future__ import annotations

from typing import Optional

import numpy as np

from . import (ADASERVE_BF16, ADASERVE_F32, MAX_TREE_NODES, adaserve_node_argmax,
               adaserve_tree_accept, adaserve_tree_attn_verify,
               adaserve_tree_attn_workspace_bytes, adaserve_tree_verify_step)


def to_device(a: np.ndarray, dtype: str, device):
    """Host array -> device tensor; uint16 arrays are bf16 bit patterns."""
    import torch
    if dtype == "bf16" and a.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


class DeviceBatch:
    """All inputs and outputs of one verify pass, resident in device memory."""

    def __init__(self, batch, device="cuda", max_accept: int = MAX_TREE_NODES):
        import torch
        self.batch = batch
        self.device = device
        self.dtype_code = ADASERVE_BF16 if batch.dtype == "bf16" else ADASERVE_F32
        i32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(device)
        self.node_indptr_host = np.ascontiguousarray(batch.node_indptr, dtype=np.int32)
        self.prefix_len_host = np.ascontiguousarray(batch.prefix_len, dtype=np.int32)
        self.node_indptr = i32(batch.node_indptr)
        self.parent = i32(batch.parent)
        self.prefix_len = i32(batch.prefix_len)
        self.block_table = i32(batch.block_table)
        self.draft_tokens = i32(batch.draft_tokens)
        dt = batch.dtype
        self.q = to_device(batch.q, dt, device)
        self.k_tree = to_device(batch.k_tree, dt, device)
        self.v_tree = to_device(batch.v_tree, dt, device)
        self.k_pages = to_device(batch.k_pages, dt, device)
        self.v_pages = to_device(batch.v_pages, dt, device)
        self.logits = to_device(batch.logits, dt, device)
        T, B = batch.total_nodes, batch.num_requests
        self.out = torch.empty_like(self.q)
        ws = adaserve_tree_attn_workspace_bytes(self.node_indptr_host, self.prefix_len_host,
                                                batch.num_q_heads, batch.num_kv_heads,
                                                batch.head_dim, batch.page_size, self.dtype_code)
        self.workspace_bytes = ws
        self.workspace = torch.zeros(max(ws, 256), dtype=torch.uint8, device=device) if ws else None
        self.max_accept = int(max_accept)
        self.target_argmax = torch.empty(T, dtype=torch.int32, device=device)
        self.accept_len = torch.empty(B, dtype=torch.int32, device=device)
        self.accept_tokens = torch.empty(B, self.max_accept, dtype=torch.int32, device=device)
        self.accept_nodes = torch.empty(B, self.max_accept, dtype=torch.int32, device=device)

    def attention(self, stream=None) -> None:
        adaserve_tree_attn_verify(
            node_indptr=self.node_indptr, node_indptr_host=self.node_indptr_host,
            parent=self.parent, q=self.q, k_tree=self.k_tree, v_tree=self.v_tree,
            k_pages=self.k_pages, v_pages=self.v_pages, block_table=self.block_table,
            prefix_len=self.prefix_len, prefix_len_host=self.prefix_len_host,
            sm_scale=self.batch.sm_scale, out=self.out, workspace=self.workspace, stream=stream)

    def argmax(self, stream=None) -> None:
        adaserve_node_argmax(self.logits, self.batch.vocab, self.target_argmax, stream=stream)

    def accept(self, stream=None) -> None:
        adaserve_tree_accept(node_indptr=self.node_indptr, parent=self.parent,
                             draft_tokens=self.draft_tokens, target_argmax=self.target_argmax,
                             max_accept=self.max_accept, accept_len=self.accept_len,
                             accept_tokens=self.accept_tokens, accept_nodes=self.accept_nodes,
                             stream=stream)

    def step(self, stream=None) -> None:
        """One verification pass: attention, argmax, acceptance (three calls)."""
        self.attention(stream)
        self.argmax(stream)
        self.accept(stream)

    def fused_step(self, stream=None) -> None:
        """The same pass through adaserve_tree_verify_step (one call)."""
        adaserve_tree_verify_step(
            node_indptr=self.node_indptr, node_indptr_host=self.node_indptr_host, parent=self.parent,
            q=self.q, k_tree=self.k_tree, v_tree=self.v_tree, k_pages=self.k_pages, v_pages=self.v_pages,
            block_table=self.block_table, prefix_len=self.prefix_len, prefix_len_host=self.prefix_len_host,
            sm_scale=self.batch.sm_scale, logits=self.logits, vocab=self.batch.vocab,
            draft_tokens=self.draft_tokens, max_accept=self.max_accept, out=self.out,
            target_argmax=self.target_argmax, accept_len=self.accept_len, accept_tokens=self.accept_tokens,
            accept_nodes=self.accept_nodes, workspace=self.workspace, stream=stream)

    def results(self):
        """Host copies: (out as float32 ndarray, argmax, accept_len, tokens, nodes)."""
        import torch
        torch.cuda.synchronize()
        out = self.out.float().cpu().numpy()
        return (out, self.target_argmax.cpu().numpy(), self.accept_len.cpu().numpy(),
                self.accept_tokens.cpu().numpy(), self.accept_nodes.cpu().numpy())
