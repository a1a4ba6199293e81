"""TEST INFRASTRUCTURE ONLY: the CPU oracle for batched tree verification.

A plain, slow, obviously correct evaluation (``oracle.c``, fp64, OpenMP)
of tree attention, per-node argmax and longest-accepted-path acceptance,
written from the paper's definitions (section 2 draft token trees;
section 3 Theorem 1 path acceptance; section 4.3 step 4 verification;
section 5.1 logits returned per node; Appendix B parents before children),
plus the accepted-path KV commit (``commit_kv``, plain numpy: section 5.1,
a request's verified tokens carried into its next iteration), the two selection
phases of Algorithm 2 (``select_trees``, section 4.3 steps 2-3) and one
beam-search speculation step (``beam_step``, section 4.3 step 1).

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It shares no code with the HIP
library and never imports it.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB_PATH = os.path.join(_HERE, "_build", "liboracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile ``oracle.c`` with gcc into ``oracle/_build/liboracle.so``."""
    if not force and os.path.exists(_LIB_PATH):
        return _LIB_PATH
    os.makedirs(os.path.dirname(_LIB_PATH), exist_ok=True)
    tmp = _LIB_PATH + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-Wall", "-Wextra",
           _SRC, "-o", tmp, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    path = os.environ.get("ADASERVE_ORACLE_LIB")   # an instrumented build (CPU sanitizer run)
    if not path:
        path = _LIB_PATH
        if not os.path.exists(path):
            build()
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    i32, i64, f64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_double
    lib.oracle_tree_attn.restype = i32
    lib.oracle_tree_attn.argtypes = [i32, P, P, P, P, i64, i32, P, P, P, P, P, i32,
                                     i32, i32, i32, i32, f64, i32, P, P]
    lib.oracle_node_argmax.restype = None
    lib.oracle_node_argmax.argtypes = [P, i64, i32, i32, i32, P]
    for name in ("oracle_tree_accept", "oracle_tree_accept_bruteforce"):
        fn = getattr(lib, name)
        fn.restype = None
        fn.argtypes = [i32, P, P, P, P, i32, P, P, P]
    lib.oracle_set_num_threads.restype = None
    lib.oracle_set_num_threads.argtypes = [i32]
    lib.oracle_get_num_threads.restype = i32
    lib.oracle_get_num_threads.argtypes = []
    _lib = lib
    return lib


def _ptr(a: np.ndarray) -> ctypes.c_void_p:
    return ctypes.c_void_p(a.ctypes.data)


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.int32)


def set_num_threads(n: int) -> None:
    _load().oracle_set_num_threads(int(n))


def num_threads() -> int:
    return int(_load().oracle_get_num_threads())


def tree_attn(*, node_indptr, parent, prefix_len, block_table, q, k_tree, v_tree,
              k_pages, v_pages, dtype: str, num_q_heads: int, num_kv_heads: int,
              head_dim: int, page_size: int, sm_scale: float,
              nodes: Optional[Sequence[int]] = None) -> np.ndarray:
    """Attention output (float64 ``[len(nodes), Hq, D]``) of the selected
    global node ids (all nodes when ``nodes`` is None)."""
    lib = _load()
    indptr = _i32(node_indptr)
    par = _i32(parent)
    L = _i32(prefix_len)
    bt = _i32(block_table)
    if bt.ndim != 2:
        raise ValueError("block_table must be 2-D")
    T = int(indptr[-1])
    sel = _i32(np.arange(T) if nodes is None else nodes)
    is_bf16 = 1 if dtype == "bf16" else 0
    want = np.uint16 if is_bf16 else np.float32
    arrs = [np.ascontiguousarray(a, dtype=want) for a in (q, k_tree, v_tree, k_pages, v_pages)]
    out = np.zeros((sel.size, num_q_heads, head_dim), dtype=np.float64)
    rc = lib.oracle_tree_attn(int(indptr.size - 1), _ptr(indptr), _ptr(par), _ptr(L), _ptr(bt),
                              int(bt.shape[1]), int(arrs[3].shape[0]),
                              *[_ptr(a) for a in arrs], is_bf16,
                              int(num_q_heads), int(num_kv_heads), int(head_dim), int(page_size),
                              float(sm_scale), int(sel.size), _ptr(sel), _ptr(out))
    if rc != 0:
        raise ValueError("oracle_tree_attn: malformed input")
    return out


def tree_attn_batch(batch, nodes: Optional[Sequence[int]] = None) -> np.ndarray:
    """``tree_attn`` on a ``VerifyBatch``."""
    return tree_attn(node_indptr=batch.node_indptr, parent=batch.parent,
                     prefix_len=batch.prefix_len, block_table=batch.block_table,
                     q=batch.q, k_tree=batch.k_tree, v_tree=batch.v_tree,
                     k_pages=batch.k_pages, v_pages=batch.v_pages, dtype=batch.dtype,
                     num_q_heads=batch.num_q_heads, num_kv_heads=batch.num_kv_heads,
                     head_dim=batch.head_dim, page_size=batch.page_size,
                     sm_scale=batch.sm_scale, nodes=nodes)


def node_argmax(logits: np.ndarray, vocab: int, dtype: str,
                rows: Optional[Sequence[int]] = None) -> np.ndarray:
    """First-maximum argmax of each logits row (or of the selected rows)."""
    lib = _load()
    want = np.uint16 if dtype == "bf16" else np.float32
    lg = np.ascontiguousarray(logits, dtype=want)
    if rows is not None:
        lg = np.ascontiguousarray(lg[np.asarray(rows, dtype=np.int64)])
    out = np.empty(lg.shape[0], dtype=np.int32)
    lib.oracle_node_argmax(_ptr(lg), int(lg.shape[1]), int(lg.shape[0]), int(vocab),
                           1 if dtype == "bf16" else 0, _ptr(out))
    return out


def _accept(fn_name, node_indptr, parent, draft_tokens, target_argmax, max_accept):
    lib = _load()
    indptr, par = _i32(node_indptr), _i32(parent)
    draft, amax = _i32(draft_tokens), _i32(target_argmax)
    B = int(indptr.size - 1)
    alen = np.empty(B, dtype=np.int32)
    tok = np.empty((B, max_accept), dtype=np.int32)
    nodes = np.empty((B, max_accept), dtype=np.int32)
    getattr(lib, fn_name)(B, _ptr(indptr), _ptr(par), _ptr(draft), _ptr(amax), int(max_accept),
                          _ptr(alen), _ptr(tok), _ptr(nodes))
    return alen, tok, nodes


def tree_accept(node_indptr, parent, draft_tokens, target_argmax, max_accept: int):
    """Topological acceptance: returns ``(accept_len, accept_tokens, accept_nodes)``."""
    return _accept("oracle_tree_accept", node_indptr, parent, draft_tokens, target_argmax,
                   max_accept)


def tree_accept_bruteforce(node_indptr, parent, draft_tokens, target_argmax, max_accept: int):
    """Acceptance by enumerating every root-to-leaf path (same outputs)."""
    return _accept("oracle_tree_accept_bruteforce", node_indptr, parent, draft_tokens,
                   target_argmax, max_accept)


def commit_kv(*, node_indptr, accept_len, accept_nodes, k_tree, v_tree, k_pages, v_pages,
              block_table, prefix_len, page_size: int):
    """Accepted-path KV commit (section 5.1: once verified, a request's tokens
    return with it to the pool of requests that the next iteration draws
    from; section 2: the root is the
    last generated token, so the accepted path root..i* is what the next
    iteration's prefix must hold).

    Reading: request r with len = accept_len[r] >= 1 commits rows k = 0, 1, ...
    in order: the tree row of local node accept_nodes[r, k] goes to cache
    position L_r + k (page block_table[r, (L_r + k) // page_size], slot
    (L_r + k) % page_size), every kv-head, K and V.  The first row whose node
    is outside the tree, whose position is past the block-table row or whose
    page id is outside the pool ends the commit.  A request with len < 1,
    len > max_accept or len > 128 (the tree-size limit) commits nothing.

    Works on copies: returns ``(k_pages, v_pages, new_prefix_len)`` with
    new_prefix_len[r] = L_r + rows committed.  Element-wise copies of whatever
    dtype the arrays hold (bf16 as uint16 bit patterns), so the result is
    bit-exact by construction.
    """
    indptr = np.asarray(node_indptr, dtype=np.int64)
    alen = np.asarray(accept_len, dtype=np.int64)
    nodes = np.asarray(accept_nodes, dtype=np.int64)
    bt = np.asarray(block_table, dtype=np.int64).reshape(len(alen), -1)
    plen = np.asarray(prefix_len, dtype=np.int64)
    kp, vp = np.array(k_pages, copy=True), np.array(v_pages, copy=True)
    num_pages = kp.shape[0]
    max_accept = nodes.shape[1]
    new_len = plen.copy()
    for r in range(len(alen)):
        n_r = int(indptr[r + 1] - indptr[r])
        length, L = int(alen[r]), int(plen[r])
        if length < 1 or length > max_accept or length > 128 or L < 0 or n_r < 1:
            continue
        done = 0
        for k in range(length):
            node = int(nodes[r, k])
            t = L + k
            e = t // page_size
            if not (0 <= node < n_r) or e >= bt.shape[1]:
                break
            page = int(bt[r, e])
            if not (0 <= page < num_pages):
                break
            row = int(indptr[r]) + node
            kp[page, :, t % page_size, :] = k_tree[row]
            vp[page, :, t % page_size, :] = v_tree[row]
            done += 1
        new_len[r] = L + done
    return kp, vp, new_len.astype(np.int32)



def select_trees(*, cand_indptr, cand_parent, cand_prob, need, budget: int, n_max: int,
                 max_nodes: int):
    """SLO-customised selection then throughput-optimised selection
    (Algorithm 2 after its speculation phase; section 4.3 steps 2 and 3).

    Every request starts with its root (one budget unit each).  Requests are
    visited in descending order of need (section 4.3 step 2: slower requests
    first; equal needs keep request order); each adds its best remaining
    candidate while the added path probabilities sum below need[r], the tree
    holds fewer than n_max nodes (root included) and budget remains.  Then the
    best remaining candidates of the whole batch are added while budget
    remains (step 3).

    Readings: the budget loops run while budget > 0 (the printed `B >= 0`
    would select one node more than the budget); "best" = highest path
    probability, ties to the smaller depth (a parent before its child), then
    (step 3) the smaller request, then the smaller local candidate index; the
    sum is accumulated in float32 in the order of selection, starting from
    0 (need[r] excludes the root's 1).  Output trees list the root first, then
    the selected candidates ordered by (depth, candidate index); tree_parent
    holds tree-local parents (root -1), tree_cand the candidate index (root -1).

    A request whose candidate tree is malformed -- more than 127 candidates, a
    parent that is not -1 or an earlier candidate, or a path probability
    outside (0, 1] or above its parent's (the root's is 1) -- takes no part:
    no budget, tree_size -1, rows of -1; an index array that does not start at
    0, decreases, or does not end at the candidate count voids every request.
    A NaN need asks for nothing and ranks last.
    """
    indptr = np.asarray(cand_indptr, dtype=np.int64)
    par = np.asarray(cand_parent, dtype=np.int64)
    prob = np.asarray(cand_prob, dtype=np.float32)
    need = np.asarray(need, dtype=np.float32)
    need = np.where(np.isnan(need), np.float32(-np.inf), need)   # a NaN need asks for nothing, ranks last
    B = int(indptr.size - 1)
    if B > 0 and (indptr[0] != 0 or indptr[-1] != par.size or (np.diff(indptr) < 0).any()):
        return (np.full(B, -1, np.int32), np.full((B, max_nodes), -1, np.int32),
                np.full((B, max_nodes), -1, np.int32))
    depth = np.zeros(par.size, dtype=np.int64)
    ok = np.ones(B, dtype=bool)
    for r in range(B):
        lo, hi = int(indptr[r]), int(indptr[r + 1])
        if hi - lo > 127 or hi < lo:
            ok[r] = False
            continue
        for i in range(lo, hi):
            p = int(par[i])
            fp = np.float32(1.0) if p == -1 else (prob[lo + p] if 0 <= p < i - lo else None)
            if fp is None or not (np.float32(0) < prob[i] <= fp):
                ok[r] = False
                break
            depth[i] = 1 if p < 0 else depth[lo + p] + 1
    added = np.zeros(par.size, dtype=bool)
    for r in range(B):           # candidates of malformed requests are never eligible
        if not ok[r]:
            added[int(indptr[r]):int(indptr[r + 1])] = True
    size = np.ones(B, dtype=np.int64)
    left = int(budget) - int(ok.sum())

    def best(cands):
        # highest probability; ties: smaller depth, then the lower index
        return min(cands, key=lambda i: (-float(prob[i]), int(depth[i]), i)) if cands else None

    order = sorted((r for r in range(B) if ok[r]), key=lambda r: (-float(need[r]), r))
    for r in order:
        acc = np.float32(0.0)
        while acc < need[r] and size[r] < n_max and left > 0:
            v = best([i for i in range(int(indptr[r]), int(indptr[r + 1])) if not added[i]])
            if v is None:
                break
            added[v] = True
            size[r] += 1
            acc = np.float32(acc + prob[v])
            left -= 1
    while left > 0:
        rest = [i for i in range(par.size) if not added[i]]
        if not rest:
            break
        v = best(rest)               # global index order = (request, local index)
        added[v] = True
        size[int(np.searchsorted(indptr, v, side="right") - 1)] += 1
        left -= 1

    tree_size = np.zeros(B, dtype=np.int32)
    tree_parent = np.full((B, max_nodes), -1, dtype=np.int32)
    tree_cand = np.full((B, max_nodes), -1, dtype=np.int32)
    for r in range(B):
        if not ok[r]:
            tree_size[r] = -1
            continue
        lo = int(indptr[r])
        sel = [i for i in range(lo, int(indptr[r + 1])) if added[i]]
        sel.sort(key=lambda i: (int(depth[i]), i))
        if 1 + len(sel) > max_nodes:
            raise ValueError("max_nodes too small")
        tid = {i: k + 1 for k, i in enumerate(sel)}
        tree_size[r] = 1 + len(sel)
        for i in sel:
            p = int(par[i])
            tree_parent[r, tid[i]] = 0 if p < 0 else tid[lo + p]
            tree_cand[r, tid[i]] = i - lo
    return tree_size, tree_parent, tree_cand


def beam_log_path_prob(logits, beam_logprob):
    """Log path probability of every child of every beam node (section 4.3
    step 1): log f(child) = log f(beam) + log softmax(draft logits of the
    beam)[token], in float64.  logits [B, w_in, V] (float values),
    beam_logprob [B, w_in].  A row with no finite logit, or a beam of log
    path probability -inf, has only children of probability 0 (-inf)."""
    x = np.asarray(logits, dtype=np.float64)
    lp = np.asarray(beam_logprob, dtype=np.float64)
    m = x.max(axis=2, keepdims=True)
    dead = ~np.isfinite(m)
    m = np.where(dead, 0.0, m)
    with np.errstate(divide="ignore", invalid="ignore"):
        lse = m + np.log(np.exp(x - m).sum(axis=2, keepdims=True))
        score = lp[:, :, None] + (x - lse)
    return np.where(dead, -np.inf, score)


def beam_step(*, logits, beam_logprob, w_out: int):
    """One beam-search speculation step (section 4.3 step 1): every beam node b
    of a request expands into all |V| tokens with path probability
    f(b) * softmax(draft logits of b)[t]; the w_out children with the highest
    path probability are kept.

    logits: [B, w_in, V] (float32 values; bf16 bit patterns are widened by
    the caller); beam_logprob: [B, w_in] natural-log path probabilities of the
    beam nodes (-inf for an unused slot).  Scores come from
    beam_log_path_prob (float64).
    Reading: ties go to the smaller beam index, then the smaller token id;
    outputs are sorted best first; children of path probability 0 (log -inf)
    are never kept, and slots past the last kept child hold parent -1,
    token -1, logprob -inf.  Returns (parent [B, w_out] int32, token
    [B, w_out] int32, logprob [B, w_out] float64).
    """
    score = beam_log_path_prob(logits, beam_logprob)       # [B, w_in, V]
    B, w_in, V = score.shape
    parent = np.full((B, w_out), -1, np.int32)
    token = np.full((B, w_out), -1, np.int32)
    out = np.full((B, w_out), -np.inf, np.float64)
    bb, tt = np.meshgrid(np.arange(w_in), np.arange(V), indexing="ij")
    for r in range(B):
        s = score[r].ravel()
        # lexicographic: highest score, then smaller beam, then smaller token
        order = np.lexsort((tt.ravel(), bb.ravel(), -s))[:w_out]
        order = order[np.isfinite(s[order])]
        k = order.size
        parent[r, :k] = bb.ravel()[order]
        token[r, :k] = tt.ravel()[order]
        out[r, :k] = s[order]
    return parent, token, out


def _sampled_tree_ok(par, n):
    if n < 1 or n > 128 or par[0] != -1:
        return False
    return all(0 <= par[i] < i for i in range(1, n))


def tree_accept_sampled(*, node_indptr, parent, draft_tokens, target_logits, draft_logits, vocab: int,
                        u_accept, u_bonus, max_accept: int):
    """Tree verification for sampled decoding: multi-step speculative
    sampling over the draft token tree (section 4.3 step 4 delegates
    verification to tree-based prior work; the reading here is the
    token-tree form of speculative sampling, lossless when each node's
    children were drawn independently from the draft distribution at that
    node).

    Row u of target_logits / draft_logits holds the target / draft model's
    logits after node u's root path (already divided by the sampling
    temperature); softmax gives p_u and q_u.  From the root: the children of
    the current node u are tried in index order; child c with token t is
    accepted when u_accept[c] * q_u(t) < p_res(t), i.e. with probability
    min(1, p_res(t) / q_u(t)); after a rejection p_res becomes
    max(0, p_res - q_u), renormalised.  An accepted child becomes the current
    node (its token is emitted); when no child is accepted (or u is a leaf)
    the bonus token is drawn from p_res by inverse CDF: the smallest v whose
    cumulative probability exceeds u_bonus[u], and the walk ends.  p_res
    starts as p_u at every node.  A rejection that leaves p_res without mass
    (possible only through rounding) ends the walk with the bonus drawn from
    p_res before it.

    Outputs follow tree_accept: accept_len = accepted drafts + 1, accept_nodes
    = the path from the root, accept_tokens = the accepted drafts' tokens then
    the bonus token; -1 for a malformed tree (as tree_accept), a draft token
    of a non-root node outside [0, vocab), a tree deeper than
    max_accept - 1, or a node with children whose draft row has no logit
    above -inf (q is then no distribution; NaN counts as none).  For callers comparing against float32 arithmetic, also
    returns per request the smallest relative margin of its acceptance tests
    (inf when it took none) and the cumulative distribution the bonus token
    was drawn from (None for a malformed request).  float64 throughout.
    """
    indptr = np.asarray(node_indptr, dtype=np.int64)
    par_all = np.asarray(parent, dtype=np.int64)
    draft = np.asarray(draft_tokens, dtype=np.int64)
    ua = np.asarray(u_accept, dtype=np.float64)
    ub = np.asarray(u_bonus, dtype=np.float64)
    B = indptr.size - 1
    alen = np.full(B, -1, np.int32)
    tok = np.full((B, max_accept), -1, np.int32)
    nodes = np.full((B, max_accept), -1, np.int32)
    margin = np.full(B, np.inf)
    bonus_cdf = [None] * B

    def softmax(row):
        x = np.asarray(row[:vocab], dtype=np.float64)
        e = np.exp(x - x.max())
        return e / e.sum()

    def draw(res, u):
        cdf = np.cumsum(res)
        v = int(np.searchsorted(cdf, u, side="right"))
        last = int(np.nonzero(res > 0)[0][-1])
        return min(v, last), cdf

    for r in range(B):
        base, n = int(indptr[r]), int(indptr[r + 1] - indptr[r])
        par = par_all[base:base + n]
        if not _sampled_tree_ok(par, n):
            continue
        depth = np.zeros(n, np.int64)
        for i in range(1, n):
            depth[i] = depth[par[i]] + 1
        if depth.max() > max_accept - 1 or any(not (0 <= draft[base + i] < vocab) for i in range(1, n)):
            continue
        if any(not np.any(np.asarray(draft_logits[base + j][:vocab], dtype=np.float64) > -np.inf)
               for j in set(int(x) for x in par[1:])):
            continue
        u, path, out, m = 0, [0], [], np.inf
        while True:
            p = softmax(target_logits[base + u])
            children = [i for i in range(u + 1, n) if par[i] == u]
            res = p
            nxt = None
            if children:
                q = softmax(draft_logits[base + u])
                for c in children:
                    t = int(draft[base + c])
                    lhs, rhs = ua[base + c] * q[t], res[t]
                    m = min(m, abs(rhs - lhs) / max(rhs, lhs, 1e-300))
                    if lhs < rhs:
                        nxt = c
                        break
                    left = np.maximum(res - q, 0.0)
                    if left.sum() <= 0.0:
                        break
                    res = left / left.sum()
            if nxt is None:
                v, cdf = draw(res, ub[base + u])
                bonus_cdf[r] = cdf
                out.append(v)
                break
            out.append(int(draft[base + nxt]))
            path.append(nxt)
            u = nxt
        k = len(path)
        alen[r] = k
        nodes[r, :k] = path
        tok[r, :k] = out
        margin[r] = m
    return alen, tok, nodes, margin, bonus_cdf
