"""Seeded synthetic inputs for batched tree verification.

This module only *draws* inputs: token trees, prefix lengths, a paged KV
pool, queries, per-node logits and draft tokens.  It holds none of the
verification arithmetic (no attention, no argmax, no acceptance), so both
the HIP path and the CPU oracle can consume what it produces without
sharing any of the method's code.

Shapes follow the paper's setting (speculation trees rooted at the last
generated token, section 2; budget = total tree nodes, Eq. 1; three SLO
classes, Table "slo"); the five named workloads mirror the Llama-3-8B and
70B attention shapes the evaluation uses (section 6.1).

Conventions shared by everything that consumes a ``VerifyBatch``:

* bf16 tensors are ``np.uint16`` arrays holding the raw bf16 bit patterns,
  produced from float32 draws by round-to-nearest-even.
* Trees are stored per request as local parent arrays: local node 0 is the
  root with parent -1 and every other node ``i`` has ``0 <= parent[i] < i``
  (a parent is always drafted before its children, Appendix B).
* The KV prefix lives in pages of ``page_size`` tokens, layout
  ``[num_pages, num_kv_heads, page_size, head_dim]``; request ``r`` owns the
  physical pages ``block_table[r, :ceil(L_r / page_size)]``.  Slots past
  ``L_r`` in a request's last page and every page no request owns are
  filled with NaN, so a consumer that reads them shows it.
* Logits carry a *planted* maximum: every row is drawn from a clipped
  normal and one position per row is then set to a value strictly above
  the clip; in a share ``tie_rate`` of the rows the same value is planted
  at two (sometimes three) distinct positions, the rate at which natural
  bf16 rows of a large vocabulary tie at their maximum.  ``planted_argmax``
  is the lowest planted position (an integer minimum over the positions
  drawn here) and draft tokens are drawn from it, so no argmax is ever
  computed here.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np

BF16_NAN = np.uint16(0x7FC0)


_CHUNK = 1 << 22


def _round_chunk(u: np.ndarray, t: np.ndarray, out: np.ndarray) -> None:
    np.right_shift(u, np.uint32(16), out=t)
    np.bitwise_and(t, np.uint32(1), out=t)
    np.add(t, u, out=t)
    np.add(t, np.uint32(0x7FFF), out=t)
    np.right_shift(t, np.uint32(16), out=t)
    out[...] = t


def f32_to_bf16_bits(x: np.ndarray, out: Optional[np.ndarray] = None) -> np.ndarray:
    """Round float32 values to bf16 (round to nearest, ties to even).

    Returns the bf16 bit patterns as uint16.  Inputs here are always finite.
    Works through the array in chunks so large tensors need no full-size
    temporaries.
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    if out is None:
        out = np.empty(x.shape, dtype=np.uint16)
    fi = x.reshape(-1).view(np.uint32)
    fo = out.reshape(-1)
    t = np.empty(min(_CHUNK, max(fi.size, 1)), dtype=np.uint32)
    for s in range(0, fi.size, _CHUNK):
        e = min(s + _CHUNK, fi.size)
        _round_chunk(fi[s:e], t[:e - s], fo[s:e])
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float32."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


# ---------------------------------------------------------------------------
# Tree shapes
# ---------------------------------------------------------------------------

def chain_tree(n: int) -> np.ndarray:
    """A chain of ``n`` nodes: node i's parent is i-1 (a draft *sequence*)."""
    p = np.arange(-1, n - 1, dtype=np.int32)
    return p


def random_tree(rng: np.random.Generator, n: int, max_depth: Optional[int] = None) -> np.ndarray:
    """Random rooted tree of ``n`` nodes in drafting order.

    Node i > 0 takes its parent uniformly among earlier nodes whose depth is
    below ``max_depth`` (all earlier nodes when ``max_depth`` is None), so the
    tree never gets deeper than ``max_depth`` (root depth 0).  The depth of
    each new node is tracked while the tree is drawn; it is bookkeeping for
    the cap, not part of the verification step.
    """
    parent = np.empty(n, dtype=np.int32)
    parent[0] = -1
    level = np.zeros(n, dtype=np.int64)
    for i in range(1, n):
        if max_depth is None:
            j = int(rng.integers(0, i))
        else:
            eligible = np.nonzero(level[:i] < max_depth)[0]
            j = int(eligible[rng.integers(0, eligible.size)])
        parent[i] = j
        level[i] = level[j] + 1
    return parent


# ---------------------------------------------------------------------------
# The batch container
# ---------------------------------------------------------------------------

@dataclass
class VerifyBatch:
    """Every input of one verification pass, as host arrays."""

    name: str
    dtype: str                      # "bf16" or "f32"
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    page_size: int
    sm_scale: float
    vocab: int
    p_match: float
    node_indptr: np.ndarray         # int32 [B+1]
    parent: np.ndarray              # int32 [T] local parent ids
    prefix_len: np.ndarray          # int32 [B]
    block_table: np.ndarray         # int32 [B, stride]
    q: np.ndarray                   # [T, Hq, D]       (uint16 bf16 bits or float32)
    k_tree: np.ndarray              # [T, Hkv, D]
    v_tree: np.ndarray              # [T, Hkv, D]
    k_pages: np.ndarray             # [P, Hkv, ps, D]
    v_pages: np.ndarray             # [P, Hkv, ps, D]
    logits: np.ndarray              # [T, row_stride]  (uint16 bf16 bits or float32)
    planted_argmax: np.ndarray      # int32 [T]  lowest planted maximum position
    draft_tokens: np.ndarray        # int32 [T]
    planted_ties: Optional[np.ndarray] = None   # int32 [T]  planted maximum positions per row
    meta: dict = field(default_factory=dict)

    @property
    def num_requests(self) -> int:
        return int(self.node_indptr.size - 1)

    @property
    def total_nodes(self) -> int:
        return int(self.node_indptr[-1])

    @property
    def num_pages(self) -> int:
        return int(self.k_pages.shape[0])

    @property
    def row_stride(self) -> int:
        return int(self.logits.shape[1])

    @property
    def elem_bytes(self) -> int:
        return 2 if self.dtype == "bf16" else 4

    def tree_sizes(self) -> np.ndarray:
        return np.diff(self.node_indptr)

    def request_parents(self, r: int) -> np.ndarray:
        a, b = int(self.node_indptr[r]), int(self.node_indptr[r + 1])
        return self.parent[a:b]


def _draw_values(rng: np.random.Generator, shape, std: float, dtype: str) -> np.ndarray:
    """N(0, std^2) draws, rounded to bf16 when ``dtype`` is bf16 (chunked)."""
    n = int(np.prod(shape))
    if dtype == "f32":
        x = rng.standard_normal(size=n, dtype=np.float32)
        if std != 1.0:
            x *= np.float32(std)
        return x.reshape(shape)
    out = np.empty(n, dtype=np.uint16)
    buf = np.empty(min(_CHUNK, max(n, 1)), dtype=np.float32)
    t = np.empty_like(buf, dtype=np.uint32)
    for s in range(0, n, _CHUNK):
        m = min(_CHUNK, n - s)
        rng.standard_normal(dtype=np.float32, out=buf[:m])
        if std != 1.0:
            buf[:m] *= np.float32(std)
        _round_chunk(buf[:m].view(np.uint32), t[:m], out[s:s + m])
    return out.reshape(shape)


def make_batch(
    *,
    parents: Sequence[np.ndarray],
    prefix_lens: Sequence[int],
    num_q_heads: int,
    num_kv_heads: int,
    head_dim: int,
    page_size: int = 16,
    dtype: str = "bf16",
    vocab: int = 128256,
    p_match: float = 0.7,
    qkv_std: Optional[float] = None,
    logit_std: float = 2.0,
    seed: int = 0,
    extra_pages: Optional[int] = None,
    row_pad: int = 0,
    name: str = "custom",
    rng: Optional[np.random.Generator] = None,
    reserve_tokens: int = 0,
    tie_rate: float = 0.0,
) -> VerifyBatch:
    """Draw every tensor of one verify batch for the given tree shapes.

    ``parents`` holds one local parent array per request; ``prefix_lens`` the
    number of tokens already in each request's KV cache.  ``reserve_tokens``
    extends every request's block table to cover that many positions past its
    prefix (pages for the accepted path to be committed to; NaN-filled like
    every slot past the prefix).  With the default 0 nothing changes.
    ``tie_rate`` is the share of logit rows whose maximum is planted at two
    (one in 30 of them: three) distinct positions instead of one.
    """
    if dtype not in ("bf16", "f32"):
        raise ValueError("dtype must be 'bf16' or 'f32'")
    if rng is None:
        rng = np.random.Generator(np.random.PCG64(seed))
    B = len(parents)
    if len(prefix_lens) != B:
        raise ValueError("one prefix length per request")
    sizes = np.array([len(p) for p in parents], dtype=np.int64)
    indptr = np.zeros(B + 1, dtype=np.int32)
    indptr[1:] = np.cumsum(sizes)
    T = int(indptr[-1])
    parent = (np.concatenate([np.asarray(p, dtype=np.int32) for p in parents])
              if B else np.zeros(0, dtype=np.int32))
    L = np.asarray(prefix_lens, dtype=np.int32)
    Hq, Hkv, D, ps = num_q_heads, num_kv_heads, head_dim, page_size
    if qkv_std is None:
        qkv_std = 1.0 if dtype == "f32" else 1.0 / math.sqrt(head_dim)

    # Paged prefix: a shuffled pool with poisoned spare pages.
    npages_req = [(int(l) + int(reserve_tokens) + ps - 1) // ps for l in L]
    live = int(sum(npages_req))
    if extra_pages is None:
        extra_pages = 1 + live // 16
    total_pages = live + extra_pages
    perm = rng.permutation(total_pages).astype(np.int32)
    stride = max(1, max(npages_req) if B else 1)
    block_table = np.full((B, stride), -1, dtype=np.int32)
    cursor = 0
    for r in range(B):
        n = npages_req[r]
        block_table[r, :n] = perm[cursor:cursor + n]
        cursor += n

    q = _draw_values(rng, (T, Hq, D), qkv_std, dtype)
    k_tree = _draw_values(rng, (T, Hkv, D), qkv_std, dtype)
    v_tree = _draw_values(rng, (T, Hkv, D), qkv_std, dtype)
    k_pages = _draw_values(rng, (total_pages, Hkv, ps, D), qkv_std, dtype)
    v_pages = _draw_values(rng, (total_pages, Hkv, ps, D), qkv_std, dtype)
    nan = BF16_NAN if dtype == "bf16" else np.float32(np.nan)
    owned = np.zeros(total_pages, dtype=bool)
    for r in range(B):
        n = npages_req[r]
        owned[block_table[r, :n]] = True
        # every slot from position L_r on (the prefix ends inside page L_r // ps)
        for e in range(int(L[r]) // ps, n):
            first = int(L[r]) - e * ps if e == int(L[r]) // ps else 0
            k_pages[block_table[r, e], :, first:, :] = nan
            v_pages[block_table[r, e], :, first:, :] = nan
    k_pages[~owned] = nan
    v_pages[~owned] = nan

    # Logits with a planted maximum per row (drawn a block of rows at a
    # time); tied rows get the same value at one or two more positions.
    row_stride = vocab + row_pad
    planted = (rng.integers(0, vocab, size=T, dtype=np.int64).astype(np.int32)
               if vocab else np.zeros(T, np.int32))
    ties = np.ones(T, dtype=np.int32)
    extra = {}
    if tie_rate > 0 and vocab >= 3:
        tied = np.nonzero(rng.random(T) < tie_rate)[0]
        for i in tied:
            k = 3 if rng.random() < 1.0 / 30 else 2
            pos = {int(planted[i])}
            while len(pos) < k:
                pos.add(int(rng.integers(0, vocab)))
            extra[int(i)] = sorted(pos)
            ties[i] = k
            planted[i] = min(pos)
    logits = np.empty((T, row_stride), dtype=np.uint16 if dtype == "bf16" else np.float32)
    clip = np.float32(7.5 * logit_std)
    rows_per = max(1, _CHUNK // max(row_stride, 1))
    for a in range(0, T, rows_per):
        b = min(T, a + rows_per)
        body = rng.standard_normal(size=(b - a, row_stride), dtype=np.float32)
        body *= np.float32(logit_std)
        np.clip(body, -clip, clip, out=body)
        if vocab:
            body[np.arange(b - a), planted[a:b]] = np.float32(8.0 * logit_std)
            for i in range(a, b):
                for pos in extra.get(i, ()):
                    body[i - a, pos] = np.float32(8.0 * logit_std)
        if dtype == "bf16":
            f32_to_bf16_bits(body, out=logits[a:b])
        else:
            logits[a:b] = body
    if row_pad:
        logits[:, vocab:] = BF16_NAN if dtype == "bf16" else np.float32(np.nan)

    # Draft tokens: each non-root node repeats its parent's planted maximum
    # with probability p_match, else a uniform token (which may coincide).
    draft = rng.integers(0, max(vocab, 1), size=T, dtype=np.int64).astype(np.int32)
    hit = rng.random(size=T) < p_match
    for r in range(B):
        a, b = int(indptr[r]), int(indptr[r + 1])
        for i in range(a + 1, b):
            if hit[i]:
                draft[i] = planted[a + parent[i]]

    return VerifyBatch(
        name=name, dtype=dtype, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=D,
        page_size=ps, sm_scale=1.0 / math.sqrt(D), vocab=vocab, p_match=p_match,
        node_indptr=indptr, parent=parent, prefix_len=L, block_table=block_table,
        q=q, k_tree=k_tree, v_tree=v_tree, k_pages=k_pages, v_pages=v_pages,
        logits=logits, planted_argmax=planted, draft_tokens=draft, planted_ties=ties,
        meta={"seed": seed},
    )


# ---------------------------------------------------------------------------
# The five named workloads
# ---------------------------------------------------------------------------

WORKLOAD_NAMES = {
    1: "tiny-f32 (1 req, 8/8 heads, D=64, L=256, 16-node random tree, V=1024)",
    2: "llama3-8b-bf16 (16 req, 32/8 heads, D=128, L~U[512,2048], 8-64 nodes depth<=8, V=128256)",
    3: "mixed-slo-8b-bf16 (64 req: 16 tight 64-128 nodes d<=6, 32 medium 16-32 d<=8, 16 relaxed 1-4 chains; L~U[256,4096])",
    4: "llama3-70b-shape-bf16 (32 req, 64/8 heads, D=128, L~U[2048,8192], 32-96 nodes depth<=10, p=0.6)",
    5: "long-context-bf16 (8 req, 32/8 heads, D=128, L=32768, 32 nodes: even chains, odd random, p=0.8)",
}

# Share of bf16 N(0, 2) logit rows over a 128256-token vocabulary whose
# maximum value occurs more than once (about 6-8.5% in samples of a few
# hundred rows, almost always twice); the bf16 workloads plant ties at this
# rate.
NATURAL_TIE_RATE = 0.085

SHORT_NAMES = {1: "tiny_f32", 2: "llama3_8b", 3: "mixed_slo", 4: "llama3_70b_shape", 5: "long_context"}

# Decoder layers of the model whose attention shape a workload takes
# (Llama-3 8B: 32, Llama-3 70B: 80); only a labelled whole-model projection
# uses them.
MODEL_LAYERS = {2: 32, 3: 32, 4: 80, 5: 32}


def make_config(n: int, seed: Optional[int] = None, tp: int = 1) -> VerifyBatch:
    """Draw the named workload ``n`` (1..5) with seed ``12162 + n``.

    ``tp`` > 1 draws one tensor-parallel rank's share of it instead: the
    same trees and prefix lengths, 1/tp of the q- and kv-heads (whole head
    groups) and the first ceil(V / tp) columns' worth of vocabulary (a
    vocab-sharded LM head's local logits)."""
    if seed is None:
        seed = 12162 + n
    rng = np.random.Generator(np.random.PCG64(seed))
    if n == 1:
        parents = [random_tree(rng, 16)]
        lens = [256]
        kw = dict(num_q_heads=8, num_kv_heads=8, head_dim=64, dtype="f32", vocab=1024,
                  p_match=0.7, logit_std=1.0)
    elif n == 2:
        B = 16
        sizes = rng.integers(8, 65, size=B)
        parents = [random_tree(rng, int(s), max_depth=8) for s in sizes]
        lens = [int(x) for x in rng.integers(512, 2049, size=B)]
        kw = dict(num_q_heads=32, num_kv_heads=8, head_dim=128, dtype="bf16", vocab=128256,
                  p_match=0.7, logit_std=2.0)
    elif n == 3:
        classes = np.array([0] * 16 + [1] * 32 + [2] * 16)
        rng.shuffle(classes)
        parents = []
        for c in classes:
            if c == 0:
                parents.append(random_tree(rng, int(rng.integers(64, 129)), max_depth=6))
            elif c == 1:
                parents.append(random_tree(rng, int(rng.integers(16, 33)), max_depth=8))
            else:
                parents.append(chain_tree(int(rng.integers(1, 5))))
        lens = [int(x) for x in rng.integers(256, 4097, size=classes.size)]
        kw = dict(num_q_heads=32, num_kv_heads=8, head_dim=128, dtype="bf16", vocab=128256,
                  p_match=0.7, logit_std=2.0)
    elif n == 4:
        B = 32
        sizes = rng.integers(32, 97, size=B)
        parents = [random_tree(rng, int(s), max_depth=10) for s in sizes]
        lens = [int(x) for x in rng.integers(2048, 8193, size=B)]
        kw = dict(num_q_heads=64, num_kv_heads=8, head_dim=128, dtype="bf16", vocab=128256,
                  p_match=0.6, logit_std=2.0)
    elif n == 5:
        B = 8
        parents = [chain_tree(32) if r % 2 == 0 else random_tree(rng, 32) for r in range(B)]
        lens = [32768] * B
        kw = dict(num_q_heads=32, num_kv_heads=8, head_dim=128, dtype="bf16", vocab=128256,
                  p_match=0.8, logit_std=2.0)
    else:
        raise ValueError("workloads are numbered 1..5")
    if tp > 1:
        if kw["num_kv_heads"] % tp:
            raise ValueError("tp must divide the kv-head count")
        kw["num_q_heads"] //= tp
        kw["num_kv_heads"] //= tp
        kw["vocab"] = -(-kw["vocab"] // tp)
    if kw["dtype"] == "bf16":
        kw["tie_rate"] = NATURAL_TIE_RATE
    b = make_batch(parents=parents, prefix_lens=lens, page_size=16, seed=seed,
                   name=SHORT_NAMES[n], rng=rng, **kw)
    b.meta["workload"] = WORKLOAD_NAMES[n] + (" (one of %d tensor-parallel ranks)" % tp if tp > 1 else "")
    b.meta["config"] = n
    b.meta["tp"] = tp
    return b


def make_tie_logits(rng: np.random.Generator, rows: int, vocab: int, dtype: str = "bf16",
                    max_ties: int = 4, row_pad: int = 0):
    """Rows whose maximum appears at 1..max_ties random positions.

    Returns ``(logits, positions)`` where ``positions[i]`` lists the tied
    maximum positions of row i (unsorted).  Half of the tied rows mix +0.0
    and -0.0 maxima when the body is made non-positive, to exercise the
    signed-zero comparison.
    """
    body = rng.standard_normal(size=(rows, vocab + row_pad), dtype=np.float32) * np.float32(2.0)
    np.clip(body, -15.0, 15.0, out=body)
    positions: List[np.ndarray] = []
    for i in range(rows):
        k = int(rng.integers(1, max_ties + 1))
        pos = rng.choice(vocab, size=k, replace=False)
        if i % 4 == 3:
            # all-negative row whose maximum is a mix of +0 and -0
            body[i, :vocab] = -np.abs(body[i, :vocab]) - np.float32(0.5)
            for j, p in enumerate(pos):
                body[i, p] = np.float32(-0.0) if j % 2 == 0 else np.float32(0.0)
        else:
            top = np.float32(16.0 + float(rng.integers(0, 4)))
            body[i, pos] = top
        positions.append(pos)
    logits = f32_to_bf16_bits(body) if dtype == "bf16" else body
    if row_pad:
        logits[:, vocab:] = BF16_NAN if dtype == "bf16" else np.float32(np.nan)
    return logits, positions


# ---------------------------------------------------------------------------
# Candidate token trees for the selection phases
# ---------------------------------------------------------------------------

@dataclass
class CandidateBatch:
    """Speculation output for a batch: every request's candidate token tree
    (root excluded), with each candidate's path probability, plus the
    selection inputs.

    cand_parent holds LOCAL parents: -1 for a child of the root, else the
    index of an earlier candidate of the same request.  need[r] is the sum of
    path probabilities the request's added nodes must reach (A_cap(r) minus
    the root's 1).  budget counts every selected node, the roots included.
    """
    cand_indptr: np.ndarray   # [B + 1] int32
    cand_parent: np.ndarray   # [C] int32
    cand_prob: np.ndarray     # [C] float32, in (0, 1]
    need: np.ndarray          # [B] float32
    budget: int
    n_max: int
    depth: int
    width: int

    @property
    def num_requests(self) -> int:
        return int(self.cand_indptr.size - 1)


def make_candidates(rng: np.random.Generator, num_requests: int, depth: int, width: int,
                    budget: Optional[int] = None, n_max: Optional[int] = None,
                    prob_levels: Optional[int] = None) -> CandidateBatch:
    """Beam-search-shaped candidate trees (section 4.3 step 1): depth layers
    of `width` candidates, each layer's parents drawn from the layer above
    (higher path probability more likely), each layer ordered by path
    probability.  Conditional probabilities are uniform in (0, 1]; with
    `prob_levels` they are multiples of 1/prob_levels (ties on purpose).
    need[r] ~ U[0, depth] (an A_cap(r) between 1 and depth + 1)."""
    indptr = [0]
    parents, probs = [], []
    for _ in range(num_requests):
        f_prev = np.ones(1)
        base = 0
        p_req, f_req = [], []
        for layer in range(depth):
            if layer == 0:
                par = np.full(width, -1, dtype=np.int64)
                f_par = np.ones(width)
            else:
                w_prev = f_prev / f_prev.sum()
                pick = rng.choice(f_prev.size, size=width, p=w_prev)
                par = base + pick
                f_par = f_prev[pick]
            if prob_levels:
                cond = rng.integers(1, prob_levels + 1, size=width) / prob_levels
            else:
                cond = 1.0 - rng.random(width)          # (0, 1]
            f = (f_par * cond).astype(np.float32).astype(np.float64)
            order = np.argsort(-f, kind="stable")
            par, f = par[order], f[order]
            if layer > 0:
                base += f_prev.size
            p_req.append(par)
            f_req.append(f)
            f_prev = f
        parents.append(np.concatenate(p_req).astype(np.int32))
        probs.append(np.concatenate(f_req).astype(np.float32))
        indptr.append(indptr[-1] + depth * width)
    need = (rng.random(num_requests) * depth).astype(np.float32)
    if budget is None:
        budget = num_requests * (1 + depth * width // 2)
    if n_max is None:
        n_max = 1 + depth * width
    return CandidateBatch(cand_indptr=np.asarray(indptr, dtype=np.int32),
                          cand_parent=np.concatenate(parents) if parents else np.zeros(0, np.int32),
                          cand_prob=np.concatenate(probs) if probs else np.zeros(0, np.float32),
                          need=need, budget=int(budget), n_max=int(n_max), depth=depth, width=width)


# ---------------------------------------------------------------------------
# Draft logits for one beam-search speculation step
# ---------------------------------------------------------------------------

@dataclass
class BeamBatch:
    """Inputs of one beam-search step (section 4.3 step 1): the draft model's
    logits after every beam node, and each beam's log path probability.

    logits: [num_requests * beam_in, row_stride] (bf16 bit patterns as
    uint16, or float32); columns past ``vocab`` hold NaN.  beam_logprob:
    [num_requests, beam_in] float32, natural-log path probabilities, best
    beam first; -inf marks an unused beam slot.
    """
    logits: np.ndarray
    beam_logprob: np.ndarray
    vocab: int
    dtype: str

    @property
    def num_requests(self) -> int:
        return int(self.beam_logprob.shape[0])

    @property
    def beam_in(self) -> int:
        return int(self.beam_logprob.shape[1])

    def logits_f32(self) -> np.ndarray:
        """[num_requests, beam_in, vocab] float32 view of the logit values."""
        x = bf16_bits_to_f32(self.logits) if self.dtype == "bf16" else self.logits
        return x[:, :self.vocab].reshape(self.num_requests, self.beam_in, self.vocab)


def make_beam_batch(rng: np.random.Generator, num_requests: int, beam_in: int, vocab: int,
                    dtype: str = "bf16", std: float = 2.0, row_pad: int = 0,
                    root_step: bool = False, dead_beams: int = 0) -> BeamBatch:
    """Draft logits ~ N(0, std) per row (rounded to bf16 for "bf16"); beam
    log path probabilities are sorted cumulative sums of log U(0, 1] (the
    shape a beam at depth > 1 has), or 0 for the root step.  `dead_beams`
    trailing beam slots per request are marked unused (-inf)."""
    rows = num_requests * beam_in
    stride = vocab + row_pad
    body = rng.standard_normal(size=(rows, stride), dtype=np.float32) * np.float32(std)
    body[:, vocab:] = np.float32(np.nan)
    logits = f32_to_bf16_bits(body) if dtype == "bf16" else body
    if dtype == "bf16" and row_pad:
        logits[:, vocab:] = BF16_NAN
    if root_step:
        lp = np.zeros((num_requests, beam_in), dtype=np.float32)
    else:
        steps = np.log(1.0 - rng.random((num_requests, beam_in, 3)))
        lp = -np.sort(-steps.sum(axis=2), axis=1).astype(np.float32)
    if dead_beams:
        lp[:, beam_in - dead_beams:] = -np.inf
    return BeamBatch(logits=logits, beam_logprob=lp, vocab=vocab, dtype=dtype)


# ---------------------------------------------------------------------------
# Inputs of sampled-decoding verification
# ---------------------------------------------------------------------------

def make_draft_logits(rng: np.random.Generator, logits: np.ndarray, vocab: int, dtype: str,
                      noise_std: float) -> np.ndarray:
    """Draft-model logits shaped like ``logits``: the target's values plus
    N(0, noise_std) noise (a draft model that mostly agrees with the target),
    rounded to bf16 for "bf16"; columns past ``vocab`` keep the target's."""
    x = bf16_bits_to_f32(logits) if dtype == "bf16" else np.asarray(logits, dtype=np.float32)
    y = x.copy()
    y[:, :vocab] += (rng.standard_normal(size=(x.shape[0], vocab), dtype=np.float32) * np.float32(noise_std))
    return f32_to_bf16_bits(y) if dtype == "bf16" else y


def make_uniforms(rng: np.random.Generator, n: int) -> np.ndarray:
    """n float32 uniforms in [0, 1) (the random numbers sampled verification
    consumes: one acceptance test per node, one bonus draw per node)."""
    return np.minimum(rng.random(n, dtype=np.float32), np.float32(1.0) - np.float32(2.0 ** -24))
