#!/usr/bin/env python3
"""Benchmark: verified tree tokens/s of one batched tree-verification pass on
one MI355X, with the dominant kernel's roofline and the CPU oracle's rate.

A step is one full verification pass over one batch: paged tree attention
(+ split-KV combine), per-node argmax over the vocabulary, acceptance.
Inputs are seeded synthetic tensors shaped like the workload named by
``--workload`` (default: the long-context batch, 8 requests over 32768-token
prefixes, the bandwidth-bound headline), resident in device memory before
timing starts.  A step is one adaserve_tree_verify_step call (attention,
argmax and acceptance in two launches: the argmax workgroups share the
attention's grid); ``--unfused`` runs the three entry points one after
another instead, and ``--unfused --overlap`` runs the per-node argmax (which
reads only the logits) on a second stream of the same priority beside the
attention, joined before the acceptance.  Consecutive steps cycle through several
copies of the inputs so that no step finds its K/V or logits in the 256 MB
last-level (MALL) cache left behind by the previous one.  Every timed
region follows 30 ms of continuous GPU work (see warm()); by default the
warm-up is as many steps as that takes, then 200 steps are timed.

Prints ONE JSON line on stdout.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_MFMA_PEAK_TFLOPS = 2500.0  # dense
FP32_PEAK_TFLOPS = 157.3
METRIC = "verified tree tokens/sec + % peak HBM GB/s, tree-verify attention, 1 MI355X"
MALL_BYTES = 256 << 20
EVENT_EVERY = 5                 # the last 1/EVENT_EVERY of the timed steps carry per-kernel events
WARM_MS = 30.0                  # continuous GPU work before any timed region (see warm())


def parse_args():
    p = argparse.ArgumentParser(description=__doc__)
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=None,
                   help="untimed warm-up steps (default: as many as keep the GPU busy for %d ms, at least 10)"
                        % WARM_MS)
    p.add_argument("--workload", type=int, default=5, choices=[1, 2, 3, 4, 5],
                   help="1 tiny-f32, 2 llama3-8b, 3 mixed-slo, 4 70b-shape, 5 long-context (default)")
    p.add_argument("--unfused", action="store_true",
                   help="time the step as three calls (attention, argmax, acceptance) instead of one")
    p.add_argument("--no-parts", action="store_true",
                   help="skip timing the step's parts alone (profiling runs: keeps the kernel statistics "
                        "to the step's own launches)")
    p.add_argument("--overlap", action="store_true",
                   help="with --unfused: run argmax on a second stream beside attention instead of after it")
    p.add_argument("--mfma-workload", type=int, default=4, choices=[0, 1, 2, 3, 4, 5],
                   help="also time tree attention alone on this (matrix-core bound) workload and "
                        "report its MFMA fraction; 0 = skip")
    p.add_argument("--tp-share", type=int, default=4,
                   help="also time one rank's share of the 70B-shaped workload under this tensor-parallel "
                        "degree (attention with heads / N, argmax over vocabulary / N); 0 = skip")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=12.0,
                   help="approximate CPU time budget of the oracle baseline sample")
    return p.parse_args()


class KernelTimer:
    """A HIP timing event created with hipEventDisableSystemFence: recording it
    skips the system-scope cache writeback and invalidation that a default
    event performs (HIP documents the flag for events used only to time),
    so the recorded durations are the kernels' own and the instrumented step
    is barely slowed (measured on MI355X: ~1.5 us per record instead of
    ~3.5 us).  Uses the HIP runtime torch has loaded."""
    _hip = None
    DISABLE_SYSTEM_FENCE = 0x20000000

    @classmethod
    def _runtime(cls):
        if cls._hip is None:
            import ctypes
            path = None
            with open("/proc/self/maps") as f:
                for line in f:
                    if "libamdhip64" in line:
                        path = line.split()[-1]
                        break
            if path is None:
                raise RuntimeError("the HIP runtime is not loaded")
            cls._hip = ctypes.CDLL(path)
        return cls._hip

    def __init__(self):
        import ctypes
        self._ct = ctypes
        self.h = ctypes.c_void_p()
        if self._runtime().hipEventCreateWithFlags(ctypes.byref(self.h), ctypes.c_uint(self.DISABLE_SYSTEM_FENCE)):
            raise RuntimeError("hipEventCreateWithFlags failed")

    def record(self, stream):
        if self._runtime().hipEventRecord(self.h, self._ct.c_void_p(stream.cuda_stream)):
            raise RuntimeError("hipEventRecord failed")

    def elapsed_time(self, end) -> float:
        ms = self._ct.c_float()
        if self._runtime().hipEventElapsedTime(self._ct.byref(ms), self.h, end.h):
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value


def algorithmic_costs(b):
    """Bytes and flops the method must move / compute, per step."""
    import numpy as np
    s = b.elem_bytes
    Hq, Hkv, D = b.num_q_heads, b.num_kv_heads, b.head_dim
    n = b.tree_sizes().astype(np.int64)
    L = b.prefix_len.astype(np.int64)
    # depth of every node (for the tree part of the flop count)
    depth_sum = 0
    for r in range(b.num_requests):
        par = b.request_parents(r)
        dep = np.zeros(len(par), np.int64)
        for i in range(1, len(par)):
            dep[i] = dep[par[i]] + 1
        depth_sum += int((dep + 1).sum())
    attn_bytes = int((2 * L * Hkv * D * s).sum() + (n * (2 * Hq + 2 * Hkv) * D * s).sum()
                     + 4 * ((L + 15) // 16).sum() + 4 * n.sum() + 8 * b.num_requests)
    attn_flops = int((4 * D * Hq * n * L).sum()) + 4 * D * Hq * depth_sum
    argmax_bytes = int(b.total_nodes) * b.vocab * s + 4 * int(b.total_nodes)
    accept_bytes = 16 * int(b.total_nodes)
    return dict(attn_bytes=attn_bytes, attn_flops=attn_flops, argmax_bytes=argmax_bytes,
                accept_bytes=accept_bytes)


def is_bf16_in(b):
    return b.dtype == "bf16"


def make_replicas(dev, count):
    """``count`` device copies of the per-step input tensors (copy 0 = originals)."""
    reps = [dict(q=dev.q, k_tree=dev.k_tree, v_tree=dev.v_tree, k_pages=dev.k_pages,
                 v_pages=dev.v_pages, logits=dev.logits)]
    for _ in range(count - 1):
        reps.append({k: v.clone() for k, v in reps[0].items()})
    return reps


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _oracle_pass(b, nodes=None):
    """One oracle pass (attention of `nodes` (all: None) over every q-head,
    argmax of their rows, acceptance of the whole batch); per-stage seconds."""
    import oracle
    t0 = time.perf_counter()
    oracle.tree_attn_batch(b, nodes=nodes)
    t1 = time.perf_counter()
    amax = oracle.node_argmax(b.logits, b.vocab, b.dtype, rows=nodes)
    t2 = time.perf_counter()
    if nodes is not None:
        amax = b.planted_argmax   # the rows not scanned: acceptance needs every node's choice
    oracle.tree_accept(b.node_indptr, b.parent, b.draft_tokens, amax, 128)
    t3 = time.perf_counter()
    return t1 - t0, t2 - t1, t3 - t2


def cpu_baseline(b, budget_s, one_thread=True):
    """The oracle (untuned) on a bounded sample of the same workload.

    When one full pass (attention of every node, argmax of every row,
    acceptance of every request) fits the budget, full passes are repeated
    until the budget is used; otherwise an even spread of nodes (attention
    and argmax of their rows) is timed with the acceptance of the whole
    batch, and the rate is scaled to the whole batch.  Per-stage seconds are
    per full pass.  With `one_thread`, the same oracle on one thread times
    the tiny workload (whole batch) and an even spread of 64 nodes of the
    Llama-3-8B-shaped workload.
    """
    import numpy as np
    import oracle
    threads = oracle.num_threads()
    T = b.total_nodes
    probe = np.unique(np.linspace(0, T - 1, min(T, 8)).round().astype(np.int64))
    ta, tm, _ = _oracle_pass(b, probe)
    per_node = max((ta + tm) / probe.size, 1e-6)
    if per_node * T <= budget_s:
        passes, sa, sm, sc = 0, 0.0, 0.0, 0.0
        while sa + sm + sc < budget_s or passes == 0:
            ta, tm, tc = _oracle_pass(b)
            sa, sm, sc, passes = sa + ta, sm + tm, sc + tc, passes + 1
        t_total = sa + sm + sc
        value = T * passes / t_total
        stages = {"attention": sa / passes, "argmax": sm / passes, "accept": sc / passes}
        sample = ("the whole batch (attention of all %d nodes over all q-heads, vocab argmax of "
                  "every row, acceptance of every request), %d full passes, fp64, %.1f s wall"
                  % (T, passes, t_total))
    else:
        want = int(min(T, max(1, budget_s / per_node)))
        sel = np.unique(np.linspace(0, T - 1, want).round().astype(np.int64))
        ta, tm, tc = _oracle_pass(b, sel)
        value = 1.0 / ((ta + tm) / sel.size + tc / T)
        stages = {"attention": ta * T / sel.size, "argmax": tm * T / sel.size, "accept": tc}
        sample = ("%d of %d tree nodes (attention over all q-heads + vocab argmax of their rows, "
                  "evenly spread over the batch) plus acceptance of the whole batch; fp64; "
                  "%.1f s wall; stage times scaled to the whole batch" % (sel.size, T, ta + tm + tc))
    res = {"value": value, "unit": "tree tokens/s", "cores": int(threads), "kind": "oracle",
           "sample": sample, "cpu_model": cpu_model(),
           "stage_s_per_pass": stages}
    if one_thread:
        from paper_2501_12162_amd.workload import WORKLOAD_NAMES, make_config
        one = {}
        oracle.set_num_threads(1)
        try:
            for n in (1, 2):
                bn = b if b.meta.get("config") == n else make_config(n)
                Tn = bn.total_nodes
                sel = None if n == 1 else np.unique(np.linspace(0, Tn - 1, 64).round().astype(np.int64))
                reps, ta, tm, tc = 0, 0.0, 0.0, 0.0
                while reps == 0 or (n == 1 and ta + tm + tc < 0.5):
                    a_, m_, c_ = _oracle_pass(bn, sel)
                    ta, tm, tc, reps = ta + a_, tm + m_, tc + c_, reps + 1
                k = Tn if sel is None else sel.size
                rate = 1.0 / ((ta + tm) / (k * reps) + tc / (Tn * reps))
                one[WORKLOAD_NAMES[n].split(" ")[0]] = {
                    "value": rate, "unit": "tree tokens/s",
                    "sample": ("whole batch, %d passes" % reps) if sel is None
                    else "%d of %d nodes evenly spread + acceptance of the whole batch" % (k, Tn)}
        finally:
            oracle.set_num_threads(threads)
        res["one_thread"] = one
    return res


def measured_traffic(workload: int, kernel: str):
    """HBM bytes per launch of `kernel` from the committed counter summary,
    or None when there is none or the kernel sources changed since.  The
    one-call step ("tree_verify_step": its two launches) is profiled in
    profiles/traffic_workload<N>.json; the attention call alone
    ("tree_attn": main kernel + split-KV merge) and the standalone argmax in
    profiles/traffic_attention_workload<N>.json (a --unfused run)."""
    from paper_2501_12162_amd.profiling import kernel_source_hash
    name = "traffic_workload%d.json" if kernel == "tree_verify_step" else "traffic_attention_workload%d.json"
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles", name % workload)
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("kernel_source_sha") != kernel_source_hash():
        return None
    fused_profile = "node_argmax" not in t["kernels"]
    if fused_profile != (kernel == "tree_verify_step"):
        return None
    k = t["kernels"].get("tree_attn" if kernel == "tree_verify_step" else kernel)
    if k is None:
        return None
    total = k["bytes"]
    if kernel in ("tree_attn", "tree_verify_step") and "tree_attn_combine" in t["kernels"]:
        total += t["kernels"]["tree_attn_combine"]["bytes"]
    return total


def attention_alone(n, calls=30, tp=1):
    """Tree attention alone, back to back, on workload `n` (its K/V exceed the
    MALL, so no call finds the previous one's data there): mean event-timed
    duration per call and its roofline fractions.  With tp > 1: one
    tensor-parallel rank's share of the workload (heads and vocabulary / tp),
    and its argmax over the local vocabulary columns timed the same way."""
    import numpy as np
    import torch
    from paper_2501_12162_amd.device import DeviceBatch
    from paper_2501_12162_amd.workload import WORKLOAD_NAMES, make_config
    b = make_config(n, tp=tp)
    costs = algorithmic_costs(b)
    d = DeviceBatch(b)
    stream = torch.cuda.current_stream()

    def timed(fn):
        warm(lambda k: d.attention(stream))
        ev = [KernelTimer() for _ in range(calls + 1)]
        hold_gpu()
        ev[0].record(stream)
        for i in range(calls):
            fn()
            ev[i + 1].record(stream)
        torch.cuda.synchronize()
        return np.array([ev[i].elapsed_time(ev[i + 1]) for i in range(calls)]) * 1e3
    us = timed(lambda: d.attention(stream))
    mean = float(us.mean())
    res = {"workload": b.meta["workload"], "tree_attn_us": mean, "tree_attn_p50_us": float(np.median(us)),
           "mfma_frac": costs["attn_flops"] / (mean * 1e-6) / 1e12 / BF16_MFMA_PEAK_TFLOPS,
           "hbm_frac": costs["attn_bytes"] / (mean * 1e-6) / 1e9 / HBM_PEAK_GBS,
           "alg_flops": costs["attn_flops"], "alg_bytes": costs["attn_bytes"],
           "traffic": measured_traffic(n, "tree_attn") if tp == 1 else None, "calls": calls}
    if tp > 1:
        am = timed(lambda: d.argmax(stream))
        res.update({"tp": tp, "q_heads": b.num_q_heads, "kv_heads": b.num_kv_heads, "vocab_columns": b.vocab,
                    "node_argmax_us": float(am.mean()),
                    "node_argmax_hbm_frac": costs["argmax_bytes"] / (float(am.mean()) * 1e-6) / 1e9 / HBM_PEAK_GBS})
    return res


def _finite(x):
    """The JSON line with NaN / inf (parts not timed) written as null."""
    if isinstance(x, dict):
        return {k: _finite(v) for k, v in x.items()}
    if isinstance(x, (list, tuple)):
        return [_finite(v) for v in x]
    if isinstance(x, float) and not math.isfinite(x):
        return None
    return x


def warm(fn, ms=WARM_MS, min_calls=10):
    """Calls fn(0), fn(1), ... until the GPU has been kept busy for about
    `ms` (and at least `min_calls` calls); returns the number of calls.

    After any idle spell (the host drawing a workload, a synchronisation
    followed by host work, a 100 ms pause) the GPU runs the same work slower
    for its first ~10 ms: on the long-context batch the first ~40 one-call
    steps take ~250 us each, later ones ~221 us, and 70B-shape attention
    reads up to 20% slow, which is the behaviour of a clock that ramps up
    under load.  Timed regions therefore follow this much work."""
    import torch
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    k = 0
    while k < min_calls or time.perf_counter() - t0 < ms * 1e-3:
        for _ in range(4):
            fn(k)
            k += 1
        torch.cuda.synchronize()
    return k


def hold_gpu(ms=3.0):
    """Keeps the current stream busy for about `ms` (torch's bounded spin
    kernel), so that calls enqueued after it are timed back to back on the
    GPU rather than at the rate the host issues them."""
    import torch
    torch.cuda._sleep(int(ms * 2.4e6))


def progress(msg):
    print("bench: " + msg, file=sys.stderr, flush=True)


def main():
    args = parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the tree-verification path is not sharded "
              "across GPUs here (run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    import paper_2501_12162_amd as ada
    from paper_2501_12162_amd.device import DeviceBatch
    from paper_2501_12162_amd.workload import WORKLOAD_NAMES, make_config

    if not os.path.exists(ada.library_path()):
        from paper_2501_12162_amd.build import build
        build()
    ada.load_library()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev_name = torch.cuda.get_device_name(0)

    progress("drawing workload %d" % args.workload)
    b = make_config(args.workload)
    costs = algorithmic_costs(b)
    dev = DeviceBatch(b)
    step_bytes = sum(t.numel() * t.element_size() for t in
                     (dev.q, dev.k_tree, dev.v_tree, dev.k_pages, dev.v_pages, dev.logits))
    n_rep = max(2, math.ceil(3 * MALL_BYTES / step_bytes) + 1)
    reps = make_replicas(dev, n_rep)
    stream = torch.cuda.current_stream()
    # argmax beside attention: a second stream of the default priority, forked
    # after the previous step's acceptance (which reads the argmax output)
    # and joined before this step's acceptance
    side = torch.cuda.Stream() if (args.overlap and args.unfused) else None
    fork, join = torch.cuda.Event(), torch.cuda.Event()
    fused = not args.unfused

    def attention(rp):
        ada.adaserve_tree_attn_verify(
            node_indptr=dev.node_indptr, node_indptr_host=dev.node_indptr_host, parent=dev.parent,
            q=rp["q"], k_tree=rp["k_tree"], v_tree=rp["v_tree"], k_pages=rp["k_pages"],
            v_pages=rp["v_pages"], block_table=dev.block_table, prefix_len=dev.prefix_len,
            prefix_len_host=dev.prefix_len_host, sm_scale=b.sm_scale, out=dev.out,
            workspace=dev.workspace, stream=stream)

    def accept(s):
        ada.adaserve_tree_accept(node_indptr=dev.node_indptr, parent=dev.parent,
                                 draft_tokens=dev.draft_tokens, target_argmax=dev.target_argmax,
                                 max_accept=dev.max_accept, accept_len=dev.accept_len,
                                 accept_tokens=dev.accept_tokens, accept_nodes=dev.accept_nodes,
                                 stream=s)

    def run_step(i, ev=None):
        """One pass; `ev` = timers: two around the one-call step, or six
        around attention, argmax and acceptance (--unfused)."""
        rp = reps[i % n_rep]
        if fused:
            if ev is not None:
                ev[0].record(stream)
            ada.adaserve_tree_verify_step(
                node_indptr=dev.node_indptr, node_indptr_host=dev.node_indptr_host, parent=dev.parent,
                q=rp["q"], k_tree=rp["k_tree"], v_tree=rp["v_tree"], k_pages=rp["k_pages"],
                v_pages=rp["v_pages"], block_table=dev.block_table, prefix_len=dev.prefix_len,
                prefix_len_host=dev.prefix_len_host, sm_scale=b.sm_scale, logits=rp["logits"], vocab=b.vocab,
                draft_tokens=dev.draft_tokens, max_accept=dev.max_accept, out=dev.out,
                target_argmax=dev.target_argmax, accept_len=dev.accept_len, accept_tokens=dev.accept_tokens,
                accept_nodes=dev.accept_nodes, workspace=dev.workspace, stream=stream)
            if ev is not None:
                ev[1].record(stream)
            return
        am = stream if side is None else side
        if side is not None:
            fork.record(stream)
            side.wait_event(fork)
        if ev is not None:
            ev[0].record(stream)
        attention(rp)
        if ev is not None:
            ev[1].record(stream)
            ev[2].record(am)
        ada.adaserve_node_argmax(rp["logits"], b.vocab, dev.target_argmax, stream=am)
        if ev is not None:
            ev[3].record(am)
        if side is not None:
            join.record(side)
            stream.wait_event(join)
        if ev is not None:
            ev[4].record(stream)
        accept(stream)
        if ev is not None:
            ev[5].record(stream)

    # calibration copy of a known size (reference for HBM byte counters)
    calib_src = torch.empty(256 << 20, dtype=torch.uint8, device="cuda").fill_(1)
    calib_dst = torch.empty_like(calib_src)
    calib_dst.copy_(calib_src)

    if args.warmup is None:
        args.warmup = warm(run_step)
    else:
        for i in range(args.warmup):
            run_step(i)
        torch.cuda.synchronize()
    progress("timing %d steps after %d warm-up steps" % (args.steps, args.warmup))

    # Per-kernel HIP events (fence-free, see KernelTimer) on the last
    # 1/EVENT_EVERY of the timed steps only, so that the throughput is not
    # charged for the measurement itself (four default events per step slow
    # a 79 us step to 93 us; four fence-free ones to 85 us).  The
    # instrumented steps are consecutive: a lone instrumented step between
    # plain ones reads its first kernel ~6 us long (its first timestamp is
    # taken before the previous step has drained), consecutive ones agree
    # with the rocprofv3 kernel trace.
    n_inst = max(1, args.steps // EVENT_EVERY)
    sampled_steps = list(range(args.steps - n_inst, args.steps))
    events = {i: [KernelTimer() for _ in range(2 if fused else 6)] for i in sampled_steps}
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        run_step(args.warmup + i, events.get(i))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    # The accepted-path KV commit runs after the step (it is not part of the
    # verification pass the metric times): its own events, on the last
    # replica, with the last step's acceptance.  Rows land in slots past each
    # prefix, which attention never reads.
    rp = reps[(args.warmup + args.steps - 1) % n_rep]
    new_len = torch.empty_like(dev.prefix_len)
    commit_ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]

    def commit():
        ada.adaserve_commit_accepted_kv(
            node_indptr=dev.node_indptr, accept_len=dev.accept_len, accept_nodes=dev.accept_nodes,
            k_tree=rp["k_tree"], v_tree=rp["v_tree"], k_pages=rp["k_pages"], v_pages=rp["v_pages"],
            block_table=dev.block_table, prefix_len=dev.prefix_len, new_prefix_len=new_len)
    commit()
    warm(run_step)   # back to the GPU's loaded clock after the host work above
    hold_gpu()   # the host enqueues every timed call before the GPU starts them
    commit_ev[0].record(stream)
    for _ in range(10):
        commit()
    commit_ev[1].record(stream)
    torch.cuda.synchronize()
    commit_us = commit_ev[0].elapsed_time(commit_ev[1]) * 1e3 / 10
    committed_rows = int((new_len - dev.prefix_len).sum().item())

    # Draft-tree selection (before a pass; not part of the timed step): a
    # candidate batch of the workload's request count, depth 8 x beam width 8,
    # with the workload's total tree size as the budget.
    from paper_2501_12162_amd.workload import make_candidates
    cands = make_candidates(np.random.Generator(np.random.PCG64(args.workload)), b.num_requests, 8, 8,
                            budget=b.total_nodes)
    tdev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    c_ip, c_par, c_prob, c_need = (tdev(cands.cand_indptr), tdev(cands.cand_parent),
                                   tdev(cands.cand_prob), tdev(cands.need))
    s_size = torch.empty(b.num_requests, dtype=torch.int32, device="cuda")
    s_par = torch.empty(b.num_requests, 128, dtype=torch.int32, device="cuda")
    s_cand = torch.empty_like(s_par)

    def select():
        ada.adaserve_select_trees(cand_indptr=c_ip, cand_parent=c_par, cand_prob=c_prob, need=c_need,
                                  budget=cands.budget, n_max=cands.n_max, tree_size=s_size,
                                  tree_parent=s_par, tree_cand=s_cand)
    select()
    warm(run_step)
    hold_gpu()   # the host enqueues every timed call before the GPU starts them
    commit_ev[0].record(stream)
    for _ in range(10):
        select()
    commit_ev[1].record(stream)
    torch.cuda.synchronize()
    select_us = commit_ev[0].elapsed_time(commit_ev[1]) * 1e3 / 10

    # One beam-search speculation step (before selection; not part of the
    # timed step): draft logits of the workload's requests x 8 beams over
    # the workload's vocabulary, keeping 8 children per request.  Calls cycle
    # through enough copies of the logits that none is read from the MALL.
    from paper_2501_12162_amd.workload import make_beam_batch
    bb = make_beam_batch(np.random.Generator(np.random.PCG64(100 + args.workload)), b.num_requests, 8,
                         b.vocab, dtype=b.dtype)
    beam_bytes = bb.logits.nbytes
    beam_reps = max(2, math.ceil(3 * MALL_BYTES / beam_bytes) + 1)
    bl = torch.from_numpy(bb.logits.view(np.int16) if is_bf16_in(b) else bb.logits).cuda()
    if is_bf16_in(b):
        bl = bl.view(torch.bfloat16)
    beam_logits = [bl] + [bl.clone() for _ in range(beam_reps - 1)]
    beam_lp = tdev(bb.beam_logprob)
    code = ada.ADASERVE_BF16 if is_bf16_in(b) else ada.ADASERVE_F32
    beam_ws = torch.empty(ada.adaserve_beam_step_workspace_bytes(b.num_requests, 8, b.vocab, 8, code),
                          dtype=torch.uint8, device="cuda")
    b_par = torch.empty(b.num_requests, 8, dtype=torch.int32, device="cuda")
    b_tok = torch.empty_like(b_par)
    b_lp = torch.empty(b.num_requests, 8, dtype=torch.float32, device="cuda")

    def beam(i):
        ada.adaserve_beam_step(logits=beam_logits[i % beam_reps], vocab=b.vocab, beam_logprob=beam_lp,
                               out_parent=b_par, out_token=b_tok, out_logprob=b_lp, workspace=beam_ws)
    beam(0)
    warm(run_step)
    hold_gpu()   # the host enqueues every timed call before the GPU starts them
    commit_ev[0].record(stream)
    for i in range(20):
        beam(i + 1)
    commit_ev[1].record(stream)
    torch.cuda.synchronize()
    beam_us = commit_ev[0].elapsed_time(commit_ev[1]) * 1e3 / 20

    # Sampled-decoding verification of the same batch (the stochastic
    # counterpart of argmax + acceptance; not part of the timed greedy step):
    # draft logits a noisy copy of the target's, one uniform per node for the
    # acceptance test and one for the bonus draw.
    from paper_2501_12162_amd.workload import make_draft_logits, make_uniforms
    srng = np.random.Generator(np.random.PCG64(200 + args.workload))
    dl = make_draft_logits(srng, b.logits, b.vocab, b.dtype, 0.5)
    d_logits = torch.from_numpy(dl.view(np.int16) if is_bf16_in(b) else dl).cuda()
    if is_bf16_in(b):
        d_logits = d_logits.view(torch.bfloat16)
    del dl
    u_acc = tdev(make_uniforms(srng, b.total_nodes))
    u_bon = tdev(make_uniforms(srng, b.total_nodes))
    s_len = torch.empty_like(dev.accept_len)
    s_tok = torch.empty_like(dev.accept_tokens)
    s_nodes = torch.empty_like(dev.accept_nodes)
    s_ws = torch.empty(ada.adaserve_tree_accept_sampled_workspace_bytes(b.total_nodes), dtype=torch.uint8,
                       device="cuda")

    def sampled():
        ada.adaserve_tree_accept_sampled(node_indptr=dev.node_indptr, parent=dev.parent, draft_tokens=dev.draft_tokens,
                                         target_logits=rp["logits"], draft_logits=d_logits, vocab=b.vocab,
                                         u_accept=u_acc, u_bonus=u_bon, max_accept=dev.max_accept, accept_len=s_len,
                                         accept_tokens=s_tok, accept_nodes=s_nodes, workspace=s_ws)
    sampled()
    warm(run_step)
    hold_gpu()   # the host enqueues every timed call before the GPU starts them
    commit_ev[0].record(stream)
    for _ in range(10):
        sampled()
    commit_ev[1].record(stream)
    torch.cuda.synchronize()
    sampled_us = commit_ev[0].elapsed_time(commit_ev[1]) * 1e3 / 10
    sampled_len = s_len.cpu().numpy()
    # algorithmic bytes of the call: every target row and the draft rows of
    # the nodes with children (a leaf's draft distribution enters no test)
    starts = np.repeat(b.node_indptr[:-1], np.diff(b.node_indptr))
    internal = np.unique((starts + b.parent)[b.parent >= 0]).size
    sampled_bytes = (b.total_nodes + internal) * b.vocab * (2 if is_bf16_in(b) else 4)

    if fused:
        # the step's parts timed alone, call after call on the same inputs
        # (each call's own events; the replicas keep the MALL cold)
        step_ms = np.array([e[0].elapsed_time(e[1]) for e in events.values()])

        def alone(fn, calls=30):
            ev = [KernelTimer() for _ in range(calls + 1)]
            warm(run_step)
            hold_gpu()   # the host enqueues every timed call before the GPU starts them
            ev[0].record(stream)
            for k in range(calls):
                fn(reps[k % n_rep])
                ev[k + 1].record(stream)
            torch.cuda.synchronize()
            return np.array([ev[k].elapsed_time(ev[k + 1]) for k in range(calls)])
        if args.no_parts:
            attn_ms = argmax_ms = accept_ms = np.full(1, np.nan)
        else:
            attn_ms = alone(attention)
            argmax_ms = alone(lambda rp: ada.adaserve_node_argmax(rp["logits"], b.vocab, dev.target_argmax,
                                                                  stream=stream))
            accept_ms = alone(lambda rp: accept(stream))
    else:
        attn_ms = np.array([e[0].elapsed_time(e[1]) for e in events.values()])
        argmax_ms = np.array([e[2].elapsed_time(e[3]) for e in events.values()])
        accept_ms = np.array([e[4].elapsed_time(e[5]) for e in events.values()])
        step_ms = np.array([e[0].elapsed_time(e[5]) for e in events.values()])

    # Reference rate of the box: torch's device-to-device copy of 256 MiB
    # (bytes read + written per second), timed after the steps so that the
    # calibration copy stays the last copy before the first attention launch.
    warm(lambda k: calib_dst.copy_(calib_src))
    hold_gpu()
    commit_ev[0].record(stream)
    for _ in range(10):
        calib_dst.copy_(calib_src)
    commit_ev[1].record(stream)
    torch.cuda.synchronize()
    copy_gbs = 2 * calib_src.numel() * 10 / (commit_ev[0].elapsed_time(commit_ev[1]) * 1e-3) / 1e9

    # sanity: the last step's argmax must equal the planted maxima
    got = dev.target_argmax.cpu().numpy()
    if not np.array_equal(got, b.planted_argmax):
        print("bench.py: argmax mismatch, results invalid", file=sys.stderr)
        sys.exit(3)
    alen = dev.accept_len.cpu().numpy()

    extra = None
    if args.mfma_workload and args.mfma_workload != args.workload:
        del reps, dev
        progress("attention alone on workload %d" % args.mfma_workload)
        extra = attention_alone(args.mfma_workload)

    T = b.total_nodes
    ms_per_step = wall * 1e3 / args.steps
    value = T * args.steps / wall
    attn_us, argmax_us, accept_us, step_us = (float(x.mean()) * 1e3
                                              for x in (attn_ms, argmax_ms, accept_ms, step_ms))
    attn_gbs = costs["attn_bytes"] / (attn_us * 1e-6) / 1e9
    argmax_gbs = costs["argmax_bytes"] / (argmax_us * 1e-6) / 1e9
    attn_tflops = costs["attn_flops"] / (attn_us * 1e-6) / 1e12
    is_bf16 = b.dtype == "bf16"
    mfma_peak = BF16_MFMA_PEAK_TFLOPS if is_bf16 else FP32_PEAK_TFLOPS
    ridge = mfma_peak * 1e12 / (HBM_PEAK_GBS * 1e9)
    attn_ai = costs["attn_flops"] / costs["attn_bytes"]
    step_bytes_alg = costs["attn_bytes"] + costs["argmax_bytes"] + costs["accept_bytes"]
    if fused:
        # the dominant unit is the one-call step (its two launches carry the
        # attention, the argmax and the acceptance): all of its algorithmic
        # bytes over the step call's event-timed duration
        step_ai = costs["attn_flops"] / step_bytes_alg
        if step_ai > ridge:
            tf = costs["attn_flops"] / (step_us * 1e-6) / 1e12
            roof = {"kernel": "tree_verify_step", "bound": "mfma", "achieved": tf, "peak": mfma_peak,
                    "unit": "TFLOP/s", "frac": tf / mfma_peak}
        else:
            gbs = step_bytes_alg / (step_us * 1e-6) / 1e9
            roof = {"kernel": "tree_verify_step", "bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS,
                    "unit": "GB/s", "frac": gbs / HBM_PEAK_GBS}
    elif attn_us >= argmax_us:
        if attn_ai > ridge:
            roof = {"kernel": "tree_attn", "bound": "mfma", "achieved": attn_tflops, "peak": mfma_peak,
                    "unit": "TFLOP/s", "frac": attn_tflops / mfma_peak}
        else:
            roof = {"kernel": "tree_attn", "bound": "hbm", "achieved": attn_gbs, "peak": HBM_PEAK_GBS,
                    "unit": "GB/s", "frac": attn_gbs / HBM_PEAK_GBS}
    else:
        roof = {"kernel": "node_argmax", "bound": "hbm", "achieved": argmax_gbs, "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": argmax_gbs / HBM_PEAK_GBS}
    roof["traffic"] = measured_traffic(args.workload, roof["kernel"])

    line = {
        "metric": METRIC,
        "value": value,
        "unit": "tree tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if is_bf16 else "f32",
        "data": "synthetic (seeded; shapes of the named workload)",
        "config": {
            "workload": WORKLOAD_NAMES[args.workload],
            "requests": b.num_requests,
            "tree_tokens": T,
            "prefix_tokens": int(b.prefix_len.sum()),
            "q_heads": b.num_q_heads, "kv_heads": b.num_kv_heads, "head_dim": b.head_dim,
            "page_size": b.page_size, "vocab": b.vocab,
            "input_copies": n_rep,
            "instrumented_steps": len(sampled_steps),
            "step": "one adaserve_tree_verify_step call" if fused else
                    "three calls (attention, argmax, acceptance)",
            "argmax_beside_attention": bool(args.overlap and args.unfused),
        },
        "roofline": roof,
        "kernels": {
            "step_us": step_us, "step_alg_bytes": step_bytes_alg,
            "step_hbm_frac": step_bytes_alg / (step_us * 1e-6) / 1e9 / HBM_PEAK_GBS,
            "parts_timed": "alone, call after call" if fused else "inside the timed steps",
            "tree_attn_us": attn_us, "tree_attn_hbm_frac": attn_gbs / HBM_PEAK_GBS,
            "tree_attn_mfma_frac": attn_tflops / mfma_peak, "tree_attn_ai_flop_per_byte": attn_ai,
            "tree_attn_alg_bytes": costs["attn_bytes"], "tree_attn_alg_flops": costs["attn_flops"],
            "node_argmax_us": argmax_us, "node_argmax_hbm_frac": argmax_gbs / HBM_PEAK_GBS,
            "node_argmax_alg_bytes": costs["argmax_bytes"],
            "tree_accept_us": accept_us,
            "kv_commit_us": commit_us,
            "kv_commit_rows": committed_rows,
            "kv_commit_bytes": committed_rows * 4 * b.num_kv_heads * b.head_dim * (2 if is_bf16 else 4),
            "select_us": select_us,
            "select_candidates": int(cands.cand_prob.size),
            "sampled_accept_us": sampled_us,
            "sampled_accepted_tokens": int(sampled_len.sum()),
            "sampled_accept_alg_bytes": int(sampled_bytes),
            "sampled_accept_hbm_frac": sampled_bytes / (sampled_us * 1e-6) / 1e9 / HBM_PEAK_GBS,
            "beam_step_us": beam_us,
            "beam_step_rows": int(bb.logits.shape[0]),
            "beam_step_hbm_frac": beam_bytes / (beam_us * 1e-6) / 1e9 / HBM_PEAK_GBS,
            "percentiles_us": {
                name: {"p10": float(np.percentile(x, 10)) * 1e3, "p50": float(np.median(x)) * 1e3,
                       "p90": float(np.percentile(x, 90)) * 1e3}
                for name, x in (("tree_attn", attn_ms), ("node_argmax", argmax_ms), ("tree_accept", accept_ms),
                                ("step", step_ms))
            },
        },
        "reference": {"device_copy_gbs": copy_gbs,
                      "note": "torch device-to-device copy of 256 MiB, bytes read + written per second"},
        "accepted_tokens_per_step": int(alen.sum()),
        "accepted_tokens_per_s": float(alen.sum()) * args.steps / wall,
        "device": dev_name,
    }
    from paper_2501_12162_amd.workload import MODEL_LAYERS
    layers = MODEL_LAYERS.get(args.workload)
    if layers and math.isfinite(attn_us):
        proj_us = layers * attn_us + argmax_us + accept_us
        line["model_projection"] = {
            "label": "projection, not a measurement: the attention call timed above repeated for every "
                     "decoder layer, plus one argmax and one acceptance; the model's other layers left out",
            "layers": layers, "step_us": proj_us, "tree_tokens_per_s": T / (proj_us * 1e-6)}
    if extra is not None:
        line["mfma_bound_attention"] = extra
    if args.tp_share > 1:
        progress("one tensor-parallel rank's share of workload 4")
        line["tp_rank_share"] = attention_alone(4, tp=args.tp_share)
    if not args.no_cpu_baseline:
        progress("oracle baseline on the host cores")
        line["cpu_baseline"] = cpu_baseline(b, args.cpu_seconds)
    print(json.dumps(_finite(line)), flush=True)


if __name__ == "__main__":
    main()
