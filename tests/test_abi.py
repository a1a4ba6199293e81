"""C-ABI checks that need no GPU: the library loads, exports every function
include/adaserve.h declares, and rejects bad arguments on the host before
any HIP call (so nothing here touches a device)."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2501_12162_amd as ada

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "adaserve.h")
FAKE = 0x1000   # never dereferenced: every call below fails validation first


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(ada.library_path()):
        from paper_2501_12162_amd.build import build
        build()
    return ada.load_library()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(adaserve_\w+)\s*\(", text)))


def test_header_and_binding_agree():
    assert declared_functions() == sorted(ada.SIGNATURES)


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def _ws(ip, pl, hq=32, hkv=8, d=128, ps=16, dtype=ada.ADASERVE_BF16):
    ip = np.asarray(ip, np.int32)
    pl = np.asarray(pl, np.int32)
    return ada.load_library().adaserve_tree_attn_workspace_bytes(
        int(pl.size), ip.ctypes.data, pl.ctypes.data, hq, hkv, d, ps, dtype)


SIZE_MAX = ctypes.c_size_t(-1).value


def test_workspace_query(lib):
    assert _ws([0, 10], [100]) == 0                       # short prefix: no split
    assert _ws([0, 32], [32768]) > 0                      # long prefix is split
    assert _ws([0, 32], [32768], dtype=ada.ADASERVE_F32) == 0
    assert _ws([0, 10], [100], hq=30, hkv=8) == SIZE_MAX
    assert _ws([0, 10], [100], d=96) == SIZE_MAX
    assert _ws([0, 10], [100], ps=32) == SIZE_MAX
    assert _ws([0, 129], [100]) == SIZE_MAX
    assert _ws([0, 0], [100]) == SIZE_MAX
    assert _ws([1, 5], [100]) == SIZE_MAX
    assert _ws([0, 5], [-1]) == SIZE_MAX
    assert b"prefix_len" in lib.adaserve_last_error()
    assert _ws([], []) == 0


def _verify(lib, **kw):
    ip = np.asarray(kw.pop("ip", [0, 4]), np.int32)
    pl = np.asarray(kw.pop("pl", [20]), np.int32)
    args = dict(node_indptr=FAKE, parent=FAKE, q=FAKE, k_tree=FAKE, v_tree=FAKE, k_pages=FAKE,
                v_pages=FAKE, num_pages=4, block_table=FAKE, bt_stride=2, prefix_len=FAKE,
                hq=8, hkv=2, d=128, ps=16, scale=0.1, dtype=ada.ADASERVE_BF16, out=FAKE,
                ws=None, ws_bytes=0)
    args.update(kw)
    return lib.adaserve_tree_attn_verify(
        int(pl.size), args["node_indptr"], ip.ctypes.data, args["parent"], args["q"], args["k_tree"],
        args["v_tree"], args["k_pages"], args["v_pages"], args["num_pages"], args["block_table"],
        args["bt_stride"], args["prefix_len"], pl.ctypes.data, args["hq"], args["hkv"], args["d"],
        args["ps"], args["scale"], args["dtype"], args["out"], args["ws"], args["ws_bytes"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(hq=6, hkv=4), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(hq=0), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(hq=64, hkv=2), ada.ADASERVE_ERR_UNSUPPORTED),
    (dict(d=80), ada.ADASERVE_ERR_UNSUPPORTED),
    (dict(ps=8), ada.ADASERVE_ERR_UNSUPPORTED),
    (dict(dtype=7), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(ip=[0, 200]), ada.ADASERVE_ERR_UNSUPPORTED),
    (dict(ip=[0, 0]), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(ip=[2, 6]), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(pl=[-3]), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(pl=[33], bt_stride=2), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(bt_stride=-1), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(num_pages=-1), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(num_pages=0), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(scale=float("nan")), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(scale=0.0), ada.ADASERVE_ERR_UNSUPPORTED),
    (dict(scale=-0.125), ada.ADASERVE_ERR_UNSUPPORTED),
    (dict(q=None), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(out=None), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(parent=None), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(k_pages=None), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(block_table=None), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(q=FAKE + 2), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(ip=[0, 32], pl=[32768], bt_stride=2048), ada.ADASERVE_ERR_WORKSPACE),
])
def test_verify_rejects_bad_arguments(lib, kw, code):
    assert _verify(lib, **kw) == code
    assert lib.adaserve_last_error()


def _verify_noalloc(lib, ip, pl, hq=8, hkv=2, d=128, scale=0.1, bt_stride=None):
    ip = np.asarray(ip, np.int32)
    pl = np.asarray(pl, np.int32)
    if bt_stride is None:
        bt_stride = max(1, int(-(-pl.max() // 16))) if pl.size else 1
    return lib.adaserve_tree_attn_verify_noalloc(
        int(pl.size), FAKE, ip.ctypes.data, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 4, FAKE, bt_stride, FAKE,
        pl.ctypes.data, hq, hkv, d, 16, scale, ada.ADASERVE_BF16, FAKE, None)


def test_verify_noalloc_rejects_batches_past_the_scratch(lib):
    # a plan needing more split-KV partials than the static scratch holds is
    # refused before anything is enqueued, with the sizes in the message
    ip = np.arange(0, 65 * 128, 128)
    pl = np.full(64, 200000)
    need = _ws(ip, pl, hq=8, hkv=2)
    assert need > ada.TREE_ATTN_SCRATCH_BYTES
    assert _verify_noalloc(lib, ip, pl) == ada.ADASERVE_ERR_WORKSPACE
    msg = lib.adaserve_last_error()
    assert b"scratch" in msg and str(need).encode() in msg
    # and it validates like the workspace entry point
    assert _verify_noalloc(lib, [0, 4], [20], hq=6, hkv=4) == ada.ADASERVE_ERR_INVALID_ARGUMENT
    assert _verify_noalloc(lib, [0, 4], [20], scale=0.0) == ada.ADASERVE_ERR_UNSUPPORTED
    assert _verify_noalloc(lib, [0, 4], [20], d=80) == ada.ADASERVE_ERR_UNSUPPORTED


def _step(lib, **kw):
    ip = np.asarray(kw.pop("ip", [0, 4]), np.int32)
    pl = np.asarray(kw.pop("pl", [20]), np.int32)
    args = dict(scale=0.1, dtype=ada.ADASERVE_BF16, hq=8, hkv=2, d=128, logits=FAKE, stride=1000, vocab=1000,
                draft=FAKE, max_accept=8, out=FAKE, amax=FAKE, alen=FAKE, atok=FAKE, anodes=FAKE, ws=None,
                ws_bytes=0, q=FAKE)
    args.update(kw)
    return lib.adaserve_tree_verify_step(
        int(pl.size), FAKE, ip.ctypes.data, FAKE, args["q"], FAKE, FAKE, FAKE, FAKE, 4, FAKE, 2, FAKE,
        pl.ctypes.data, args["hq"], args["hkv"], args["d"], 16, args["scale"], args["dtype"], args["logits"],
        args["stride"], args["vocab"], args["draft"], args["max_accept"], args["out"], args["amax"], args["alen"],
        args["atok"], args["anodes"], args["ws"], args["ws_bytes"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(hq=6, hkv=4), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(scale=0.0), ada.ADASERVE_ERR_UNSUPPORTED),
    (dict(vocab=0), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(stride=999), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(max_accept=0), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(logits=None), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(logits=FAKE + 1), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(draft=None), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(amax=None), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(amax=FAKE + 2), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(alen=None), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(atok=None), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(anodes=None), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(out=None), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(q=FAKE + 2), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(ip=[0, 32], pl=[32768]), ada.ADASERVE_ERR_INVALID_ARGUMENT),   # block table too narrow
    (dict(dtype=ada.ADASERVE_F32, logits=FAKE + 2), ada.ADASERVE_ERR_INVALID_ARGUMENT),
])
def test_verify_step_rejects_bad_arguments(lib, kw, code):
    assert _step(lib, **kw) == code
    assert lib.adaserve_last_error()


def test_verify_step_empty_batch_is_a_noop(lib):
    assert _step(lib, ip=[0], pl=[]) == ada.ADASERVE_OK


def test_verify_empty_batch_is_a_noop(lib):
    assert _verify(lib, ip=[0], pl=[]) == ada.ADASERVE_OK


def test_argmax_rejects_bad_arguments(lib):
    f = lib.adaserve_node_argmax
    assert f(FAKE, 10, -1, 10, 1, FAKE, None) == ada.ADASERVE_ERR_INVALID_ARGUMENT
    assert f(FAKE, 10, 0, 10, 1, FAKE, None) == ada.ADASERVE_OK          # nothing to do
    assert f(FAKE, 10, 3, 0, 1, FAKE, None) == ada.ADASERVE_ERR_INVALID_ARGUMENT
    assert f(FAKE, 9, 3, 10, 1, FAKE, None) == ada.ADASERVE_ERR_INVALID_ARGUMENT
    assert f(None, 10, 3, 10, 1, FAKE, None) == ada.ADASERVE_ERR_INVALID_ARGUMENT
    assert f(FAKE, 10, 3, 10, 1, None, None) == ada.ADASERVE_ERR_INVALID_ARGUMENT
    assert f(FAKE, 10, 3, 10, 5, FAKE, None) == ada.ADASERVE_ERR_INVALID_ARGUMENT
    assert f(FAKE + 1, 10, 3, 10, 1, FAKE, None) == ada.ADASERVE_ERR_INVALID_ARGUMENT


def test_accept_rejects_bad_arguments(lib):
    f = lib.adaserve_tree_accept
    assert f(-1, 4, FAKE, FAKE, FAKE, FAKE, 4, FAKE, FAKE, FAKE, None) == ada.ADASERVE_ERR_INVALID_ARGUMENT
    assert f(1, -4, FAKE, FAKE, FAKE, FAKE, 4, FAKE, FAKE, FAKE, None) == ada.ADASERVE_ERR_INVALID_ARGUMENT
    assert f(1, 4, FAKE, FAKE, FAKE, FAKE, 0, FAKE, FAKE, FAKE, None) == ada.ADASERVE_ERR_INVALID_ARGUMENT
    assert f(1, 4, None, FAKE, FAKE, FAKE, 4, FAKE, FAKE, FAKE, None) == ada.ADASERVE_ERR_INVALID_ARGUMENT
    assert f(1, 4, FAKE, None, FAKE, FAKE, 4, FAKE, FAKE, FAKE, None) == ada.ADASERVE_ERR_INVALID_ARGUMENT
    assert f(1, 4, FAKE, FAKE, FAKE, FAKE, 4, None, FAKE, FAKE, None) == ada.ADASERVE_ERR_INVALID_ARGUMENT
    assert f(0, 0, None, None, None, None, 4, None, None, None, None) == ada.ADASERVE_OK


def _commit(lib, **kw):
    args = dict(B=1, indptr=FAKE, alen=FAKE, nodes=FAKE, max_accept=4, k_tree=FAKE, v_tree=FAKE,
                k_pages=FAKE, v_pages=FAKE, num_pages=4, bt=FAKE, bt_stride=2, plen=FAKE, hkv=2,
                d=128, ps=16, dtype=ada.ADASERVE_BF16, new_len=FAKE)
    args.update(kw)
    return lib.adaserve_commit_accepted_kv(
        args["B"], args["indptr"], args["alen"], args["nodes"], args["max_accept"], args["k_tree"],
        args["v_tree"], args["k_pages"], args["v_pages"], args["num_pages"], args["bt"],
        args["bt_stride"], args["plen"], args["hkv"], args["d"], args["ps"], args["dtype"],
        args["new_len"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(B=-1), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(max_accept=0), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(num_pages=-1), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(bt_stride=-2), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(hkv=0), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(d=0), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(ps=0), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(dtype=3), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(d=12), ada.ADASERVE_ERR_UNSUPPORTED),                               # 24-byte rows
    (dict(d=6, dtype=ada.ADASERVE_F32), ada.ADASERVE_ERR_UNSUPPORTED),
    (dict(alen=None), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(new_len=None), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(k_pages=None), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(bt=None), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(v_tree=FAKE + 8), ada.ADASERVE_ERR_INVALID_ARGUMENT),
])
def test_commit_rejects_bad_arguments(lib, kw, code):
    assert _commit(lib, **kw) == code
    assert lib.adaserve_last_error()


def test_commit_empty_batch_is_a_noop(lib):
    assert _commit(lib, B=0, indptr=None, alen=None) == ada.ADASERVE_OK


def _select(lib, **kw):
    args = dict(B=2, C=10, indptr=FAKE, par=FAKE, prob=FAKE, need=FAKE, budget=8, n_max=4,
                max_nodes=128, size=FAKE, tpar=FAKE, tcand=FAKE)
    args.update(kw)
    return lib.adaserve_select_trees(args["B"], args["C"], args["indptr"], args["par"], args["prob"],
                                     args["need"], args["budget"], args["n_max"], args["max_nodes"],
                                     args["size"], args["tpar"], args["tcand"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(B=-1), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(B=513), ada.ADASERVE_ERR_UNSUPPORTED),
    (dict(C=-1), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(C=8193), ada.ADASERVE_ERR_UNSUPPORTED),
    (dict(budget=-1), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(n_max=0), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(max_nodes=127), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(indptr=None), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(prob=None), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(tcand=None), ada.ADASERVE_ERR_INVALID_ARGUMENT),
])
def test_select_rejects_bad_arguments(lib, kw, code):
    assert _select(lib, **kw) == code
    assert lib.adaserve_last_error()


def test_select_empty_batch_is_a_noop(lib):
    assert _select(lib, B=0, C=0, indptr=None, par=None, prob=None) == ada.ADASERVE_OK


def _beam_ws(lib, B=2, w_in=4, V=1000, w_out=8, dtype=ada.ADASERVE_BF16):
    return lib.adaserve_beam_step_workspace_bytes(B, w_in, V, w_out, dtype)


def test_beam_workspace_query(lib):
    # one scan part per 65536 bf16 (32768 fp32) logits of a row: a (max, sum)
    # pair per part, 256-byte aligned, then w_out sorted entries per part
    assert _beam_ws(lib, B=2, w_in=4, V=65536, w_out=8) == 256 + 2 * 4 * 1 * 8 * 8
    assert _beam_ws(lib, B=2, w_in=4, V=65537, w_out=8) == 256 + 2 * 4 * 2 * 8 * 8
    assert _beam_ws(lib, B=2, w_in=4, V=65536, w_out=8, dtype=ada.ADASERVE_F32) == 256 + 2 * 4 * 2 * 8 * 8
    assert _beam_ws(lib, V=1 << 20) != SIZE_MAX
    assert _beam_ws(lib, V=(1 << 20) + 1) == SIZE_MAX
    assert _beam_ws(lib, B=0) == 0
    assert _beam_ws(lib, w_in=0) == SIZE_MAX
    assert _beam_ws(lib, w_in=65) == SIZE_MAX
    assert _beam_ws(lib, w_out=65) == SIZE_MAX
    assert _beam_ws(lib, V=0) == SIZE_MAX
    assert _beam_ws(lib, dtype=7) == SIZE_MAX


def _beam(lib, **kw):
    args = dict(B=2, w_in=4, logits=0x1000 * 16, stride=1024, V=1000, dtype=ada.ADASERVE_BF16, lp=FAKE,
                w_out=8, par=FAKE, tok=FAKE, out_lp=FAKE, ws=0x100000, ws_bytes=1 << 20)
    args.update(kw)
    return lib.adaserve_beam_step(args["B"], args["w_in"], args["logits"], args["stride"], args["V"],
                                  args["dtype"], args["lp"], args["w_out"], args["par"], args["tok"],
                                  args["out_lp"], args["ws"], args["ws_bytes"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(B=-1), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(w_in=0), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(w_in=65), ada.ADASERVE_ERR_UNSUPPORTED),
    (dict(w_out=0), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(w_out=65), ada.ADASERVE_ERR_UNSUPPORTED),
    (dict(V=0), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(V=(1 << 20) + 8, stride=(1 << 20) + 8), ada.ADASERVE_ERR_UNSUPPORTED),
    (dict(stride=999), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(stride=1001), ada.ADASERVE_ERR_INVALID_ARGUMENT),      # rows not 16-byte apart
    (dict(logits=0x1000 * 16 + 2), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(dtype=3), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(logits=None), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(lp=None), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(out_lp=None), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(ws=None), ada.ADASERVE_ERR_WORKSPACE),
    (dict(ws_bytes=64), ada.ADASERVE_ERR_WORKSPACE),
    (dict(ws=0x100000 + 64), ada.ADASERVE_ERR_INVALID_ARGUMENT),  # workspace not 256-byte aligned
])
def test_beam_rejects_bad_arguments(lib, kw, code):
    assert _beam(lib, **kw) == code
    assert lib.adaserve_last_error()


def test_beam_empty_batch_is_a_noop(lib):
    assert _beam(lib, B=0, logits=None, lp=None, par=None, tok=None, out_lp=None, ws=None,
                 ws_bytes=0) == ada.ADASERVE_OK


def _sampled(lib, **kw):
    args = dict(B=2, T=10, indptr=FAKE, par=FAKE, draft=FAKE, tl=0x1000 * 16, dl=0x2000 * 16, stride=1024, V=1000,
                dtype=ada.ADASERVE_BF16, ua=FAKE, ub=FAKE, K=8, alen=FAKE, tok=FAKE, nodes=FAKE, ws=0x100000,
                ws_bytes=lib.adaserve_tree_accept_sampled_workspace_bytes(10))
    args.update(kw)
    return lib.adaserve_tree_accept_sampled(args["B"], args["T"], args["indptr"], args["par"], args["draft"],
                                            args["tl"], args["dl"], args["stride"], args["V"], args["dtype"],
                                            args["ua"], args["ub"], args["K"], args["alen"], args["tok"],
                                            args["nodes"], args["ws"], args["ws_bytes"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(B=-1), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(T=-1), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(K=0), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(V=0), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(stride=999), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(stride=1001), ada.ADASERVE_ERR_INVALID_ARGUMENT),     # rows not 16 bytes apart
    (dict(tl=0x1000 * 16 + 4), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(dtype=5), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(indptr=None), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(dl=None), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(ub=None), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(nodes=None), ada.ADASERVE_ERR_INVALID_ARGUMENT),
    (dict(ws=None), ada.ADASERVE_ERR_WORKSPACE),
    (dict(ws_bytes=10 * 8 * 16 - 1), ada.ADASERVE_ERR_WORKSPACE),  # 10 nodes, vocab 1000: 8 parts each
    (dict(ws=0x100000 + 8), ada.ADASERVE_ERR_INVALID_ARGUMENT),   # workspace not 16-byte aligned
])
def test_sampled_accept_rejects_bad_arguments(lib, kw, code):
    assert _sampled(lib, **kw) == code
    assert lib.adaserve_last_error()


def test_sampled_accept_empty_batch_is_a_noop(lib):
    assert _sampled(lib, B=0, T=0, indptr=None, par=None, draft=None, tl=None, dl=None, ua=None, ub=None,
                    alen=None, tok=None, nodes=None, ws=None, ws_bytes=0) == ada.ADASERVE_OK


def test_sampled_accept_workspace_query(lib):
    assert lib.adaserve_tree_accept_sampled_workspace_bytes(0) == 0
    # 16 bytes per node and statistics part, sized for the most parts a node
    # can take (64: one per token range of a draw's pass)
    assert lib.adaserve_tree_accept_sampled_workspace_bytes(586) == 586 * 64 * 16
    assert lib.adaserve_tree_accept_sampled_workspace_bytes(1) == 64 * 16
    assert lib.adaserve_tree_accept_sampled_workspace_bytes(-1) == SIZE_MAX
