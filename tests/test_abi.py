"""The C-ABI library (CPU side): it loads, exports every symbol its headers
declare, and rejects bad arguments before enqueueing anything, so these calls
never touch a GPU."""
import ctypes
import os
import re

import pytest

import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    names = []
    for h in sorted(os.listdir(os.path.join(ROOT, "include"))):
        if not h.endswith(".h"):
            continue
        src = open(os.path.join(ROOT, "include", h)).read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        names += re.findall(r"\b((?:moe|dsa)_[a-z0-9_]+)\s*\(", src)
    return sorted(set(names))


@pytest.fixture(scope="module")
def M():
    import paper_2608_14560_amd as M
    if not os.path.exists(M.LIB_PATH):
        from paper_2608_14560_amd import build
        build.build()
    return M


def test_every_declared_symbol_is_exported(M):
    L = M.lib()
    names = _declared_functions()
    assert "moe_fused_fp8" in names and "moe_route" in names and "moe_workspace_size" in names
    for n in names:
        assert hasattr(L, n), n
    assert set(M.EXPORTED) == set(names)


def test_stage_names(M):
    assert M.num_stages() == 7
    assert M.stage_names()[3].startswith("gemm1")


def _shape(**kw):
    import paper_2608_14560_amd as M
    base = M.Shape.of(W.CONFIGS["decode"])
    d = {f: getattr(base, f) for f in M.Shape.__dataclass_fields__}
    d.update(kw)
    return M.Shape(**d)


@pytest.mark.parametrize("kw", [
    dict(H=7000), dict(I=100), dict(T=-1), dict(num_experts=255), dict(n_group=0),
    dict(topk_group=9), dict(topk_group=0), dict(top_k=0), dict(top_k=129),
    dict(num_local_experts=0), dict(local_expert_offset=250),
    dict(local_expert_offset=-1), dict(routed_scaling_factor=float("inf")),
    dict(num_experts=16, n_group=16, num_local_experts=8, topk_group=2, top_k=2),  # group size 1
])
def test_invalid_shapes(M, kw):
    s = _shape(**kw)
    assert M.workspace_size(s) == 0
    rc = M.lib().moe_fused_fp8(ctypes.byref(s.c()), *([None] * 9), None, None, 0, None)
    assert rc == M.MOE_ERR_INVALID_ARG


@pytest.mark.parametrize("kw", [dict(num_experts=2048, n_group=8, num_local_experts=32),
                                dict(top_k=17, topk_group=8)])
def test_unsupported_shapes(M, kw):
    s = _shape(**kw)
    rc = M.lib().moe_fused_fp8(ctypes.byref(s.c()), *([None] * 9), None, None, 0, None)
    assert rc == M.MOE_ERR_UNSUPPORTED


def _fake_ptrs(n, align=256):
    # aligned, never dereferenced: validation fails before anything is enqueued
    return [ctypes.c_void_p(0x10000 * (i + 1) * align) for i in range(n)]


def test_null_and_misaligned_pointers(M):
    s = _shape()
    L = M.lib()
    ws_bytes = M.workspace_size(s)
    ptrs = _fake_ptrs(9)
    ws = ctypes.c_void_p(0x7000000)
    for i in range(9):
        bad = list(ptrs)
        bad[i] = None
        assert L.moe_fused_fp8(ctypes.byref(s.c()), *bad, None, ws, ws_bytes, None) == M.MOE_ERR_INVALID_ARG
        bad[i] = ctypes.c_void_p(ptrs[i].value + 4)
        assert L.moe_fused_fp8(ctypes.byref(s.c()), *bad, None, ws, ws_bytes, None) == M.MOE_ERR_INVALID_ARG
    # workspace: null, misaligned, too small
    assert L.moe_fused_fp8(ctypes.byref(s.c()), *ptrs, None, None, ws_bytes, None) == M.MOE_ERR_INVALID_ARG
    assert L.moe_fused_fp8(ctypes.byref(s.c()), *ptrs, None, ctypes.c_void_p(0x7000010), ws_bytes,
                           None) == M.MOE_ERR_INVALID_ARG
    assert L.moe_fused_fp8(ctypes.byref(s.c()), *ptrs, None, ws, ws_bytes - 1,
                           None) == M.MOE_ERR_WORKSPACE_TOO_SMALL
    # a route_out with a null member
    ro = M.CRouteOut(*[p.value for p in _fake_ptrs(5)])
    ro.pair_row = None
    assert L.moe_fused_fp8(ctypes.byref(s.c()), *ptrs, ctypes.byref(ro), ws, ws_bytes,
                           None) == M.MOE_ERR_INVALID_ARG
    # staged entry: wrong event count
    ev = (ctypes.c_void_p * 3)(1, 2, 3)
    assert L.moe_fused_fp8_staged(ctypes.byref(s.c()), *ptrs, None, ws, ws_bytes, None, ev,
                                  3) == M.MOE_ERR_INVALID_ARG


def test_empty_batch_is_a_noop(M):
    s = _shape(T=0)
    assert M.workspace_size(s) > 0
    rc = M.lib().moe_fused_fp8(ctypes.byref(s.c()), *([None] * 9), None, None, 0, None)
    assert rc == M.MOE_OK


def test_route_rejects_bad_arguments(M):
    s = _shape()
    L = M.lib()
    ws_bytes = M.workspace_size(s)
    ro = M.CRouteOut(*[p.value for p in _fake_ptrs(5)])
    lg, bs = _fake_ptrs(2)
    ws = ctypes.c_void_p(0x7000000)
    assert L.moe_route(ctypes.byref(s.c()), lg, bs, None, ws, ws_bytes, None) == M.MOE_ERR_INVALID_ARG
    assert L.moe_route(ctypes.byref(s.c()), None, bs, ctypes.byref(ro), ws, ws_bytes,
                       None) == M.MOE_ERR_INVALID_ARG
    assert L.moe_route(ctypes.byref(s.c()), lg, bs, ctypes.byref(ro), ws, 16,
                       None) == M.MOE_ERR_WORKSPACE_TOO_SMALL


def test_router_entry_points_reject_bad_arguments(M):
    s = _shape()
    L = M.lib()
    ws_bytes = M.workspace_size(s)
    ro = M.CRouteOut(*[p.value for p in _fake_ptrs(5)])
    hid, hsc, wg, bs = _fake_ptrs(4)
    ws = ctypes.c_void_p(0x7000000)
    sc = ctypes.byref(s.c())
    # moe_route_hidden: each input null or misaligned, no route_out, small workspace
    args = [hid, hsc, wg, bs]
    for i in range(4):
        bad = list(args)
        bad[i] = None
        assert L.moe_route_hidden(sc, *bad, ctypes.byref(ro), ws, ws_bytes, None) == M.MOE_ERR_INVALID_ARG
        bad[i] = ctypes.c_void_p(args[i].value + 4)
        assert L.moe_route_hidden(sc, *bad, ctypes.byref(ro), ws, ws_bytes, None) == M.MOE_ERR_INVALID_ARG
    assert L.moe_route_hidden(sc, *args, None, ws, ws_bytes, None) == M.MOE_ERR_INVALID_ARG
    assert L.moe_route_hidden(sc, *args, ctypes.byref(ro), ws, 16, None) == M.MOE_ERR_WORKSPACE_TOO_SMALL
    # moe_fused_fp8_router: the router weight is required; a null logits pointer
    # is refused by moe_fused_fp8
    ptrs = _fake_ptrs(9)
    bad = list(ptrs)
    bad[2] = None
    assert L.moe_fused_fp8_router(sc, *bad, None, ws, ws_bytes, None) == M.MOE_ERR_INVALID_ARG
    assert L.moe_fused_fp8(sc, *bad, None, ws, ws_bytes, None) == M.MOE_ERR_INVALID_ARG
    assert L.moe_fused_fp8_router(sc, *ptrs, None, ws, 16, None) == M.MOE_ERR_WORKSPACE_TOO_SMALL
    # debug logits: null output
    assert L.moe_debug_router_logits(sc, hid, hsc, wg, None, ws, ws_bytes, None) == M.MOE_ERR_INVALID_ARG
    # empty batch: a no-op for the projection entry points too
    s0 = _shape(T=0)
    ro0 = M.CRouteOut(None, None, _fake_ptrs(1)[0].value, _fake_ptrs(1)[0].value, None)
    assert L.moe_fused_fp8_router(ctypes.byref(s0.c()), *ptrs, None, None, 0, None) == M.MOE_OK


def test_dsa_indexer_rejects_bad_arguments(M):
    L = M.lib()
    good = M.CDsaShape(4, 64, 128, 64, 2048, 36, 300)
    assert M.dsa_workspace_size(good) >= 4 * 36 * 64 * 4
    for bad, code in [(M.CDsaShape(4, 32, 128, 64, 2048, 36, 300), M.MOE_ERR_UNSUPPORTED),
                      (M.CDsaShape(4, 64, 64, 64, 2048, 36, 300), M.MOE_ERR_UNSUPPORTED),
                      (M.CDsaShape(-1, 64, 128, 64, 2048, 36, 300), M.MOE_ERR_INVALID_ARG),
                      (M.CDsaShape(4, 64, 128, 0, 2048, 36, 300), M.MOE_ERR_INVALID_ARG),
                      (M.CDsaShape(4, 64, 128, 64, 0, 36, 300), M.MOE_ERR_INVALID_ARG),
                      (M.CDsaShape(4, 64, 128, 64, 2048, 36, 0), M.MOE_ERR_INVALID_ARG)]:
        assert M.dsa_workspace_size(bad) == 0
        assert L.dsa_topk_indexer(ctypes.byref(bad), *_fake_ptrs(7), ctypes.c_void_p(0x7000000), 1 << 30,
                                  None) == code
    ptrs = _fake_ptrs(7)
    ws = ctypes.c_void_p(0x7000000)
    nbytes = M.dsa_workspace_size(good)
    for i in range(7):
        bad = list(ptrs)
        bad[i] = None
        assert L.dsa_topk_indexer(ctypes.byref(good), *bad, ws, nbytes, None) == M.MOE_ERR_INVALID_ARG
        bad[i] = ctypes.c_void_p(ptrs[i].value + 4)
        assert L.dsa_topk_indexer(ctypes.byref(good), *bad, ws, nbytes, None) == M.MOE_ERR_INVALID_ARG
    assert L.dsa_topk_indexer(ctypes.byref(good), *ptrs, ws, nbytes - 1, None) == M.MOE_ERR_WORKSPACE_TOO_SMALL
    empty = M.CDsaShape(0, 64, 128, 64, 2048, 36, 300)
    assert L.dsa_topk_indexer(ctypes.byref(empty), *([None] * 7), None, 0, None) == M.MOE_OK


def test_dsa_attention_rejects_bad_arguments(M):
    L = M.lib()
    good = M.CAttnShape(8, 16, 2048, 8462 * 64, 0.072)
    nbytes = M.dsa_attention_workspace_size(good)
    assert nbytes >= 8 * 32 * 16 * (512 * 2 + 2 * 4)  # bf16 split outputs, fp32 (max, sum)
    for bad, code in [(M.CAttnShape(8, 8, 2048, 100, 0.1), M.MOE_ERR_UNSUPPORTED),
                      (M.CAttnShape(8, 16, 70000, 100, 0.1), M.MOE_ERR_UNSUPPORTED),
                      (M.CAttnShape(-1, 16, 2048, 100, 0.1), M.MOE_ERR_INVALID_ARG),
                      (M.CAttnShape(8, 16, 0, 100, 0.1), M.MOE_ERR_INVALID_ARG),
                      (M.CAttnShape(8, 16, 2048, 0, 0.1), M.MOE_ERR_INVALID_ARG),
                      (M.CAttnShape(8, 16, 2048, 100, float("nan")), M.MOE_ERR_INVALID_ARG)]:
        assert M.dsa_attention_workspace_size(bad) == 0
        assert L.dsa_sparse_attention(ctypes.byref(bad), *_fake_ptrs(7), ctypes.c_void_p(0x7000000), 1 << 30,
                                      None) == code
    ptrs = _fake_ptrs(7)
    ws = ctypes.c_void_p(0x7000000)
    for i in range(7):
        bad = list(ptrs)
        bad[i] = None
        assert L.dsa_sparse_attention(ctypes.byref(good), *bad, ws, nbytes, None) == M.MOE_ERR_INVALID_ARG
        bad[i] = ctypes.c_void_p(ptrs[i].value + 4)
        assert L.dsa_sparse_attention(ctypes.byref(good), *bad, ws, nbytes, None) == M.MOE_ERR_INVALID_ARG
    assert L.dsa_sparse_attention(ctypes.byref(good), *ptrs, ws, nbytes - 1, None) == M.MOE_ERR_WORKSPACE_TOO_SMALL
    assert L.dsa_sparse_attention(ctypes.byref(M.CAttnShape(0, 16, 2048, 100, 0.1)), *([None] * 7), None, 0,
                                  None) == M.MOE_OK


def test_workspace_grows_with_batch(M):
    sizes = [M.workspace_size(_shape(T=t)) for t in (1, 16, 256, 4096)]
    assert sizes == sorted(sizes) and sizes[0] > 0


def test_python_binding_refuses_cpu_tensors(M):
    import torch
    cfg = W.CONFIGS["tiny"]
    s = M.Shape.of(cfg)
    x = torch.zeros(cfg.T, cfg.num_experts)
    with pytest.raises(ValueError):
        M.route(s, x, torch.zeros(cfg.num_experts), route_out=M.alloc_route_out(s, "cpu"),
                workspace=torch.zeros(256, dtype=torch.uint8))
