"""MI355X (gfx950) fused block-scaled FP8 mixture-of-experts layer.

Python binding of ``libmoe.so`` (the hand-written HIP kernels behind the C-ABI
declared in ``include/moe.h``).  This module only marshals arguments: torch
tensors provide device memory and the current stream; every step of the layer
runs in the library's kernels.  There is no fallback: if the library is not
built, or a tensor is not on the GPU, the call raises.

Entry points (same names as the C-ABI):
  workspace_size(shape)               bytes of scratch the calls need
  route(shape, logits, bias, ...)     stage (1) + stage (2) bookkeeping
  fused_fp8(shape, ...)               the whole layer, bf16 output
  fused_fp8_noalloc(shape, ...)       the same with the library's own scratch (no allocation)
  fused_fp8_staged(..., events)       same, recording an event before each kernel
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmoe.so")

MOE_OK, MOE_ERR_INVALID_ARG, MOE_ERR_UNSUPPORTED, MOE_ERR_WORKSPACE_TOO_SMALL, MOE_ERR_HIP = range(5)

EXPORTED = ("moe_workspace_size", "moe_route", "moe_route_hidden", "moe_fused_fp8",
            "moe_fused_fp8_router", "moe_fused_fp8_staged", "moe_fused_fp8_noalloc", "moe_num_stages", "moe_stage_name",
            "moe_status_string", "moe_debug_sigmoid", "moe_debug_e4m3_encode",
            "moe_debug_act_views", "moe_debug_mfma_block", "moe_debug_router_logits",
            "moe_debug_combine_from_act",
            "dsa_workspace_size", "dsa_topk_indexer", "dsa_debug_scores",
            "dsa_attention_workspace_size", "dsa_sparse_attention")


class MoEError(RuntimeError):
    def __init__(self, fn: str, code: int):
        super().__init__(f"{fn}: {status_string(code)} ({code})")
        self.code = code


class CShape(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int32), ("H", ctypes.c_int32), ("I", ctypes.c_int32),
                ("num_experts", ctypes.c_int32), ("num_local_experts", ctypes.c_int32),
                ("local_expert_offset", ctypes.c_int32), ("n_group", ctypes.c_int32),
                ("topk_group", ctypes.c_int32), ("top_k", ctypes.c_int32),
                ("routed_scaling_factor", ctypes.c_float)]


class CRouteOut(ctypes.Structure):
    _fields_ = [("topk_ids", ctypes.c_void_p), ("topk_weights", ctypes.c_void_p),
                ("expert_offsets", ctypes.c_void_p), ("perm_token", ctypes.c_void_p),
                ("pair_row", ctypes.c_void_p)]


@dataclass(frozen=True)
class Shape:
    T: int
    H: int
    I: int
    num_experts: int
    num_local_experts: int
    local_expert_offset: int
    n_group: int
    topk_group: int
    top_k: int
    routed_scaling_factor: float = 2.5

    @staticmethod
    def of(cfg) -> "Shape":
        return Shape(*(getattr(cfg, f) for f in Shape.__dataclass_fields__))

    def c(self) -> CShape:
        return CShape(self.T, self.H, self.I, self.num_experts, self.num_local_experts,
                      self.local_expert_offset, self.n_group, self.topk_group, self.top_k,
                      self.routed_scaling_factor)


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded C-ABI library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2608_14560_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        P, S, Z = ctypes.c_void_p, ctypes.POINTER(CShape), ctypes.c_size_t
        R = ctypes.POINTER(CRouteOut)
        L.moe_workspace_size.argtypes = [S]
        L.moe_workspace_size.restype = Z
        L.moe_route.argtypes = [S, P, P, R, P, Z, P]
        L.moe_route.restype = ctypes.c_int
        L.moe_fused_fp8.argtypes = [S, P, P, P, P, P, P, P, P, P, R, P, Z, P]
        L.moe_fused_fp8.restype = ctypes.c_int
        L.moe_fused_fp8_noalloc.argtypes = [S, P, P, P, P, P, P, P, P, P, R, P]
        L.moe_fused_fp8_noalloc.restype = ctypes.c_int
        L.moe_route_hidden.argtypes = [S, P, P, P, P, R, P, Z, P]
        L.moe_route_hidden.restype = ctypes.c_int
        L.moe_fused_fp8_router.argtypes = [S, P, P, P, P, P, P, P, P, P, R, P, Z, P]
        L.moe_fused_fp8_router.restype = ctypes.c_int
        L.moe_debug_router_logits.argtypes = [S, P, P, P, P, P, Z, P]
        L.moe_debug_router_logits.restype = ctypes.c_int
        DS = ctypes.POINTER(CDsaShape)
        L.dsa_workspace_size.argtypes = [DS]
        L.dsa_workspace_size.restype = ctypes.c_size_t
        L.dsa_topk_indexer.argtypes = [DS, P, P, P, P, P, P, P, P, Z, P]
        L.dsa_topk_indexer.restype = ctypes.c_int
        L.dsa_debug_scores.argtypes = [DS, P, P, P, P, P, P, P, P]
        L.dsa_debug_scores.restype = ctypes.c_int
        AS = ctypes.POINTER(CAttnShape)
        L.dsa_attention_workspace_size.argtypes = [AS]
        L.dsa_attention_workspace_size.restype = ctypes.c_size_t
        L.dsa_sparse_attention.argtypes = [AS, P, P, P, P, P, P, P, P, Z, P]
        L.dsa_sparse_attention.restype = ctypes.c_int
        L.moe_fused_fp8_staged.argtypes = [S, P, P, P, P, P, P, P, P, P, R, P, Z, P,
                                           ctypes.POINTER(P), ctypes.c_int]
        L.moe_fused_fp8_staged.restype = ctypes.c_int
        L.moe_num_stages.argtypes = []
        L.moe_num_stages.restype = ctypes.c_int
        L.moe_stage_name.argtypes = [ctypes.c_int]
        L.moe_stage_name.restype = ctypes.c_char_p
        L.moe_status_string.argtypes = [ctypes.c_int]
        L.moe_status_string.restype = ctypes.c_char_p
        L.moe_debug_sigmoid.argtypes = [P, P, ctypes.c_int64, P]
        L.moe_debug_sigmoid.restype = ctypes.c_int
        L.moe_debug_e4m3_encode.argtypes = [P, P, ctypes.c_int64, P]
        L.moe_debug_e4m3_encode.restype = ctypes.c_int
        L.moe_debug_mfma_block.argtypes = [P, P, P, ctypes.c_int64, P]
        L.moe_debug_mfma_block.restype = ctypes.c_int
        L.moe_debug_act_views.argtypes = [S, P, ctypes.POINTER(P), ctypes.POINTER(P)]
        L.moe_debug_act_views.restype = ctypes.c_int
        L.moe_debug_combine_from_act.argtypes = [S, P, P, P, P, P, P, P, P, Z, P]
        L.moe_debug_combine_from_act.restype = ctypes.c_int
        _lib = L
    return _lib


def status_string(code: int) -> str:
    return lib().moe_status_string(code).decode()


def _check(fn: str, code: int):
    if code != MOE_OK:
        raise MoEError(fn, code)


def _dev(t: torch.Tensor | None, dtype, name: str):
    if t is None:
        raise ValueError(f"{name} is required")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor (the layer has no CPU path)")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def workspace_size(shape: Shape) -> int:
    return int(lib().moe_workspace_size(ctypes.byref(shape.c())))


def alloc_workspace(shape: Shape, device="cuda") -> torch.Tensor:
    return torch.empty(max(workspace_size(shape), 256), dtype=torch.uint8, device=device)


def alloc_route_out(shape: Shape, device="cuda") -> dict:
    # at least one row each, so an empty batch still gets non-null buffers
    T, K, El = shape.T, shape.top_k, shape.num_local_experts
    R = max(T, 1)
    return dict(topk_ids=torch.empty(R, K, dtype=torch.int32, device=device)[:T],
                topk_weights=torch.empty(R, K, dtype=torch.float32, device=device)[:T],
                expert_offsets=torch.empty(El + 1, dtype=torch.int32, device=device),
                perm_token=torch.empty(R * K, dtype=torch.int32, device=device),
                pair_row=torch.empty(R, K, dtype=torch.int32, device=device)[:T])


def _route_struct(ro: dict) -> CRouteOut:
    return CRouteOut(_dev(ro["topk_ids"], torch.int32, "topk_ids"),
                     _dev(ro["topk_weights"], torch.float32, "topk_weights"),
                     _dev(ro["expert_offsets"], torch.int32, "expert_offsets"),
                     _dev(ro["perm_token"], torch.int32, "perm_token"),
                     _dev(ro["pair_row"], torch.int32, "pair_row"))


def route(shape: Shape, logits: torch.Tensor, bias: torch.Tensor, route_out: dict | None = None,
          workspace: torch.Tensor | None = None, stream=None) -> dict:
    """Stage (1) and the permutation of stage (2); returns the route-out tensors."""
    ro = route_out if route_out is not None else alloc_route_out(shape, logits.device)
    ws = workspace if workspace is not None else alloc_workspace(shape, logits.device)
    cro = _route_struct(ro)
    rc = lib().moe_route(ctypes.byref(shape.c()), _dev(logits, torch.float32, "logits"),
                         _dev(bias, torch.float32, "bias"), ctypes.byref(cro),
                         _dev(ws, torch.uint8, "workspace"), ws.numel(), _stream(stream))
    _check("moe_route", rc)
    return ro


def route_hidden(shape: Shape, hidden, hidden_scale, router_weight, bias,
                 route_out: dict | None = None, workspace: torch.Tensor | None = None,
                 stream=None) -> dict:
    """Stage (1) with the router projection on the device (fp32 router weight
    [E_g, H]), then the permutation of stage (2); returns the route-out tensors."""
    ro = route_out if route_out is not None else alloc_route_out(shape, hidden.device)
    ws = workspace if workspace is not None else alloc_workspace(shape, hidden.device)
    cro = _route_struct(ro)
    rc = lib().moe_route_hidden(ctypes.byref(shape.c()), _dev(hidden, torch.uint8, "hidden"),
                                _dev(hidden_scale, torch.float32, "hidden_scale"),
                                _dev(router_weight, torch.float32, "router_weight"),
                                _dev(bias, torch.float32, "bias"), ctypes.byref(cro),
                                _dev(ws, torch.uint8, "workspace"), ws.numel(), _stream(stream))
    _check("moe_route_hidden", rc)
    return ro


def debug_router_logits(shape: Shape, hidden, hidden_scale, router_weight,
                        workspace: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """The fp32 logits [T, E_g] that moe_route_hidden forms (test hook)."""
    ws = workspace if workspace is not None else alloc_workspace(shape, hidden.device)
    out = torch.empty(max(shape.T, 1), shape.num_experts, dtype=torch.float32,
                      device=hidden.device)[: shape.T]
    rc = lib().moe_debug_router_logits(ctypes.byref(shape.c()), _dev(hidden, torch.uint8, "hidden"),
                                       _dev(hidden_scale, torch.float32, "hidden_scale"),
                                       _dev(router_weight, torch.float32, "router_weight"),
                                       _dev(out, torch.float32, "logits"),
                                       _dev(ws, torch.uint8, "workspace"), ws.numel(),
                                       _stream(stream))
    _check("moe_debug_router_logits", rc)
    return out


def _fused_args(shape, hidden, hidden_scale, logits, bias, w13, w13_scale, w2, w2_scale, out,
                route_out, workspace):
    return [ctypes.byref(shape.c()),
            _dev(hidden, torch.uint8, "hidden"), _dev(hidden_scale, torch.float32, "hidden_scale"),
            _dev(logits, torch.float32, "logits"), _dev(bias, torch.float32, "bias"),
            _dev(w13, torch.uint8, "w13"), _dev(w13_scale, torch.float32, "w13_scale"),
            _dev(w2, torch.uint8, "w2"), _dev(w2_scale, torch.float32, "w2_scale"),
            _dev(out, torch.bfloat16, "out"),
            ctypes.byref(_route_struct(route_out)) if route_out is not None else None,
            ] + ([] if workspace is None else
                 [_dev(workspace, torch.uint8, "workspace"), ctypes.c_size_t(workspace.numel())])


def fused_fp8(shape: Shape, hidden, hidden_scale, logits, bias, w13, w13_scale, w2, w2_scale,
              out: torch.Tensor | None = None, route_out: dict | None = None,
              workspace: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """The whole layer (stages (1)-(4)); returns out [T, H] bf16."""
    if out is None:
        out = torch.empty(shape.T, shape.H, dtype=torch.bfloat16, device=hidden.device)
    if workspace is None:
        workspace = alloc_workspace(shape, hidden.device)
    args = _fused_args(shape, hidden, hidden_scale, logits, bias, w13, w13_scale, w2, w2_scale,
                       out, route_out, workspace)
    _check("moe_fused_fp8", lib().moe_fused_fp8(*args, _stream(stream)))
    return out


def fused_fp8_noalloc(shape: Shape, hidden, hidden_scale, logits, bias, w13, w13_scale, w2,
                      w2_scale, out: torch.Tensor, route_out: dict | None = None,
                      stream=None) -> torch.Tensor:
    """The whole layer with the library's own per-GPU scratch instead of a
    workspace (moe_fused_fp8_noalloc): for callers that cannot allocate, so
    `out` [T, H] bf16 is required.  Overlapping calls on one GPU race."""
    args = _fused_args(shape, hidden, hidden_scale, logits, bias, w13, w13_scale, w2, w2_scale,
                       out, route_out, None)
    _check("moe_fused_fp8_noalloc", lib().moe_fused_fp8_noalloc(*args, _stream(stream)))
    return out


def fused_fp8_router(shape: Shape, hidden, hidden_scale, router_weight, bias, w13, w13_scale,
                     w2, w2_scale, out: torch.Tensor | None = None,
                     route_out: dict | None = None, workspace: torch.Tensor | None = None,
                     stream=None) -> torch.Tensor:
    """The whole layer with the router projection on the device; returns out
    [T, H] bf16."""
    if out is None:
        out = torch.empty(shape.T, shape.H, dtype=torch.bfloat16, device=hidden.device)
    if workspace is None:
        workspace = alloc_workspace(shape, hidden.device)
    args = _fused_args(shape, hidden, hidden_scale, router_weight, bias, w13, w13_scale, w2,
                       w2_scale, out, route_out, workspace)
    _check("moe_fused_fp8_router", lib().moe_fused_fp8_router(*args, _stream(stream)))
    return out


class FusedCall:
    """A prepared moe_fused_fp8 call: the arguments are validated and marshalled
    once, each call() only enqueues the layer on the stream.  The tensors must
    stay alive (and keep their addresses) while the object is used; their
    contents may change between calls."""

    def __init__(self, shape: Shape, hidden, hidden_scale, logits, bias, w13, w13_scale, w2,
                 w2_scale, out, workspace, route_out: dict | None = None, stream=None,
                 router: bool = False):
        """router=True: `logits` is the fp32 router weight [E_g, H] and each call
        runs moe_fused_fp8_router (no staged variant)."""
        self._keep = (shape.c(), route_out and _route_struct(route_out))
        args = _fused_args(shape, hidden, hidden_scale, logits, bias, w13, w13_scale, w2,
                           w2_scale, out, route_out, workspace)
        args[0] = ctypes.byref(self._keep[0])
        if route_out is not None:
            args[10] = ctypes.byref(self._keep[1])
        self._args = (*args, _stream(stream))
        self._fn = lib().moe_fused_fp8_router if router else lib().moe_fused_fp8
        self._staged = None if router else lib().moe_fused_fp8_staged
        self.out = out

    def __call__(self):
        rc = self._fn(*self._args)
        if rc:
            raise MoEError("moe_fused_fp8", rc)
        return self.out

    def staged(self, events_array, n: int):
        """events_array: a ctypes array of n raw hipEvent_t handles."""
        rc = self._staged(*self._args, events_array, n)
        if rc:
            raise MoEError("moe_fused_fp8_staged", rc)
        return self.out


def event_array(events: list):
    """ctypes array of the raw HIP handles of torch.cuda.Events (created here)."""
    for ev in events:
        if ev.cuda_event == 0:
            ev.record()
    return (ctypes.c_void_p * len(events))(*[ev.cuda_event for ev in events])


def num_stages() -> int:
    return lib().moe_num_stages()


def stage_names() -> list[str]:
    return [lib().moe_stage_name(i).decode() for i in range(num_stages())]


def fused_fp8_staged(shape: Shape, hidden, hidden_scale, logits, bias, w13, w13_scale, w2,
                     w2_scale, out, workspace, events: list, route_out: dict | None = None,
                     stream=None) -> torch.Tensor:
    """fused_fp8 recording ``events[i]`` (torch.cuda.Event, timing enabled) on the
    stream before kernel i and ``events[-1]`` after the last kernel."""
    n = num_stages() + 1
    if len(events) != n:
        raise ValueError(f"need {n} events")
    for ev in events:  # torch creates the HIP event lazily, on its first record
        if ev.cuda_event == 0:
            ev.record()
    arr = (ctypes.c_void_p * n)(*[ev.cuda_event for ev in events])
    args = _fused_args(shape, hidden, hidden_scale, logits, bias, w13, w13_scale, w2, w2_scale,
                       out, route_out, workspace)
    _check("moe_fused_fp8_staged",
           lib().moe_fused_fp8_staged(*args, _stream(stream), arr, n))
    return out


# ----------------------------------------------------------------- test hooks
def debug_sigmoid(x: torch.Tensor, stream=None) -> torch.Tensor:
    y = torch.empty_like(x)
    _check("moe_debug_sigmoid", lib().moe_debug_sigmoid(
        _dev(x, torch.float32, "x"), _dev(y, torch.float32, "y"), x.numel(), _stream(stream)))
    return y


def debug_e4m3_encode(x: torch.Tensor, stream=None) -> torch.Tensor:
    q = torch.empty(x.shape, dtype=torch.uint8, device=x.device)
    _check("moe_debug_e4m3_encode", lib().moe_debug_e4m3_encode(
        _dev(x, torch.float32, "x"), _dev(q, torch.uint8, "q"), x.numel(), _stream(stream)))
    return q


def debug_mfma_block(a: torch.Tensor, b: torch.Tensor, stream=None) -> torch.Tensor:
    """a, b: [n, 16, 128] uint8 e4m3 codes -> d [n, 16, 16] with d = a @ b^T per case."""
    n = a.shape[0]
    d = torch.empty(n, 16, 16, dtype=torch.float32, device=a.device)
    _check("moe_debug_mfma_block", lib().moe_debug_mfma_block(
        _dev(a, torch.uint8, "a"), _dev(b, torch.uint8, "b"), _dev(d, torch.float32, "d"), n,
        _stream(stream)))
    return d


def debug_act_views(shape: Shape, workspace: torch.Tensor):
    """(act [P_max, I] uint8, act_scale [P_max, I/128] f32) views into the workspace."""
    a, s = ctypes.c_void_p(), ctypes.c_void_p()
    _check("moe_debug_act_views", lib().moe_debug_act_views(
        ctypes.byref(shape.c()), _dev(workspace, torch.uint8, "workspace"),
        ctypes.byref(a), ctypes.byref(s)))
    base = workspace.data_ptr()
    P = max(shape.T * shape.top_k, 1)
    act = workspace[a.value - base: a.value - base + P * shape.I].view(P, shape.I)
    sc = workspace[s.value - base: s.value - base + P * (shape.I // 128) * 4]
    return act, sc.view(torch.float32).view(P, shape.I // 128)


def debug_combine_from_act(shape: Shape, logits, bias, act, act_scale, w2, w2_scale,
                           out: torch.Tensor | None = None, workspace: torch.Tensor | None = None,
                           stream=None) -> torch.Tensor:
    """GEMM2 and the weighted combine on a given intermediate act [T*k, I] uint8 /
    act_scale [T*k, I/128] f32 (permuted row order of ``route``); routing is
    recomputed from logits/bias.  Returns out [T, H] bf16 (test hook)."""
    if out is None:
        out = torch.empty(shape.T, shape.H, dtype=torch.bfloat16, device=logits.device)
    if workspace is None:
        workspace = alloc_workspace(shape, logits.device)
    P = shape.T * shape.top_k
    if tuple(act.shape) != (P, shape.I) or tuple(act_scale.shape) != (P, shape.I // 128):
        raise ValueError("act must be [T*top_k, I] and act_scale [T*top_k, I/128]")
    rc = lib().moe_debug_combine_from_act(
        ctypes.byref(shape.c()), _dev(logits, torch.float32, "logits"), _dev(bias, torch.float32, "bias"),
        _dev(act, torch.uint8, "act"), _dev(act_scale, torch.float32, "act_scale"),
        _dev(w2, torch.uint8, "w2"), _dev(w2_scale, torch.float32, "w2_scale"),
        _dev(out, torch.bfloat16, "out"), _dev(workspace, torch.uint8, "workspace"),
        ctypes.c_size_t(workspace.numel()), _stream(stream))
    _check("moe_debug_combine_from_act", rc)
    return out


# ---------------------------------------------------------------- DSA TopK indexer
class CDsaShape(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("num_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("page_size", ctypes.c_int32), ("topk", ctypes.c_int32), ("max_pages", ctypes.c_int32),
                ("num_pages", ctypes.c_int32)]


def dsa_shape(q: torch.Tensor, k_cache: torch.Tensor, block_table: torch.Tensor, topk: int) -> CDsaShape:
    B, NH, D = q.shape
    return CDsaShape(B, NH, D, k_cache.shape[1], topk, block_table.shape[1], k_cache.shape[0])


def dsa_workspace_size(shape: CDsaShape) -> int:
    return int(lib().dsa_workspace_size(ctypes.byref(shape)))


def _dsa_ptrs(q, weights, k_cache, k_scale, block_table, seq_lens):
    return [_dev(q, torch.uint8, "q"), _dev(weights, torch.float32, "weights"),
            _dev(k_cache, torch.uint8, "k_cache"), _dev(k_scale, torch.float32, "k_scale"),
            _dev(block_table, torch.int32, "block_table"), _dev(seq_lens, torch.int32, "seq_lens")]


def dsa_topk_indexer(q, weights, k_cache, k_scale, block_table, seq_lens, topk: int = 2048,
                     out: torch.Tensor | None = None, workspace: torch.Tensor | None = None,
                     stream=None) -> torch.Tensor:
    """DSA TopK Indexer (paper Section 3.1.3): int32 [B, topk] physical cache
    indices of each sequence's topk best tokens, ascending position order,
    padded with -1."""
    shape = dsa_shape(q, k_cache, block_table, topk)
    if out is None:
        out = torch.empty(max(shape.B, 1), topk, dtype=torch.int32, device=q.device)[: shape.B]
    if workspace is None:
        workspace = torch.empty(max(dsa_workspace_size(shape), 256), dtype=torch.uint8, device=q.device)
    rc = lib().dsa_topk_indexer(ctypes.byref(shape), *_dsa_ptrs(q, weights, k_cache, k_scale, block_table,
                                                                seq_lens),
                                _dev(out, torch.int32, "out"), _dev(workspace, torch.uint8, "workspace"),
                                workspace.numel(), _stream(stream))
    _check("dsa_topk_indexer", rc)
    return out


def dsa_debug_scores(q, weights, k_cache, k_scale, block_table, seq_lens, stream=None) -> torch.Tensor:
    """Scores [B, max_pages * page_size] of every token (test hook); entries past a
    sequence's length are left as allocated (NaN here)."""
    shape = dsa_shape(q, k_cache, block_table, 1)
    scores = torch.full((max(shape.B, 1), shape.max_pages * shape.page_size), float("nan"),
                        dtype=torch.float32, device=q.device)[: shape.B]
    rc = lib().dsa_debug_scores(ctypes.byref(shape), *_dsa_ptrs(q, weights, k_cache, k_scale, block_table,
                                                                seq_lens),
                                _dev(scores, torch.float32, "scores"), _stream(stream))
    _check("dsa_debug_scores", rc)
    return scores


# ---------------------------------------------------------------- DSA sparse attention
class CAttnShape(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int32), ("num_heads", ctypes.c_int32), ("topk", ctypes.c_int32),
                ("num_rows", ctypes.c_int32), ("sm_scale", ctypes.c_float)]


def attention_shape(q_nope: torch.Tensor, ckv: torch.Tensor, indices: torch.Tensor, sm_scale: float) -> CAttnShape:
    T, H, _ = q_nope.shape
    rows = ckv.numel() // ckv.shape[-1]
    return CAttnShape(T, H, indices.shape[1], rows, float(sm_scale))


def dsa_attention_workspace_size(shape: CAttnShape) -> int:
    return int(lib().dsa_attention_workspace_size(ctypes.byref(shape)))


def dsa_sparse_attention(q_nope, q_pe, ckv, kpe, indices, sm_scale: float, out=None, lse=None,
                         workspace=None, stream=None):
    """DSA sparse attention (paper Section 3.1.2): (out bf16 [T, H, 512],
    lse float32 [T, H], base 2)."""
    if q_nope.dim() != 3 or q_nope.shape[2] != 512 or ckv.shape[-1] != 512 or indices.dim() != 2:
        raise ValueError("q_nope must be [T, H, 512], ckv [..., 512] and indices [T, topk]")
    shape = attention_shape(q_nope, ckv, indices, sm_scale)
    T, H = shape.T, shape.num_heads
    if tuple(q_pe.shape) != (T, H, 64) or kpe.numel() != shape.num_rows * 64 or kpe.shape[-1] != 64 \
            or indices.shape[0] != T:
        raise ValueError("q_pe must be [T, H, 64], kpe [rows, 64] over the rows of ckv and indices [T, topk]")
    if (out is not None and tuple(out.shape) != (T, H, 512)) or (lse is not None and tuple(lse.shape) != (T, H)):
        raise ValueError("out must be [T, H, 512] and lse [T, H]")
    if out is None:
        out = torch.empty(max(T, 1), H, 512, dtype=torch.bfloat16, device=q_nope.device)[:T]
    if lse is None:
        lse = torch.empty(max(T, 1), H, dtype=torch.float32, device=q_nope.device)[:T]
    if workspace is None:
        workspace = torch.empty(max(dsa_attention_workspace_size(shape), 256), dtype=torch.uint8,
                                device=q_nope.device)
    rc = lib().dsa_sparse_attention(ctypes.byref(shape), _dev(q_nope, torch.bfloat16, "q_nope"),
                                    _dev(q_pe, torch.bfloat16, "q_pe"), _dev(ckv, torch.bfloat16, "ckv"),
                                    _dev(kpe, torch.bfloat16, "kpe"), _dev(indices, torch.int32, "indices"),
                                    _dev(out, torch.bfloat16, "out"), _dev(lse, torch.float32, "lse"),
                                    _dev(workspace, torch.uint8, "workspace"), workspace.numel(),
                                    _stream(stream))
    _check("dsa_sparse_attention", rc)
    return out, lse
