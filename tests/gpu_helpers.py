"""Shared helpers of the GPU parity tests: seeded inputs on the device, host
copies for the oracle, and the output tolerance check."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
import workloads as W

# |gpu - ref| <= ATOL + RTOL * |ref| elementwise, ref = the oracle's bf16 output
ATOL, RTOL = 1e-2, 2e-2

_cache: dict = {}


def log(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def inputs(cfg: W.MoEConfig, seed: int) -> W.MoEInputs:
    """Seeded inputs generated on the GPU (cached: the big configs take seconds)."""
    key = (cfg, seed)
    if key not in _cache:
        if len(_cache) > 2:
            _cache.clear()
            torch.cuda.empty_cache()
        _cache[key] = W.generate(cfg, seed, device="cuda")
    return _cache[key]


def oracle_route(cfg, inp):
    s = oracle.shape_of(cfg)
    ids, w = oracle.route(s, inp.logits.cpu().numpy(), inp.bias.cpu().numpy())
    offs, perm, pr = oracle.permute(s, ids)
    return dict(topk_ids=ids, topk_weights=w, expert_offsets=offs, perm_token=perm, pair_row=pr)


def experts_of(cfg, ids: np.ndarray, tokens) -> list[int]:
    le = ids[np.asarray(tokens)].ravel() - cfg.local_expert_offset
    return sorted(set(int(e) for e in le if 0 <= e < cfg.num_local_experts))


def oracle_forward(cfg, inp, tokens=None, ref_ids=None):
    """The oracle's output for ``tokens`` (all by default); weights are copied to
    the host only for the experts those tokens use (from the oracle's routing)."""
    if ref_ids is None:
        ref_ids = oracle_route(cfg, inp)["topk_ids"]
    toks = np.arange(cfg.T) if tokens is None else np.asarray(tokens)
    h = W.host_arrays(inp, experts=experts_of(cfg, ref_ids, toks))
    out, ids, w = oracle.forward(oracle.shape_of(cfg), **h, tokens=toks.astype(np.int32))
    return out, ids, w


def assert_out_close(gpu_rows: torch.Tensor, ref_bits: np.ndarray, what: str = ""):
    g = gpu_rows.float().cpu().numpy()
    r = oracle.bf16_bits_to_float(ref_bits)
    err = np.abs(g - r)
    bad = err > ATOL + RTOL * np.abs(r)
    if bad.any():
        idx = np.argwhere(bad)[:8]
        raise AssertionError(
            f"{what}: {bad.sum()} of {bad.size} elements outside |d| <= {ATOL} + {RTOL}|ref|; "
            f"first at {idx.tolist()}: gpu={g[bad][:8].tolist()} ref={r[bad][:8].tolist()}")
    return float(err.max()), float(np.abs(r).max())
