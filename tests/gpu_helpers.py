"""Shared helpers of the GPU parity tests: seeded inputs on the device, host
copies for the oracle, and the layer's parity checks.

The layer's parity (stages (1)-(4) of the paper's Section 3.1.1) is checked in
three parts, all against the oracle:
  * routing and permutation bit for bit;
  * the re-quantised FP8 intermediate: every code and block scale of the
    device must lie in the oracle's admissible set (the codes any FP8 block
    GEMM1 within the oracle's stated error model produces), and the share of
    codes that differ from the oracle's own (flips) stays below FLIP_GATE;
  * the bf16 output: |gpu - ref| <= ATOL + RTOL |ref| + widen, ref the
    oracle's output and widen the oracle's bound on how far the observed
    (admissible) intermediate differences can move it:
    widen[t, n] = sum_j |w_j| sum_i |dq_gpu[i] - dq_ref[i]| |W2[n, i]| over
    the token's resident pairs j (dq = code value times block scale);
and, separately, GEMM2 + combine alone (moe_debug_combine_from_act) on the
oracle's own intermediate against the oracle, with the plain tolerance.
"""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
import workloads as W

# |gpu - ref| <= ATOL + RTOL * |ref| elementwise, ref = the oracle's bf16 output
ATOL, RTOL = 1e-2, 2e-2
# largest share of re-quantised codes allowed to differ from the oracle's own
# (each such code is still admissible); pinned on the CPU by
# test_flip_rate_separates_rounding_from_bias
FLIP_GATE = 0.01

_cache: dict = {}
_DEC = torch.arange(256, dtype=torch.int32).to(torch.uint8).view(torch.float8_e4m3fn).double().numpy()


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


def run_fused(M, cfg, inp):
    s = M.Shape.of(cfg)
    ro = M.alloc_route_out(s)
    ws = M.alloc_workspace(s)
    out = M.fused_fp8(s, inp.hidden, inp.hidden_scale, inp.logits, inp.bias, inp.w13,
                      inp.w13_scale, inp.w2, inp.w2_scale, route_out=ro, workspace=ws)
    torch.cuda.synchronize()
    return out, ro, ws


def check_route(cfg, ro, ref):
    ids = ro["topk_ids"].cpu().numpy()
    assert (ids == ref["topk_ids"]).all(), f"topk_ids differ at {np.argwhere(ids != ref['topk_ids'])[:5]}"
    w = ro["topk_weights"].cpu().numpy()
    assert (w.view(np.int32) == ref["topk_weights"].view(np.int32)).all(), "topk_weights differ"
    offs = ro["expert_offsets"].cpu().numpy()
    assert (offs == ref["expert_offsets"]).all(), "expert_offsets differ"
    P = int(offs[-1])
    assert (ro["perm_token"].cpu().numpy()[:P] == ref["perm_token"]).all(), "perm_token differs"
    assert (ro["pair_row"].cpu().numpy() == ref["pair_row"]).all(), "pair_row differs"


def assert_out_close(gpu_rows, ref_bits: np.ndarray, what: str = "", widen=None):
    g = gpu_rows.float().cpu().numpy() if isinstance(gpu_rows, torch.Tensor) else gpu_rows
    r = oracle.bf16_bits_to_float(ref_bits)
    err = np.abs(g - r)
    tol = ATOL + RTOL * np.abs(r)
    if widen is not None:
        tol = tol + widen * (1.0 + 1e-6)
    bad = err > tol
    if bad.any():
        idx = np.argwhere(bad)[:8]
        raise AssertionError(
            f"{what}: {bad.sum()} of {bad.size} elements outside |d| <= {ATOL} + {RTOL}|ref|"
            f"{' + widen' if widen is not None else ''}; first at {idx.tolist()}: "
            f"gpu={g[bad][:8].tolist()} ref={r[bad][:8].tolist()}")
    return float(err.max()), float(np.abs(r).max()), float((err / tol).max())


def _rows_of(ref, toks):
    pr = ref["pair_row"][toks]
    rows = np.sort(pr[pr >= 0]).astype(np.int64)
    experts = np.searchsorted(ref["expert_offsets"], rows, side="right") - 1
    return rows, experts.astype(np.int32)


def _dequant_abs(w2, s2):
    """|W2| dequantised, float32 [H, I]."""
    v = np.abs(_DEC[w2]).astype(np.float32)
    return v * np.repeat(np.repeat(s2, 128, 0), 128, 1)


def layer_parity(M, cfg, inp, tokens=None, staged=True, what=""):
    """Runs the layer once and checks it against the oracle on ``tokens`` (all
    by default): routing, the admissible intermediate, the output within the
    widened tolerance, and (staged) GEMM2 + combine alone on the oracle's
    intermediate.  Returns a dict of statistics."""
    what = what or cfg.name
    shape_o = oracle.shape_of(cfg)
    s = M.Shape.of(cfg)
    out, ro, ws = run_fused(M, cfg, inp)
    ref = oracle_route(cfg, inp)
    check_route(cfg, ro, ref)
    toks = np.arange(cfg.T, dtype=np.int32) if tokens is None else np.asarray(tokens, np.int32)
    rows, rexp = _rows_of(ref, toks)
    P = int(ref["expert_offsets"][-1])
    need = sorted(set(rexp.tolist()))
    h = W.host_arrays(inp, experts=need)
    log(f"{what}: P={P}, checking {len(toks)} tokens, {len(rows)} pairs on {len(need)} experts")

    # the FP8 intermediate: admissible, few flips
    adm = oracle.admissible_batch(shape_o, h["hidden"], h["hidden_scale"], h["w13"], h["w13_scale"],
                                  tokens=ref["perm_token"][rows], experts=rexp)
    act_v, sc_v = M.debug_act_views(s, ws)
    ridx = torch.from_numpy(rows).cuda()
    q_g = act_v.index_select(0, ridx).cpu().numpy() if len(rows) else np.zeros((0, cfg.I), np.uint8)
    s_g = sc_v.index_select(0, ridx).cpu().numpy() if len(rows) else np.zeros((0, cfg.I // 128), np.float32)
    v_g = _DEC[q_g]
    code_ok = (v_g >= adm["v_lo"]) & (v_g <= adm["v_hi"])
    scale_ok = ((s_g >= adm["s_lo"]) & (s_g <= adm["s_hi"])) | ((s_g == 1.0) & (adm["zero_ok"] > 0))
    assert code_ok.all(), (f"{what}: {(~code_ok).sum()} codes outside the admissible set, first "
                           f"(row, i) {np.argwhere(~code_ok)[:4].tolist()}")
    assert scale_ok.all(), f"{what}: {(~scale_ok).sum()} block scales outside the admissible set"
    flips = int((v_g != _DEC[adm["q"]]).sum())
    total = int(v_g.size)
    scale_diff = int((s_g.view(np.int32) != adm["qs"].view(np.int32)).sum())
    assert flips <= FLIP_GATE * max(total, 1), f"{what}: {flips} of {total} codes flipped"

    # the oracle's intermediate in permuted order (the rows checked here)
    act_o = np.zeros((max(cfg.T * cfg.top_k, 1), cfg.I), np.uint8)
    sc_o = np.ones((max(cfg.T * cfg.top_k, 1), cfg.I // 128), np.float32)
    act_o[rows] = adm["q"]
    sc_o[rows] = adm["qs"]

    # the output: oracle's GEMM2 + combine on its own intermediate (bit-identical
    # to its forward pass), tolerance widened by the observed differences
    ref_out = oracle.combine_from_act(shape_o, act_o, sc_o, h["w2"], h["w2_scale"], ref["expert_offsets"],
                                      ref["pair_row"], ref["topk_weights"], tokens=toks)
    dq = np.abs(v_g * np.repeat(s_g, 128, 1) - _DEC[adm["q"]] * np.repeat(adm["qs"], 128, 1))
    contrib = np.zeros((len(rows), cfg.H), np.float64)
    nz = dq.max(1) > 0
    for e in need:
        sel = np.flatnonzero((rexp == e) & nz)
        if sel.size:
            contrib[sel] = dq[sel].astype(np.float32) @ _dequant_abs(h["w2"][e], h["w2_scale"][e]).T
    row_pos = {int(r): i for i, r in enumerate(rows)}
    widen = np.zeros((len(toks), cfg.H), np.float64)
    for ti, t in enumerate(toks):
        for j in range(cfg.top_k):
            r = int(ref["pair_row"][t, j])
            if r >= 0 and nz[row_pos[r]]:
                widen[ti] += abs(float(ref["topk_weights"][t, j])) * contrib[row_pos[r]]
    g_rows = out.index_select(0, torch.from_numpy(toks).long().cuda())
    err, mag, used = assert_out_close(g_rows, ref_out, what, widen=widen)
    r_f = oracle.bf16_bits_to_float(ref_out)
    plain_bad = int((np.abs(g_rows.float().cpu().numpy() - r_f) > ATOL + RTOL * np.abs(r_f)).sum())
    # tokens without a resident expert are exactly zero
    none = toks[(ref["pair_row"][toks] < 0).all(1)]
    if none.size:
        assert (out[torch.from_numpy(none).long().cuda()] == 0).all()

    stats = dict(P=P, pairs=len(rows), flips=flips, codes=total, scale_diffs=scale_diff,
                 max_err=err, max_ref=mag, tol_used=used, beyond_plain_tol=plain_bad)
    if staged:
        out_s = M.debug_combine_from_act(s, inp.logits, inp.bias, torch.from_numpy(act_o).cuda(),
                                         torch.from_numpy(sc_o).cuda(), inp.w2, inp.w2_scale)
        torch.cuda.synchronize()
        e2, _, u2 = assert_out_close(out_s.index_select(0, torch.from_numpy(toks).long().cuda()),
                                     ref_out, f"{what} staged")
        stats.update(staged_max_err=e2, staged_tol_used=u2)
    log(f"{what}: {stats}")
    return stats
